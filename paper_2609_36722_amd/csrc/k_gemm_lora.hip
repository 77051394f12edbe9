// K2: bf16 MFMA projection GEMM with the rank-r LoRA update fused into its
// epilogue (query-side adaptation, section 4 eq. 4):
//   out[i][n] = x[i] . w[n]  +  (n < lora_cols ? t[i] . b[n] : 0),
//   t = scale * x A^T  (computed first by lora_down_kernel).
//
// The GEMM is computed as C^T = W x^T so that the MFMA accumulator of a lane
// holds four consecutive output features of one token (8-byte stores).  Both
// operands are K-contiguous in memory ([rows][hidden]), so tiles go to LDS
// without a transpose.  Workgroup tile BN (features) x BM (tokens) x 64 (k),
// four waves in a 2 x 2 grid, 32x32x16 MFMAs, fp32 accumulation, LDS double
// buffered with register prefetch of the next k-tile.  LDS rows are 128 bytes
// (eight 16-byte chunks); chunk c of row r is stored at c ^ (r & 7) so that
// the 32 rows an MFMA operand read touches spread over all banks.
//
// The LoRA term enters as extra MFMA k-steps after the main loop: A operand
// = rows of B (rank padded to 16 with zeros), B operand = t as a bf16 hi/lo
// pair, so t keeps ~16 significant bits and the update stays in fp32.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int BK = 64;
constexpr int kChunksPerRow = BK / 8;  // 16-byte chunks per LDS row

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

template <int BM, int BN>
__global__ __launch_bounds__(256, 2) void gemm_lora_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w,
                                                           int M, int N, int K, const bf16_t* __restrict__ b,
                                                           int rank, int r_pad, int lora_cols,
                                                           const bf16_t* __restrict__ t_hi,
                                                           const bf16_t* __restrict__ t_lo, bf16_t* __restrict__ out,
                                                           int n_mt, int n_nt) {
  constexpr int FN = BN / 64;  // 32-row MFMA blocks per wave along features
  constexpr int FM = BM / 64;  // along tokens
  constexpr int ROWS = BN + BM;
  constexpr int LOADS = ROWS * kChunksPerRow / 256;  // 16-byte chunks per thread per k-tile
  static_assert(ROWS * kChunksPerRow % 256 == 0, "tile must split evenly over 256 threads");

  __shared__ u32x4 lds[2][ROWS * kChunksPerRow];

  // XCD-aware tile order: consecutive workgroups land on different XCDs, so
  // give each XCD a contiguous run of tiles that share weight rows.
  const int total = n_mt * n_nt;
  int lin = blockIdx.x;
  if ((total & 7) == 0) lin = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const int nt = lin / n_mt;
  const int mt = lin - nt * n_mt;
  const int n0 = nt * BN;
  const int m0 = mt * BM;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave >> 1;  // feature half
  const int wm = wave & 1;   // token half
  const int l32 = lane & 31;
  const int hi = lane >> 5;

  // global source of each of this thread's chunks
  const u32x4* src[LOADS];
  int dst[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int c = tid + 256 * i;
    const int row = c / kChunksPerRow;
    const int ch = c % kChunksPerRow;
    const bf16_t* base;
    if (row < BN) {
      base = w + (int64_t)(n0 + row) * K;
    } else {
      int m = m0 + row - BN;
      m = m < M ? m : M - 1;  // rows past the end are computed but never stored
      base = x + (int64_t)m * K;
    }
    src[i] = reinterpret_cast<const u32x4*>(base) + ch;
    dst[i] = row * kChunksPerRow + swz(row, ch);
  }

  f32x16 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x16{};

  u32x4 pre[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) pre[i] = src[i][0];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) lds[0][dst[i]] = pre[i];
  __syncthreads();

  const int n_kt = K / BK;
  for (int kt = 0; kt < n_kt; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < n_kt) {
#pragma unroll
      for (int i = 0; i < LOADS; ++i) pre[i] = src[i][(kt + 1) * kChunksPerRow];
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = 2 * ks + hi;
      bf16x8 af[FN], bfr[FM];
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const int row = wn * (BN / 2) + i * 32 + l32;
        af[i] = as_bf16x8(lds[cur][row * kChunksPerRow + swz(row, ch)]);
      }
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        const int row = BN + wm * (BM / 2) + j * 32 + l32;
        bfr[j] = as_bf16x8(lds[cur][row * kChunksPerRow + swz(row, ch)]);
      }
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = mfma32(af[i], bfr[j], acc[i][j]);
    }
    if (kt + 1 < n_kt) {
#pragma unroll
      for (int i = 0; i < LOADS; ++i) lds[cur ^ 1][dst[i]] = pre[i];
    }
    __syncthreads();
  }

  // ---- fused low-rank epilogue: acc += B[n][:] . t[m][:] --------------------
  if (r_pad > 0) {
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int nb = n0 + wn * (BN / 2) + i * 32;
      if (nb >= lora_cols) continue;  // lora_cols is a multiple of 32
      const int n = nb + l32;
      for (int ks = 0; ks < r_pad; ks += 16) {
        bf16x8 a;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int jj = ks + 8 * hi + e;
          const bf16_t bv = jj < rank ? b[(int64_t)n * rank + jj] : (bf16_t)0;
          a[e] = __builtin_bit_cast(__bf16, bv);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          int m = m0 + wm * (BM / 2) + j * 32 + l32;
          m = m < M ? m : M - 1;
          const int64_t off = (int64_t)m * r_pad + ks + 8 * hi;
          const bf16x8 th = as_bf16x8(*reinterpret_cast<const u32x4*>(t_hi + off));
          const bf16x8 tl = as_bf16x8(*reinterpret_cast<const u32x4*>(t_lo + off));
          acc[i][j] = mfma32(a, th, acc[i][j]);
          acc[i][j] = mfma32(a, tl, acc[i][j]);
        }
      }
    }
  }

  // ---- store: lane holds features nb + 8q + 4*hi + (0..3) of token m --------
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int m = m0 + wm * (BM / 2) + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int nb = n0 + wn * (BN / 2) + i * 32;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = nb + 8 * q + 4 * hi;
        u32x2 pk;
        pk[0] = pack_bf16x2(acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]);
        pk[1] = pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
        *reinterpret_cast<u32x2*>(out + (int64_t)m * N + n) = pk;
      }
    }
  }
}

// t = scale * x A^T for one token per wave; each lane accumulates its slice of
// the hidden dimension for every rank, then the wave reduces.

__global__ __launch_bounds__(256) void lora_down_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ a,
                                                        int n_tok, int hidden, int rank, int r_pad, float scale,
                                                        bf16_t* __restrict__ t_hi, bf16_t* __restrict__ t_lo) {
  const int lane = threadIdx.x & 63;
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= n_tok) return;
  const bf16_t* xr = x + (int64_t)tok * hidden;
  for (int j0 = 0; j0 < r_pad; j0 += 16) {
    float accj[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) accj[j] = 0.f;
    for (int k = lane * 8; k < hidden; k += 64 * 8) {
      const u32x4 xv = *reinterpret_cast<const u32x4*>(xr + k);
      float xf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xf[2 * e] = bf16_to_f32((bf16_t)(xv[e] & 0xFFFFu));
        xf[2 * e + 1] = bf16_to_f32((bf16_t)(xv[e] >> 16));
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if (j0 + j < rank) {
          const u32x4 av = *reinterpret_cast<const u32x4*>(a + (int64_t)(j0 + j) * hidden + k);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            accj[j] = fmaf(xf[2 * e], bf16_to_f32((bf16_t)(av[e] & 0xFFFFu)), accj[j]);
            accj[j] = fmaf(xf[2 * e + 1], bf16_to_f32((bf16_t)(av[e] >> 16)), accj[j]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float s = wave_sum(accj[j]) * scale;
      if (lane == j) {
        const bf16_t h = (j0 + j < rank) ? f32_to_bf16(s) : (bf16_t)0;
        const bf16_t l = (j0 + j < rank) ? f32_to_bf16(s - bf16_to_f32(h)) : (bf16_t)0;
        t_hi[(int64_t)tok * r_pad + j0 + j] = h;
        t_lo[(int64_t)tok * r_pad + j0 + j] = l;
      }
    }
  }
}

}  // namespace

hipError_t launch_lora_down(const uint16_t* x, const uint16_t* a, int n_tok, int hidden, int rank, int r_pad,
                            float scale, uint16_t* t_hi, uint16_t* t_lo, hipStream_t stream) {
  if (n_tok == 0 || r_pad == 0) return hipSuccess;
  hipLaunchKernelGGL(lora_down_kernel, dim3((n_tok + 3) / 4), dim3(256), 0, stream, x, a, n_tok, hidden, rank, r_pad,
                     scale, t_hi, t_lo);
  return hipGetLastError();
}

hipError_t launch_gemm_lora(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int hidden,
                            const uint16_t* b, int rank, int r_pad, int lora_cols, const uint16_t* t_hi,
                            const uint16_t* t_lo, uint16_t* out, hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  constexpr int BN = 128;
  const int n_nt = n_out / BN;
  // Prefer 128-token tiles once they alone give every CU two workgroups.
  const int n_mt128 = (n_tok + 127) / 128;
  if ((int64_t)n_mt128 * n_nt >= 512) {
    hipLaunchKernelGGL((gemm_lora_kernel<128, BN>), dim3(n_mt128 * n_nt), dim3(256), 0, stream, x, w, n_tok, n_out,
                       hidden, b, rank, r_pad, lora_cols, t_hi, t_lo, out, n_mt128, n_nt);
  } else {
    const int n_mt = (n_tok + 63) / 64;
    hipLaunchKernelGGL((gemm_lora_kernel<64, BN>), dim3(n_mt * n_nt), dim3(256), 0, stream, x, w, n_tok, n_out,
                       hidden, b, rank, r_pad, lora_cols, t_hi, t_lo, out, n_mt, n_nt);
  }
  return hipGetLastError();
}

}  // namespace attuner
