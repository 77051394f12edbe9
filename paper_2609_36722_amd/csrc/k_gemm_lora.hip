// K2: bf16 MFMA projection GEMM with the rank-r LoRA update fused into its
// epilogue (query-side adaptation, section 4 eq. 4):
//   out[i][n] = x[i] . w[n]  +  (n < lora_cols ? t[i] . b[n] : 0),
//   t = scale * x A^T  (lora_down_kernel, run first).
//
// The GEMM is computed as C^T = W x^T so that the MFMA accumulator of a lane
// holds four consecutive output features of one token (8-byte stores).  Both
// operands are K-contiguous in memory ([rows][hidden]), so tiles go to LDS
// without a transpose.  Workgroup tile BN (features) x BM (tokens) x 64 (k),
// four waves (WN along features x 4/WN along tokens), 32x32x16 MFMAs, fp32
// accumulation.  The k-loop
// keeps NS k-tiles in flight in a register ring (the small-token shapes of
// suffix prefill are latency-bound, not bandwidth-bound) and double-buffers
// LDS.  LDS rows are 128 bytes (eight 16-byte chunks); chunk c of row r is
// stored at c ^ ((r >> 1) & 7), so the 16 rows one operand read touches in a
// cycle land on 16 distinct bank groups.
//
// The LoRA term enters as extra MFMA k-steps after the main loop: A operand
// = rows of B (rank padded to 16 with zeros), B operand = t rounded to a
// bf16 hi/lo pair, so t keeps ~16 significant bits and the update is summed
// in fp32.  lora_down_kernel leaves t as fp32 partial sums over 256-wide
// slices of the hidden dimension; the epilogue adds the slices in order.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int BK = 64;
constexpr int kChunksPerRow = BK / 8;  // 16-byte chunks per LDS row
constexpr int kLoraSlice = 256;        // hidden elements per lora_down workgroup

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

template <int BM, int BN, int WN, int NS>
__global__ __launch_bounds__(256, 2) void gemm_lora_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w,
                                                           int M, int N, int K, const bf16_t* __restrict__ b,
                                                           int rank, int r_pad, int lora_cols,
                                                           const float* __restrict__ t_part, int n_slice,
                                                           bf16_t* __restrict__ out, int n_mt, int n_nt) {
  constexpr int WM = 4 / WN;            // waves along tokens (WN along features)
  constexpr int TN = BN / WN, TM = BM / WM;  // wave tile
  constexpr int FN = TN / 32;           // 32-row MFMA blocks per wave along features
  constexpr int FM = TM / 32;           // along tokens
  static_assert(FN >= 1 && FM >= 1 && WN * WM == 4, "bad wave layout");
  constexpr int ROWS = BN + BM;
  constexpr int LOADS = ROWS * kChunksPerRow / 256;  // 16-byte chunks per thread per k-tile
  static_assert(ROWS * kChunksPerRow % 256 == 0, "tile must split evenly over 256 threads");

  __shared__ u32x4 lds[2][ROWS * kChunksPerRow];

  // XCD-aware tile order: workgroup i runs on XCD i % 8, so give each XCD a
  // contiguous run of tiles; consecutive tiles share weight rows.
  const int total = n_mt * n_nt;
  const int per_xcd = total >> 3;
  int lin = blockIdx.x;
  if (lin < 8 * per_xcd) lin = (lin & 7) * per_xcd + (lin >> 3);
  const int nt = lin / n_mt;
  const int mt = lin - nt * n_mt;
  const int n0 = nt * BN;
  const int m0 = mt * BM;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave / WM;  // wave position along features
  const int wm = wave % WM;  // along tokens
  const int l32 = lane & 31;
  const int hi = lane >> 5;

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

  // n_kt is a multiple of NS (the launcher picks NS so); every load and LDS
  // store below is unconditional (tile indices clamped), which keeps the
  // compiler's wait counting exact: only the oldest ring slot is waited for.
  const int n_kt = K / BK;
  u32x4 ring[NS][LOADS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int i = 0; i < LOADS; ++i) ring[s][i] = src[i][s * kChunksPerRow];
#pragma unroll
  for (int i = 0; i < LOADS; ++i) lds[0][dst[i]] = ring[0][i];
  __syncthreads();

  for (int kt0 = 0; kt0 < n_kt; kt0 += NS) {
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int kt = kt0 + u;
      // ring[u] (tile kt) is already in LDS: refill it with tile kt + NS
      const int nxt = min(kt + NS, n_kt - 1);
#pragma unroll
      for (int i = 0; i < LOADS; ++i) ring[u][i] = src[i][nxt * kChunksPerRow];
      const int cur = kt & 1;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = 2 * ks + hi;
        bf16x8 af[FN], bfr[FM];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int row = wn * TN + i * 32 + l32;
          af[i] = as_bf16x8(lds[cur][row * kChunksPerRow + swz(row, ch)]);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          const int row = BN + wm * TM + j * 32 + l32;
          bfr[j] = as_bf16x8(lds[cur][row * kChunksPerRow + swz(row, ch)]);
        }
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j) acc[i][j] = mfma32(af[i], bfr[j], acc[i][j]);
      }
      // tile kt + 1 (ring slot u + 1) into the other LDS buffer; after the last
      // tile this stores a stale tile nobody reads
#pragma unroll
      for (int i = 0; i < LOADS; ++i) lds[cur ^ 1][dst[i]] = ring[(u + 1) % NS][i];
      __syncthreads();
    }
  }

  // ---- fused low-rank epilogue: acc += B[n][:] . t[m][:] --------------------
  if (r_pad > 0 && n0 < lora_cols) {
    const int64_t slice_stride = (int64_t)M * r_pad;
    for (int ks = 0; ks < r_pad; ks += 16) {
      bf16x8 th[FM], tl[FM];
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        int m = m0 + wm * TM + j * 32 + l32;
        m = m < M ? m : M - 1;
        const float* tp = t_part + (int64_t)m * r_pad + ks + 8 * hi;
        f32x4 s0 = f32x4{}, s1 = f32x4{};
        for (int z = 0; z < n_slice; ++z) {
          s0 += *reinterpret_cast<const f32x4*>(tp + z * slice_stride);
          s1 += *reinterpret_cast<const f32x4*>(tp + z * slice_stride + 4);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const __bf16 h0 = static_cast<__bf16>(s0[e]);
          const __bf16 h1 = static_cast<__bf16>(s1[e]);
          th[j][e] = h0;
          th[j][e + 4] = h1;
          tl[j][e] = static_cast<__bf16>(s0[e] - static_cast<float>(h0));
          tl[j][e + 4] = static_cast<__bf16>(s1[e] - static_cast<float>(h1));
        }
      }
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const int nb = n0 + wn * TN + i * 32;
        if (nb >= lora_cols) continue;  // lora_cols is a multiple of 32
        const int n = nb + l32;
        bf16x8 a;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int jj = ks + 8 * hi + e;
          const bf16_t bv = jj < rank ? b[(int64_t)n * rank + jj] : (bf16_t)0;
          a[e] = __builtin_bit_cast(__bf16, bv);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          acc[i][j] = mfma32(a, th[j], acc[i][j]);
          acc[i][j] = mfma32(a, tl[j], acc[i][j]);
        }
      }
    }
  }

  // ---- store: lane holds features nb + 8q + 4*hi + (0..3) of token m --------
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int m = m0 + wm * TM + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int nb = n0 + wn * TN + i * 32;
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

// t = scale * x A^T with MFMAs, as fp32 partial sums per 256-wide slice of the
// hidden dimension: workgroup (32-token block, slice), each wave multiplies a
// 64-wide part of the slice and the four waves are summed through LDS.
// t_part[slice][token][r_pad]; ranks rank .. r_pad-1 come out zero.
__global__ __launch_bounds__(256) void lora_down_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ a,
                                                        int n_tok, int hidden, int rank, int r_pad, float scale,
                                                        float* __restrict__ t_part) {
  __shared__ float red[4][2][16][64];
  const int mb = blockIdx.x, kz = blockIdx.y;
  const int m0 = mb * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int nblk = (r_pad + 31) / 32;
  const int m = min(m0 + l32, n_tok - 1);
  const bf16_t* xr = x + (int64_t)m * hidden;

  u32x4 xa[4], ab[4][2];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const int k = kz * kLoraSlice + wave * 64 + st * 16 + 8 * hf;
    const bool kin = k < hidden;
    xa[st] = kin ? *reinterpret_cast<const u32x4*>(xr + k) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int n = 32 * nb + l32;
      ab[st][nb] = (kin && nb < nblk && n < rank) ? *reinterpret_cast<const u32x4*>(a + (int64_t)n * hidden + k)
                                                 : u32x4{0u, 0u, 0u, 0u};
    }
  }
  f32x16 acc[2] = {f32x16{}, f32x16{}};
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
      if (nb < nblk) acc[nb] = mfma32(as_bf16x8(xa[st]), as_bf16x8(ab[st][nb]), acc[nb]);
  // acc[nb][v] = C[token 8(v/4) + 4hf + v%4][rank 32nb + l32]
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) red[wave][nb][v][lane] = acc[nb][v];
  __syncthreads();

  for (int e = tid; e < nblk * 1024; e += 256) {
    const int nb = e >> 10, v = (e >> 6) & 15, ln = e & 63;
    const int tok = m0 + 8 * (v >> 2) + 4 * (ln >> 5) + (v & 3);
    const int rk = 32 * nb + (ln & 31);
    if (tok < n_tok && rk < r_pad)
      t_part[((int64_t)kz * n_tok + tok) * r_pad + rk] =
          scale * (red[0][nb][v][ln] + red[1][nb][v][ln] + red[2][nb][v][ln] + red[3][nb][v][ln]);
  }
}

}  // namespace

int lora_down_slices(int hidden) { return (hidden + kLoraSlice - 1) / kLoraSlice; }

hipError_t launch_lora_down(const uint16_t* x, const uint16_t* a, int n_tok, int hidden, int rank, int r_pad,
                            float scale, float* t_part, hipStream_t stream) {
  if (n_tok == 0 || r_pad == 0) return hipSuccess;
  ATTUNER_LAUNCH("lora_down_kernel", lora_down_kernel, dim3((n_tok + 31) / 32, lora_down_slices(hidden)), dim3(256),
                 stream, x, a, n_tok, hidden, rank, r_pad, scale, t_part);
  return hipGetLastError();
}

hipError_t launch_gemm_lora(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int hidden,
                            const uint16_t* b, int rank, int r_pad, int lora_cols, const float* t_part,
                            uint16_t* out, hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  const int n_slice = lora_down_slices(hidden);
  // Tile choice (measured on gfx950 at hidden 2560, 6144 outputs): 128x128
  // tiles once they alone give every CU two workgroups; 64 tokens x 128
  // features with a 4-deep prefetch for mid-size suffixes; 64x64 tiles with an
  // 8-deep prefetch when even that leaves most CUs idle (the weight stream is
  // latency-bound there).  The prefetch depth must divide the number of
  // 64-wide k-tiles; n_out is a multiple of 128.
  const int n_kt = hidden / BK;
  const int n_mt128 = (n_tok + 127) / 128;
  const int n_mt64 = (n_tok + 63) / 64;
  const int n_nt128 = n_out / 128;
#define ATTUNER_GEMM(BM_, BN_, WN_, NS_)                                                                          \
  ATTUNER_LAUNCH("gemm_lora_kernel", (gemm_lora_kernel<BM_, BN_, WN_, NS_>),                                      \
                 dim3(((n_tok + (BM_) - 1) / (BM_)) * (n_out / (BN_))), dim3(256), stream, x, w, n_tok, n_out,     \
                 hidden, b, rank, r_pad, lora_cols, t_part, n_slice, out, (n_tok + (BM_) - 1) / (BM_), n_out / (BN_))
#define ATTUNER_GEMM_NS(BM_, BN_, WN_, NSMAX_)          \
  if (n_kt % (NSMAX_) == 0) ATTUNER_GEMM(BM_, BN_, WN_, NSMAX_);        \
  else if (n_kt % 4 == 0) ATTUNER_GEMM(BM_, BN_, WN_, 4);               \
  else if (n_kt % 2 == 0) ATTUNER_GEMM(BM_, BN_, WN_, 2);               \
  else ATTUNER_GEMM(BM_, BN_, WN_, 1);
  if ((int64_t)n_mt128 * n_nt128 >= 512) {
    if (n_kt % 2 == 0) ATTUNER_GEMM(128, 128, 2, 2);
    else ATTUNER_GEMM(128, 128, 2, 1);
  } else if ((int64_t)n_mt64 * n_nt128 >= 128) {
    ATTUNER_GEMM_NS(64, 128, 2, 4)
  } else {
    ATTUNER_GEMM_NS(64, 64, 2, 8)
  }
#undef ATTUNER_GEMM_NS
#undef ATTUNER_GEMM
  return hipGetLastError();
}

}  // namespace attuner
