// Projection for a few tokens (decode: one new token per request): out =
// x W^T with the same epilogue modes and low-rank update as the GEMM, for
// n_tok <= kGemvMaxTok.  With a handful of tokens each weight is used once
// per token, so the launch streams W from HBM and an MFMA tile would be
// mostly empty: a group of KW waves owns two consecutive output rows, its
// lanes read 16-byte chunks of both rows (consecutive lanes, consecutive
// chunks: whole 128-byte lines; the KW waves take every KW-th 1 KB piece of
// the rows, so a long row is cut into fewer sequential load batches) and of
// every token's x, accumulate bf16 dot2 products in fp32, and the rows' sums
// meet in a wave reduction (and, for KW > 1, in LDS).  The low-rank term
// (rows below lora_cols) enters before the reduction: lane j of the group's
// first wave adds t[token][j] * B[row][j], t = scale * x A^T summed once per
// workgroup (into LDS) from the slice partials of the down-projection kernel.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// t[i] = sum over the n_slice slice partials p[z * stride + i], added in slice
// order; the loads go out sixteen at a time (one round trip for up to 16
// slices, i.e. a hidden size up to 4096; missing slices add zero)
__device__ __forceinline__ float slice_sum(const float* __restrict__ p, int n_slice, int64_t stride, int64_t i) {
  float tv = 0.f;
  for (int z = 0; z < n_slice; z += 16) {
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = z + u < n_slice ? p[(z + u) * stride + i] : 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) tv += v[u];
  }
  return tv;
}

// 16-byte chunks per row and lane in flight: fewer for more tokens, which
// each add a chunk of x per chunk of W
template <int T>
constexpr int chunk_batch() {
  return T <= 8 ? 4 : 2;
}

// The operands go through scalar parameters: a bit cast applied to a vector
// element expression directly reads element 0 whatever the index (seen with
// this compiler).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

__device__ __forceinline__ float dot8(u32x4 a, u32x4 b, float c) {
#pragma unroll
  for (int e = 0; e < 4; ++e) c = dot2(a[e], b[e], c);
  return c;
}

template <int T, int KW>
__global__ __launch_bounds__(256) void gemv_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, int N,
                                                   int K, const bf16_t* __restrict__ b, int rank, int r_pad,
                                                   int lora_cols, const float* __restrict__ t_part, int n_slice,
                                                   GemmEpi epi, bf16_t* out) {
  constexpr int kGroups = 4 / KW;      // row pairs per workgroup
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int kp = wave % KW;            // which pieces of the rows this wave takes
  const int n0 = (blockIdx.x * kGroups + wave / KW) * 2;
  // t = scale * x A^T for the workgroup's rows (all below lora_cols or none:
  // lora_cols is a multiple of 32, a workgroup owns at most 8 rows), summed
  // once from the slice partials into LDS by all threads
  __shared__ float t_lds[T][64];
  __shared__ f32x2 part[4][T];
  const bool lora_rows = r_pad > 0 && (int)blockIdx.x * 2 * kGroups < lora_cols;
  if (lora_rows) {
    for (int i = threadIdx.x; i < T * r_pad; i += 256) {
      const int t = i / r_pad, j = i % r_pad;
      t_lds[t][j] = slice_sum(t_part, n_slice, (int64_t)T * r_pad, (int64_t)t * r_pad + j);
    }
    __syncthreads();
  }
  const int nc = K / 8;
  auto xchunk = [&](int t, int c) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(x + (int64_t)t * K + 8 * c);
  };
  const bf16_t* w0 = w + (int64_t)n0 * K;
  const bf16_t* w1 = w0 + K;

  float acc[2][T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[0][t] = acc[1][t] = 0.f;

  // whole batches of kChunkBatch chunks per lane (all loads issued, then the
  // products), then the chunks left one at a time
  constexpr int kChunkBatch = chunk_batch<T>();
  constexpr int kStride = 64 * KW;
  int c = lane + 64 * kp;
  for (; c + kStride * (kChunkBatch - 1) < nc; c += kStride * kChunkBatch) {
    u32x4 wa[kChunkBatch], wb[kChunkBatch], xv[kChunkBatch][T];
#pragma unroll
    for (int j = 0; j < kChunkBatch; ++j) {
      const int cj = c + kStride * j;
      wa[j] = *reinterpret_cast<const u32x4*>(w0 + 8 * cj);
      wb[j] = *reinterpret_cast<const u32x4*>(w1 + 8 * cj);
#pragma unroll
      for (int t = 0; t < T; ++t) xv[j][t] = xchunk(t, cj);
    }
#pragma unroll
    for (int j = 0; j < kChunkBatch; ++j)
#pragma unroll
      for (int t = 0; t < T; ++t) {
        acc[0][t] = dot8(wa[j], xv[j][t], acc[0][t]);
        acc[1][t] = dot8(wb[j], xv[j][t], acc[1][t]);
      }
  }
  for (; c < nc; c += kStride) {
    const u32x4 wa = *reinterpret_cast<const u32x4*>(w0 + 8 * c);
    const u32x4 wb = *reinterpret_cast<const u32x4*>(w1 + 8 * c);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const u32x4 xv = xchunk(t, c);
      acc[0][t] = dot8(wa, xv, acc[0][t]);
      acc[1][t] = dot8(wb, xv, acc[1][t]);
    }
  }

  // rows below lora_cols: lane j < rank of the group's first wave adds
  // t[token][j] * B[row][j]
  if (lora_rows && kp == 0 && lane < rank) {
    const float b0 = bf16_to_f32(b[(int64_t)n0 * rank + lane]);
    const float b1 = bf16_to_f32(b[(int64_t)(n0 + 1) * rank + lane]);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      acc[0][t] = fmaf(t_lds[t][lane], b0, acc[0][t]);
      acc[1][t] = fmaf(t_lds[t][lane], b1, acc[1][t]);
    }
  }

  float y0 = 0.f, y1 = 0.f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const float s0 = wave_sum(acc[0][t]);
    const float s1 = wave_sum(acc[1][t]);
    if (lane == t) {
      y0 = s0;
      y1 = s1;
    }
  }
  if (KW > 1) {
    // the group's waves meet in LDS; its first wave finishes the rows
    if (lane < T) part[wave][lane] = f32x2{y0, y1};
    __syncthreads();
    if (kp != 0) return;
    if (lane < T) {
#pragma unroll
      for (int q = 1; q < KW; ++q) {
        y0 += part[wave + q][lane][0];
        y1 += part[wave + q][lane][1];
      }
    }
  }
  if (lane >= T) return;
  const int t = lane;
  if (epi.mode == kEpiF32) {
    *reinterpret_cast<f32x2*>(epi.out_f32 + (int64_t)t * N + n0) = f32x2{y0, y1};
    return;
  }
  if (epi.mode == kEpiSwiglu) {
    // rows n0 (gate j) and n0 + 1 (up j), j = n0 / 2
    out[(int64_t)t * (N / 2) + n0 / 2] = f32_to_bf16(y0 / (1.0f + __expf(-y0)) * y1);
    return;
  }
  if (epi.mode == kEpiResidual) {
    const uint32_t r = *reinterpret_cast<const uint32_t*>(epi.residual + (int64_t)t * N + n0);
    y0 += __uint_as_float(r << 16);
    y1 += __uint_as_float(r & 0xFFFF0000u);
  }
  *reinterpret_cast<uint32_t*>(out + (int64_t)t * N + n0) = pack_bf16x2(y0, y1);
}

// The same product on the matrix cores, for more tokens: with 16 tokens the
// dot-product form reads every x chunk again for each row pair (x traffic
// 8 times W's), while a 16 x 16 x 32 MFMA takes 16 tokens against 16 rows at
// once.  Workgroup = 16 output rows; lane l of a wave loads 64 contiguous
// bytes of row l % 16 and of token l % 16's x at k offset 32 (l / 16) of a
// 128-wide batch, and the four 16-byte pieces feed four MFMAs (the product
// sums over k, so any k order shared by both operands is exact).  The eight
// waves take every eighth batch and meet in LDS; tokens past n_tok are zero.
template <int CB, int NW>
__global__ __launch_bounds__(64 * NW) void gemv_mfma_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w,
                                                        int T, int N, int K, const bf16_t* __restrict__ b, int rank,
                                                        int r_pad, int lora_cols, const float* __restrict__ t_part,
                                                        int n_slice, GemmEpi epi, bf16_t* out) {
  __shared__ float t_lds[16][64];
  __shared__ f32x4 part[NW][64];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int n0 = blockIdx.x * 16;
  const bool lora_rows = r_pad > 0 && n0 < lora_cols;  // lora_cols % 32 == 0: all 16 rows or none
  if (lora_rows) {
    for (int i = threadIdx.x; i < T * r_pad; i += 64 * NW) {
      const int t = i / r_pad, j = i % r_pad;
      t_lds[t][j] = slice_sum(t_part, n_slice, (int64_t)T * r_pad, (int64_t)t * r_pad + j);
    }
  }
  const int col = lane & 15, grp = lane >> 4;
  const bool tok_ok = col < T;
  const bf16_t* wr = w + (int64_t)(n0 + col) * K + 32 * grp;
  const bf16_t* xr = x + (int64_t)min(col, T - 1) * K + 32 * grp;
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
  // wave 0 adds the low-rank term at the end: its B row (rank <= 16) is
  // requested now, with the weights
  constexpr int kPreRank = 16;
  float bpre[kPreRank];
  const bool pre = lora_rows && wave == 0 && rank <= kPreRank;
  if (pre) {
#pragma unroll
    for (int j = 0; j < kPreRank; ++j) bpre[j] = j < rank ? bf16_to_f32(b[(int64_t)(n0 + col) * rank + j]) : 0.f;
  }
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nb = K / 128;
  int bi = wave;
  for (; bi + NW * (CB - 1) < nb; bi += NW * CB) {
    u32x4 wv[CB][4], xv[CB][4];
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int kb = (bi + NW * j) * 128;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wv[j][e] = *reinterpret_cast<const u32x4*>(wr + kb + 8 * e);
        xv[j][e] = *reinterpret_cast<const u32x4*>(xr + kb + 8 * e);
      }
    }
#pragma unroll
    for (int j = 0; j < CB; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(tok_ok ? xv[j][e] : zero), as_bf16x8(wv[j][e]), acc,
                                                      0, 0, 0);
  }
  for (; bi < nb; bi += NW) {
    const int kb = bi * 128;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const u32x4 wv = *reinterpret_cast<const u32x4*>(wr + kb + 8 * e);
      const u32x4 xv = *reinterpret_cast<const u32x4*>(xr + kb + 8 * e);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(tok_ok ? xv : zero), as_bf16x8(wv), acc, 0, 0, 0);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  // acc[v] = C[token 4 grp + v][row n0 + col]
  const int n = n0 + col;
  float y[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    y[v] = part[0][lane][v];
#pragma unroll
    for (int q = 1; q < NW; ++q) y[v] += part[q][lane][v];
  }
  if (pre) {
#pragma unroll
    for (int j = 0; j < kPreRank; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (j < rank && 4 * grp + v < T) y[v] = fmaf(t_lds[4 * grp + v][j], bpre[j], y[v]);
  } else if (lora_rows) {
    for (int j = 0; j < rank; ++j) {
      const float bj = bf16_to_f32(b[(int64_t)n * rank + j]);
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (4 * grp + v < T) y[v] = fmaf(t_lds[4 * grp + v][j], bj, y[v]);
    }
  }
  float yp[4];  // the partner row's value (row n ^ 1, lane l ^ 1): SwiGLU pairs
#pragma unroll
  for (int v = 0; v < 4; ++v) yp[v] = __shfl_xor(y[v], 1, 64);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int t = 4 * grp + v;
    if (t >= T) continue;
    if (epi.mode == kEpiF32) {
      epi.out_f32[(int64_t)t * N + n] = y[v];
    } else if (epi.mode == kEpiSwiglu) {
      if ((col & 1) == 0) out[(int64_t)t * (N / 2) + n / 2] = f32_to_bf16(y[v] / (1.0f + __expf(-y[v])) * yp[v]);
    } else if (epi.mode == kEpiResidual) {
      out[(int64_t)t * N + n] = f32_to_bf16(y[v] + bf16_to_f32(epi.residual[(int64_t)t * N + n]));
    } else {
      out[(int64_t)t * N + n] = f32_to_bf16(y[v]);
    }
  }
}

// From this many tokens the matrix-core form (k_dim % 128 == 0, n_out % 16
// == 0) replaces the dot-product one.
constexpr int kGemvMfmaMinTok = 9;

// Waves per row pair (measured on the model's projection shapes): one for
// more than 8 tokens, whose x chunks already fill the loads in flight; else
// four for long rows (K >= 8192, or K >= 4096 from 4 tokens on), two
// otherwise.
int gemv_kw(int n_tok, int k_dim) {
  if (n_tok > 8) return 1;
  if (k_dim >= 8192 || (n_tok >= 4 && k_dim >= 4096)) return 4;
  return 2;
}

}  // namespace

hipError_t launch_gemv(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int k_dim, const uint16_t* b,
                       int rank, int r_pad, int lora_cols, const float* t_part, GemmEpi epi, uint16_t* out,
                       hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  if (n_tok > kGemvMaxTok || n_out % 8 != 0 || k_dim % 8 != 0 || (r_pad > 0 && t_part == nullptr))
    return hipErrorInvalidValue;
  const int n_slice = lora_down_slices(k_dim, n_tok);
  if (n_tok >= kGemvMfmaMinTok && k_dim % 128 == 0 && n_out % 16 == 0) {
    ATTUNER_LAUNCH("gemv_mfma_kernel", (gemv_mfma_kernel<2, 8>), dim3((unsigned)(n_out / 16)), dim3(512), stream, x, w,
                   n_tok, n_out, k_dim, b, rank, r_pad, lora_cols, t_part, n_slice, epi, out);
    return hipGetLastError();
  }
  const int kw = gemv_kw(n_tok, k_dim);
  const dim3 grid((unsigned)(n_out * kw / 8));
#define ATTUNER_GEMV_KW(T_, KW_)                                                                             \
  ATTUNER_LAUNCH("gemv_kernel", (gemv_kernel<T_, KW_>), grid, dim3(256), stream, x, w, n_out, k_dim, b, rank, \
                 r_pad, lora_cols, t_part, n_slice, epi, out)
#define ATTUNER_GEMV_SMALL(T_) \
  case T_:                     \
    if (kw == 4)               \
      ATTUNER_GEMV_KW(T_, 4);  \
    else                       \
      ATTUNER_GEMV_KW(T_, 2);  \
    break;
#define ATTUNER_GEMV_LARGE(T_) \
  case T_:                     \
    ATTUNER_GEMV_KW(T_, 1);    \
    break;
  switch (n_tok) {
    ATTUNER_GEMV_SMALL(1)
    ATTUNER_GEMV_SMALL(2)
    ATTUNER_GEMV_SMALL(3)
    ATTUNER_GEMV_SMALL(4)
    ATTUNER_GEMV_SMALL(5)
    ATTUNER_GEMV_SMALL(6)
    ATTUNER_GEMV_SMALL(7)
    ATTUNER_GEMV_SMALL(8)
    ATTUNER_GEMV_LARGE(9)
    ATTUNER_GEMV_LARGE(10)
    ATTUNER_GEMV_LARGE(11)
    ATTUNER_GEMV_LARGE(12)
    ATTUNER_GEMV_LARGE(13)
    ATTUNER_GEMV_LARGE(14)
    ATTUNER_GEMV_LARGE(15)
    ATTUNER_GEMV_LARGE(16)
    default: return hipErrorInvalidValue;
  }
#undef ATTUNER_GEMV_KW
#undef ATTUNER_GEMV_SMALL
#undef ATTUNER_GEMV_LARGE
  return hipGetLastError();
}

}  // namespace attuner
