// Row kernels of the decoder layer around the path: the embedding lookup of
// the suffix tokens, the hidden-size RMSNorm (the layer's input and
// post-attention norms and the final norm) and the greedy pick of the first
// generated token over the vocabulary.
//
// embed_rows_kernel: one wave per token; out[t] = table[ids[t]] as 16-byte
// copies (dim a multiple of 8).
//
// rms_norm_rows_kernel: one wave per row; lane l holds the 16-byte chunks l,
// l + 64, ... of the row (all of it stays in registers), the sum of squares
// is an in-lane sum plus a wave reduction, and the output is written from
// the same registers.  dim is a multiple of 8 and at most 64 * 8 * kMaxPass.
//
// argmax: 64 workgroups per row each scan a slice of the row's 16-byte groups
// keeping (largest value, smallest index), reduced in the wave and through
// LDS; a second one-wave launch per row reduces the 64 slice results.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int kMaxPass = 16;  // dim <= 8192

__global__ __launch_bounds__(256) void embed_rows_kernel(const bf16_t* __restrict__ table,
                                                         const int32_t* __restrict__ ids, int n_tok, int dim,
                                                         bf16_t* __restrict__ out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_tok) return;
  const int lane = threadIdx.x & 63;
  const u32x4* src = reinterpret_cast<const u32x4*>(table + (int64_t)ids[t] * dim);
  u32x4* dst = reinterpret_cast<u32x4*>(out + (int64_t)t * dim);
  for (int c = lane; c < dim / 8; c += 64) dst[c] = src[c];
}

__global__ __launch_bounds__(256) void rms_norm_rows_kernel(const bf16_t* __restrict__ x, int64_t ld_x,
                                                            const int32_t* __restrict__ rows, int n_rows, int dim,
                                                            const bf16_t* __restrict__ gamma, float eps,
                                                            bf16_t* __restrict__ out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= n_rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t src_row = rows != nullptr ? rows[r] : r;
  const bf16_t* xr = x + src_row * ld_x;
  const int n_chunk = dim / 8;
  u32x4 v[kMaxPass], g[kMaxPass];
  float ss = 0.f;
  // every load first, gamma's with the row's (one round trip; chunks past
  // the row read as zeros, which add nothing), then the squares
#pragma unroll
  for (int k = 0; k < kMaxPass; ++k) {
    const int c = lane + 64 * k;
    v[k] = u32x4{0u, 0u, 0u, 0u};
    g[k] = v[k];
    if (c < n_chunk) {
      v[k] = *reinterpret_cast<const u32x4*>(xr + 8 * c);
      g[k] = *reinterpret_cast<const u32x4*>(gamma + 8 * c);
    }
  }
#pragma unroll
  for (int k = 0; k < kMaxPass; ++k) ss = accum_squares(ss, v[k]);
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)dim + eps);
  bf16_t* orow = out + (int64_t)r * dim;
#pragma unroll
  for (int k = 0; k < kMaxPass; ++k) {
    const int c = lane + 64 * k;
    if (c >= n_chunk) continue;
    *reinterpret_cast<u32x4*>(orow + 8 * c) = norm_chunk(v[k], g[k], inv);
  }
}

// (value, index) order: larger value first, then smaller index
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

constexpr int kArgmaxSlices = 64;  // workgroups per row in the first pass

__device__ __forceinline__ void wave_best(float& bv, int& bi) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
}

// First pass: workgroup (slice, row) finds the best (value, index) of its
// slice of the row's 16-byte groups (the last slice also takes the values
// past the last whole group).
__global__ __launch_bounds__(256) void argmax_slices_kernel(const float* __restrict__ logits, int n,
                                                            float* __restrict__ part_v, int32_t* __restrict__ part_i) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int sl = blockIdx.x;
  const float* row = logits + (int64_t)blockIdx.y * n;
  const int n4 = n / 4;
  const int per = (n4 + kArgmaxSlices - 1) / kArgmaxSlices;
  const int g0 = sl * per, g1 = min(n4, g0 + per);
  float bv = -INFINITY;
  int bi = n;  // no element seen
  for (int g = g0 + (int)threadIdx.x; g < g1; g += 256) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(row + 4 * g);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (better(v[e], 4 * g + e, bv, bi)) {
        bv = v[e];
        bi = 4 * g + e;
      }
  }
  if (sl == kArgmaxSlices - 1)
    for (int i = 4 * n4 + threadIdx.x; i < n; i += 256)
      if (better(row[i], i, bv, bi)) {
        bv = row[i];
        bi = i;
      }
  wave_best(bv, bi);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (better(sv[w], si[w], bv, bi)) {
        bv = sv[w];
        bi = si[w];
      }
    part_v[(int64_t)blockIdx.y * kArgmaxSlices + sl] = bv;
    part_i[(int64_t)blockIdx.y * kArgmaxSlices + sl] = bi;
  }
}

// Second pass: one wave per row over its slices' results.  The slices are
// disjoint index ranges, so the (value, smallest index) order gives the
// row's argmax whatever the order of the reduction.
__global__ __launch_bounds__(64) void argmax_merge_kernel(const float* __restrict__ part_v,
                                                          const int32_t* __restrict__ part_i, int n,
                                                          int32_t* __restrict__ ids, float* __restrict__ max_out) {
  float bv = part_v[(int64_t)blockIdx.x * kArgmaxSlices + threadIdx.x];
  int bi = part_i[(int64_t)blockIdx.x * kArgmaxSlices + threadIdx.x];
  wave_best(bv, bi);
  if (threadIdx.x == 0) {
    ids[blockIdx.x] = bi < n ? bi : 0;  // a row of NaNs only: index 0
    if (max_out != nullptr) max_out[blockIdx.x] = bv;
  }
}

}  // namespace

hipError_t launch_embed_rows(const uint16_t* table, const int32_t* ids, int n_tok, int dim, uint16_t* out,
                             hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  if (dim % 8 != 0) return hipErrorInvalidValue;
  ATTUNER_LAUNCH("embed_rows_kernel", embed_rows_kernel, dim3((unsigned)((n_tok + 3) / 4)), dim3(256), stream, table,
                 ids, n_tok, dim, out);
  return hipGetLastError();
}

hipError_t launch_rms_norm_rows(const uint16_t* x, int64_t ld_x, const int32_t* rows, int n_rows, int dim,
                                const uint16_t* gamma, float eps, uint16_t* out, hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  if (dim % 8 != 0 || dim > 64 * 8 * kMaxPass) return hipErrorInvalidValue;
  ATTUNER_LAUNCH("rms_norm_rows_kernel", rms_norm_rows_kernel, dim3((unsigned)((n_rows + 3) / 4)), dim3(256), stream,
                 x, ld_x, rows, n_rows, dim, gamma, eps, out);
  return hipGetLastError();
}

size_t argmax_scratch_bytes(int n_rows) { return (size_t)n_rows * kArgmaxSlices * (sizeof(float) + sizeof(int32_t)); }

hipError_t launch_argmax_rows(const float* logits, int n_rows, int n, int32_t* ids, float* max_out, void* scratch,
                              hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  float* part_v = static_cast<float*>(scratch);
  int32_t* part_i = reinterpret_cast<int32_t*>(part_v + (size_t)n_rows * kArgmaxSlices);
  ATTUNER_LAUNCH("argmax_slices_kernel", argmax_slices_kernel, dim3(kArgmaxSlices, (unsigned)n_rows), dim3(256),
                 stream, logits, n, part_v, part_i);
  ATTUNER_LAUNCH("argmax_merge_kernel", argmax_merge_kernel, dim3((unsigned)n_rows), dim3(kArgmaxSlices), stream,
                 part_v, part_i, n, ids, max_out);
  return hipGetLastError();
}

}  // namespace attuner

namespace attuner {

namespace {

// Deployment form of the adapter: w_out[n] = w[n] + scale * sum_j b[n][j] a[j]
// for rows n < lora_cols (one bf16 rounding of the fp32 sum), w_out[n] = w[n]
// otherwise.  Workgroup = one row; thread = 16-byte chunks of it.
__global__ __launch_bounds__(256) void merge_lora_kernel(const bf16_t* __restrict__ w, int k_dim,
                                                         const bf16_t* __restrict__ a, const bf16_t* __restrict__ b,
                                                         int rank, float scale, int lora_cols, bf16_t* w_out) {
  const int n = blockIdx.x;
  const bf16_t* wr = w + (int64_t)n * k_dim;
  bf16_t* orow = w_out + (int64_t)n * k_dim;
  const bool adapt = n < lora_cols;
  for (int c = threadIdx.x; c < k_dim / 8; c += 256) {
    const u32x4 wv = *reinterpret_cast<const u32x4*>(wr + 8 * c);
    if (!adapt) {
      *reinterpret_cast<u32x4*>(orow + 8 * c) = wv;
      continue;
    }
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < rank; ++j) {
      const float bj = bf16_to_f32(b[(int64_t)n * rank + j]);
      const u32x4 av = *reinterpret_cast<const u32x4*>(a + (int64_t)j * k_dim + 8 * c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = fmaf(bj, __uint_as_float(av[e] << 16), acc[2 * e]);
        acc[2 * e + 1] = fmaf(bj, __uint_as_float(av[e] & 0xFFFF0000u), acc[2 * e + 1]);
      }
    }
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = pack_bf16x2(__uint_as_float(wv[e] << 16) + scale * acc[2 * e],
                         __uint_as_float(wv[e] & 0xFFFF0000u) + scale * acc[2 * e + 1]);
    *reinterpret_cast<u32x4*>(orow + 8 * c) = o;
  }
}

}  // namespace

hipError_t launch_merge_lora(const uint16_t* w, int n_out, int k_dim, const uint16_t* a, const uint16_t* b, int rank,
                             float scale, int lora_cols, uint16_t* w_out, hipStream_t stream) {
  if (n_out == 0) return hipSuccess;
  if (k_dim % 8 != 0) return hipErrorInvalidValue;
  ATTUNER_LAUNCH("merge_lora_kernel", merge_lora_kernel, dim3((unsigned)n_out), dim3(256), stream, w, k_dim, a, b,
                 rank, scale, lora_cols, w_out);
  return hipGetLastError();
}

}  // namespace attuner
