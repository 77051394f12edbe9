// K3: per-head QK-RMSNorm + RoPE of the suffix tokens (section 4: the adapted
// query passes through the model's own query normalisation and RoPE), and the
// write of the suffix keys and values into their request-cache rows.
//
// One wave per (token, head slot); slots 0..Hq-1 are query heads, Hq..Hq+Hkv-1
// are KV heads (normalise + rotate k, copy v).  Lane j holds the rotary pair
// (j, j + 64) of the head, so the rotation needs no data exchange and the
// RMS is one wave reduction.  Angles come from a host-built table of
// (cos, sin) of pos * theta^(-2j/128), evaluated in fp64 and stored fp32.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

__global__ __launch_bounds__(256) void qk_norm_rope_kernel(NormRopeParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n_slots = p.n_q_heads + p.n_kv_heads;
  const int tok = (int)(wid / n_slots);
  const int slot = (int)(wid - (int64_t)tok * n_slots);
  if (tok >= p.total_q) return;

  int r = 0;
  while (r + 1 < p.n_req && tok >= p.req[r + 1].q_start) ++r;
  const NormRopeReq rq = p.req[r];
  const int i = tok - rq.q_start;
  const int pos = rq.pos0 + i;

  const bool is_q = slot < p.n_q_heads;
  const int g = slot - p.n_q_heads;
  const bf16_t* src = is_q ? p.q_raw + (int64_t)tok * p.ld_q + slot * kHeadDim
                           : p.k_raw + (int64_t)tok * p.ld_kv + g * kHeadDim;
  const bf16_t* gam = is_q ? p.gamma_q : p.gamma_k;
  bf16_t* dst = is_q ? p.q_hat + ((int64_t)tok * p.n_q_heads + slot) * kHeadDim
                     : p.k_cache + g * p.kv_head_stride + (int64_t)(rq.kv_row0 + i) * kHeadDim;

  const float x0 = bf16_to_f32(src[lane]);
  const float x1 = bf16_to_f32(src[lane + 64]);
  const float ms = wave_sum(x0 * x0 + x1 * x1) * (1.0f / kHeadDim);
  const float inv = 1.0f / sqrtf(ms + p.eps);
  const float y0 = x0 * inv * bf16_to_f32(gam[lane]);
  const float y1 = x1 * inv * bf16_to_f32(gam[lane + 64]);
  const float2 cs = p.rope[(int64_t)pos * 64 + lane];
  dst[lane] = f32_to_bf16(y0 * cs.x - y1 * cs.y);
  dst[lane + 64] = f32_to_bf16(y1 * cs.x + y0 * cs.y);

  if (!is_q) {
    const bf16_t* vs = p.v_raw + (int64_t)tok * p.ld_kv + g * kHeadDim;
    bf16_t* vd = p.v_cache + g * p.kv_head_stride + (int64_t)(rq.kv_row0 + i) * kHeadDim;
    vd[lane] = vs[lane];
    vd[lane + 64] = vs[lane + 64];
  }
}

}  // namespace

hipError_t launch_qk_norm_rope(const NormRopeParams& p, hipStream_t stream) {
  if (p.total_q == 0) return hipSuccess;
  const int64_t waves = (int64_t)p.total_q * (p.n_q_heads + p.n_kv_heads);
  ATTUNER_LAUNCH("qk_norm_rope_kernel", qk_norm_rope_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), stream, p);
  return hipGetLastError();
}

}  // namespace attuner
