// K3: per-head QK-RMSNorm + RoPE of the suffix tokens (section 4: the base
// model's q-norm and rotary embedding apply to the adapted query as they
// would to the plain one), and the
// write of the suffix keys and values into their request-cache rows.
//
// Eight lanes per (token, head slot); slots 0..Hq-1 are query heads,
// Hq..Hq+Hkv-1 are KV heads (normalise + rotate k, copy v).  Lane j of a group
// holds dimensions 8j..8j+7 and their rotary partners 64+8j..64+8j+7 (two
// 16-byte loads), so the rotation needs no data exchange and the RMS is an
// in-lane sum plus three exchanges within the group.  Angles come from a
// host-built table of (cos, sin) of pos * theta^(-2j/128), evaluated in fp64
// and stored fp32.  Rows, gamma and outputs are 16-byte aligned.  The
// arithmetic (head_norm_rope) is shared with the decode kernel, which applies
// it to the new token inside its own launch.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

__global__ __launch_bounds__(256) void qk_norm_rope_kernel(NormRopeParams p) {
  const int lane8 = threadIdx.x & 7;
  const int64_t grp = (int64_t)blockIdx.x * 32 + (threadIdx.x >> 3);
  const int n_slots = p.n_q_heads + p.n_kv_heads;
  const int tok = (int)(grp / n_slots);
  const int slot = (int)(grp - (int64_t)tok * n_slots);
  if (tok >= p.total_q) return;  // whole 8-lane groups leave together

  // the request of this token: a constant-offset argument read (scalar) for a
  // single request, a per-lane search otherwise
  NormRopeReq rq;
  if (p.n_req == 1) {
    rq = p.req[0];
  } else {
    int r = 0;
    while (r + 1 < p.n_req && tok >= p.req[r + 1].q_start) ++r;
    rq = p.req[r];
  }
  const int i = tok - rq.q_start;
  const int pos = rq.pos0 + i;

  const bool is_q = slot < p.n_q_heads;
  const int g = slot - p.n_q_heads;
  const bf16_t* src = is_q ? p.q_raw + (int64_t)tok * p.ld_q + slot * kHeadDim
                           : p.k_raw + (int64_t)tok * p.ld_kv + g * kHeadDim;
  const bf16_t* gam = is_q ? p.gamma_q : p.gamma_k;
  bf16_t* dst = is_q ? p.q_hat + ((int64_t)tok * p.n_q_heads + slot) * kHeadDim
                     : p.k_cache + g * p.kv_head_stride + (int64_t)(rq.kv_row0 + i) * kHeadDim;
  const int j0 = 8 * lane8;

  // every load of the lane first (row, gamma, angles and, for a KV slot, the
  // value row): one memory round trip
  const u32x4 xa = *reinterpret_cast<const u32x4*>(src + j0);
  const u32x4 xb = *reinterpret_cast<const u32x4*>(src + 64 + j0);
  const u32x4 ga = *reinterpret_cast<const u32x4*>(gam + j0);
  const u32x4 gb = *reinterpret_cast<const u32x4*>(gam + 64 + j0);
  const f32x4* cs4 = reinterpret_cast<const f32x4*>(p.rope + (int64_t)pos * 64 + j0);
  f32x4 cs[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) cs[e] = cs4[e];  // (cos, sin) of pairs j0 + 2e and j0 + 2e + 1
  u32x4 va = u32x4{0u, 0u, 0u, 0u}, vb = u32x4{0u, 0u, 0u, 0u};
  if (!is_q) {
    const bf16_t* vs = p.v_raw + (int64_t)tok * p.ld_kv + g * kHeadDim;
    va = *reinterpret_cast<const u32x4*>(vs + j0);
    vb = *reinterpret_cast<const u32x4*>(vs + 64 + j0);
  }
  u32x4 oa, ob;
  head_norm_rope(xa, xb, ga, gb, cs, p.eps, oa, ob);
  *reinterpret_cast<u32x4*>(dst + j0) = oa;
  *reinterpret_cast<u32x4*>(dst + 64 + j0) = ob;

  if (!is_q) {
    bf16_t* vd = p.v_cache + g * p.kv_head_stride + (int64_t)(rq.kv_row0 + i) * kHeadDim;
    *reinterpret_cast<u32x4*>(vd + j0) = va;
    *reinterpret_cast<u32x4*>(vd + 64 + j0) = vb;
  }
}

}  // namespace

hipError_t launch_qk_norm_rope(const NormRopeParams& p, hipStream_t stream) {
  if (p.total_q == 0) return hipSuccess;
  const int64_t groups = (int64_t)p.total_q * (p.n_q_heads + p.n_kv_heads);  // 8 lanes each
  ATTUNER_LAUNCH("qk_norm_rope_kernel", qk_norm_rope_kernel, dim3((unsigned)((groups + 31) / 32)), dim3(256), stream,
                 p);
  return hipGetLastError();
}

}  // namespace attuner
