// Decode attention: one new token per request attends to every key of its
// assembled cache (the artifacts, the suffix and the tokens generated so far,
// its own key included).  Generated tokens keep the adapted query projection
// (section 4: the adapter acts on every online token), so a decode step is
// the one-row case of eq. 3 over the request's whole context.
//
// One row per request reads each cached K/V byte once and does 4 flops per
// byte pair, so the kernel streams HBM: the 4 query heads of a KV head share
// every K/V load, the keys of a request are cut into chunks (split-KV), and
// the arithmetic runs on the vector ALU (an MFMA tile would be 1/8 full).
//
// decode_attention_kernel: workgroup = (request, KV head g, key chunk), 256
// threads = 32 key groups of 8 lanes.  Lane `sub` of a group holds dims
// 8 sub .. 8 sub + 7 and 64 + 8 sub .. 64 + 8 sub + 7 of the 4 query rows
// (bf16 pairs) and of the 4 output accumulators (fp32); a wave's K (and V)
// load instruction covers 8 whole 128-byte lines of 8 consecutive keys.  Per
// key: q . k as bf16 dot2 products, summed over the group's 8 lanes with
// DPP; online softmax in the log2 domain per step of 2 keys; o += p v; the
// loads of the next step are in flight during the arithmetic of this one.
// The 32 groups then merge through LDS.  A request with one chunk writes O
// (bf16); otherwise each chunk writes its unnormalised O and (max, sum) in
// fp32 and decode_combine_kernel merges the chunks of the request.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

ATTUNER_VIOLATION_WORD(g_violations_decode, read_violations_decode_impl)

constexpr int D = kHeadDim;
constexpr int G = 4;                // query heads per KV head
constexpr int LPK = 8;              // lanes per key
constexpr int NTH = 256;
constexpr int GROUPS = NTH / LPK;   // keys per workgroup per sub-step
constexpr int U = 2;                // keys per group per step
constexpr float kNegBig = -1.0e30f;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// Sum over the 8 lanes of a key group (lanes 8j .. 8j + 7): swap neighbours,
// swap pairs (quad permutations), then add the mirrored half-row.
__device__ __forceinline__ float sum8(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x141, 0xF, 0xF, false));
  return x;
}

__device__ __forceinline__ float lo_f(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_f(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

__global__ __launch_bounds__(NTH) void decode_attention_kernel(const DecodeParams p) {
  __shared__ float s_o[GROUPS][G][D];
  __shared__ f32x2 s_ml[GROUPS][G];

  const int hkv = p.n_kv_heads;
  const int g = blockIdx.x % hkv;
  const int sid = blockIdx.x / hkv;
  int r = 0;
  while (r + 1 < p.n_req && sid >= p.req[r + 1].split0) ++r;
  const DecodeReq rq = p.req[r];
  const int k0 = (sid - rq.split0) * p.chunk;
  const int k1 = min(rq.n_keys, k0 + p.chunk);
  if constexpr (kChecked) {
    // the request's keys lie inside its cache plane
    if (rq.kv_start < 0 || rq.n_keys < 1 || (int64_t)rq.kv_start + rq.n_keys > p.kv_head_stride / D) {
      if (threadIdx.x == 0) ATTUNER_VIOLATE(g_violations_decode, kViolDecodeRange);
      return;
    }
  }
  const int grp = threadIdx.x >> 3;
  const int sub = threadIdx.x & 7;

  bf16_t* kbase = p.k + g * p.kv_head_stride + (int64_t)rq.kv_start * D;
  bf16_t* vbase = p.v + g * p.kv_head_stride + (int64_t)rq.kv_start * D;
  // Steps of U keys per group, double-buffered: the loads of step i + 1 are
  // issued before the arithmetic of step i.
  struct Buf {
    u32x4 ka[U], kc[U], va[U], vc[U];
  };
  auto load = [&](int key0, Buf& b) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int key = min(key0 + u * GROUPS, k1 - 1);  // past the chunk: a valid row, masked below
      const bf16_t* kr = kbase + (int64_t)key * D;
      const bf16_t* vr = vbase + (int64_t)key * D;
      b.ka[u] = *reinterpret_cast<const u32x4*>(kr + 8 * sub);
      b.kc[u] = *reinterpret_cast<const u32x4*>(kr + 64 + 8 * sub);
      b.va[u] = *reinterpret_cast<const u32x4*>(vr + 8 * sub);
      b.vc[u] = *reinterpret_cast<const u32x4*>(vr + 64 + 8 * sub);
    }
  };
  // The first step's keys and values are requested before the query
  // prologue, which they do not depend on; the workgroup whose chunk holds
  // the new key requests them after writing that key's row (below).
  const bool last = sid - rq.split0 == rq.n_split - 1;
  const int key_first = k0 + grp;
  Buf b0, b1;
  if (!last) load(key_first, b0);

  // The new token's 4 query rows of this KV head, normalised and rotated
  // from the raw projection (every key group derives them: a few hundred
  // ALU operations against the chunk's stream), in the layout of the key
  // loads: dims 8 sub .. 8 sub + 7 and their rotary partners 64 + 8 sub ...
  f32x4 cs[4];
  {
    const f32x4* cs4 = reinterpret_cast<const f32x4*>(p.rope + (int64_t)rq.pos * 64 + 8 * sub);
#pragma unroll
    for (int e = 0; e < 4; ++e) cs[e] = cs4[e];
  }
  const bf16_t* qrow = p.q_raw + (int64_t)rq.q_row * p.ld_q + g * G * D;
  const u32x4 gqa = *reinterpret_cast<const u32x4*>(p.gamma_q + 8 * sub);
  const u32x4 gqb = *reinterpret_cast<const u32x4*>(p.gamma_q + 64 + 8 * sub);
  u32x4 qa[G], qb[G];
#pragma unroll
  for (int h = 0; h < G; ++h)
    head_norm_rope(*reinterpret_cast<const u32x4*>(qrow + h * D + 8 * sub),
                   *reinterpret_cast<const u32x4*>(qrow + h * D + 64 + 8 * sub), gqa, gqb, cs, p.eps, qa[h], qb[h]);
  // The workgroup whose chunk holds the last key (the new token's) normalises
  // and rotates that key and writes it and its value into their cache row
  // before its key loop reads the row (the workgroup barrier orders the
  // writes of group 0 before every group's loads); no other workgroup reads
  // the row.
  if (last) {
    if (grp == 0) {
      const bf16_t* kr = p.k_raw + (int64_t)rq.q_row * p.ld_kv + g * D;
      const bf16_t* vr = p.v_raw + (int64_t)rq.q_row * p.ld_kv + g * D;
      u32x4 ka, kb;
      head_norm_rope(*reinterpret_cast<const u32x4*>(kr + 8 * sub), *reinterpret_cast<const u32x4*>(kr + 64 + 8 * sub),
                     *reinterpret_cast<const u32x4*>(p.gamma_k + 8 * sub),
                     *reinterpret_cast<const u32x4*>(p.gamma_k + 64 + 8 * sub), cs, p.eps, ka, kb);
      const int64_t row = (int64_t)(rq.n_keys - 1) * D;
      *reinterpret_cast<u32x4*>(kbase + row + 8 * sub) = ka;
      *reinterpret_cast<u32x4*>(kbase + row + 64 + 8 * sub) = kb;
      *reinterpret_cast<u32x4*>(vbase + row + 8 * sub) = *reinterpret_cast<const u32x4*>(vr + 8 * sub);
      *reinterpret_cast<u32x4*>(vbase + row + 64 + 8 * sub) = *reinterpret_cast<const u32x4*>(vr + 64 + 8 * sub);
      __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));  // the stores have reached the cache
    }
    __syncthreads();
    load(key_first, b0);
  }

  float m[G], l[G], o[G][16];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = kNegBig;
    l[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) o[h][i] = 0.f;
  }

  auto step = [&](int key0, const Buf& b) __attribute__((always_inline)) {
    float sc[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool valid = key0 + u * GROUPS < k1;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = dot2(qa[h][e], b.ka[u][e], acc);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = dot2(qb[h][e], b.kc[u][e], acc);
        acc = sum8(acc);
        sc[u][h] = valid ? acc * p.score_scale : kNegBig;
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mb = sc[0][h];
#pragma unroll
      for (int u = 1; u < U; ++u) mb = fmaxf(mb, sc[u][h]);
      if (mb > m[h]) {
        const float alpha = exp2f(m[h] - mb);
        l[h] *= alpha;
#pragma unroll
        for (int i = 0; i < 16; ++i) o[h][i] *= alpha;
        m[h] = mb;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[16];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[2 * e] = lo_f(b.va[u][e]);
        vf[2 * e + 1] = hi_f(b.va[u][e]);
        vf[8 + 2 * e] = lo_f(b.vc[u][e]);
        vf[8 + 2 * e + 1] = hi_f(b.vc[u][e]);
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float pr = exp2f(sc[u][h] - m[h]);
        l[h] += pr;
#pragma unroll
        for (int i = 0; i < 16; ++i) o[h][i] = fmaf(pr, vf[i], o[h][i]);
      }
    }
  };

  constexpr int STEP = GROUPS * U;
  int key0 = key_first;
  if (key0 < k1) {
    while (true) {
      if (key0 + STEP < k1) load(key0 + STEP, b1);
      step(key0, b0);
      key0 += STEP;
      if (key0 >= k1) break;
      if (key0 + STEP < k1) load(key0 + STEP, b0);
      step(key0, b1);
      key0 += STEP;
      if (key0 >= k1) break;
    }
  }

  // merge the 32 key groups: every group's (m, l) and O slice through LDS
#pragma unroll
  for (int h = 0; h < G; ++h) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s_o[grp][h][8 * sub + i] = o[h][i];
      s_o[grp][h][64 + 8 * sub + i] = o[h][8 + i];
    }
    if (sub == 0) s_ml[grp][h] = f32x2{m[h], l[h]};
  }
  __syncthreads();
  const int h = threadIdx.x >> 6;
  const int d = 2 * (threadIdx.x & 63);
  float mm = kNegBig;
#pragma unroll 8
  for (int j = 0; j < GROUPS; ++j) mm = fmaxf(mm, s_ml[j][h][0]);
  float ll = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll 8
  for (int j = 0; j < GROUPS; ++j) {
    const f32x2 ml = s_ml[j][h];
    const float w = exp2f(ml[0] - mm);
    ll = fmaf(w, ml[1], ll);
    o0 = fmaf(w, s_o[j][h][d], o0);
    o1 = fmaf(w, s_o[j][h][d + 1], o1);
  }
  const int qh = g * G + h;
  if (rq.n_split == 1) {
    const float inv = 1.0f / ll;
    *reinterpret_cast<uint32_t*>(p.o + ((int64_t)rq.q_row * p.n_q_heads + qh) * D + d) = pack_bf16x2(o0 * inv, o1 * inv);
  } else {
    const int64_t row = (int64_t)sid * p.n_q_heads + qh;
    *reinterpret_cast<f32x2*>(p.part_o + row * D + d) = f32x2{o0, o1};
    if ((threadIdx.x & 63) == 0) *reinterpret_cast<f32x2*>(p.part_ml + row * 2) = f32x2{mm, ll};
  }
}

// Merge the chunks of each request with more than one: workgroup = (request,
// query head); its 256 threads are 8 chunk groups of 32 lanes (4 dims each),
// group j merging chunks j, j + 8, ... with the loads of up to 8 chunks in
// flight, then the 8 groups merge through LDS.
constexpr int CG = 8;     // chunk groups per workgroup
constexpr int CB = 8;     // chunks loaded per group before merging

__global__ __launch_bounds__(NTH) void decode_combine_kernel(const DecodeParams p) {
  __shared__ f32x4 s_o[CG][32];
  __shared__ f32x2 s_ml[CG];
  const int qh = blockIdx.x % p.n_q_heads;
  const DecodeReq rq = p.req[blockIdx.x / p.n_q_heads];
  if (rq.n_split <= 1) return;
  const int cg = threadIdx.x >> 5;
  const int ln = threadIdx.x & 31;
  float m = kNegBig, l = 0.f;
  f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = cg; s0 < rq.n_split; s0 += CG * CB) {
    f32x2 ml[CB];
    f32x4 ov[CB];
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      const int s = min(s0 + b * CG, rq.n_split - 1);
      const int64_t row = (int64_t)(rq.split0 + s) * p.n_q_heads + qh;
      ml[b] = *reinterpret_cast<const f32x2*>(p.part_ml + row * 2);
      ov[b] = *reinterpret_cast<const f32x4*>(p.part_o + row * D + 4 * ln);
    }
    float mb = m;
#pragma unroll
    for (int b = 0; b < CB; ++b)
      if (s0 + b * CG < rq.n_split) mb = fmaxf(mb, ml[b][0]);
    const float alpha = exp2f(m - mb);
    l *= alpha;
    o *= alpha;
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      if (s0 + b * CG >= rq.n_split) continue;
      const float w = exp2f(ml[b][0] - mb);
      l = fmaf(w, ml[b][1], l);
      o += w * ov[b];
    }
    m = mb;
  }
  s_o[cg][ln] = o;
  if (ln == 0) s_ml[cg] = f32x2{m, l};
  __syncthreads();
  if (threadIdx.x >= 32) return;
  float mm = kNegBig;
#pragma unroll
  for (int j = 0; j < CG; ++j) mm = fmaxf(mm, s_ml[j][0]);
  float ll = 0.f;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < CG; ++j) {
    const float w = exp2f(s_ml[j][0] - mm);
    ll = fmaf(w, s_ml[j][1], ll);
    acc += w * s_o[j][ln];
  }
  const float inv = 1.0f / ll;
  u32x2 pk;
  pk[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  pk[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(p.o + ((int64_t)rq.q_row * p.n_q_heads + qh) * D + 4 * ln) = pk;
}

}  // namespace

hipError_t read_violations_decode(unsigned int* bits, bool reset) {
  return read_violations_decode_impl(bits, reset);
}

hipError_t launch_decode_attention(const DecodeParams& p, hipStream_t stream) {
  if (p.total_splits == 0) return hipSuccess;
  if (p.n_q_heads != G * p.n_kv_heads) return hipErrorInvalidValue;
  ATTUNER_LAUNCH("decode_attention_kernel", decode_attention_kernel, dim3((unsigned)(p.total_splits * p.n_kv_heads)),
                 dim3(NTH), stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.total_splits > p.n_req) {
    ATTUNER_LAUNCH("decode_combine_kernel", decode_combine_kernel, dim3((unsigned)(p.n_req * p.n_q_heads)), dim3(NTH),
                   stream, p);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace attuner
