// K4: multi-segment GQA flash attention over an assembled request cache
// (eq. 3 form: softmax(q K^T / sqrt(d) + M) V with the causal mask; appendix
// A.5: scaled dot-product attention over the assembled context).  Suffix row
// i of a request sees cache keys 0 .. art_len + i: every artifact key and the
// suffix causally.
//
// Work unit = (request, block of 32 suffix tokens, KV head g, key split).
// The workgroup's four waves are the four query heads that share KV head g,
// so every K/V tile staged in LDS serves 4 x 32 query rows.  Per 64-key tile:
//   S^T = K Q^T  (MFMA A = K rows from LDS, B = Q held in registers), so the
//                accumulator of a lane holds 32 keys of ONE token and the row
//                max / row sum are in-lane plus one exchange with lane ^ 32;
//   online softmax in the log2 domain (exp2 with log2(e)/sqrt(d) folded in);
//   O^T += V^T P^T  (MFMA A = V^T from LDS, B = P^T straight from the S^T
//                accumulator, converted to bf16 in registers).
// For the last step to need no data movement, V is written to LDS transposed
// ([d][key]) with the keys of each 16-key group in the order the S^T
// accumulator hands them to the MFMA: key quads (0, 2, 1, 3).
// LDS: K [2][64 keys][16 chunks] and V^T [2][128 d][8 chunks], double
// buffered with a register prefetch of the next tile (64 KiB per workgroup);
// chunks are XOR-swizzled by row so operand reads spread over the banks.
//
// Work units of one KV head go to blockIdx.x = unit * Hkv + g: with Hkv = 8
// workgroups are dealt round-robin over the 8 XCDs, so each XCD's L2 serves a
// single KV head.  Late (heavier, causal) query blocks are dispatched first.
// With n_split > 1 the key range of a block is cut into n_split tile ranges;
// each writes a normalised fp32 partial and its (max, sum), merged by
// attn_combine_kernel.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int BQ = 32;
constexpr int BKV = 64;
constexpr int D = kHeadDim;
constexpr int KCH = D / 8;    // 16-byte chunks per K row
constexpr int VCH = BKV / 8;  // 16-byte chunks per V^T row

struct TileRegs {
  u32x4 k[4];
  u32x4 v[4];
};

__device__ __forceinline__ void load_tile(TileRegs& t, const bf16_t* __restrict__ kb, const bf16_t* __restrict__ vb,
                                          int kv0, int kv_len, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int row = c >> 4, ch = c & 15;
    const int key = kv0 + row;
    t.k[i] = key < kv_len ? *reinterpret_cast<const u32x4*>(kb + (int64_t)key * D + ch * 8) : u32x4{0u, 0u, 0u, 0u};
  }
  const int quad = tid >> 4, dc = tid & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int key = kv0 + 4 * quad + i;
    t.v[i] = key < kv_len ? *reinterpret_cast<const u32x4*>(vb + (int64_t)key * D + dc * 8) : u32x4{0u, 0u, 0u, 0u};
  }
}

__device__ __forceinline__ void store_tile(const TileRegs& t, u32x4* __restrict__ ks, u32x2* __restrict__ vts,
                                           int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int row = c >> 4, ch = c & 15;
    ks[row * KCH + (ch ^ (row & 15))] = t.k[i];
  }
  // V: this thread holds keys 4*quad .. 4*quad+3 at d = 8*dc .. 8*dc+7; write
  // them as 8 rows of V^T, each 4 keys (8 bytes) wide.
  const int quad = tid >> 4, dc = tid & 15;
  const int grp = quad >> 2;                       // 16-key group
  const int pq = (0x3120 >> (4 * (quad & 3))) & 3; // key quad -> position quad: 0,2,1,3
  const int chunk = 2 * grp + (pq >> 1);
  const int half = pq & 1;
#pragma unroll
  for (int dd = 0; dd < 8; ++dd) {
    const int w = dd >> 1;
    const int sh = (dd & 1) * 16;
    const uint32_t e0 = (t.v[0][w] >> sh) & 0xFFFFu;
    const uint32_t e1 = (t.v[1][w] >> sh) & 0xFFFFu;
    const uint32_t e2 = (t.v[2][w] >> sh) & 0xFFFFu;
    const uint32_t e3 = (t.v[3][w] >> sh) & 0xFFFFu;
    const int d = 8 * dc + dd;
    u32x2 pr;
    pr[0] = e0 | (e1 << 16);
    pr[1] = e2 | (e3 << 16);
    vts[(d * VCH + (chunk ^ (d & 7))) * 2 + half] = pr;
  }
}

__global__ __launch_bounds__(256, 2) void attention_kernel(AttnParams p) {
  __shared__ u32x4 k_lds[2][BKV * KCH];
  __shared__ u32x4 vt_lds[2][D * VCH];

  const int hkv = p.n_kv_heads;
  const int g = blockIdx.x % hkv;
  int unit = blockIdx.x / hkv;
  int r = 0;
  while (r + 1 < p.n_req && unit >= p.req[r + 1].wg_start) ++r;
  const AttnReq rq = p.req[r];
  unit -= rq.wg_start;
  const int split = unit % p.n_split;
  const int qb = rq.n_qblk - 1 - unit / p.n_split;
  const int t0 = qb * BQ;
  const int blk_rows = min(BQ, rq.q_len - t0);
  const int kv_len = rq.art_len + t0 + blk_rows;  // keys any row of the block sees
  const int n_tiles = (kv_len + BKV - 1) / BKV;
  const int per = (n_tiles + p.n_split - 1) / p.n_split;
  const int tb = min(n_tiles, split * per);
  const int te = min(n_tiles, tb + per);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int h = g * 4 + wave;
  const int t = t0 + l32;  // this lane's suffix token (index within the request)
  const bool row_ok = l32 < blk_rows;
  const int64_t qrow = (int64_t)(rq.q_start + t);

  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row_ok) v = *reinterpret_cast<const u32x4*>(p.q + (qrow * p.n_q_heads + h) * D + ks * 16 + hf * 8);
    qf[ks] = as_bf16x8(v);
  }

  const bf16_t* kb = p.k + g * p.kv_head_stride + (int64_t)rq.kv_start * D;
  const bf16_t* vb = p.v + g * p.kv_head_stride + (int64_t)rq.kv_start * D;

  float m_i = -INFINITY, l_i = 0.f;
  f32x16 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x16{};

  const float sc = p.score_scale;
  const int vis_lim = rq.art_len + t;  // last visible key of this row

  if (tb < te) {
    TileRegs regs;
    load_tile(regs, kb, vb, tb * BKV, kv_len, tid);
    store_tile(regs, k_lds[0], reinterpret_cast<u32x2*>(vt_lds[0]), tid);
    __syncthreads();

    for (int tile = tb; tile < te; ++tile) {
      const int cur = (tile - tb) & 1;
      const int kv0 = tile * BKV;
      if (tile + 1 < te) load_tile(regs, kb, vb, kv0 + BKV, kv_len, tid);

      // ---- S^T = K Q^T --------------------------------------------------
      f32x16 s[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        s[kh] = f32x16{};
        const int row = kh * 32 + l32;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const bf16x8 a = as_bf16x8(k_lds[cur][row * KCH + ((2 * ks + hf) ^ (row & 15))]);
          s[kh] = mfma32(a, qf[ks], s[kh]);
        }
      }

      // ---- mask + online softmax (log2 domain) -----------------------------
      const bool need_mask = kv0 + BKV - 1 > rq.art_len + t0;
      float mx = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float z = s[kh][v] * sc;
          if (need_mask) {
            const int key = kv0 + kh * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
            if (key > vis_lim) z = -INFINITY;
          }
          s[kh][v] = z;
          mx = fmaxf(mx, z);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_i, mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_i - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = exp2f(s[kh][v] - m_use);
          s[kh][v] = e;
          rs += e;
        }
      }
      rs += __shfl_xor(rs, 32, 64);
      l_i = l_i * alpha + rs;
      m_i = m_new;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[db][v] *= alpha;

      // ---- O^T += V^T P^T -------------------------------------------------
      bf16x8 pk[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = pack_bf16x2(s[j >> 1][(j & 1) * 8 + 2 * e], s[j >> 1][(j & 1) * 8 + 2 * e + 1]);
        pk[j] = as_bf16x8(w);
      }
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int d = db * 32 + l32;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bf16x8 a = as_bf16x8(vt_lds[cur][d * VCH + ((2 * j + hf) ^ (d & 7))]);
          acc[db] = mfma32(a, pk[j], acc[db]);
        }
      }

      if (tile + 1 < te) store_tile(regs, k_lds[cur ^ 1], reinterpret_cast<u32x2*>(vt_lds[cur ^ 1]), tid);
      __syncthreads();
    }
  }

  if (!row_ok) return;
  const float inv_l = l_i > 0.f ? 1.0f / l_i : 0.f;
  if (p.n_split == 1) {
    bf16_t* orow = p.o + (qrow * p.n_q_heads + h) * D;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        u32x2 pr;
        pr[0] = pack_bf16x2(acc[db][4 * q] * inv_l, acc[db][4 * q + 1] * inv_l);
        pr[1] = pack_bf16x2(acc[db][4 * q + 2] * inv_l, acc[db][4 * q + 3] * inv_l);
        *reinterpret_cast<u32x2*>(orow + db * 32 + 8 * q + 4 * hf) = pr;
      }
    }
    if (p.lse != nullptr && hf == 0) p.lse[qrow * p.n_q_heads + h] = (m_i + log2f(l_i)) * 0.69314718055994531f;
  } else {
    const int64_t prow = ((int64_t)split * p.total_q + qrow) * p.n_q_heads + h;
    float* po = p.part_o + prow * D;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v;
        v[0] = acc[db][4 * q] * inv_l;
        v[1] = acc[db][4 * q + 1] * inv_l;
        v[2] = acc[db][4 * q + 2] * inv_l;
        v[3] = acc[db][4 * q + 3] * inv_l;
        *reinterpret_cast<f32x4*>(po + db * 32 + 8 * q + 4 * hf) = v;
      }
    }
    if (hf == 0) {
      p.part_ml[prow * 2] = m_i;
      p.part_ml[prow * 2 + 1] = l_i;
    }
  }
}

// Merge the n_split partials of one (token, head) per wave: weights
// l_s * 2^(m_s - max m); lane j owns output dims 2j, 2j + 1.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // token * Hq + head
  if (row >= (int64_t)p.total_q * p.n_q_heads) return;
  const int64_t stride = (int64_t)p.total_q * p.n_q_heads;
  float mmax = -INFINITY;
  for (int s = 0; s < p.n_split; ++s) mmax = fmaxf(mmax, p.part_ml[(s * stride + row) * 2]);
  float wsum = 0.f, o0 = 0.f, o1 = 0.f;
  for (int s = 0; s < p.n_split; ++s) {
    const float m = p.part_ml[(s * stride + row) * 2];
    const float l = p.part_ml[(s * stride + row) * 2 + 1];
    const float w = (m == -INFINITY) ? 0.f : l * exp2f(m - mmax);
    const float2 v = *reinterpret_cast<const float2*>(p.part_o + (s * stride + row) * D + 2 * lane);
    o0 = fmaf(w, v.x, o0);
    o1 = fmaf(w, v.y, o1);
    wsum += w;
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  *reinterpret_cast<uint32_t*>(p.o + row * D + 2 * lane) = pack_bf16x2(o0 * inv, o1 * inv);
  if (p.lse != nullptr && lane == 0) p.lse[row] = (mmax + log2f(wsum)) * 0.69314718055994531f;
}

}  // namespace

hipError_t launch_attention(const AttnParams& p, hipStream_t stream) {
  if (p.n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(attention_kernel, dim3((unsigned)(p.n_units * p.n_kv_heads)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn_combine(const AttnParams& p, hipStream_t stream) {
  const int64_t rows = (int64_t)p.total_q * p.n_q_heads;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace attuner
