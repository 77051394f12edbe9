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
//   online softmax in the log2 domain: p = 2^(s * log2(e)/sqrt(d) - m) as one
//                FMA and one v_exp_f32; the O rescale is skipped when no row
//                max of the wave moved;
//   O^T += V^T P^T  (MFMA A = V^T, B = P^T straight from the S^T accumulator
//                converted to bf16 in registers).
// The S^T accumulator hands a lane the keys of each 16-key group in the order
// (4hf + 0..3, 8 + 4hf + 0..3), hf = lane / 32; the V^T operand is read in that
// same key order with the gfx950 LDS transpose read (ds_read_b64_tr_b16): a
// 16-lane group pointing at a 4-key x 16-dim block of the natural [key][d]
// tile receives one dimension per lane across the 4 keys.  So K and V both
// sit in LDS in their natural layout, written with 16-byte stores.
// LDS: K [2][64][16 chunks], V [2][64][16 chunks] (64 KiB per workgroup),
// double buffered with a register prefetch of the next tile.  16-byte chunks
// are XOR-swizzled by row (K: row & 15, for b128 operand reads of 16 rows;
// V: 4 * (row & 3), for transpose reads of 4 rows x 2 chunks).
//
// Work units of one KV head go to blockIdx.x = unit * Hkv + g: with Hkv = 8
// workgroups are dealt round-robin over the 8 XCDs, so each XCD's L2 serves a
// single KV head.  Late (heavier, causal) query blocks are dispatched first.
// With n_split > 1 the key range of a block is cut into n_split tile ranges;
// each writes a normalised fp32 partial and its (max, sum), and a second
// kernel merges them.  (Merging inside this kernel would need agent-scope
// release/acquire between workgroups, which on gfx950 writes back and
// invalidates the XCD's L2 and costs the other workgroups their K/V reuse.)

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int BQ = 32;
constexpr int BKV = 64;
constexpr int D = kHeadDim;
constexpr int CH = D / 8;  // 16-byte chunks per K/V row

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) bf16_t lds_bf16;
typedef float f32x2 __attribute__((ext_vector_type(2)));

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
    const bool ok = key < kv_len;
    const int64_t off = (int64_t)key * D + ch * 8;
    t.k[i] = ok ? *reinterpret_cast<const u32x4*>(kb + off) : u32x4{0u, 0u, 0u, 0u};
    t.v[i] = ok ? *reinterpret_cast<const u32x4*>(vb + off) : u32x4{0u, 0u, 0u, 0u};
  }
}

__device__ __forceinline__ void store_tile(const TileRegs& t, u32x4* __restrict__ ks, u32x4* __restrict__ vs,
                                           int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int row = c >> 4, ch = c & 15;
    ks[row * CH + (ch ^ (row & 15))] = t.k[i];
    vs[row * CH + (ch ^ ((row & 3) << 2))] = t.v[i];
  }
}

// O row (token qrow, head h) from the O^T accumulator: lane holds d =
// 32 db + 8 q + 4 hf + (0..3); also the natural-log LSE of the row.
__device__ __forceinline__ void store_output(const AttnParams& p, int64_t qrow, int h, int hf, const f32x16* acc,
                                             float scale, float m_log2, float l) {
  bf16_t* orow = p.o + (qrow * p.n_q_heads + h) * D;
#pragma unroll
  for (int db = 0; db < 4; ++db) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      u32x2 pr;
      pr[0] = pack_bf16x2(acc[db][4 * q] * scale, acc[db][4 * q + 1] * scale);
      pr[1] = pack_bf16x2(acc[db][4 * q + 2] * scale, acc[db][4 * q + 3] * scale);
      *reinterpret_cast<u32x2*>(orow + db * 32 + 8 * q + 4 * hf) = pr;
    }
  }
  if (p.lse != nullptr && hf == 0) p.lse[qrow * p.n_q_heads + h] = (m_log2 + __log2f(l)) * 0.69314718055994531f;
}

__global__ __launch_bounds__(256, 2) void attention_kernel(AttnParams p) {
  __shared__ u32x4 k_lds[2][BKV * CH];
  __shared__ u32x4 v_lds[2][BKV * CH];

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

  // transpose-read addressing of the V^T operand (see the header): lane r of
  // its 16-lane group points at key row (r >> 2) of a 4-key block and dims
  // d0 + 4 (r & 3) .. +3, d0 = 32 db + 16 * group.
  const int r16 = lane & 15;
  const int grp = (lane >> 4) & 1;
  const int vrow = r16 >> 2;  // == key & 3 of the row it reads
  int vcol[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int chunk = 4 * db + 2 * grp + ((r16 & 3) >> 1);
    vcol[db] = ((chunk ^ (vrow << 2)) << 3) + ((r16 & 1) << 2);
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
    store_tile(regs, k_lds[0], v_lds[0], tid);
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
          const bf16x8 a = as_bf16x8(k_lds[cur][row * CH + ((2 * ks + hf) ^ (row & 15))]);
          s[kh] = mfma32(a, qf[ks], s[kh]);
        }
      }

      // ---- mask + online softmax (log2 domain) -----------------------------
      if (kv0 + BKV - 1 > rq.art_len + t0) {
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kv0 + kh * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
            if (key > vis_lim) s[kh][v] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kh][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_i, mx * sc);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_i - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = __builtin_amdgcn_exp2f(fmaf(s[kh][v], sc, -m_use));
          s[kh][v] = e;
          rs += e;
        }
      rs += __shfl_xor(rs, 32, 64);
      l_i = l_i * alpha + rs;
      m_i = m_new;
      if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[db][v] *= alpha;
      }

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
      const lds_bf16* vbase = (const lds_bf16*)(v_lds[cur]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row_a = 16 * j + 4 * hf + vrow;  // keys 16j + 4hf + 0..3
        const int row_b = row_a + 8;                // keys 16j + 8 + 4hf + 0..3
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const v4i16 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_v4i16*)(vbase + row_a * D + vcol[db]));
          const v4i16 vbv = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_v4i16*)(vbase + row_b * D + vcol[db]));
          v4i16 lo = va, hi2 = vbv;
          typedef short v8i16 __attribute__((ext_vector_type(8)));
          const v8i16 a8 = __builtin_shufflevector(lo, hi2, 0, 1, 2, 3, 4, 5, 6, 7);
          acc[db] = mfma32(__builtin_bit_cast(bf16x8, a8), pk[j], acc[db]);
        }
      }

      if (tile + 1 < te) store_tile(regs, k_lds[cur ^ 1], v_lds[cur ^ 1], tid);
      __syncthreads();
    }
  }

  const float inv_l = l_i > 0.f ? 1.0f / l_i : 0.f;
  if (p.n_split == 1) {
    if (row_ok) store_output(p, qrow, h, hf, acc, inv_l, m_i, l_i);
    return;
  }

  // ---- split-KV: publish the normalised partial and its (max, sum) --------
  if (!row_ok) return;
  const int64_t prow = (int64_t)split * p.total_q * p.n_q_heads + qrow * p.n_q_heads + h;
  float* po = p.part_o + prow * D;
#pragma unroll
  for (int db = 0; db < 4; ++db) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = acc[db][4 * q + e] * inv_l;
      *reinterpret_cast<f32x4*>(po + db * 32 + 8 * q + 4 * hf) = v;
    }
  }
  if (hf == 0) *reinterpret_cast<f32x2*>(p.part_ml + prow * 2) = f32x2{m_i, l_i};
}

// Merge the n_split partials of one (token, head) per wave: weight of split s
// is l_s * 2^(m_s - max_s m_s); lane j owns output dims 2j, 2j + 1.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // token * Hq + head
  const int64_t stride = (int64_t)p.total_q * p.n_q_heads;
  if (row >= stride) return;
  float mmax = -INFINITY;
  for (int s = 0; s < p.n_split; ++s) mmax = fmaxf(mmax, p.part_ml[(s * stride + row) * 2]);
  float wsum = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll 4
  for (int s = 0; s < p.n_split; ++s) {
    const f32x2 ml = *reinterpret_cast<const f32x2*>(p.part_ml + (s * stride + row) * 2);
    const float w = (ml[0] == -INFINITY) ? 0.f : ml[1] * __builtin_amdgcn_exp2f(ml[0] - mmax);
    const f32x2 v = *reinterpret_cast<const f32x2*>(p.part_o + (s * stride + row) * D + 2 * lane);
    o0 = fmaf(w, v[0], o0);
    o1 = fmaf(w, v[1], o1);
    wsum += w;
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  *reinterpret_cast<uint32_t*>(p.o + row * D + 2 * lane) = pack_bf16x2(o0 * inv, o1 * inv);
  if (p.lse != nullptr && lane == 0) p.lse[row] = (mmax + __log2f(wsum)) * 0.69314718055994531f;
}

}  // namespace

hipError_t launch_attention(const AttnParams& p, hipStream_t stream) {
  if (p.n_units == 0) return hipSuccess;
  ATTUNER_LAUNCH("attention_kernel", attention_kernel, dim3((unsigned)(p.n_units * p.n_kv_heads)), dim3(256), stream,
                 p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_split == 1) return e;
  const int64_t rows = (int64_t)p.total_q * p.n_q_heads;
  ATTUNER_LAUNCH("attn_combine_kernel", attn_combine_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), stream, p);
  return hipGetLastError();
}

}  // namespace attuner
