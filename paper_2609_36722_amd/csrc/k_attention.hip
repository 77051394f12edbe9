// K4: multi-segment GQA flash attention over an assembled request cache
// (eq. 3 form: softmax(q K^T / sqrt(d) + M) V with the causal mask; appendix
// A.5: scaled dot-product attention over the assembled context).  Suffix row
// i of a request sees cache keys 0 .. art_len + i: every artifact key and the
// suffix causally.  Rows of several online spans of one prompt may share a
// request entry (packed back to back): each row then sees the keys up to its
// own position, which only grows from row to row.
//
// Work unit = (request, block of 64 suffix tokens, KV head g, key split), one
// workgroup of eight waves: the four query heads that share KV head g times
// two 32-token halves, so every K/V tile staged in LDS serves 256 query rows.
// K/V tiles (64 keys) are copied global -> LDS by the DMA form of the load
// (global_load_lds, 16 bytes per lane) into a four-stage ring: while tile i
// is multiplied and tile i - 1 finishes, tiles i+1 and i+2 are in flight, with
// no staging registers and one barrier per tile.  Per tile and wave:
//   S^T = K Q^T  (MFMA A = K rows from LDS, B = Q held in registers), so the
//                accumulator of a lane holds 32 keys of ONE token and the row
//                max / row sum are in-lane plus one exchange with lane ^ 32;
//   online softmax in the log2 domain: p = 2^(s * log2(e)/sqrt(d) - m) as one
//                FMA and one v_exp_f32.  Only a range's first tile and the
//                masked diagonal tiles take a row max; the other tiles use
//                the current reference m, and only if some tile's p sum
//                passes a bound does the workgroup run its key range again
//                with a row max per tile, so neither the max nor the O
//                rescale costs anything in the common case.
//                Each lane sums p over its own 32 keys of a tile into its
//                partial l; the two lanes of a token combine their partials
//                once at the end;
//   O^T += V^T P^T  (MFMA A = V^T, B = P^T straight from the S^T accumulator
//                converted to bf16 in registers).
// The loop is software-pipelined inside each wave: QK of tile i is issued
// next to the exponentials of tile i - 1, and PV of tile i - 1 next to the row
// max of tile i, so that each MFMA has vector-ALU work beside it that does
// not depend on it (gfx950 overlaps the two only in part, measured at about
// 60% of the MFMA time).  Tiles reaching the causal diagonal take a plain
// masked step.
// The S^T accumulator hands a lane the keys of each 16-key group in the order
// (4hf + 0..3, 8 + 4hf + 0..3), hf = lane / 32; the V^T operand is read in that
// same key order with the gfx950 LDS transpose read (ds_read_b64_tr_b16): a
// 16-lane group pointing at a 4-key x 16-dim block of the natural [key][d]
// tile receives one dimension per lane across the 4 keys.  16-byte chunks are
// XOR-swizzled by row (K: row & 15, for b128 operand reads of 16 rows; V:
// 4 * (row & 3), for transpose reads of 4 rows x 2 chunks): no bank conflicts.
//
// Work units of one KV head go to blockIdx.x = unit * Hkv + g: with Hkv = 8
// workgroups are dealt round-robin over the 8 XCDs, so each XCD's L2 serves a
// single KV head.  Late (heavier, causal) query blocks are dispatched first.
// With key splits the key range of a block is cut into its request's n_split
// tile ranges; each writes its normalised partial (bf16) and (max, sum)
// (fp32), and a second kernel merges them.  (Merging inside this kernel would need
// agent-scope release/acquire between workgroups, which on gfx950 writes back
// and invalidates the XCD's L2 and costs the other workgroups their K/V reuse.)
//
// A second instantiation (GATHER) also copies another layer's artifact pages
// from the pool into the request cache, so that a layer-by-layer prefill has
// layer l + 1's cache assembled by the end of layer l's attention: each wave
// moves 1 KiB chunks through three LDS slots of its own with the same DMA
// form of the load, issued after a tile's K/V copies, and stores each chunk
// from LDS three tiles later.

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

ATTUNER_VIOLATION_WORD(g_violations_attn, read_violations_attn_impl)

constexpr int BQ = 64;       // suffix tokens per workgroup (two 32-token halves)
constexpr int BKV = 64;      // keys per tile
constexpr int NSTAGE = 4;    // K/V tiles in LDS: i - 1 (its PV), i (its QK), i + 1 and i + 2 in flight
constexpr int D = kHeadDim;
constexpr int CH = D / 8;    // 16-byte chunks per K/V row
constexpr int NTHREADS = 512;
constexpr float kLazyMax = 8.0f;   // tiles that take a row max: m moves only past this margin (log2 units)
constexpr float kSumLim = 4096.f;  // unmasked tiles: a lane's tile sum above this sends the workgroup through a second pass

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) bf16_t lds_bf16;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;
typedef float f32x2 __attribute__((ext_vector_type(2)));

// One 16-byte-per-lane global -> LDS copy with a wave-uniform 64-bit base in
// SGPRs and a per-lane 32-bit byte offset (the saddr form): the offsets stay
// fixed from tile to tile, only the scalar base moves.  The LDS base goes in
// through an M0-bound input operand, as in lds_dma16.
__device__ __forceinline__ void lds_dma16_s(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile(
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(sbase), "{m0}"(lds_base)
      : "memory");
}

// Per-lane byte offsets (within a 64-key tile) of the K/V tile DMA.  Wave w
// moves 1 KiB blocks w and w + 8 of each 16 KiB tile; lane i of a block lands
// at byte 16 i of it, i.e. row 4 * block + i / 16, physical chunk i % 16, so
// the lane fetches the logical chunk the swizzle maps there (K: chunk ^
// (row & 15), V: chunk ^ 4 (row & 3); the same for both blocks of a lane).
struct DmaLane {
  int row0;                 // tile row of block w (block w + 8: row0 + 32)
  uint32_t kchunk, vchunk;  // byte offset of the fetched chunk within its row
};

__device__ __forceinline__ DmaLane dma_lane(int wave, int lane) {
  DmaLane d;
  d.row0 = 4 * wave + (lane >> 4);
  const int phys = lane & 15;
  d.kchunk = 16u * (phys ^ (d.row0 & 15));
  d.vchunk = 16u * (phys ^ ((d.row0 & 3) << 2));
  return d;
}

// Issue the DMA of one 64-key K and V tile (keys kv0 .. kv0+63 of the
// request; rows past kv_len - 1 re-read row kv_len - 1, whose values the mask
// discards) straight into LDS.  Exactly 4 loads per wave per tile.
__device__ __forceinline__ void dma_tile(const bf16_t* kb, const bf16_t* vb, int kv0, int kv_len, uint32_t k_dst,
                                         uint32_t v_dst, const DmaLane& d, int wave) {
  const bf16_t* ks = kb + (int64_t)kv0 * D;
  const bf16_t* vs = vb + (int64_t)kv0 * D;
  const bool full = kv0 + BKV <= kv_len;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = d.row0 + 32 * j;
    const int src = full ? row : min(kv0 + row, kv_len - 1) - kv0;
    const uint32_t roff = (uint32_t)src * (D * 2);
    const uint32_t blk = (uint32_t)(wave + 8 * j);
    lds_dma16_s(ks, roff + d.kchunk, k_dst + 1024u * blk);
    lds_dma16_s(vs, roff + d.vchunk, v_dst + 1024u * blk);
  }
}

// ---- per-wave phases of one 64-key tile (32 query rows per wave) -----------

// S^T = K Q^T: MFMA A = K rows from LDS, B = Q in registers; the accumulator
// of a lane holds keys 32 kh + 8 (v / 4) + 4 hf + v % 4 of ONE token.
__device__ __forceinline__ void qk_tile(const u32x4* kt, const bf16x8 (&qf)[8], int l32, int hf, f32x16 (&s)[2]) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {
    s[kh] = f32x16{};
    const int row = kh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8 a = as_bf16x8(kt[row * CH + ((2 * ks + hf) ^ (row & 15))]);
      s[kh] = mfma32(a, qf[ks], s[kh]);
    }
  }
}

__device__ __forceinline__ void mask_tile(f32x16 (&s)[2], int kv0, int vis_lim, int hf) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = kv0 + kh * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
      if (key > vis_lim) s[kh][v] = -INFINITY;
    }
}

// Row max, lazy reference update (the reference m only moves when the tile
// max exceeds it by more than `lazy` in log2 units: l and O accumulate against
// the same reference, so the result is unchanged), l *= alpha, and the scores
// turned into exponents s * log2(e)/sqrt(d) - m.  Returns alpha.  l is the
// lane's own partial sum; lanes l32 and l32 + 32 hold the same token and get
// the same m (the max is exchanged), so one alpha serves both partials.
__device__ __forceinline__ float max_tile(f32x16 (&s)[2], float sc, float& m_i, float& l_i, float lazy) {
  float mx = -INFINITY;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kh][v]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_tile = mx * sc;
  const float m_new = m_tile > m_i + lazy ? m_tile : m_i;
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = __builtin_amdgcn_exp2f(m_i - m_use);
  l_i *= alpha;
  m_i = m_new;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int v = 0; v < 16; ++v) s[kh][v] = fmaf(s[kh][v], sc, -m_use);
  return alpha;
}

// Exponents of a tile against the current reference m (finite), no max.
__device__ __forceinline__ void shift_tile(f32x16 (&s)[2], float sc, float m_i) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int v = 0; v < 16; ++v) s[kh][v] = fmaf(s[kh][v], sc, -m_i);
}

// p = 2^(exponent) and the bf16 P^T operand (16-key groups j).  Returns the
// lane's sum of p over its 32 keys.
__device__ __forceinline__ float exp_tile(f32x16 (&s)[2], bf16x8 (&pk)[4]) {
  float rs = 0.f;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[kh][v] = __builtin_amdgcn_exp2f(s[kh][v]);
      rs += s[kh][v];
    }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = pack_bf16x2(s[j >> 1][(j & 1) * 8 + 2 * e], s[j >> 1][(j & 1) * 8 + 2 * e + 1]);
    pk[j] = as_bf16x8(w);
  }
  return rs;
}

// O^T += V^T P^T.  The S^T accumulator hands a lane the keys of each 16-key
// group in the order (4hf + 0..3, 8 + 4hf + 0..3); V^T is read in that key
// order with the LDS transpose read.
__device__ __forceinline__ void pv_tile(const lds_bf16* vt, const bf16x8 (&pk)[4], int hf, int vrow,
                                        const int (&vcol)[4], f32x16 (&acc)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row_a = 16 * j + 4 * hf + vrow;  // keys 16j + 4hf + 0..3
    const int row_b = row_a + 8;                // keys 16j + 8 + 4hf + 0..3
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const v4i16 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vt + row_a * D + vcol[db]));
      const v4i16 vbv = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vt + row_b * D + vcol[db]));
      typedef short v8i16 __attribute__((ext_vector_type(8)));
      const v8i16 a8 = __builtin_shufflevector(va, vbv, 0, 1, 2, 3, 4, 5, 6, 7);
      acc[db] = mfma32(__builtin_bit_cast(bf16x8, a8), pk[j], acc[db]);
    }
  }
}

__device__ __forceinline__ void rescale(f32x16 (&acc)[4], float alpha) {
  if (__any(alpha != 1.0f)) {
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[db][v] *= alpha;
  }
}

// GATHER: the launch also copies another layer's pages into the request cache
// (AttnParams g_*): each wave takes every eighth chunk of its workgroup's
// range, one per tile.  A chunk is fetched into one of the wave's three LDS
// slots by the DMA form of the load right after the tile's K/V copies, and
// stored from there two tiles later, when the tile's wait has covered it:
// loads complete in the order issued, and a store can only lengthen a wait.
template <bool GATHER>
__global__ __launch_bounds__(NTHREADS, 1) void attention_kernel(AttnParams p) {
  __shared__ u32x4 k_lds[NSTAGE][BKV * CH];
  __shared__ u32x4 v_lds[NSTAGE][BKV * CH];
  constexpr int kGSlots = 3;
  __shared__ u32x4 g_lds[GATHER ? NTHREADS / 64 * kGSlots * 64 : 1];

  const int hkv = p.n_kv_heads;
  const int g = blockIdx.x % hkv;
  int unit = blockIdx.x / hkv;
  int r = 0;
  while (r + 1 < p.n_req && unit >= p.req[r + 1].wg_start) ++r;
  const AttnReq rq = p.req[r];
  unit -= rq.wg_start;
  const int split = unit % rq.n_split;
  const int qb = rq.n_qblk - 1 - unit / rq.n_split;
  const int t0 = qb * BQ;
  const int blk_rows = min(BQ, rq.q_len - t0);
  // last visible key of row tt of the request (rows past the end take the
  // last row's); grows with tt
  auto lim = [&](int tt) __attribute__((always_inline)) {
    tt = min(tt, rq.q_len - 1);
    if (rq.n_span == 0) return rq.art_len + tt;
    const int row = rq.q_start + tt;
    int base_row = p.span_row[rq.span0], base_off = p.span_off[rq.span0];
    for (int j = rq.span0 + 1; j < rq.span0 + rq.n_span; ++j)
      if (p.span_row[j] <= row) {
        base_row = p.span_row[j];
        base_off = p.span_off[j];
      }
    return base_off + row - base_row;
  };
  const int kv_len = lim(t0 + blk_rows - 1) + 1;  // keys any row of the block sees
  if constexpr (kChecked) {
    // the request's q rows and key range lie inside the launch's buffers
    if (rq.q_start < 0 || rq.q_start + rq.q_len > p.total_q || rq.kv_start < 0 ||
        (int64_t)rq.kv_start + kv_len > p.kv_head_stride / D) {
      if (threadIdx.x == 0) ATTUNER_VIOLATE(g_violations_attn, kViolAttnRange);
      return;
    }
  }
  const int n_tiles = (kv_len + BKV - 1) / BKV;
  const int per = (n_tiles + rq.n_split - 1) / rq.n_split;
  const int tb = min(n_tiles, split * per);
  const int te = min(n_tiles, tb + per);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // 0..7, kept in SGPRs
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int h = g * 4 + (wave & 3);
  const int t0w = t0 + 32 * (wave >> 2);  // first token of this wave's half
  const int t = t0w + l32;                // this lane's suffix token (index within the request)
  const bool row_ok = t - t0 < blk_rows;
  const int64_t qrow = (int64_t)(rq.q_start + t);

  const bf16_t* kb = p.k + g * p.kv_head_stride + (int64_t)rq.kv_start * D;
  const bf16_t* vb = p.v + g * p.kv_head_stride + (int64_t)rq.kv_start * D;
  const uint32_t k_base = lds_addr(k_lds[0]), v_base = lds_addr(v_lds[0]);
  constexpr uint32_t kStage = BKV * CH * 16;  // bytes per stage of K (and of V)
  const DmaLane dl = dma_lane(wave, lane);

  // Gather state (wave-uniform): the wave's chunks are g_first + 8 n for
  // n < g_count; chunk n is fetched at the wave's sync n into slot n % 3 and
  // stored at sync n + 3 (or after the loops).  g_prev: the previous sync
  // fetched a chunk after its tile's K/V copies.
  int g_first = 0, g_count = 0, g_syncs = 0;
  bool g_prev = false;
  if constexpr (GATHER) {
    const int cb = blockIdx.x * p.g_per_wg;
    const int ce = min(p.g_chunks, cb + p.g_per_wg);
    g_first = cb + wave;
    g_count = ce > g_first ? (ce - g_first + NTHREADS / 64 - 1) / (NTHREADS / 64) : 0;
  }
  // the copied layer's pool pages and cache planes, and chunk c's 16-byte
  // piece for this lane in each (offsets in 16-byte units); returns whether
  // this lane's row holds a token (rows past n_valid do not)
  const int g_nslab = 2 * hkv;
  const u32x4* g_src = reinterpret_cast<const u32x4*>(p.g_pool) +
                       (int64_t)p.g_layer * p.g_pool_pages * g_nslab * (kPageTokens * CH);
  u32x4* g_dst = reinterpret_cast<u32x4*>(p.g_req_kv) + (int64_t)p.g_layer * g_nslab * p.g_cache_rows * CH;
  auto g_addr = [&](int c, uint32_t& so, uint32_t& dof) __attribute__((always_inline)) {
    const int e = c >> p.g_shift;
    const int rem = c & ((1 << p.g_shift) - 1);
    const int sl = rem >> 2, qt = rem & 3;
    // through the constant address space: a scalar load, waited for with
    // the LDS counter, so the vector-memory wait of the K/V ring is left alone
    const __attribute__((address_space(4))) int32_t* ent =
        (const __attribute__((address_space(4))) int32_t*)p.g_table + 4 * e;  // {page, n_valid, dst_row, req}
    const int row = 4 * qt + (lane >> 4);
    if constexpr (kChecked) {
      // an HBM pool page of this layer, rows inside a page and the cache plane
      const bool ok = ent[0] >= 0 && (ent[0] & ~kPageIdMask) == 0 && ent[0] < p.g_pool_pages && ent[1] >= 0 &&
                      ent[1] <= kPageTokens && ent[2] >= 0 && (int64_t)ent[2] + ent[1] <= p.g_cache_rows;
      if (!ok) {
        if (lane == 0) ATTUNER_VIOLATE(g_violations_attn, kViolCopyEntry);
        so = (uint32_t)(lane & 15);  // a fetch stays inside page 0; nothing is stored
        dof = 0;
        return false;
      }
    }
    const bool valid = row < ent[1];
    const uint32_t rr = valid ? (uint32_t)row : 0u;
    so = ((uint32_t)((ent[0] & kPageIdMask) * g_nslab + sl) * kPageTokens + rr) * CH + (uint32_t)(lane & 15);
    dof = ((uint32_t)sl * (uint32_t)p.g_cache_rows + (uint32_t)ent[2] + rr) * CH + (uint32_t)(lane & 15);
    return valid;
  };
  const uint32_t g_base = lds_addr(g_lds) + (uint32_t)wave * kGSlots * 1024u;
  // store the wave's chunk n from its slot (its fetch is complete)
  auto g_store = [&](int n) __attribute__((always_inline)) {
    uint32_t so, dof;
    const bool valid = g_addr(g_first + n * (NTHREADS / 64), so, dof);
    // the lane's 16-byte piece of the slot, at 16 (lane >> 4) + (lane & 15):
    // formed here from the two values the addresses above use, in an opaque
    // step, so that the compiler keeps no register for it across the tile
    // loop (it spilled one, and a reload's wait drains the K/V ring)
    uint32_t piece;
    asm volatile("v_lshl_or_b32 %0, %1, 4, %2" : "=v"(piece) : "v"(lane >> 4), "v"(lane & 15));
    const u32x4 v = *(const __attribute__((address_space(3))) u32x4*)(uintptr_t)(
        g_base + (uint32_t)(n % kGSlots) * 1024u + piece * 16u);
    if (valid) __builtin_nontemporal_store(v, g_dst + dof);
  };

  // Prologue: the Q rows and the DMA of tile tb fly together and one wait
  // covers both (Q is then in registers, so the compiler needs no
  // vector-memory wait inside the tile loop); tile tb + 1 follows.
  bf16x8 qf[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row_ok) v = *reinterpret_cast<const u32x4*>(p.q + (qrow * p.n_q_heads + h) * D + ks * 16 + hf * 8);
    qf[ks] = as_bf16x8(v);
  }
  if (tb < te) dma_tile(kb, vb, tb * BKV, kv_len, k_base, v_base, dl, wave);
  __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));

  // transpose-read addressing of the V^T operand: lane r of its 16-lane group
  // points at key row (r >> 2) of a 4-key block and dims d0 + 4 (r & 3) .. +3,
  // d0 = 32 db + 16 * group.
  const int r16 = lane & 15;
  const int grp = (lane >> 4) & 1;
  const int vrow = r16 >> 2;  // == key & 3 of the row it reads
  int vcol[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int chunk = 4 * db + 2 * grp + ((r16 & 3) >> 1);
    vcol[db] = ((chunk ^ (vrow << 2)) << 3) + ((r16 & 1) << 2);
  }

  float m_i = -INFINITY, l_i = 0.f;
  f32x16 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x16{};

  const float sc = p.score_scale;
  const int vis_lim = lim(t);  // last visible key of this row

  const int mask_from = lim(t0w);  // tiles ending past this key need the mask
  // tiles before tp end at or before the diagonal of every row of the wave
  const int tp = min(max((mask_from + 1) / BKV, tb), te);

  if (tb + 1 < te) dma_tile(kb, vb, (tb + 1) * BKV, kv_len, k_base + kStage, v_base + kStage, dl, wave);

  // Start of tile `tile`: this wave's copies of it done (those of tile + 1,
  // if any, may still fly), then everyone's; the stage of tile - 2 is free
  // and receives tile + 2.
  auto tile_sync = [&](int tile) __attribute__((always_inline)) {
    // The loads after this tile's copies: tile + 1's four and, with the
    // gather, the chunk the previous sync fetched after them; waiting for
    // all but those leaves only tile + 1 in flight.  The chunk fetched two
    // syncs ago is complete as well (tile + 1's copies came after it).
    if (tile + 1 < te) {
      if (GATHER && g_prev) __builtin_amdgcn_s_waitcnt(vmcnt_wait(5));
      else __builtin_amdgcn_s_waitcnt(vmcnt_wait(4));
    } else {
      __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
    }
    barrier_no_fence();
    if (tile + 2 < te) {
      const uint32_t nb = (uint32_t)((tile - tb + 2) & (NSTAGE - 1)) * kStage;
      dma_tile(kb, vb, (tile + 2) * BKV, kv_len, k_base + nb, v_base + nb, dl, wave);
    }
    if constexpr (GATHER) {
      const int n = g_syncs;
      if (n >= kGSlots && n - kGSlots < g_count) g_store(n - kGSlots);  // frees slot n % 3
      g_prev = false;
      if (n < g_count) {
        uint32_t so, dof;
        (void)g_addr(g_first + n * (NTHREADS / 64), so, dof);
        lds_dma16(g_src + so, g_base + (uint32_t)(n % kGSlots) * 1024u);
        g_prev = tile + 2 < te;  // the next sync counts it only if it follows tile + 2's copies
      }
      g_syncs = n + 1;
    }
  };
  auto kst = [&](int tile) __attribute__((always_inline)) { return k_lds[(tile - tb) & (NSTAGE - 1)]; };
  auto vst = [&](int tile) __attribute__((always_inline)) {
    return (const lds_bf16*)v_lds[(tile - tb) & (NSTAGE - 1)];
  };

  // Unmasked tiles, software-pipelined inside the wave: QK of `tile` is
  // issued alongside the exponentials of tile - 1, and PV of tile - 1
  // alongside the exponents of `tile`.  S^T alternates between sa and sb.
  // Only the first tile takes a row max: later tiles' exponents are taken
  // against the current reference m.  A lane whose sum over a tile exceeds
  // kSumLim (some p large, or an overflow) marks itself; if any lane of the
  // workgroup did, the whole range is run again with a row max per tile (the
  // second pass below), so every p kept is at most kSumLim.
  bool bad = false;
  for (bool redo = false;; redo = true) {
    if (!redo && tb < tp) {
      f32x16 sa[2], sb[2];
      bf16x8 pk[4];
      tile_sync(tb);
      qk_tile(kst(tb), qf, l32, hf, sa);
      max_tile(sa, sc, m_i, l_i, kLazyMax);
      auto finish = [&](f32x16 (&so)[2]) __attribute__((always_inline)) {
        const float rs = exp_tile(so, pk);
        bad = bad || !(rs <= kSumLim);
        l_i += rs;
      };
      auto step = [&](f32x16 (&sn)[2], f32x16 (&so)[2], int tile) __attribute__((always_inline)) {
        tile_sync(tile);
        qk_tile(kst(tile), qf, l32, hf, sn);
        finish(so);
        pv_tile(vst(tile - 1), pk, hf, vrow, vcol, acc);
        shift_tile(sn, sc, m_i);
      };
      int tile = tb + 1;
      for (; tile + 1 < tp; tile += 2) {
        step(sb, sa, tile);
        step(sa, sb, tile + 1);
      }
      if (tile < tp) {
        step(sb, sa, tile);
        finish(sb);
      } else {
        finish(sa);
      }
      pv_tile(vst(tp - 1), pk, hf, vrow, vcol, acc);
    }

    // tiles reaching the diagonal (all tiles in the second pass): one row max
    // per tile, plain steps
    for (int tile = redo ? tb : tp; tile < te; ++tile) {
      f32x16 s[2];
      bf16x8 pk[4];
      tile_sync(tile);
      const int kv0 = tile * BKV;
      qk_tile(kst(tile), qf, l32, hf, s);
      if (kv0 + BKV - 1 > mask_from) mask_tile(s, kv0, vis_lim, hf);
      rescale(acc, max_tile(s, sc, m_i, l_i, kLazyMax));
      l_i += exp_tile(s, pk);
      pv_tile(vst(tile), pk, hf, vrow, vcol, acc);
    }
    // every wave has left the ring when this returns
    if (redo || !__syncthreads_or(bad)) break;
    m_i = -INFINITY;
    l_i = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x16{};
    g_prev = false;  // the last fetch came before the new copies
    if (tb < te) dma_tile(kb, vb, tb * BKV, kv_len, k_base, v_base, dl, wave);
    if (tb + 1 < te) dma_tile(kb, vb, (tb + 1) * BKV, kv_len, k_base + kStage, v_base + kStage, dl, wave);
  }
  if constexpr (GATHER) {
    // the chunks still in LDS, then the rest of the wave's chunks directly,
    // eight loads in flight at a time (short key ranges leave most of the
    // copy to this loop, and one chunk at a time would pay a memory latency
    // per kilobyte)
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
    for (int n = max(0, g_syncs - kGSlots); n < min(g_syncs, g_count); ++n) g_store(n);
    constexpr int kGBatch = 8;
    for (int n0 = g_syncs; n0 < g_count; n0 += kGBatch) {
      u32x4 v[kGBatch];
      uint32_t dof[kGBatch];
      bool ok[kGBatch];
#pragma unroll
      for (int i = 0; i < kGBatch; ++i) {
        // every lane loads (a row past n_valid reads row 0 of its page; past
        // the wave's last chunk, that chunk again): only the stores are masked
        uint32_t so;
        const int n = min(n0 + i, g_count - 1);
        ok[i] = g_addr(g_first + n * (NTHREADS / 64), so, dof[i]) && n0 + i < g_count;
        v[i] = __builtin_nontemporal_load(g_src + so);
      }
#pragma unroll
      for (int i = 0; i < kGBatch; ++i)
        if (ok[i]) __builtin_nontemporal_store(v[i], g_dst + dof[i]);
    }
  }
  l_i += __shfl_xor(l_i, 32, 64);  // the two lanes of a token hold its two partial sums

  // ---- epilogue: O / l (the output, or with n_split > 1 this split's
  // normalised partial) goes through LDS, so that each store below is 16
  // bytes per lane of a whole 256-byte row.  The O^T accumulator holds, per
  // lane, dims 32 db + 8 q + 4 hf + 0..3 of one token: 8-byte slot 8 db + 2 q
  // + hf of that token's row.  Slot s of row r is kept at s ^ r (rows of 32
  // slots), so the 32 lanes of a half-wave, one row each, write 32 distinct
  // slots (no bank conflicts); a 16-byte chunk c of row r then sits at chunk
  // c ^ (r >> 1), its two halves swapped when r is odd.
  const float inv_l = l_i > 0.f ? 1.0f / l_i : 0.f;
  constexpr int kRowBytes = D * 2;
  static_assert(8 * 32 * kRowBytes <= (int)sizeof(k_lds), "epilogue staging must fit the K ring");
  __syncthreads();  // every wave is done with the K/V ring
  char* stage = reinterpret_cast<char*>(&k_lds[0][0]) + wave * 32 * kRowBytes;
#pragma unroll
  for (int db = 0; db < 4; ++db) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      u32x2 pr;
      pr[0] = pack_bf16x2(acc[db][4 * q] * inv_l, acc[db][4 * q + 1] * inv_l);
      pr[1] = pack_bf16x2(acc[db][4 * q + 2] * inv_l, acc[db][4 * q + 3] * inv_l);
      const int slot = (8 * db + 2 * q + hf) ^ l32;
      *reinterpret_cast<u32x2*>(stage + l32 * kRowBytes + slot * 8) = pr;
    }
  }
  const int64_t head_rows = (int64_t)p.total_q * p.n_q_heads;  // rows of one split's partial
  bf16_t* dst = p.n_split == 1 ? p.o : p.part_o + (int64_t)split * head_rows * D;
  const int sub = lane >> 4;  // row within a group of 4; 16 lanes x 16 bytes per row
  const int c16 = lane & 15;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int rr = 4 * j + sub;  // token t0w + rr
    u32x4 v = *reinterpret_cast<const u32x4*>(stage + rr * kRowBytes + (c16 ^ (rr >> 1)) * 16);
    if (rr & 1) v = u32x4{v[2], v[3], v[0], v[1]};
    if (t0w + rr - t0 < blk_rows) {
      const int64_t orow = (int64_t)(rq.q_start + t0w + rr) * p.n_q_heads + h;
      *reinterpret_cast<u32x4*>(dst + orow * D + c16 * 8) = v;
    }
  }
  if (!row_ok || hf != 0) return;
  const int64_t hrow = qrow * p.n_q_heads + h;
  if (p.n_split == 1) {
    if (p.lse != nullptr) p.lse[hrow] = (m_i + __log2f(l_i)) * 0.69314718055994531f;
  } else {
    *reinterpret_cast<f32x2*>(p.part_ml + ((int64_t)split * head_rows + hrow) * 2) = f32x2{m_i, l_i};
    // slices past this request's own split count: empty (the merge skips them)
    if (split == 0)
      for (int s = rq.n_split; s < p.n_split; ++s)
        *reinterpret_cast<f32x2*>(p.part_ml + ((int64_t)s * head_rows + hrow) * 2) = f32x2{-INFINITY, 0.f};
  }
}

// Merge the n_split partials: weight of split s is l_s * 2^(m_s - max_s m_s).
// Workgroup b serves KV head g = b % Hkv and 4 tokens (with Hkv = 8, on the
// XCD whose workgroups wrote those partials; the partials still come back
// through the memory side, as the attention kernel's end writes its L2 back).
// A wave merges the 4 query heads of one token; 16 lanes per (token, head)
// row, lane owning dims 8 (lane % 16) .. +7; every split's data is requested
// before any is used.
constexpr int kMaxSplit = kMaxAttnSplit;

template <int NS>
__global__ __launch_bounds__(256, 2) void attn_combine_kernel(AttnParams p) {
  const int g = blockIdx.x % p.n_kv_heads;
  const int t = (blockIdx.x / p.n_kv_heads) * 4 + (threadIdx.x >> 6);
  if (t >= p.total_q) return;
  const int lane = threadIdx.x & 63;
  const int h = g * 4 + (lane >> 4);
  const int d0 = 8 * (lane & 15);
  const int64_t row = (int64_t)t * p.n_q_heads + h;
  const int64_t stride = (int64_t)p.total_q * p.n_q_heads;
  // the split count is a template constant: every load is issued before the
  // first one is waited for
  f32x2 ml[NS];
  u32x4 v[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    ml[s] = *reinterpret_cast<const f32x2*>(p.part_ml + (s * stride + row) * 2);
    v[s] = *reinterpret_cast<const u32x4*>(p.part_o + (s * stride + row) * D + d0);
  }
  __builtin_amdgcn_sched_barrier(0);  // keep every load ahead of the first use
  float mmax = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) mmax = fmaxf(mmax, ml[s][0]);
  float wsum = 0.f;
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    // an empty slice (no keys, or past its request's split count) holds no
    // partial worth reading: its values are skipped, not weighted by zero
    const bool empty = ml[s][0] == -INFINITY;
    const float w = empty ? 0.f : ml[s][1] * __builtin_amdgcn_exp2f(ml[s][0] - mmax);
    wsum += w;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = fmaf(w, __uint_as_float(v[s][e] << 16), o[2 * e]);
      const float hi = fmaf(w, __uint_as_float(v[s][e] & 0xFFFF0000u), o[2 * e + 1]);
      o[2 * e] = empty ? o[2 * e] : lo;
      o[2 * e + 1] = empty ? o[2 * e + 1] : hi;
    }
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  u32x4 pr;
#pragma unroll
  for (int e = 0; e < 4; ++e) pr[e] = pack_bf16x2(o[2 * e] * inv, o[2 * e + 1] * inv);
  *reinterpret_cast<u32x4*>(p.o + row * D + d0) = pr;
  if (p.lse != nullptr && (lane & 15) == 0) p.lse[row] = (mmax + __log2f(wsum)) * 0.69314718055994531f;
}

}  // namespace

hipError_t read_violations_attention(unsigned int* bits, bool reset) {
  return read_violations_attn_impl(bits, reset);
}

hipError_t launch_attention(const AttnParams& p, hipStream_t stream) {
  if (p.n_units == 0) return hipSuccess;
  if (p.g_table != nullptr)
    ATTUNER_LAUNCH("attention_gather_kernel", attention_kernel<true>, dim3((unsigned)(p.n_units * p.n_kv_heads)),
                   dim3(NTHREADS), stream, p);
  else
    ATTUNER_LAUNCH("attention_kernel", attention_kernel<false>, dim3((unsigned)(p.n_units * p.n_kv_heads)),
                   dim3(NTHREADS), stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_split == 1) return e;
  if (p.n_split > kMaxSplit || p.n_q_heads != 4 * p.n_kv_heads) return hipErrorInvalidValue;
  const int64_t wgs = (int64_t)((p.total_q + 3) / 4) * p.n_kv_heads;
#define ATTUNER_COMBINE(NS_)                                                                                   \
  case NS_:                                                                                                    \
    ATTUNER_LAUNCH("attn_combine_kernel", attn_combine_kernel<NS_>, dim3((unsigned)wgs), dim3(256), stream, p); \
    break;
  switch (p.n_split) {
    ATTUNER_COMBINE(2) ATTUNER_COMBINE(3) ATTUNER_COMBINE(4) ATTUNER_COMBINE(5) ATTUNER_COMBINE(6)
    ATTUNER_COMBINE(7) ATTUNER_COMBINE(8) ATTUNER_COMBINE(9) ATTUNER_COMBINE(10) ATTUNER_COMBINE(11)
    ATTUNER_COMBINE(12) ATTUNER_COMBINE(13) ATTUNER_COMBINE(14) ATTUNER_COMBINE(15) ATTUNER_COMBINE(16)
    default: return hipErrorInvalidValue;
  }
#undef ATTUNER_COMBINE
  return hipGetLastError();
}

}  // namespace attuner
