// K2: bf16 MFMA projection GEMM with the rank-r LoRA update fused into its
// epilogue (query-side adaptation, section 4 eq. 4):
//   out[i][n] = x[i] . w[n]  +  (n < lora_cols ? t[i] . b[n] : 0),
//   t = scale * x A^T  (computed by the GEMM's own k-loop for r <= 32, else
//   by lora_down_kernel first).
//
// The GEMM is computed as C^T = W x^T so that the MFMA accumulator of a lane
// holds four consecutive output features of one token (8-byte stores).  Both
// operands are K-contiguous in memory ([rows][hidden]), so tiles go to LDS
// without a transpose.  Workgroup tile BN (features) x BM (tokens) x 64 (k),
// 32x32x16 MFMAs, fp32 accumulation, the operand tiles copied global -> LDS
// by the DMA form of the load.  Two kernels: gemm_lora_kernel (one wave per
// wave tile) and gemm_kg2_kernel (96 x 64 wave tiles, two groups of waves on
// alternate k-steps).  At suffix sizes the operand ingest per CU is the
// ceiling (measured on gfx950: about 58 GB/s per CU, 15 TB/s out of the L2s,
// the same rate hipBLASLt's kernels reach on these shapes), so the tile shape
// is chosen to minimise ingested bytes, M N K 2 (1/BM + 1/BN), while keeping
// every CU busy, and the copies are spread between the MFMAs so that the
// compute hides under the ingest.  LDS rows are 128 bytes (eight 16-byte
// chunks); chunk c of row r is stored at c ^ ((r >> 1) & 7), so the 16 rows
// one operand read touches in a cycle land on 16 distinct bank groups.
//
// The LoRA term enters as extra MFMA k-steps after the main loop: A operand
// = rows of B (rank padded to 16 with zeros), B operand = t rounded to a
// bf16 hi/lo pair, so t keeps ~16 significant bits and the update is summed
// in fp32.  lora_down_kernel leaves t as fp32 partial sums over slices of
// the hidden dimension (256 or 1024 wide); the epilogue adds the slices in
// order.

#include <type_traits>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int BK = 64;
constexpr int kChunksPerRow = BK / 8;  // 16-byte chunks per LDS row
constexpr int kLoraSlice = 256;        // hidden elements per lora_down chunk (four waves x 64)
constexpr int kLoraSliceWide = 1024;   // hidden elements per lora_down workgroup above kGemvMaxTok tokens
constexpr int kLoraRows = 32;          // A rows staged per k-tile when the down-projection is fused
constexpr int kGroupM = 4;             // token tiles per group of the tile order

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Fused low-rank epilogue and store of one wave's FN x FM blocks of C^T:
// acc += B[n][:] . t[m][:] for features n < lora_cols, then bf16 stores (lane
// holds features nb + 8q + 4*hi + (0..3) of token m).  n_base / m_base: the
// wave tile's first feature / token.
template <int FN, int FM>
__device__ __forceinline__ void lora_epilogue_store(f32x16 (&acc)[FN][FM], int n_base, int m_base, int ml_base,
                                                    int l32, int hi, int M, int N, const bf16_t* __restrict__ b,
                                                    int rank, int r_pad, int lora_cols,
                                                    const float* __restrict__ t_part, int n_slice,
                                                    const float* t_lds, const GemmEpi& epi, bf16_t* out) {
  if (r_pad > 0 && n_base < lora_cols) {
    const int64_t slice_stride = (int64_t)M * r_pad;
    // B rows as 16-byte loads when they are whole 16-byte runs
    const bool b_vec = (rank & 7) == 0 && (reinterpret_cast<uintptr_t>(b) & 15) == 0;
    for (int ks = 0; ks < r_pad; ks += 16) {
      bf16x8 th[FM], tl[FM];
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        f32x4 s0 = f32x4{}, s1 = f32x4{};
        if (t_lds != nullptr) {
          // fused: t[token][rank] staged in LDS by this workgroup
          const float* tr = t_lds + (ml_base + j * 32 + l32) * (kLoraRows + 1) + ks + 8 * hi;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s0[e] = tr[e];
            s1[e] = tr[4 + e];
          }
        } else {
          int m = m_base + j * 32 + l32;
          m = m < M ? m : M - 1;
          const float* tp = t_part + (int64_t)m * r_pad + ks + 8 * hi;
          for (int z = 0; z < n_slice; ++z) {
            s0 += *reinterpret_cast<const f32x4*>(tp + z * slice_stride);
            s1 += *reinterpret_cast<const f32x4*>(tp + z * slice_stride + 4);
          }
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
        const int nb = n_base + i * 32;
        if (nb >= lora_cols) continue;  // lora_cols is a multiple of 32
        const int n = nb + l32;
        bf16x8 a;
        const int j0 = ks + 8 * hi;  // this lane's 8 ranks j0 .. j0 + 7 of B row n
        if (b_vec) {
          // rank % 8 == 0: the 8 ranks are all below rank or all past it
          u32x4 v = u32x4{0u, 0u, 0u, 0u};
          if (j0 < rank) v = *reinterpret_cast<const u32x4*>(b + (int64_t)n * rank + j0);
          a = as_bf16x8(v);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const bf16_t bv = j0 + e < rank ? b[(int64_t)n * rank + j0 + e] : (bf16_t)0;
            a[e] = __builtin_bit_cast(__bf16, bv);
          }
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          acc[i][j] = mfma32(a, th[j], acc[i][j]);
          acc[i][j] = mfma32(a, tl[j], acc[i][j]);
        }
      }
    }
  }

#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int m = m_base + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int nb = n_base + i * 32;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = nb + 8 * q + 4 * hi;  // features n .. n + 3 of token m
        float c[4] = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if (epi.mode == kEpiF32) {
          *reinterpret_cast<f32x4*>(epi.out_f32 + (int64_t)m * N + n) = f32x4{c[0], c[1], c[2], c[3]};
          continue;
        }
        if (epi.mode == kEpiSwiglu) {
          // (gate, up) pairs (n, n + 1) and (n + 2, n + 3) -> outputs n / 2, n / 2 + 1
          const float s0 = c[0] / (1.0f + __expf(-c[0])) * c[1];
          const float s1 = c[2] / (1.0f + __expf(-c[2])) * c[3];
          *reinterpret_cast<uint32_t*>(out + (int64_t)m * (N / 2) + n / 2) = pack_bf16x2(s0, s1);
          continue;
        }
        if (epi.mode == kEpiResidual) {
          const u32x2 r = *reinterpret_cast<const u32x2*>(epi.residual + (int64_t)m * N + n);
          c[0] += __uint_as_float(r[0] << 16);
          c[1] += __uint_as_float(r[0] & 0xFFFF0000u);
          c[2] += __uint_as_float(r[1] << 16);
          c[3] += __uint_as_float(r[1] & 0xFFFF0000u);
        }
        u32x2 pk;
        pk[0] = pack_bf16x2(c[0], c[1]);
        pk[1] = pack_bf16x2(c[2], c[3]);
        *reinterpret_cast<u32x2*>(out + (int64_t)m * N + n) = pk;
      }
    }
  }
}

// Both operand tiles are copied global -> LDS by the DMA form of the load
// (16 bytes per lane, no staging registers) into an NST-stage ring, so NST - 1
// k-tiles are in flight per workgroup while one is multiplied.  WN x WM waves;
// one barrier per k-tile.  A k-tile stage is (BN + BM) rows of 128 bytes,
// moved as 1 KiB blocks of 8 rows (lane i -> row 8 blk + i / 8, physical
// chunk i % 8, holding the logical chunk the swizzle maps there).
template <int BM, int BN, int WN, int WM, int NST, bool ILV>
__global__ __launch_bounds__(64 * WN * WM, 1) void gemm_lora_kernel(const bf16_t* __restrict__ x,
                                                                   const bf16_t* __restrict__ w, int M, int N, int K,
                                                                   const bf16_t* __restrict__ a, float scale,
                                                                   const bf16_t* __restrict__ b, int rank, int r_pad,
                                                                   int lora_cols, const float* __restrict__ t_part,
                                                                   int n_slice, GemmEpi epi, bf16_t* out, int n_mt,
                                                                   int n_nt, int kt_split) {
  constexpr int NW = WN * WM;
  constexpr int TN = BN / WN, TM = BM / WM;
  constexpr int FN = TN / 32, FM = TM / 32;
  static_assert(FN >= 1 && FM >= 1 && TN % 32 == 0 && TM % 32 == 0, "bad wave layout");
  // stage rows: W rows [0, BN), x rows [BN, BN + BM), and (fused LoRA) the
  // kLoraRows rows of A [BN + BM, BN + BM + kLoraRows)
  constexpr int ROWS = BN + BM + kLoraRows;
  static_assert((BN + BM) % 8 == 0, "stage must be whole 1 KiB blocks");
  constexpr int STAGE = ROWS * kChunksPerRow;
  static_assert(BM * (kLoraRows + 1) * 4 <= STAGE * 16, "t staging must fit one stage");
  __shared__ u32x4 lds[NST * STAGE];

  // Tile order.  Workgroup i runs on XCD i % 8: each XCD gets a contiguous
  // run of the order below, so the ~32 workgroups one XCD runs at a time
  // share operand panels in its L2.  The order walks groups of kGroupM token
  // tiles across all feature tiles, token tile fastest: 32 concurrent
  // workgroups cover about kGroupM x 8 tiles (kGroupM x-panels, 8 W-panels).
  // Split-K (kt_split > 0): workgroup blockIdx.x / total takes k-tiles
  // [split * kt_split, (split + 1) * kt_split) of tile blockIdx.x % total and
  // writes its fp32 partial to slice `split` of epi.out_f32.
  const int total = n_mt * n_nt;
  const int per_xcd = total >> 3;
  const int split = kt_split > 0 ? (int)blockIdx.x / total : 0;
  int lin = kt_split > 0 ? (int)blockIdx.x % total : (int)blockIdx.x;
  if (lin < 8 * per_xcd) lin = (lin & 7) * per_xcd + (lin >> 3);
  const int in_group = kGroupM * n_nt;
  const int first_m = (lin / in_group) * kGroupM;
  const int gm = min(n_mt - first_m, kGroupM);
  const int mt = first_m + (lin % in_group) % gm;
  const int nt = (lin % in_group) / gm;
  const int n0 = nt * BN;
  const int m0 = mt * BM;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wn = wave / WM;
  const int wm = wave % WM;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int kt0 = split * kt_split;
  const int n_kt = kt_split > 0 ? min(K / BK - kt0, kt_split) : K / BK;
  const uint32_t lds0 = lds_addr(lds);

  f32x16 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x16{};

  // Fused down-projection (t_part == null): this workgroup needs t for its
  // tokens, so the k-loop also stages A's rows and, for each 32-token block,
  // one wave that holds its x fragments accumulates t^T = A x^T next to its
  // main MFMAs.  t then goes through LDS to the epilogue.
  const bool fused = t_part == nullptr && r_pad > 0 && n0 < lora_cols;
  f32x16 tacc[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) tacc[j] = f32x16{};

  auto kloop = [&](auto la_tag) __attribute__((always_inline)) {
    constexpr bool LA = decltype(la_tag)::value;
    constexpr int NBLK = (BN + BM + (LA ? kLoraRows : 0)) / 8;
    constexpr int PW = (NBLK + NW - 1) / NW;  // DMA instructions per wave per stage
    static_assert((NST - 2) * PW <= 63, "vmcnt range");
    // DMA sources of this lane (blocks past the stage repeat the last block:
    // same bytes to the same place)
    const bf16_t* src[PW];
    uint32_t doff[PW];
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int blk = min(wave + NW * j, NBLK - 1);
      const int row = 8 * blk + (lane >> 3);
      const int lg = swz(row, lane & 7);
      const bf16_t* base;
      if (row < BN) {
        base = w + (int64_t)(n0 + row) * K;
      } else if (row < BN + BM) {
        const int m = min(m0 + row - BN, M - 1);  // rows past the end are computed, never stored
        base = x + (int64_t)m * K;
      } else {
        // A rows past rank repeat row rank - 1: finite, and met by zero B columns
        base = a + (int64_t)min(row - BN - BM, rank - 1) * K;
      }
      src[j] = base + 8 * lg + (int64_t)kt0 * BK;
      doff[j] = 1024u * blk;
    }
#pragma unroll
    for (int st = 0; st < NST - 1; ++st) {
      const int kt = min(st, n_kt - 1);
#pragma unroll
      for (int j = 0; j < PW; ++j) lds_dma16(src[j] + kt * BK, lds0 + (uint32_t)(st * STAGE * 16) + doff[j]);
    }
    // t block j (32 tokens) is accumulated by the wave column wn == j % WN
    // of the wave row that holds those tokens: the extra MFMAs spread over
    // min(FM, WN) wave columns
    int slot = 0, nslot = NST - 1;
    for (int kt = 0; kt < n_kt; ++kt) {
      // own copies of tile kt done, then everyone's; slot nslot (tile kt - 1) is free
      __builtin_amdgcn_s_waitcnt(vmcnt_wait((NST - 2) * PW));
      barrier_no_fence();
      const int nk = min(kt + NST - 1, n_kt - 1);
      const u32x4* cur = lds + slot * STAGE;
      // ILV: the stage's copies are spread over the k-steps (one after
      // every second MFMA, the rest after the last k-step), so that a wave
      // whose copies wait for room in the memory pipeline has MFMAs in
      // flight; otherwise all are issued here
      int d = ILV ? 0 : PW;
      if (!ILV) {
#pragma unroll
        for (int j = 0; j < PW; ++j) lds_dma16(src[j] + nk * BK, lds0 + (uint32_t)(nslot * STAGE * 16) + doff[j]);
      }
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = 2 * ks + hi;
        bf16x8 af[FN], bfr[FM];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int row = wn * TN + i * 32 + l32;
          af[i] = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          const int row = BN + wm * TM + j * 32 + l32;
          bfr[j] = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
        }
        int q = 0;
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j) {
            acc[i][j] = mfma32(af[i], bfr[j], acc[i][j]);
            if (ILV && (q & 1) == 1 && d < PW) {
              __builtin_amdgcn_sched_barrier(0);
              lds_dma16(src[d] + nk * BK, lds0 + (uint32_t)(nslot * STAGE * 16) + doff[d]);
              __builtin_amdgcn_sched_barrier(0);
              ++d;
            }
            ++q;
          }
        if (LA && wn < FM) {
          const int row = BN + BM + l32;
          const bf16x8 ar = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
#pragma unroll
          for (int j = 0; j < FM; ++j)
            if (j % WN == wn) tacc[j] = mfma32(ar, bfr[j], tacc[j]);
        }
      }
#pragma unroll
      for (int e = 0; e < PW; ++e)
        if (e >= d) lds_dma16(src[e] + nk * BK, lds0 + (uint32_t)(nslot * STAGE * 16) + doff[e]);
      slot = slot + 1 == NST ? 0 : slot + 1;
      nslot = nslot + 1 == NST ? 0 : nslot + 1;
    }
    // the clamped copies of the last iterations must land before the LDS is
    // reused or the workgroup ends (its LDS may be handed to the next one)
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
  };

  const float* t_lds = nullptr;
  if (fused) {
    kloop(std::integral_constant<bool, true>{});
    // t^T accumulator: lane holds ranks 8 (v / 4) + 4 hi + v % 4 of token
    // l32 of each 32-token block; staged as fp32 t[token][rank], row stride
    // kLoraRows + 1
    float* ts = reinterpret_cast<float*>(lds);
    barrier_no_fence();
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      if (j % WN != wn) continue;
      const int ml = wm * TM + j * 32 + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) ts[ml * (kLoraRows + 1) + 8 * (v >> 2) + 4 * hi + (v & 3)] = scale * tacc[j][v];
    }
    __syncthreads();
    t_lds = ts;
  } else {
    kloop(std::integral_constant<bool, false>{});
  }

  if (kt_split > 0) epi.out_f32 += (int64_t)split * M * N;
  lora_epilogue_store<FN, FM>(acc, n0 + wn * TN, m0 + wm * TM, wm * TM, l32, hi, M, N, b, rank, r_pad, lora_cols,
                              t_part, n_slice, t_lds, epi, out);
}

// The same product with two k-groups of waves.  Each wave holds a 96 x 64
// (features x tokens) tile of C^T, which reads 5 LDS fragments per 6 MFMAs
// (3 per 2 for the 32 x 64 tile above), and the waves of group g take
// k-steps g and g + 2 of every 64-deep k-tile, so that two waves share each
// SIMD and cover each other's LDS latency.  After the k-loop the groups
// exchange halves through LDS: group g gives its partner its partial sums of
// token block 1 - g and adds the partner's partial sums of token block g,
// then applies the epilogue to block g.  The fused LoRA down-projection is
// split the same way (each group's t^T over its k-steps, summed in LDS).
template <int BM, int BN, int WN, int WM, int NST>
__global__ __launch_bounds__(128 * WN * WM, 1) void gemm_kg2_kernel(const bf16_t* __restrict__ x,
                                                                   const bf16_t* __restrict__ w, int M, int N, int K,
                                                                   const bf16_t* __restrict__ a, float scale,
                                                                   const bf16_t* __restrict__ b, int rank, int r_pad,
                                                                   int lora_cols, const float* __restrict__ t_part,
                                                                   int n_slice, GemmEpi epi, bf16_t* out, int n_mt,
                                                                   int n_nt, int kt_split) {
  constexpr int NWG = WN * WM;  // waves per k-group
  constexpr int NW = 2 * NWG;
  constexpr int TN = BN / WN, TM = BM / WM;
  constexpr int FN = TN / 32, FM = TM / 32;
  static_assert(FM == 2 && FN >= 1 && TN % 32 == 0, "each group finishes one of a wave's two token blocks");
  constexpr int ROWS = BN + BM + kLoraRows;
  static_assert((BN + BM) % 8 == 0, "stage must be whole 1 KiB blocks");
  constexpr int STAGE = ROWS * kChunksPerRow;
  __shared__ u32x4 lds[NST * STAGE];
  // after the k-loop: t staging [BM][kLoraRows + 1] floats, then the exchange
  // [2 groups][NWG waves][FN][16][64 lanes] floats
  constexpr int kTsFloats = (BM * (kLoraRows + 1) + 63) / 64 * 64;
  static_assert((kTsFloats + 2 * NWG * FN * 16 * 64) * 4 <= NST * STAGE * 16, "exchange must fit the ring");

  const int total = n_mt * n_nt;
  const int per_xcd = total >> 3;
  const int split = kt_split > 0 ? (int)blockIdx.x / total : 0;
  int lin = kt_split > 0 ? (int)blockIdx.x % total : (int)blockIdx.x;
  if (lin < 8 * per_xcd) lin = (lin & 7) * per_xcd + (lin >> 3);
  const int in_group = kGroupM * n_nt;
  const int first_m = (lin / in_group) * kGroupM;
  const int gm = min(n_mt - first_m, kGroupM);
  const int mt = first_m + (lin % in_group) % gm;
  const int nt = (lin % in_group) / gm;
  const int n0 = nt * BN;
  const int m0 = mt * BM;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int kg = wave / NWG;
  const int wv = wave % NWG;
  const int wn = wv / WM;
  const int wm = wv % WM;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int kt0 = split * kt_split;
  const int n_kt = kt_split > 0 ? min(K / BK - kt0, kt_split) : K / BK;
  const uint32_t lds0 = lds_addr(lds);

  f32x16 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x16{};
  const bool fused = t_part == nullptr && r_pad > 0 && n0 < lora_cols;
  f32x16 tacc[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) tacc[j] = f32x16{};

  auto kloop = [&](auto la_tag) __attribute__((always_inline)) {
    constexpr bool LA = decltype(la_tag)::value;
    constexpr int NBLK = (BN + BM + (LA ? kLoraRows : 0)) / 8;
    constexpr int PW = (NBLK + NW - 1) / NW;
    static_assert((NST - 2) * PW <= 63, "vmcnt range");
    const bf16_t* src[PW];
    uint32_t doff[PW];
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int blk = min(wave + NW * j, NBLK - 1);
      const int row = 8 * blk + (lane >> 3);
      const int lg = swz(row, lane & 7);
      const bf16_t* base;
      if (row < BN) {
        base = w + (int64_t)(n0 + row) * K;
      } else if (row < BN + BM) {
        const int m = min(m0 + row - BN, M - 1);
        base = x + (int64_t)m * K;
      } else {
        base = a + (int64_t)min(row - BN - BM, rank - 1) * K;
      }
      src[j] = base + 8 * lg + (int64_t)kt0 * BK;
      doff[j] = 1024u * blk;
    }
#pragma unroll
    for (int st = 0; st < NST - 1; ++st) {
      const int kt = min(st, n_kt - 1);
#pragma unroll
      for (int j = 0; j < PW; ++j) lds_dma16(src[j] + kt * BK, lds0 + (uint32_t)(st * STAGE * 16) + doff[j]);
    }
    int slot = 0, nslot = NST - 1;
    for (int kt = 0; kt < n_kt; ++kt) {
      __builtin_amdgcn_s_waitcnt(vmcnt_wait((NST - 2) * PW));
      barrier_no_fence();
      const int nk = min(kt + NST - 1, n_kt - 1);
      const u32x4* cur = lds + slot * STAGE;
      // fragments of both k-steps (the second read while the first multiplies)
      bf16x8 af[2][FN], bfr[2][FM], ar[2];
      auto load = [&](int s2) __attribute__((always_inline)) {
        const int ch = 2 * (kg + 2 * s2) + hi;
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int row = wn * TN + i * 32 + l32;
          af[s2][i] = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
        }
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          const int row = BN + wm * TM + j * 32 + l32;
          bfr[s2][j] = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
        }
        if (LA && wn < FM) {
          const int row = BN + BM + l32;
          ar[s2] = as_bf16x8(cur[row * kChunksPerRow + swz(row, ch)]);
        }
      };
      constexpr int HALF = (PW + 1) / 2;
      load(0);
      load(1);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        int q = 0;
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j) {
            acc[i][j] = mfma32(af[s2][i], bfr[s2][j], acc[i][j]);
            if (q % 2 == 1) {
              const int d = s2 * HALF + q / 2;
              if (d < PW && q / 2 < HALF) {
                __builtin_amdgcn_sched_barrier(0);
                lds_dma16(src[d] + nk * BK, lds0 + (uint32_t)(nslot * STAGE * 16) + doff[d]);
                __builtin_amdgcn_sched_barrier(0);
              }
            }
            ++q;
          }
        if (LA && wn < FM) {
#pragma unroll
          for (int j = 0; j < FM; ++j)
            if (j % WN == wn) tacc[j] = mfma32(ar[s2], bfr[s2][j], tacc[j]);
        }
        // DMAs of this half not yet issued (more than FN * FM / 2 of them)
#pragma unroll
        for (int e = (FN * FM) / 2; e < HALF; ++e) {
          const int d = s2 * HALF + e;
          if (d < PW) lds_dma16(src[d] + nk * BK, lds0 + (uint32_t)(nslot * STAGE * 16) + doff[d]);
        }
      }
      slot = slot + 1 == NST ? 0 : slot + 1;
      nslot = nslot + 1 == NST ? 0 : nslot + 1;
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
  };

  if (fused) kloop(std::integral_constant<bool, true>{});
  else kloop(std::integral_constant<bool, false>{});
  __syncthreads();  // every wave is done with the ring

  float* ts = reinterpret_cast<float*>(lds);
  float* xch = ts + kTsFloats;
  const float* t_lds = nullptr;
  if (fused) {
    // t^T accumulator: lane holds ranks 8 (v / 4) + 4 hi + v % 4 of token
    // l32 of each 32-token block; staged as t[token][rank] (row stride
    // kLoraRows + 1), group 0's sums first, group 1's added
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      if (kg == g) {
#pragma unroll
        for (int j = 0; j < FM; ++j) {
          if (j % WN != wn || wn >= FM) continue;
          const int ml = wm * TM + j * 32 + l32;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            float* d = ts + ml * (kLoraRows + 1) + 8 * (v >> 2) + 4 * hi + (v & 3);
            *d = g == 0 ? scale * tacc[j][v] : *d + scale * tacc[j][v];
          }
        }
      }
      __syncthreads();
    }
    t_lds = ts;
  }

  if (kt_split > 0) epi.out_f32 += (int64_t)split * M * N;
  auto finish = [&](auto j_tag) __attribute__((always_inline)) {
    constexpr int J = decltype(j_tag)::value;  // the token block this group finishes
    float* give = xch + ((kg * NWG + wv) * FN) * 1024;
    float* take = xch + (((1 - kg) * NWG + wv) * FN) * 1024;
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) give[(i * 16 + v) * 64 + lane] = acc[i][1 - J][v];
    __syncthreads();
    f32x16 mine[FN][1];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) mine[i][0][v] = acc[i][J][v] + take[(i * 16 + v) * 64 + lane];
    lora_epilogue_store<FN, 1>(mine, n0 + wn * TN, m0 + wm * TM + 32 * J, wm * TM + 32 * J, l32, hi, M, N, b, rank,
                               r_pad, lora_cols, t_part, n_slice, t_lds, epi, out);
  };
  if (kg == 0) finish(std::integral_constant<int, 0>{});
  else finish(std::integral_constant<int, 1>{});
}

// t = scale * x A^T with MFMAs, as fp32 partial sums per slice of the hidden
// dimension (slice_w wide: 256 for the few-token GEMV, which has few token
// blocks to spread, kLoraSliceWide otherwise, so that a GEMM epilogue sums
// fewer partials): workgroup (32-token block, slice), each wave multiplies a
// 64-wide part of every 256-wide chunk of the slice and the four waves are
// summed through LDS.  t_part[slice][token][r_pad]; ranks rank .. r_pad-1
// come out zero.
__global__ __launch_bounds__(256) void lora_down_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ a,
                                                        int n_tok, int hidden, int rank, int r_pad, float scale,
                                                        int slice_w, float* __restrict__ t_part) {
  __shared__ float red[4][2][16][64];
  const int mb = blockIdx.x, kz = blockIdx.y;
  const int m0 = mb * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int nblk = (r_pad + 31) / 32;
  const int m = min(m0 + l32, n_tok - 1);
  const bf16_t* xr = x + (int64_t)m * hidden;

  f32x16 acc[2] = {f32x16{}, f32x16{}};
  for (int c0 = kz * slice_w; c0 < min(hidden, (kz + 1) * slice_w); c0 += kLoraSlice) {
    u32x4 xa[4], ab[4][2];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int k = c0 + wave * 64 + st * 16 + 8 * hf;
      const bool kin = k < hidden;
      xa[st] = kin ? *reinterpret_cast<const u32x4*>(xr + k) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int n = 32 * nb + l32;
        ab[st][nb] = (kin && nb < nblk && n < rank) ? *reinterpret_cast<const u32x4*>(a + (int64_t)n * hidden + k)
                                                   : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        if (nb < nblk) acc[nb] = mfma32(as_bf16x8(xa[st]), as_bf16x8(ab[st][nb]), acc[nb]);
  }
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

static int lora_slice_width(int n_tok) { return n_tok <= kGemvMaxTok ? kLoraSlice : kLoraSliceWide; }

int lora_down_slices(int hidden, int n_tok) {
  const int w = lora_slice_width(n_tok);
  return (hidden + w - 1) / w;
}

hipError_t launch_lora_down(const uint16_t* x, const uint16_t* a, int n_tok, int hidden, int rank, int r_pad,
                            float scale, float* t_part, hipStream_t stream) {
  if (n_tok == 0 || r_pad == 0) return hipSuccess;
  ATTUNER_LAUNCH("lora_down_kernel", lora_down_kernel,
                 dim3((n_tok + 31) / 32, lora_down_slices(hidden, n_tok)), dim3(256), stream, x, a, n_tok, hidden,
                 rank, r_pad, scale, lora_slice_width(n_tok), t_part);
  return hipGetLastError();
}

namespace {

// Sum of the n_split fp32 partials [n_split][M][N] and the epilogue of epi
// (thread = 4 consecutive outputs of one token).
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int n_split, int M, int N,
                                                            GemmEpi epi, bf16_t* out) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;  // quad index
  if (q >= (int64_t)M * N / 4) return;
  const int64_t m = q / (N / 4);
  const int n = (int)(q % (N / 4)) * 4;
  const int64_t plane = (int64_t)M * N;
  f32x4 c = *reinterpret_cast<const f32x4*>(part + m * N + n);
  for (int s = 1; s < n_split; ++s) c += *reinterpret_cast<const f32x4*>(part + s * plane + m * N + n);
  if (epi.mode == kEpiF32) {
    *reinterpret_cast<f32x4*>(epi.out_f32 + m * N + n) = c;
    return;
  }
  if (epi.mode == kEpiSwiglu) {
    const float s0 = c[0] / (1.0f + __expf(-c[0])) * c[1];
    const float s1 = c[2] / (1.0f + __expf(-c[2])) * c[3];
    *reinterpret_cast<uint32_t*>(out + m * (N / 2) + n / 2) = pack_bf16x2(s0, s1);
    return;
  }
  if (epi.mode == kEpiResidual) {
    const u32x2 r = *reinterpret_cast<const u32x2*>(epi.residual + m * N + n);
    c[0] += __uint_as_float(r[0] << 16);
    c[1] += __uint_as_float(r[0] & 0xFFFF0000u);
    c[2] += __uint_as_float(r[1] << 16);
    c[3] += __uint_as_float(r[1] & 0xFFFF0000u);
  }
  u32x2 pk;
  pk[0] = pack_bf16x2(c[0], c[1]);
  pk[1] = pack_bf16x2(c[2], c[3]);
  *reinterpret_cast<u32x2*>(out + m * N + n) = pk;
}

// rate: the operand ingest per CU the tile model assumes (measured on
// gfx950; the two-k-group kernel overlaps its MFMAs with the copies best)
struct Tile {
  int bm, bn;
  double rate;
};
constexpr Tile kTiles[] = {{256, 256, 42e9}, {128, 256, 52e9}, {256, 96, 52e9}, {128, 128, 52e9}, {128, 96, 52e9},
                           {64, 96, 52e9},   {64, 64, 52e9},   {128, 192, 60e9}, {128, 96, 60e9}};
constexpr int kNumTiles = (int)(sizeof(kTiles) / sizeof(kTiles[0]));


hipError_t launch_tile(int tile, int kt_split, int grid, const uint16_t* x, const uint16_t* w, int n_tok, int n_out,
                       int hidden, const uint16_t* a, float scale, const uint16_t* b, int rank, int r_pad,
                       int lora_cols, const float* t_part, int n_slice, GemmEpi epi, uint16_t* out,
                       hipStream_t stream) {
#define ATTUNER_GEMM(BM_, BN_, WN_, WM_, NST_, ILV_)                                                           \
  ATTUNER_LAUNCH("gemm_lora_kernel", (gemm_lora_kernel<BM_, BN_, WN_, WM_, NST_, ILV_>), dim3((unsigned)grid), \
                 dim3(64 * (WN_) * (WM_)), stream, x, w, n_tok, n_out, hidden, a, scale, b, rank, r_pad,       \
                 lora_cols, t_part, n_slice, epi, out, (n_tok + (BM_) - 1) / (BM_), n_out / (BN_), kt_split)
#define ATTUNER_GEMM_KG2(BM_, BN_, WN_, WM_, NST_)                                                             \
  ATTUNER_LAUNCH("gemm_kg2_kernel", (gemm_kg2_kernel<BM_, BN_, WN_, WM_, NST_>), dim3((unsigned)grid),       \
                 dim3(128 * (WN_) * (WM_)), stream, x, w, n_tok, n_out, hidden, a, scale, b, rank, r_pad,      \
                 lora_cols, t_part, n_slice, epi, out, (n_tok + (BM_) - 1) / (BM_), n_out / (BN_), kt_split)
  switch (tile) {
    case 0: ATTUNER_GEMM(256, 256, 4, 2, 2, true); break;
    case 1: ATTUNER_GEMM(128, 256, 4, 2, 3, false); break;
    case 2: ATTUNER_GEMM(256, 96, 3, 4, 3, false); break;
    case 3: ATTUNER_GEMM(128, 128, 2, 2, 4, false); break;
    case 4: ATTUNER_GEMM(128, 96, 3, 2, 4, false); break;
    case 5: ATTUNER_GEMM(64, 96, 3, 2, 5, false); break;
    case 6: ATTUNER_GEMM(64, 64, 2, 2, 6, false); break;
    case 7: ATTUNER_GEMM_KG2(128, 192, 2, 2, 3); break;
    case 8: ATTUNER_GEMM_KG2(128, 96, 1, 2, 4); break;
    default: return hipErrorInvalidValue;  // callers keep n_out a multiple of 64: 64x64 always fits
  }
#undef ATTUNER_GEMM
#undef ATTUNER_GEMM_KG2
  return hipGetLastError();
}

}  // namespace

// Tile and key split of a product, by a model fitted to gfx950 runs.  One
// workgroup per CU at a time; a workgroup's time is the larger of its operand
// ingest ((BM + BN) * k-range * 2 bytes at the tile's rate: about 52 GB/s per
// CU, 42 GB/s for the 256 x 256 tile whose ring holds only two k-tiles, 60
// GB/s for the two-k-group tiles) and its MFMA work
// (2 BM BN k-range at about 6 TFLOP/s per CU); a launch takes ceil(workgroups
// / 256) such rounds plus a fixed 4 us.  Without a low-rank term, and when a
// tile's workgroups would leave CUs idle, the k range may be split across
// workgroups: shorter k-loops, paid for by the fp32 partials (split * M * N *
// 8 bytes written and read at about 4 TB/s) and a 3 us reduce launch.  The
// plan minimises the model; ties go to the earlier tile and to no split.  On
// gfx950 it picks the measured fastest plan for the q/k/v projection (6144
// outputs, hidden 2560 / 4096) at T = 64 (64x64), 256 (64x96), 512 (the
// two-k-group 128x96), 1024 (the two-k-group 128x192) and 33792 (256x256),
// and for the o/gate-up/down products of the 4B and 8B layers at 256 and
// 1024 tokens (e.g. down at 256 tokens: 128x128 in 6 splits, 28.9 us against
// 46.5 us unsplit).
GemmPlan plan_gemm(int n_tok, int n_out, int k_dim, bool lora) {
  constexpr double kMfmaPerCu = 6e12, kFixed = 4e-6;
  constexpr double kPartBw = 4e12, kReduceLaunch = 3e-6;
  constexpr int kSplits[] = {1, 2, 3, 4, 6, 8, 12, 16};
  const int n_kt = k_dim / BK;
  GemmPlan best{-1, 1, 0};
  double best_t = 0.0;
  for (int i = 0; i < kNumTiles; ++i) {
    if (n_out % kTiles[i].bn != 0) continue;
    const int64_t tiles = (int64_t)((n_tok + kTiles[i].bm - 1) / kTiles[i].bm) * (n_out / kTiles[i].bn);
    const double rate = kTiles[i].rate;
    for (int s : kSplits) {
      // splits only add workgroups where the tiles alone leave CUs idle
      if (s > 1 && (lora || n_kt < 4 * s || tiles >= 256)) break;
      const int kts = (n_kt + s - 1) / s;
      const int used = (n_kt + kts - 1) / kts;  // splits that hold k-tiles
      // fp32 partials of every split: bounded, so that a reserved workspace holds any plan
      if (used > 1 && (int64_t)used * n_tok * n_out * 4 > kGemmSplitWsMaxBytes) break;
      const int64_t wgs = tiles * used;
      const double k_range = (double)kts * BK;
      const double per_wg = std::max((kTiles[i].bm + kTiles[i].bn) * k_range * 2 / rate,
                                     2.0 * kTiles[i].bm * kTiles[i].bn * k_range / kMfmaPerCu);
      double t = (double)((wgs + 255) / 256) * per_wg + kFixed;
      if (used > 1) t += (double)used * n_tok * n_out * 8 / kPartBw + kReduceLaunch;
      if (best.tile < 0 || t < best_t * (1.0 - 1e-9)) {
        best = GemmPlan{i, used, used > 1 ? kts : 0};
        best_t = t;
      }
    }
  }
  return best;
}

namespace {

hipError_t launch_gemm_any(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int hidden, const uint16_t* a,
                           float scale, const uint16_t* b, int rank, int r_pad, int lora_cols, const float* t_part,
                           GemmEpi epi, uint16_t* out, const GemmPlan* plan, float* split_ws, hipStream_t stream) {
  if (n_tok == 0) return hipSuccess;
  if (n_tok <= kGemvMaxTok)
    return launch_gemv(x, w, n_tok, n_out, hidden, b, rank, r_pad, lora_cols, t_part, epi, out, stream);
  const int n_slice = lora_down_slices(hidden, n_tok);
  const GemmPlan pl = plan ? *plan : plan_gemm(n_tok, n_out, hidden, r_pad > 0);
  if (pl.tile < 0) return hipErrorInvalidValue;
  const int tiles = ((n_tok + kTiles[pl.tile].bm - 1) / kTiles[pl.tile].bm) * (n_out / kTiles[pl.tile].bn);
  if (pl.n_split <= 1)
    return launch_tile(pl.tile, 0, tiles, x, w, n_tok, n_out, hidden, a, scale, b, rank, r_pad, lora_cols, t_part,
                       n_slice, epi, out, stream);
  if (split_ws == nullptr || r_pad > 0) return hipErrorInvalidValue;
  const GemmEpi part{kEpiF32, nullptr, split_ws};
  hipError_t e = launch_tile(pl.tile, pl.kt_split, tiles * pl.n_split, x, w, n_tok, n_out, hidden, nullptr, 0.f,
                             nullptr, 0, 0, 0, nullptr, n_slice, part, nullptr, stream);
  if (e != hipSuccess) return e;
  const int64_t quads = (int64_t)n_tok * n_out / 4;
  ATTUNER_LAUNCH("splitk_reduce_kernel", splitk_reduce_kernel, dim3((unsigned)((quads + 255) / 256)), dim3(256), stream,
                 split_ws, pl.n_split, n_tok, n_out, epi, out);
  return hipGetLastError();
}

}  // namespace

// The 256 x 256 tile's eight waves keep its MFMAs busy, so the redundant
// down-projection (every feature tile of the adapted columns computes t for
// its tokens) shows in full there: at 5368 tokens x 4096 -> 6144 (rank 16)
// 268 us fused against 244 us for lora_down_kernel + the GEMM reading t.  The
// other tiles hide it (1024 tokens, rank 32: 63.6 us fused, 67.4 separate).
bool gemm_fuses_lora(int n_tok, int n_out, int hidden) {
  return plan_gemm(n_tok, n_out, hidden, true).tile != 0;
}

hipError_t launch_gemm_lora(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int hidden,
                            const uint16_t* a, float scale, const uint16_t* b, int rank, int r_pad, int lora_cols,
                            const float* t_part, uint16_t* out, hipStream_t stream) {
  const GemmPlan pl = plan_gemm(n_tok, n_out, hidden, true);  // no key split here
  return launch_gemm_any(x, w, n_tok, n_out, hidden, a, scale, b, rank, r_pad, lora_cols, t_part,
                         GemmEpi{kEpiBf16, nullptr, nullptr}, out, &pl, nullptr, stream);
}

hipError_t launch_gemm(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int k_dim, GemmEpi epi,
                       uint16_t* out, const GemmPlan& plan, float* split_ws, hipStream_t stream) {
  return launch_gemm_any(x, w, n_tok, n_out, k_dim, nullptr, 0.f, nullptr, 0, 0, 0, nullptr, epi, out, &plan,
                         split_ws, stream);
}

}  // namespace attuner
