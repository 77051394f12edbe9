// Internal launch interface between the host runtime and the gfx950 kernels.
// Every launcher validates nothing: the runtime has checked shapes and bounds
// before calling it.  Each returns the hipError_t of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attuner {

constexpr int kMaxReq = 64;
constexpr int kHeadDim = 128;    // the kernels are built for this head size
constexpr int kPageTokens = 16;  // tokens per pool page

// Launch tracing: while tracing is on for the calling thread (attuner_trace_*),
// the runtime records a named HIP event pair on the launch stream around every
// kernel launch; otherwise these are a pointer test.
void trace_launch_begin(const char* kernel, hipStream_t stream);
void trace_launch_end(const char* kernel, hipStream_t stream);

#define ATTUNER_LAUNCH(name, kernel, grid, block, stream, ...)              \
  do {                                                                      \
    trace_launch_begin(name, stream);                                       \
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);        \
    trace_launch_end(name, stream);                                         \
  } while (0)

// Violation words of the bounds-checked build (common.h): OR the file's bits
// into *bits, clearing them when `reset`; the current device's copy.  The
// ordinary build adds nothing.
hipError_t read_violations_gather(unsigned int* bits, bool reset);
hipError_t read_violations_attention(unsigned int* bits, bool reset);
hipError_t read_violations_decode(unsigned int* bits, bool reset);

// ---- a0 / a2: pool store and block-table gather ---------------------------

// Copy one artifact (k, v: [n_layers][n_kv][n_tokens][128]) into its pages.
// pool layout: [n_layers][pool_pages][2][n_kv][16][128].
hipError_t launch_store_pages(const uint16_t* k, const uint16_t* v, int n_tokens, const int32_t* pages_dev,
                              int n_pages, uint16_t* pool, int64_t pool_pages, int n_layers, int n_kv,
                              hipStream_t stream);

// Copy every entry {page, n_valid, dst_row, request} of the block table, for
// layers layer_begin .. layer_begin + n_layers - 1, into req_kv
// [model layers][2][n_kv][cache_rows][128].  A page with kHostPageFlag set
// is page (page & ~kHostPageFlag) of the host pool (pinned host memory, same
// layout, read by the kernel over the host link); others are HBM pool pages.
constexpr int32_t kHostPageFlag = 1 << 30;
// A page with kStagePageFlag set is page (page & kPageIdMask) of the staging
// pool: device memory that host pages were copied into for the current
// assembly (same layout as the other pools).
constexpr int32_t kStagePageFlag = 1 << 29;
constexpr int32_t kPageIdMask = kStagePageFlag - 1;
hipError_t launch_gather(const int32_t* table_dev, int64_t n_entries, const uint16_t* pool, int64_t pool_pages,
                         const uint16_t* host_pool, int64_t host_pages, const uint16_t* stage_pool,
                         int64_t stage_pages, int layer_begin, int n_layers, int n_kv, uint16_t* req_kv,
                         int64_t cache_rows, hipStream_t stream);

// ---- a3: LoRA-down and the projection GEMM --------------------------------

// t = scale * x a^T as fp32 partial sums over slices of the hidden
// dimension: t_part[lora_down_slices(hidden, n_tok)][n_tok][r_pad]; ranks
// rank .. r_pad-1 are zero.  The slice count never exceeds that of one token.
int lora_down_slices(int hidden, int n_tok);
// Whether the projection GEMM of this shape computes t itself (rank <=
// kGemmFusedLoraMaxRank); otherwise launch_lora_down runs first.
bool gemm_fuses_lora(int n_tok, int n_out, int hidden);
hipError_t launch_lora_down(const uint16_t* x, const uint16_t* a, int n_tok, int hidden, int rank, int r_pad,
                            float scale, float* t_part, hipStream_t stream);

// out[i][n] = x[i] . w[n] + (n < lora_cols ? t[i] . b[n] : 0) (r_pad = 0: no
// adapter).  t is the sum of the slices of t_part when t_part is given;
// with t_part null (and r_pad <= kGemmFusedLoraMaxRank) the kernel computes
// t = scale * x a^T itself, except for n_tok <= kGemvMaxTok, which needs
// t_part.
constexpr int kGemmFusedLoraMaxRank = 32;
hipError_t launch_gemm_lora(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int hidden,
                            const uint16_t* a, float scale, const uint16_t* b, int rank, int r_pad, int lora_cols,
                            const float* t_part, uint16_t* out, hipStream_t stream);

// ---- the decoder layer around the path: plain GEMMs with other epilogues --

// What the GEMM stores for C = x W^T ([n_tok][n_out], fp32 accumulate):
//   kEpiBf16      out = C (bf16)
//   kEpiResidual  out = C + residual (bf16; residual [n_tok][n_out], may be out)
//   kEpiSwiglu    W rows interleave gate and up (row 2j = gate_j, 2j+1 = up_j):
//                 out[i][j] = silu(C[i][2j]) * C[i][2j+1] (bf16, [n_tok][n_out/2])
//   kEpiF32       out_f32 = C (fp32)
enum GemmEpiMode : int { kEpiBf16 = 0, kEpiResidual = 1, kEpiSwiglu = 2, kEpiF32 = 3 };
struct GemmEpi {
  int mode;
  const uint16_t* residual;
  float* out_f32;
};
// Tile (index into the launcher's tile list) and key split of a product:
// n_split > 1 splits the k range into chunks of kt_split 64-wide k-tiles and
// needs a workspace of n_split * n_tok * n_out floats (never with a low-rank
// term).  plan_gemm picks both by the ingest cost model.
struct GemmPlan {
  int tile;
  int n_split;
  int kt_split;
};
GemmPlan plan_gemm(int n_tok, int n_out, int k_dim, bool lora);
hipError_t launch_gemm(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int k_dim, GemmEpi epi,
                       uint16_t* out, const GemmPlan& plan, float* split_ws, hipStream_t stream);

// The same product for at most kGemvMaxTok tokens as a weight-streaming
// GEMV (any mode; the low-rank term needs t_part from launch_lora_down);
// n_out and k_dim multiples of 8.  launch_gemm_lora and launch_gemm route
// such token counts here; from 9 tokens (k_dim % 128 == 0, n_out % 16 ==
// 0) the GEMV runs on the matrix cores.
constexpr int kGemvMaxTok = 16;

// Key splits of a plain product: at most kMaxGemmSplit, and their fp32
// partials (splits x n_tok x n_out x 4 bytes) at most kGemmSplitWsMaxBytes.
constexpr int kMaxGemmSplit = 16;
constexpr int64_t kGemmSplitWsMaxBytes = (int64_t)64 << 20;
hipError_t launch_gemv(const uint16_t* x, const uint16_t* w, int n_tok, int n_out, int k_dim, const uint16_t* b,
                       int rank, int r_pad, int lora_cols, const float* t_part, GemmEpi epi, uint16_t* out,
                       hipStream_t stream);

// w_out[n] = w[n] + scale * b[n] . a for n < lora_cols, w[n] otherwise
// ([n_out][k_dim] bf16; w_out may be w).
hipError_t launch_merge_lora(const uint16_t* w, int n_out, int k_dim, const uint16_t* a, const uint16_t* b, int rank,
                             float scale, int lora_cols, uint16_t* w_out, hipStream_t stream);

// out[t] = table[ids[t]] (rows of dim bf16 elements; ids in range).
hipError_t launch_embed_rows(const uint16_t* table, const int32_t* ids, int n_tok, int dim, uint16_t* out,
                             hipStream_t stream);

// out[r] = x[rows[r]] * rsqrt(mean(x[rows[r]]^2) + eps) * gamma over `dim`
// elements (rows null: r itself); bf16 in and out, fp32 arithmetic.
hipError_t launch_rms_norm_rows(const uint16_t* x, int64_t ld_x, const int32_t* rows, int n_rows, int dim,
                                const uint16_t* gamma, float eps, uint16_t* out, hipStream_t stream);

// ids[r] = the smallest index of the largest value of logits[r][0 .. n-1]
// (fp32), max_out[r] = that value (max_out may be null).  scratch: device
// memory of argmax_scratch_bytes(n_rows) for the per-slice results.
size_t argmax_scratch_bytes(int n_rows);
hipError_t launch_argmax_rows(const float* logits, int n_rows, int n, int32_t* ids, float* max_out, void* scratch,
                              hipStream_t stream);

// ---- a4: QK-RMSNorm + RoPE ------------------------------------------------

struct NormRopeReq {
  int32_t q_start;   // first row of the request in q_raw / k_raw / v_raw / q_hat
  int32_t q_len;     // suffix tokens
  int32_t kv_row0;   // cache row of suffix token 0
  int32_t pos0;      // rotary position of suffix token 0
};

struct NormRopeParams {
  const uint16_t* q_raw;
  const uint16_t* k_raw;
  const uint16_t* v_raw;
  int64_t ld_q, ld_kv;
  const uint16_t* gamma_q;
  const uint16_t* gamma_k;
  const float2* rope;        // [max_pos][64] (cos, sin)
  uint16_t* q_hat;           // [T_q][Hq][128]
  uint16_t* k_cache;         // K head 0 of the layer; head stride kv_head_stride
  uint16_t* v_cache;
  int64_t kv_head_stride;    // elements between heads (= cache rows * 128)
  int32_t n_q_heads, n_kv_heads;
  int32_t total_q;
  float eps;
  int32_t n_req;
  NormRopeReq req[kMaxReq];
};

hipError_t launch_qk_norm_rope(const NormRopeParams& p, hipStream_t stream);

// ---- a5: attention ---------------------------------------------------------

struct AttnReq {
  int32_t q_start;   // first row in q_hat / o
  int32_t q_len;
  int32_t kv_start;  // cache row of key 0 of the request
  int32_t art_len;   // cached artifact keys; row i sees keys 0 .. art_len + i
  int32_t n_qblk;    // ceil(q_len / 64)
  int32_t wg_start;  // first work unit of the request (units = qblocks * n_split)
  int32_t n_split;   // key splits of the request's blocks (<= AttnParams::n_split)
  // n_span == 0: row i sees keys 0 .. art_len + i.  Otherwise the rows are
  // online spans packed back to back (span_row / span_off entries span0 ..
  // span0 + n_span - 1): a row of the span starting at q row R with offset
  // F sees keys 0 .. F + (row - R); positions only grow with the row.
  int32_t span0;
  int32_t n_span;
};

struct AttnParams {
  const uint16_t* q;       // [T_q][Hq][128]
  const uint16_t* k;       // K head 0; head stride kv_head_stride
  const uint16_t* v;
  int64_t kv_head_stride;
  uint16_t* o;             // [T_q][Hq][128]
  float* lse;              // [T_q][Hq] or null
  uint16_t* part_o;        // [n_split][T_q][Hq][128] bf16, normalised (n_split > 1)
  float* part_ml;          // [n_split][T_q][Hq][2]      (n_split > 1)
  int32_t n_q_heads, n_kv_heads;
  int32_t total_q;
  int32_t n_split;         // largest split count of any request: partial slices
  int32_t n_units;         // work units per KV head
  float score_scale;       // log2(e) / sqrt(d)
  int32_t n_req;
  AttnReq req[kMaxReq];
  int32_t span_row[kMaxReq];  // first q row of each packed span
  int32_t span_off[kMaxReq];  // its offset (first position) in its request's cache rows
  // Optional: copy one layer's pages (HBM pool) into the request cache beside
  // the attention, in 1 KiB chunks (4 rows of one (K|V, head) slab of one
  // block-table entry): g_chunks = entries * 2 * n_kv * 4, g_per_wg of them
  // per workgroup.  g_table null: none.  The host keeps one layer's pool and
  // cache offsets below 2^32 16-byte units.
  const int32_t* g_table;  // block table {page, n_valid, dst_row, request} per entry
  const uint16_t* g_pool;
  int64_t g_pool_pages;
  uint16_t* g_req_kv;
  int64_t g_cache_rows;
  int32_t g_chunks;        // < 2^31
  int32_t g_per_wg;
  int32_t g_layer;
  int32_t g_shift;         // log2(chunks per entry), 4 * 2 * n_kv a power of two
};

// Attention, plus the split-KV merge kernel when n_split > 1 (at most
// kMaxAttnSplit splits).
constexpr int kMaxAttnSplit = 16;
hipError_t launch_attention(const AttnParams& p, hipStream_t stream);

// ---- decode: one new token per request over its whole cache ----------------

struct DecodeReq {
  int32_t q_row;     // row of the request's token in q_raw / k_raw / v_raw / o
  int32_t kv_start;  // cache row of key 0 of the request
  int32_t n_keys;    // keys it attends to (its own, written by the launch, is the last)
  int32_t split0;    // first key chunk of the request in the launch
  int32_t n_split;   // chunks of the request (ceil(n_keys / chunk))
  int32_t pos;       // RoPE position of the new token
};

// The new token's q/k/v rows come raw from the projection: the kernel applies
// the per-head RMSNorm (gamma_q, gamma_k) and RoPE (table rope[pos][64] of
// (cos, sin)) and writes k and v into cache row kv_start + n_keys - 1.
struct DecodeParams {
  const uint16_t* q_raw;   // row r at q_raw + r * ld_q: [Hq][128]
  const uint16_t* k_raw;   // row r at k_raw + r * ld_kv: [Hkv][128]
  const uint16_t* v_raw;
  int64_t ld_q, ld_kv;
  const uint16_t* gamma_q;
  const uint16_t* gamma_k;
  const float2* rope;
  float eps;
  uint16_t* k;             // K head 0 of the cache; head stride kv_head_stride
  uint16_t* v;
  int64_t kv_head_stride;
  uint16_t* o;             // [rows][Hq][128]
  float* part_o;           // [total_splits][Hq][128] fp32, unnormalised
  float* part_ml;          // [total_splits][Hq][2] (max in log2 units, sum)
  int32_t n_q_heads, n_kv_heads;
  int32_t chunk;           // keys per chunk
  float score_scale;       // log2(e) / sqrt(d)
  int32_t n_req;
  int32_t total_splits;
  DecodeReq req[kMaxReq];
};

// Decode attention, plus the chunk merge when a request has several chunks.
hipError_t launch_decode_attention(const DecodeParams& p, hipStream_t stream);

}  // namespace attuner
