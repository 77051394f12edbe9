/*
 * attuner.h -- C ABI of the Attuner suffix-prefill library (libattuner.so).
 *
 * What it computes (Attuner, "Recomputation-Free KV Cache Reuse via
 * Query-Side Adaptation"): prefill of a request's online suffix over a frozen,
 * position-independent artifact cache.
 *   - Artifacts are encoded once, alone, with keys rotated at their own local
 *     positions 0..L-1 (section 2, eq. 2, PIC; appendix C.1, PIC).  The library
 *     keeps their per-layer K/V in a paged pool in device memory.
 *   - A request's cached blocks are put together in prompt order without
 *     re-encoding or re-rotation (section 2, the PIC box; appendix A.3,
 *     "Cache construction and reuse").
 *   - Suffix tokens get the query-side LoRA projection q = W_q h + s B (A h),
 *     s = alpha / r (section 4, eq. 4); keys and values use the plain
 *     projections, and stored artifact K/V is never modified.
 *   - q and k pass through the per-head RMSNorm and RoPE (section 4), then
 *     scaled dot-product GQA attention runs over [artifact keys ; suffix keys]
 *     with every artifact key visible and a causal mask inside the suffix
 *     (eq. 3 gives the form; appendix A.5, Deployment).
 *   - attuner_full_prefill runs the same kernels on a whole request with no
 *     cache (section 2, Full; appendix C.1, Full): the speed baseline, and,
 *     on an artifact alone at position 0, the artifact encoder.
 *
 * Conventions shared by every call:
 *   - All tensors are bfloat16 (raw 16-bit patterns) unless stated, row-major,
 *     densely packed unless a leading dimension ("ld", in elements) is given.
 *   - "device" pointers are device memory owned by the caller; the library
 *     never frees them.  "host" pointers are read before the call returns.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *     enqueues work on `stream` and returns without waiting for it, except
 *     where noted; results are valid once the stream has reached that point.
 *   - Workspaces: the context owns scratch buffers (split partials, LoRA
 *     slice partials, the full-prefill projection, logits, the RoPE table).
 *     A call that needs more than they hold grows them with hipMalloc and
 *     never waits for the device (a replaced buffer stays allocated until
 *     attuner_reserve or attuner_destroy, since queued work may read it).
 *     attuner_reserve sizes them all up front.
 *   - Graph capture: while `stream` is capturing a HIP graph, a call that
 *     would have to grow a workspace or extend the RoPE table fails with
 *     ERANGE, and a call that copies host arrays to the device
 *     (attuner_store_artifact(_host), attuner_assemble_*, attuner_embed,
 *     attuner_rms_norm with a row list) fails with EINVAL; nothing is
 *     enqueued then.  Every other call, within reserved limits, captures.
 *   - Every call returns a status; on failure nothing is enqueued, and
 *     attuner_last_error() describes the cause.  Arguments are validated on
 *     the host before any launch.
 *   - One context may be used from one host thread and one stream at a time:
 *     its internal workspaces are shared by all of its calls.
 *   - Model geometry is fixed at create time; the kernels require
 *     head_dim == 128, page_tokens == 16, n_q_heads == 4 * n_kv_heads and
 *     hidden % 64 == 0.
 */
#ifndef ATTUNER_H
#define ATTUNER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATTUNER_OK = 0,
  ATTUNER_EINVAL = -1,  /* bad argument: null pointer, shape, rank, geometry  */
  ATTUNER_ENOMEM = -2,  /* page pool full, or a device allocation failed       */
  ATTUNER_ENOENT = -3,  /* unknown artifact id                                */
  ATTUNER_EDEVICE = -4, /* a HIP runtime call failed                          */
  ATTUNER_ERANGE = -5   /* a size beyond a documented limit                   */
} attuner_status;

typedef struct {
  int32_t n_layers;    /* transformer layers whose K/V the pool holds          */
  int32_t hidden;      /* model width H (projection input size)                */
  int32_t n_q_heads;   /* Hq                                                   */
  int32_t n_kv_heads;  /* Hkv; Hq / Hkv query heads share one K/V head         */
  int32_t head_dim;    /* d (must be 128)                                      */
  int32_t page_tokens; /* tokens per pool page (must be 16)                    */
  float rope_theta;    /* rotary base (Qwen3: 1e6)                             */
  float rms_eps;       /* RMSNorm epsilon (Qwen3: 1e-6)                        */
} attuner_model_cfg;

typedef struct attuner_ctx attuner_ctx;

/* Largest number of requests in one assemble / attention call. */
#define ATTUNER_MAX_REQUESTS 64
/* Largest LoRA rank. */
#define ATTUNER_MAX_RANK 64

/* Thread-local description of the last failed call on this thread ("" if none). */
const char* attuner_last_error(void);

/* Create a context on HIP device `device` with a pool of `pool_pages` pages.
 * A page holds page_tokens tokens of K and V for every layer and KV head:
 * n_layers * 2 * n_kv_heads * page_tokens * head_dim * 2 bytes (see
 * attuner_pool_info).  The pool is the only memory allocated here; it is
 * released by attuner_destroy.  Synchronous.
 * Errors: EINVAL (geometry), ERANGE (pool_pages outside [0, 2^29)), ENOMEM
 * (allocation), EDEVICE. */
attuner_status attuner_create(const attuner_model_cfg* cfg, int64_t pool_pages, int32_t device,
                              attuner_ctx** out);

/* Release the context, its pool and workspaces.  Waits for the device. */
void attuner_destroy(attuner_ctx* ctx);

/* Limits for attuner_reserve.  A zero field reserves nothing of its kind. */
typedef struct {
  int32_t max_tokens;   /* token rows of one projection, norm/attention, full-prefill, linear, gate/up,
                           embedding or row-norm call                                               */
  int32_t max_position; /* one past the largest token position of any call (RoPE table)             */
  int32_t max_rank;     /* largest LoRA rank of attuner_qproj_lora / attuner_full_prefill            */
  int32_t max_out;      /* largest n_out of attuner_linear, 2 * n_inter of attuner_gate_up_swiglu    */
  int32_t max_lm_rows;  /* rows of one attuner_lm_head_argmax call                                  */
  int32_t max_vocab;    /* vocab of attuner_lm_head_argmax                                          */
} attuner_limits;

/* Size every workspace and the RoPE table of the context for calls within
 * `limits`, so that such calls allocate nothing (what a caller needs before
 * capturing them into a HIP graph, see the conventions above).  Also frees
 * buffers that earlier growth replaced.  Synchronous: waits for the device.
 * Errors: EINVAL (negative limit), ERANGE (max_rank > ATTUNER_MAX_RANK),
 * ENOMEM, EDEVICE. */
attuner_status attuner_reserve(attuner_ctx* ctx, const attuner_limits* limits);

/* Pool geometry and occupancy (host outputs; any may be NULL). */
attuner_status attuner_pool_info(const attuner_ctx* ctx, int64_t* pool_pages, int64_t* free_pages,
                                 int64_t* page_bytes);

/* --------------------------------------------------------------------------
 * a0: store a frozen artifact (cache construction, section 2 eq. 2, PIC).
 *
 * k, v: device [n_layers][n_kv_heads][n_tokens][head_dim], k already
 * normalised and rotated at local positions 0..n_tokens-1.  The values are
 * copied bit for bit into ceil(n_tokens / page_tokens) pool pages (unused
 * rows of the last page are zero).  The caller keeps ownership of k and v and
 * may reuse them once the stream has passed this call.  *artifact_id receives
 * a new id (>= 0).
 * Errors: EINVAL (n_tokens <= 0, null pointer), ENOMEM (pool full).
 * ------------------------------------------------------------------------ */
attuner_status attuner_store_artifact(attuner_ctx* ctx, int32_t n_tokens, const void* k, const void* v,
                                      void* stream, int32_t* artifact_id);

/* Return an artifact's pages to the pool.  Work already enqueued that reads
 * them must have completed before the pages are reused by a later store.
 * Errors: ENOENT. */
attuner_status attuner_release_artifact(attuner_ctx* ctx, int32_t artifact_id);

/* Physical page ids of an artifact as block tables carry them (host pool
 * pages with ATTUNER_HOST_PAGE_FLAG set), in token order (host output of up
 * to max_pages entries), its page count and its token count.  Errors:
 * ENOENT, ERANGE (max_pages too small; *n_pages still set). */
attuner_status attuner_artifact_pages(const attuner_ctx* ctx, int32_t artifact_id, int32_t* pages_out,
                                      int32_t max_pages, int32_t* n_pages, int32_t* n_tokens);

/* --------------------------------------------------------------------------
 * Artifact caches kept in CPU RAM: the paper stores the artifact caches in
 * host memory and copies what a request uses to the GPU inside the timed
 * region (appendix A.2: CPU RAM cache lookup and GPU transfer are timed).
 *
 * attuner_host_pool_create gives the context a second pool of host_pages
 * pages (same page size and layout as the HBM pool) in pinned host memory
 * mapped for the device (hipHostMalloc), released by attuner_destroy; once
 * per context.  attuner_store_artifact_host stores an artifact there (k, v
 * as for attuner_store_artifact, device memory; the copy runs on `stream`);
 * its id is used like any other: every assembly call gathers its pages
 * straight from host memory over the host link into the request cache (the
 * same gather kernel; per layer with attuner_gather_layers, so a layer's
 * transfer can overlap earlier layers' compute).  Block tables carry host
 * pages as (page | ATTUNER_HOST_PAGE_FLAG).  attuner_release_artifact returns
 * pages to the pool they came from.
 * Errors: EINVAL (no host pool / a second one), ERANGE (host_pages outside
 * [1, 2^29)), ENOMEM (pinned allocation, host pool full), EDEVICE.
 * ------------------------------------------------------------------------ */
#define ATTUNER_HOST_PAGE_FLAG (1 << 30)

attuner_status attuner_host_pool_create(attuner_ctx* ctx, int64_t host_pages);

attuner_status attuner_store_artifact_host(attuner_ctx* ctx, int32_t n_tokens, const void* k, const void* v,
                                           void* stream, int32_t* artifact_id);

attuner_status attuner_host_pool_info(const attuner_ctx* ctx, int64_t* host_pages, int64_t* free_pages);

/* --------------------------------------------------------------------------
 * a1 + a2: assemble request caches (section 2, the PIC box; appendix A.3).
 *
 * A batch of n_req requests, CSR over host arrays: request r uses artifacts
 * artifact_ids[req_ptr[r] .. req_ptr[r+1]) in that (prompt) order; ids may
 * repeat; a request may have none.  suffix_cap[r] rows are reserved after
 * its artifacts for the suffix tokens.
 *
 * Request r owns rows [cu_ctx[r], cu_ctx[r+1]) of the assembled cache, with
 * cu_ctx[0] = 0 and cu_ctx[r+1] = cu_ctx[r] + art_len[r] + suffix_cap[r];
 * its artifacts fill rows cu_ctx[r] .. cu_ctx[r] + art_len[r] - 1 back to
 * back.  The cache (req_kv, device) is laid out
 *     [n_layers][2 (K, V)][n_kv_heads][cache_rows][head_dim]
 * with cache_rows = cu_ctx[n_req].  attuner_assemble_plan returns n_entries
 * and cache_rows so the caller can size its buffers.
 *
 * The block table (device, n_entries x 4 int32) gets one entry per logical
 * page, in request, artifact, page order:
 *     { physical page, valid tokens, first destination row, request }.
 * It is built on the host and copied to block_table asynchronously; the
 * gather kernel then copies every page of every layer into req_kv (one
 * launch).  Rows outside the artifacts (the suffix rows) are not written.
 * cu_ctx (host, n_req + 1) and art_len (host, n_req) receive the layout.
 * Errors: EINVAL, ENOENT (unknown id), ERANGE (n_req > ATTUNER_MAX_REQUESTS,
 * or cache_rows does not match the plan).
 * ------------------------------------------------------------------------ */
attuner_status attuner_assemble_plan(const attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                     const int32_t* artifact_ids, const int32_t* suffix_cap,
                                     int64_t* n_entries, int64_t* cache_rows);

attuner_status attuner_assemble_kv(attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                   const int32_t* artifact_ids, const int32_t* suffix_cap,
                                   int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                   void* req_kv, int64_t cache_rows, void* stream);

/* --------------------------------------------------------------------------
 * a1 and a2 apart (same method and layout as attuner_assemble_kv, which is
 * attuner_assemble_table followed by attuner_gather_layers over all layers).
 *
 * attuner_assemble_table plans the batch on the host and copies the block
 * table to block_table on `stream`; it fills cu_ctx and art_len as
 * attuner_assemble_kv does and copies no cache rows.
 *
 * attuner_gather_layers copies the pages of layers layer_begin ..
 * layer_begin + n_layers - 1 into req_kv, leaving the other layers' rows
 * untouched, so a caller can gather layer l on one stream while earlier
 * layers compute on another (ordering the two with events).  block_table,
 * n_entries and cache_rows must be the block table, entry count and cache
 * rows of the last attuner_assemble_table call on this context, and the
 * device table must not have been modified since (the copy trusts its
 * entries); anything else is refused with EINVAL.  Errors: EINVAL (also a
 * null or unaligned req_kv), ERANGE (layers outside [0, n_layers)).
 * ------------------------------------------------------------------------ */
attuner_status attuner_assemble_table(attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                      const int32_t* artifact_ids, const int32_t* suffix_cap,
                                      int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                      int64_t cache_rows, void* stream);

attuner_status attuner_gather_layers(attuner_ctx* ctx, const int32_t* block_table, int64_t n_entries,
                                     int32_t layer_begin, int32_t n_layers, void* req_kv,
                                     int64_t cache_rows, void* stream);

/* --------------------------------------------------------------------------
 * Host-pool artifacts moved by bulk copies into HBM (the transfer of
 * appendix A.2, done per layer so that it overlaps the compute of earlier
 * layers; a bulk copy holds far fewer wave slots than the gather kernel
 * reading host memory page by page, and a page that several requests use
 * crosses the host link once).
 *
 * attuner_stage_pool_create gives the context a staging pool of stage_pages
 * pages in HBM (same page size and layout as the other pools; released by
 * attuner_destroy); once per context.
 *
 * attuner_assemble_table_staged is attuner_assemble_table, except that every
 * distinct host page the batch uses gets a staging page (the i-th smallest
 * host page id gets staging page i; a page used by several requests is
 * staged once) and the block table names the staging page, as
 * (page | ATTUNER_STAGE_PAGE_FLAG); HBM-pool pages are unchanged.
 * *staged_pages (may be null) receives the number of distinct host pages.
 * It also records the copies that attuner_stage_layers makes: one per
 * maximal range of consecutive host page ids.
 *
 * attuner_stage_layers copies layers layer_begin .. layer_begin + n_layers - 1
 * of those host pages into the staging pool with hipMemcpyAsync on `stream`
 * (from the pinned host pool: one copy per run and layer; the HIP runtime
 * chooses the engine; for these copies it uses the DMA engines, so they
 * occupy no compute units).  attuner_gather_layers over the staged table then moves the staged
 * pages of a layer into the request cache like any HBM page; the caller
 * orders each layer's gather after that layer's staging copy (same stream,
 * or an event).  The call is the last staged assembly's: once another
 * assembly call is made on the context it is refused with EINVAL.  Under
 * graph capture the copies of the current plan are recorded; a replay makes
 * those same copies, so a captured graph belongs to one batch plan (the same
 * artifacts in the same order give the same plan).  The staging pool is
 * shared by every call on the context: a staged assembly must not start
 * while copies or gathers of the previous one may still be running unless
 * both use the same plan.
 * Errors: EINVAL (no staging pool / a second one; the last assembly not
 * staged), ERANGE (stage_pages outside [1, 2^29); more distinct host pages
 * than stage_pages; layers outside [0, n_layers)), ENOMEM, EDEVICE; otherwise
 * as attuner_assemble_table.
 *
 * attuner_stage_pool_info: the staging pool's size and the number of copy
 * runs per layer of the current plan (0 when the last assembly was not
 * staged).
 * ------------------------------------------------------------------------ */
#define ATTUNER_STAGE_PAGE_FLAG (1 << 29)

attuner_status attuner_stage_pool_create(attuner_ctx* ctx, int64_t stage_pages);

attuner_status attuner_assemble_table_staged(attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                             const int32_t* artifact_ids, const int32_t* suffix_cap,
                                             int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                             int64_t cache_rows, int64_t* staged_pages, void* stream);

attuner_status attuner_stage_layers(attuner_ctx* ctx, int32_t layer_begin, int32_t n_layers, void* stream);

attuner_status attuner_stage_pool_info(const attuner_ctx* ctx, int64_t* stage_pages, int64_t* runs);

/* --------------------------------------------------------------------------
 * Prompts that interleave cached artifacts with online spans (appendix A.3:
 * system text, headers, separators and the question sit between and around
 * the cached artifacts and are computed online, while the artifacts' KV is
 * put together in the original prompt order; appendix A.5: attention with
 * the causal mask and the position ids of the assembled context).
 *
 * Request r is the segment list segments[req_ptr[r] .. req_ptr[r+1]) in
 * prompt order: an entry >= 0 is an artifact id, an entry -n < 0 an online
 * span of n tokens.  Request r owns cache rows [cu_ctx[r], cu_ctx[r+1]): its
 * whole prompt, artifact pages where the artifacts sit and rows left for the
 * online spans where they sit (same cache layout as attuner_assemble_kv).
 * attuner_assemble_segments_plan returns n_entries, cache_rows and the
 * number of online spans.  attuner_assemble_segments builds the block table
 * (entries as in attuner_assemble_kv, copied to block_table on `stream`),
 * gathers every layer into req_kv, fills cu_ctx (host, n_req + 1) and spans
 * (host, n_spans x 3: request, offset of the span inside its request,
 * length; in request and prompt order), and records the table for
 * attuner_gather_layers.  Online rows are not written.
 * Errors: EINVAL, ENOENT (unknown id), ERANGE (n_req > ATTUNER_MAX_REQUESTS,
 * cache_rows does not match the plan).
 * ------------------------------------------------------------------------ */
attuner_status attuner_assemble_segments_plan(const attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                              const int32_t* segments, int64_t* n_entries,
                                              int64_t* cache_rows, int32_t* n_spans);

attuner_status attuner_assemble_segments(attuner_ctx* ctx, int32_t n_req, const int32_t* req_ptr,
                                         const int32_t* segments, int32_t* block_table, int32_t* cu_ctx,
                                         int32_t* spans, void* req_kv, int64_t cache_rows, void* stream);

/* --------------------------------------------------------------------------
 * a3: LoRA-adapted projection (section 4, eq. 4; fused q/k/v weights).
 *
 *   out[i][n] = sum_k x[i][k] w[n][k]
 *             + (n < lora_cols ? scale * sum_j (sum_k x[i][k] a[j][k]) b[n][j] : 0)
 *
 * x: device [n_tok][hidden]; w: device [n_out][hidden]; a: device
 * [rank][hidden]; b: device [lora_cols][rank]; out: device [n_tok][n_out].
 * Accumulation is fp32; out is rounded to bf16 once.  rank == 0 (a, b may be
 * NULL) is the plain projection, i.e. the merged-weight deployment form.
 * With w = [W_q; W_k; W_v] and lora_cols = n_q_heads * head_dim the keys and
 * values stay unadapted, as the method requires.
 * Requires n_out % 128 == 0, lora_cols % 32 == 0, lora_cols <= n_out,
 * 0 <= rank <= ATTUNER_MAX_RANK, n_tok >= 0.  Uses a context workspace
 * (grown with hipMalloc on first use at a larger n_tok or rank).
 * ------------------------------------------------------------------------ */
attuner_status attuner_qproj_lora(attuner_ctx* ctx, int32_t n_tok, const void* x, const void* w,
                                  int32_t n_out, const void* a, const void* b, int32_t rank, float scale,
                                  int32_t lora_cols, void* out, void* stream);

/* Deployment form of the adapter (appendix A.5: the learned update is merged
 * into the query projection, W_Q <- W_Q + (alpha/r) B A, for online
 * inference; attuner_qproj_lora with rank 0 then runs the merged weights).
 * w_out[n][k] = w[n][k] + scale * sum_j b[n][j] a[j][k] for rows n <
 * lora_cols (fp32 sum, one bf16 rounding), w_out[n][k] = w[n][k] for the
 * other rows.  w, w_out: device [n_out][k_dim] bf16 (w_out may be w); a:
 * [rank][k_dim]; b: [lora_cols][rank].  k_dim a multiple of 8; 0 <= rank <=
 * ATTUNER_MAX_RANK (rank 0: a copy).  Errors: EINVAL, ERANGE. */
attuner_status attuner_merge_lora(attuner_ctx* ctx, const void* w, int32_t n_out, int32_t k_dim,
                                  const void* a, const void* b, int32_t rank, float scale,
                                  int32_t lora_cols, void* w_out, void* stream);

/* --------------------------------------------------------------------------
 * a4: per-head QK-RMSNorm + RoPE of the suffix (section 4: the base model's
 * q-norm and rotary embedding apply to the adapted query unchanged).
 *
 * Per request r (host arrays of n_req entries, cu_q of n_req + 1): suffix
 * tokens are rows cu_q[r] .. cu_q[r+1]-1 of q_raw/k_raw/v_raw; token i of the
 * request sits at position pos0[r] + i.
 *   q_hat = rope(gamma_q * q / sqrt(mean(q^2) + eps))   per query head
 *   k_hat = rope(gamma_k * k / sqrt(mean(k^2) + eps))   per KV head
 * rope pairs dimension j with j + 64 and turns it by (pos) * theta^(-2j/128)
 * (angles from an fp64 host table, stored fp32).
 * q_raw: device, row stride ld_q, Hq*d columns; k_raw, v_raw: device, row
 * stride ld_kv, Hkv*d columns; gamma_q, gamma_k: device [head_dim].  All five
 * 16-byte aligned and ld_q, ld_kv multiples of 8 (else ATTUNER_EINVAL).
 * q_hat: device [T_q][Hq][d].  k_hat and v of request r's token i are written
 * to cache row cu_ctx[r] + art_len[r] + i of layer `layer` of req_kv
 * (layout of attuner_assemble_kv).  Requires art_len[r] + (cu_q[r+1] -
 * cu_q[r]) <= cu_ctx[r+1] - cu_ctx[r].
 * ------------------------------------------------------------------------ */
attuner_status attuner_qk_norm_rope(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                    const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                    const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                    int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* q_hat,
                                    void* req_kv, int64_t cache_rows, void* stream);

/* --------------------------------------------------------------------------
 * a5: multi-segment GQA attention over an assembled cache (eq. 3 form with
 * the causal mask; appendix A.5).
 *
 * Suffix token i of request r, query head h, reads KV head h / (Hq / Hkv) at
 * cache rows cu_ctx[r] + j for j = 0 .. art_len[r] + i: all artifact keys and
 * the suffix causally.  o[t][h][:] = sum_j softmax_j(q_hat . k_j / sqrt(d)) v_j.
 * q_hat: device [T_q][Hq][d]; o: device [T_q][Hq][d] (bf16);
 * lse: device [T_q][Hq] fp32 natural-log sum of exp of the scaled scores, or
 * NULL.  o may alias q_hat exactly (same pointer).  The cached rows
 * art_len[r] .. art_len[r] + q_len - 1 must already hold the suffix keys and
 * values (attuner_qk_norm_rope writes them).
 * ------------------------------------------------------------------------ */
attuner_status attuner_attention(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                 const int32_t* cu_ctx, const int32_t* art_len, const void* q_hat,
                                 const void* req_kv, int64_t cache_rows, void* o, float* lse, void* stream);

/* a4 + a5 in one call: q_raw/k_raw/v_raw as in attuner_qk_norm_rope; the
 * normalised queries are staged in `o`, which then receives the attention
 * output [T_q][Hq][d]. */
attuner_status attuner_suffix_attn(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                   const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                   const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                   int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                   int64_t cache_rows, void* o, float* lse, void* stream);

/* attuner_suffix_attn for `layer` that also performs
 * attuner_gather_layers(ctx, block_table, n_entries, gather_layer, 1, req_kv,
 * cache_rows, stream): the layer-by-layer prefill of section 2 (equation 3)
 * copies each layer's cached artifact pages (appendix A.2) before that
 * layer's attention, and this call lets the copy of the next layer ride in
 * the attention launch of this one, where it overlaps the attention's
 * matrix work.  Results are bit-identical to the two calls made apart.
 *   block_table, n_entries, cache_rows: those of the last
 *   attuner_assemble_table call (else ATTUNER_EINVAL), as for
 *   attuner_gather_layers.  gather_layer in [0, n_layers) (else
 *   ATTUNER_ERANGE) and != layer (else ATTUNER_EINVAL): the attention
 *   reads `layer`'s rows while the copy writes gather_layer's.
 * The copy rides in the attention launch when every page of that table is
 * in the HBM pool, 8 n_kv_heads is a power of two, one layer's pool and
 * cache planes are below 4 GiB, and the attention's key tiles can carry at
 * least half of the copy (each wave moves 1 KiB per tile it passes);
 * otherwise (host or staged pages, other shapes, no suffix tokens, short
 * key ranges) the copy runs as a gather launch of its own on `stream`,
 * before the attention.  Other arguments, outputs and errors as
 * attuner_suffix_attn. */
attuner_status attuner_suffix_attn_gather(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                          const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                          const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                          int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                          int64_t cache_rows, void* o, float* lse, const int32_t* block_table,
                                          int64_t n_entries, int32_t gather_layer, void* stream);

/* Size of the fixed device buffer of attuner_suffix_attn_noalloc (per device). */
#define ATTUNER_NOALLOC_SCRATCH_BYTES (24 << 20)

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * attuner_suffix_attn with its key-split partials in a fixed device buffer
 * of ATTUNER_NOALLOC_SCRATCH_BYTES (24 MiB) instead of a context workspace;
 * arguments, outputs and errors as attuner_suffix_attn.  The call allocates
 * nothing and never waits for the device.  The buffer is part of the
 * library's code object: one copy per device, located when the first
 * context is created on that device and held until the process ends.
 *   - The split plan is limited to plans whose partials fit the buffer:
 *     n_split x (query rows) x Hq x (2 head_dim + 8) bytes <= 24 MiB.  A batch
 *     whose usual plan does not fit runs with fewer key splits (same result
 *     within the parity bar); every batch the other call takes is accepted.
 *   - Token positions must lie in the context's RoPE table (4096 positions
 *     from create; attuner_reserve extends it); this call does not extend
 *     it: ERANGE otherwise.
 *   - Every call on a device shares that device's buffer, which keeps the
 *     last call's contents: calls that overlap on one device (other streams,
 *     contexts or threads) race and must be ordered by the caller.  Nothing
 *     in it has to start at zero: a call reads only partials it wrote.
 * Errors: as attuner_suffix_attn; ERANGE (position past the RoPE table);
 * EDEVICE (the buffer's device address could not be looked up). */
attuner_status attuner_suffix_attn_noalloc(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                           const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                           const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                           int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                           int64_t cache_rows, void* o, float* lse, void* stream);

/* --------------------------------------------------------------------------
 * a6: full-context prefill of one layer with the same kernels (section 2,
 * Full; appendix C.1, Full).
 *
 * x: device [n_tok][hidden] at positions pos0 .. pos0 + n_tok - 1; wqkv: device
 * [(Hq + 2 Hkv) d][hidden] (rows W_q, then W_k, then W_v); a, b, rank, scale
 * as in attuner_qproj_lora on the query rows (rank 0 = no adapter, the
 * paper's Full).  Plain causal attention over the n_tok tokens.
 * o: device [n_tok][Hq][d]; k_out, v_out: device [n_kv_heads][n_tok][d]
 * (normalised/rotated keys and raw values: with pos0 = 0 on an artifact
 * alone, the K/V attuner_store_artifact expects for one layer);
 * lse: device [n_tok][Hq] fp32 or NULL.  o, k_out, v_out, gamma_q and gamma_k
 * must be 16-byte aligned (else ATTUNER_EINVAL).  Uses context workspaces.
 * ------------------------------------------------------------------------ */
attuner_status attuner_full_prefill(attuner_ctx* ctx, int32_t n_tok, int32_t pos0, const void* x,
                                    const void* wqkv, const void* a, const void* b, int32_t rank,
                                    float scale, const void* gamma_q, const void* gamma_k, void* o,
                                    void* k_out, void* v_out, float* lse, void* stream);

/* --------------------------------------------------------------------------
 * a4 + a5 for online spans at any offsets (the interleaved prompts above;
 * the suffix of attuner_suffix_attn is the case of one span at the end).
 *
 * Span s (host arrays of n_spans <= ATTUNER_MAX_REQUESTS entries, cu_q of
 * n_spans + 1): its tokens are rows cu_q[s] .. cu_q[s+1]-1 of q_raw/k_raw/
 * v_raw/o; its request's cache rows start at kv_start[s] and the span sits
 * offset[s] rows into them; token i has position pos0[s] + i (pos0 NULL:
 * offset[s] + i, the assembled position).  The call normalises and rotates
 * q and k, writes k_hat and v to rows kv_start[s] + offset[s] + i of layer
 * `layer` (every span's rows first), then token i of span s attends to rows
 * kv_start[s] .. kv_start[s] + offset[s] + i: everything before it in its
 * prompt (artifact keys as stored, earlier spans' keys as just written) and
 * its own span causally.  Requires kv_start[s] + offset[s] + (cu_q[s+1] -
 * cu_q[s]) <= cache_rows.  q_raw/k_raw/v_raw/ld/gamma as in
 * attuner_qk_norm_rope; o: device [T][Hq][d] (also stages the normalised
 * queries); lse: device [T][Hq] fp32 or NULL.
 * ------------------------------------------------------------------------ */
attuner_status attuner_span_attn(attuner_ctx* ctx, int32_t layer, int32_t n_spans, const int32_t* cu_q,
                                 const int32_t* kv_start, const int32_t* offset, const int32_t* pos0,
                                 const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                 int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                 int64_t cache_rows, void* o, float* lse, void* stream);

/* --------------------------------------------------------------------------
 * Decode with the adapted queries: every generated token keeps the adapted
 * query projection (section 4: the adapter acts on all online tokens), and
 * attends to its request's whole assembled context (eq. 3 with one query
 * row).  One new token per request; its q/k/v rows come from
 * attuner_qproj_lora on those tokens (row r = request r).
 *
 * Request r has ctx_len[r] keys already in its cache rows cu_ctx[r] ..
 * (artifacts, suffix and earlier generated tokens, as attuner_assemble_kv and
 * earlier calls left them).  The call normalises and rotates the new q and k
 * at position pos[r] (NULL: ctx_len[r]), writes k_hat and v into cache row
 * cu_ctx[r] + ctx_len[r] of layer `layer`, and writes
 * o[r][h][:] = sum_j softmax_j(q_hat . k_j / sqrt(d)) v_j over the
 * ctx_len[r] + 1 keys j = 0 .. ctx_len[r].  Requires ctx_len[r] + 1 <=
 * cu_ctx[r+1] - cu_ctx[r] (the suffix capacity given to the assembly must
 * cover the generated tokens) and n_q_heads = 4 n_kv_heads.  q_raw/k_raw/
 * v_raw/ld_q/ld_kv/gamma as in attuner_qk_norm_rope (the normalisation and
 * rotation run inside the decode launch); o: device [n_req][Hq][d] bf16, not
 * overlapping q_raw, k_raw or v_raw.  Long contexts are split into key
 * chunks merged in fp32 (context workspace).
 * ------------------------------------------------------------------------ */
attuner_status attuner_decode_attn(attuner_ctx* ctx, int32_t layer, int32_t n_req, const int32_t* cu_ctx,
                                   const int32_t* ctx_len, const int32_t* pos, const void* q_raw,
                                   int64_t ld_q, const void* k_raw, const void* v_raw, int64_t ld_kv,
                                   const void* gamma_q, const void* gamma_k, void* req_kv,
                                   int64_t cache_rows, void* o, void* stream);

/* --------------------------------------------------------------------------
 * The decoder layer around the path (the models the method adapts are Qwen3
 * decoder stacks, section 5.1; the greedy first token ends the timed region
 * of the paper's time-to-first-token, appendix A.2).  With
 * these calls a caller chains real layers: h -> rms_norm -> (a3..a5) ->
 * linear(o, W_o, residual h) -> rms_norm -> gate_up_swiglu -> linear(.,
 * W_down, residual) -> next layer; then rms_norm of the last token of each
 * request and lm_head_argmax.  All tensors are bf16 device buffers, 16-byte
 * aligned, rows contiguous; errors EINVAL / ERANGE before any launch.
 *
 * attuner_embed: out[t] = table[token_ids[t]] for t < n_tok: the suffix
 *   tokens' embedding rows, the residual stream entering layer 0.  token_ids:
 *   host int32, each in [0, vocab) (else ERANGE); table: [vocab][hidden];
 *   out: [n_tok][hidden].  Copies the ids through a context workspace.
 *
 * attuner_rms_norm: out[r] = x[rows[r]] / sqrt(mean(x[rows[r]]^2) + eps) * gamma
 *   over the model's hidden size (<= 8192), fp32 arithmetic.  x holds
 *   n_x_rows rows of stride ld_x (>= hidden, multiple of 8); rows (host int32,
 *   n_rows entries, each in [0, n_x_rows)) or NULL for rows 0 .. n_rows - 1;
 *   out: [n_rows][hidden].  eps is the context's rms_eps.
 *
 * attuner_linear: out[n_tok][n_out] = x[n_tok][k_dim] w[n_out][k_dim]^T
 *   (+ residual[n_tok][n_out] when residual is not NULL; residual may be
 *   out).  fp32 accumulation, one bf16 rounding.  k_dim and n_out: positive
 *   multiples of 64.
 *
 * attuner_gate_up_swiglu: out[n_tok][n_inter] = silu(x W_gate^T) * (x W_up^T)
 *   with silu(z) = z / (1 + e^-z) (the SwiGLU MLP).  w_gu: [2 n_inter][k_dim]
 *   with gate row j at row 2j and up row j at row 2j + 1.  n_inter: a
 *   positive multiple of 32; k_dim: a positive multiple of 64.
 *
 * attuner_lm_head_argmax: ids[r] = argmax_v x[r] . w_lm[v] over v < vocab
 *   (fp32 logits; ties go to the smallest index), max_logit[r] = that logit
 *   (max_logit may be NULL).  x: [n_rows][hidden]; w_lm: [vocab][hidden];
 *   vocab a positive multiple of 64; ids (int32) and max_logit (fp32) on the
 *   device.  Uses a context workspace of n_rows * vocab floats.
 * ------------------------------------------------------------------------ */
attuner_status attuner_embed(attuner_ctx* ctx, int32_t n_tok, const int32_t* token_ids,
                             const void* table, int32_t vocab, void* out, void* stream);

attuner_status attuner_rms_norm(attuner_ctx* ctx, const void* x, int64_t n_x_rows, int64_t ld_x,
                                const int32_t* rows, int32_t n_rows, const void* gamma, void* out,
                                void* stream);

attuner_status attuner_linear(attuner_ctx* ctx, int32_t n_tok, const void* x, int32_t k_dim,
                              const void* w, int32_t n_out, const void* residual, void* out,
                              void* stream);

attuner_status attuner_gate_up_swiglu(attuner_ctx* ctx, int32_t n_tok, const void* x, int32_t k_dim,
                                      const void* w_gu, int32_t n_inter, void* out, void* stream);

attuner_status attuner_lm_head_argmax(attuner_ctx* ctx, int32_t n_rows, const void* x,
                                      const void* w_lm, int32_t vocab, int32_t* ids,
                                      float* max_logit, void* stream);

/* --------------------------------------------------------------------------
 * Kernel timing.  Between attuner_trace_begin and attuner_trace_end, every
 * kernel this library launches from the calling thread is bracketed by a
 * pair of HIP events on its stream.  attuner_trace_end waits for the
 * recorded events and returns, per kernel name, the launch count, the summed
 * and the largest event-to-event time, sorted by total time (host array of
 * up to max_entries; *n_entries receives the number of kernels).  Do not
 * trace while a stream is being captured into a graph.
 * Errors: EINVAL (no trace open on this thread for ctx), ERANGE (max_entries
 * too small; *n_entries still set), EDEVICE.
 * ------------------------------------------------------------------------ */
typedef struct {
  char kernel[48];
  int64_t launches;
  double total_ms;
  double max_ms;
} attuner_kernel_time;

attuner_status attuner_trace_begin(attuner_ctx* ctx);
attuner_status attuner_trace_end(attuner_ctx* ctx, attuner_kernel_time* out, int32_t max_entries,
                                 int32_t* n_entries);

/* --------------------------------------------------------------------------
 * Bounds-checked build (a debugging aid; no passage of the paper defines it:
 * it guards the paged assembly of section 2 and appendix A.3).
 * libattuner_checked.so is this library compiled with device-side tests,
 * before each use, of every block-table entry the gather and the attention
 * launch's page copy read (page id within its pool, n_valid within a page,
 * destination rows within the request-cache plane), of the page ids the
 * store writes, and of the query rows and key ranges the attention and
 * decode launches read (within the buffers they were given).  A failed test
 * sets one of the bits below in a word in device memory and the access is
 * skipped (that entry, or the whole workgroup), so a corrupted table or range
 * is reported instead of faulting; results of skipped work are undefined.
 * Same entry points and arguments as libattuner.so.
 * ------------------------------------------------------------------------ */
#define ATTUNER_VIOL_GATHER_PAGE (1u << 0)   /* gather: page id past its pool, or that pool absent */
#define ATTUNER_VIOL_GATHER_ROWS (1u << 1)   /* gather: n_valid past a page, or rows past the cache plane */
#define ATTUNER_VIOL_STORE_PAGE (1u << 2)    /* store: page id past the pool */
#define ATTUNER_VIOL_ATTN_RANGE (1u << 3)    /* attention: query rows or key range past its buffers */
#define ATTUNER_VIOL_COPY_ENTRY (1u << 4)    /* attention's page copy: entry outside its pool or cache plane */
#define ATTUNER_VIOL_DECODE_RANGE (1u << 5)  /* decode: key range past the cache plane */

/* *checked = 1 in libattuner_checked.so, 0 in libattuner.so.  No device work.
 * Errors: EINVAL (null checked). */
attuner_status attuner_bounds_checked(int32_t* checked);

/* Waits for all work on `device` to finish (a blocking diagnostic call; not
 * for use while a stream is capturing), then stores in *bits the OR of the
 * ATTUNER_VIOL_* bits the kernels have set on that device since the last
 * reset, and clears them when reset != 0.  The ordinary build stores 0 and
 * touches no device.
 * Errors: EINVAL (null bits, device out of range), EDEVICE (a HIP error,
 * including one left by earlier work on the device). */
attuner_status attuner_bounds_violations(int32_t device, int32_t reset, uint32_t* bits);

#ifdef __cplusplus
}
#endif

#endif /* ATTUNER_H */
