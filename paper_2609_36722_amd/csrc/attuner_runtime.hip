// Host runtime of libattuner: context, paged artifact pool, block-table
// builder, workspaces, launch planning and the C ABI declared in attuner.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <queue>
#include <set>
#include <string>
#include <vector>

#include "attuner.h"
#include "kernels.h"

using namespace attuner;

namespace {

thread_local std::string g_last_error;

attuner_status fail(attuner_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(ATTUNER_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Positions of the RoPE table built at create time (attuner_reserve or a
// later call may extend it).
constexpr int64_t kRopeInitPositions = 4096;
// Largest (splits x query rows) of an attention launch with key splits: the
// partials then take at most this many rows of Hq x (2 d + 8) bytes.
constexpr int64_t kAttnSplitRowsMax = 16384;

// true when `stream` is capturing work into a HIP graph.  A failed query
// counts as capturing (the caller then refuses to allocate).
bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &st) != hipSuccess) {
    (void)hipGetLastError();
    return true;
  }
  return st != hipStreamCaptureStatusNone;
}

// Growable device buffer.  Growth never waits for the device: the old
// buffer, which work already enqueued may still read, goes to a retired list
// that is freed when the context is destroyed or attuner_reserve runs.
struct DeviceBuf {
  void* ptr = nullptr;
  size_t cap = 0;
  hipError_t grow(size_t bytes, std::vector<void*>& retired) {
    if (bytes <= cap) return hipSuccess;
    const size_t want = std::max(bytes, cap * 2);
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, want);
    if (e != hipSuccess) return e;
    if (ptr) retired.push_back(ptr);
    ptr = p;
    cap = want;
    return hipSuccess;
  }
  void release() {
    if (ptr) (void)hipFree(ptr);
    ptr = nullptr;
    cap = 0;
  }
};

// Pinned host staging for small host->device uploads (block tables, page
// lists).  Two slots used in turn; a slot is refilled only after the copy
// that last read it has completed.
struct Staging {
  void* host[2] = {nullptr, nullptr};
  size_t cap[2] = {0, 0};
  hipEvent_t done[2] = {nullptr, nullptr};
  bool pending[2] = {false, false};
  int next = 0;

  // (callers check first that `stream` is not capturing: a captured copy
  // would re-read this slot at every replay, long after it was refilled)
  hipError_t upload(const void* src, size_t bytes, void* dst_dev, hipStream_t stream) {
    if (bytes == 0) return hipSuccess;
    const int s = next;
    next ^= 1;
    hipError_t e;
    if (pending[s]) {
      e = hipEventSynchronize(done[s]);
      if (e != hipSuccess) return e;
      pending[s] = false;
    }
    if (done[s] == nullptr) {
      e = hipEventCreateWithFlags(&done[s], hipEventDisableTiming);
      if (e != hipSuccess) return e;
    }
    if (cap[s] < bytes) {
      if (host[s]) (void)hipHostFree(host[s]);
      host[s] = nullptr;
      cap[s] = 0;
      const size_t want = std::max(bytes, (size_t)1 << 16);
      e = hipHostMalloc(&host[s], want, hipHostMallocDefault);
      if (e != hipSuccess) {
        host[s] = nullptr;
        return e;
      }
      cap[s] = want;
    }
    memcpy(host[s], src, bytes);
    e = hipMemcpyAsync(dst_dev, host[s], bytes, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return e;
    e = hipEventRecord(done[s], stream);
    if (e != hipSuccess) return e;
    pending[s] = true;
    return hipSuccess;
  }
  void release() {
    for (int s = 0; s < 2; ++s) {
      if (pending[s]) (void)hipEventSynchronize(done[s]);
      if (done[s]) (void)hipEventDestroy(done[s]);
      if (host[s]) (void)hipHostFree(host[s]);
      host[s] = nullptr;
      done[s] = nullptr;
    }
  }
};

struct Artifact {
  std::vector<int32_t> pages;  // page indices in its pool
  int32_t n_tokens;
  bool host = false;           // pages of the host pool
  // the page id as block tables carry it
  int32_t table_page(int32_t pg) const { return host ? (pg | kHostPageFlag) : pg; }
};

// Named HIP event pairs around kernel launches (attuner_trace_*).  Events
// come from a pool that is reused from one trace to the next.
struct Tracer {
  struct Rec {
    const char* name;
    hipEvent_t start, stop;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
  hipError_t err = hipSuccess;

  hipEvent_t take() {
    if (pool_used < pool.size()) return pool[pool_used++];
    hipEvent_t e = nullptr;
    // no system-scope fence at each record: the markers then perturb the
    // kernels they bracket (and their caches) as little as possible
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) {
      err = r;
      return nullptr;
    }
    pool.push_back(e);
    ++pool_used;
    return e;
  }
  void release() {
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    pool.clear();
    recs.clear();
    pool_used = 0;
  }
};

thread_local Tracer* g_tracer = nullptr;

}  // namespace

namespace attuner {

void trace_launch_begin(const char* kernel, hipStream_t stream) {
  Tracer* t = g_tracer;
  if (t == nullptr) return;
  Tracer::Rec r{kernel, t->take(), t->take()};
  if (r.start == nullptr || r.stop == nullptr) return;
  hipError_t e = hipEventRecord(r.start, stream);
  if (e != hipSuccess) t->err = e;
  t->recs.push_back(r);
}

void trace_launch_end(const char* kernel, hipStream_t stream) {
  Tracer* t = g_tracer;
  if (t == nullptr || t->recs.empty() || t->recs.back().name != kernel) return;
  hipError_t e = hipEventRecord(t->recs.back().stop, stream);
  if (e != hipSuccess) t->err = e;
}

}  // namespace attuner

// ---- fixed device scratch of attuner_suffix_attn_noalloc --------------------
// One copy per device, allocated with the code object and held until the
// process ends.  Host code never uses the name `scratch` as an address (on
// the host it is only a stand-in for the symbol): its device address is
// looked up once per device and kept in g_scratch.
static __device__ __align__(256) char scratch[ATTUNER_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;

struct ScratchSlot {
  bool looked_up = false;
  hipError_t err = hipSuccess;
  void* ptr = nullptr;
};

std::mutex g_scratch_mu;
ScratchSlot g_scratch[kMaxDevices];

// Look up the device address of `scratch` on `device`, which must be the
// current device; once per device (later calls return the first result).
hipError_t locate_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ScratchSlot& sl = g_scratch[device];
  if (!sl.looked_up) {
    void* ptr = nullptr;
    sl.err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (sl.err != hipSuccess) {
      (void)hipGetLastError();
      ptr = nullptr;
    }
    sl.ptr = ptr;
    sl.looked_up = true;
  }
  return sl.err;
}

void* scratch_ptr(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch[device].looked_up && g_scratch[device].err == hipSuccess ? g_scratch[device].ptr : nullptr;
}

}  // namespace

struct attuner_ctx {
  attuner_model_cfg cfg;
  int device = 0;
  int64_t pool_pages = 0;
  int64_t page_bytes = 0;  // one page, all layers
  uint16_t* pool = nullptr;
  std::set<int32_t> free_pages;
  // host pool: pinned, mapped host memory (host pointer and its device alias)
  int64_t host_pages = 0;
  uint16_t* host_pool = nullptr;
  uint16_t* host_pool_dev = nullptr;
  std::set<int32_t> host_free;
  // staging pool in HBM (same layout) for host pages moved by the copy
  // engines, and the copies the last staged assembly planned: runs of
  // {first host page, first staging page, pages}
  int64_t stage_pages = 0;
  uint16_t* stage_pool = nullptr;
  std::vector<std::array<int32_t, 3>> stage_runs;
  bool last_staged = false;
  std::map<int32_t, Artifact> artifacts;
  int32_t next_id = 0;

  std::vector<void*> retired;       // device buffers replaced by growth (freed at destroy / reserve)
  std::vector<void*> retired_host;  // pinned RoPE uploads (freed likewise)
  DeviceBuf ws_pages;   // page list of the artifact being stored
  DeviceBuf ws_lora;    // LoRA-down slice partials
  DeviceBuf ws_part;    // split-KV partials
  DeviceBuf ws_qkv;     // full prefill: fused projection output
  DeviceBuf ws_logits;  // LM-head logits (fp32)
  DeviceBuf ws_split;   // key-split partials of a plain product (fp32)
  DeviceBuf ws_rows;    // token ids of an embedding lookup / rows of a row-subset RMSNorm
  DeviceBuf rope;       // (cos, sin) table [rope_pos][64]
  int64_t rope_pos = 0;
  // the block table the last attuner_assemble_table call wrote (the only one
  // attuner_gather_layers accepts)
  const int32_t* last_table = nullptr;
  int64_t last_entries = -1, last_rows = -1;
  bool last_hbm_only = false;  // every page of that table is an HBM-pool page
  // key splits chosen for the last attention batch shape (q_len, art_len per
  // request), reused while the shape repeats (every layer of a stack)
  std::vector<int32_t> split_shape;
  std::vector<int> split_plan;
  std::vector<int> split_order;  // launch order of the requests' workgroups
  Staging staging;
  Tracer tracer;
};

namespace {

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

int q_dim(const attuner_ctx* c) { return c->cfg.n_q_heads * c->cfg.head_dim; }
int kv_dim(const attuner_ctx* c) { return c->cfg.n_kv_heads * c->cfg.head_dim; }

// Grow a workspace to `bytes` for a call on `stream` (no device wait; see
// DeviceBuf).  Refused while the stream is capturing a graph: the allocation
// would not be part of the graph, so the caller reserves first.
attuner_status grow(attuner_ctx* c, DeviceBuf& buf, size_t bytes, hipStream_t stream, const char* what) {
  if (bytes <= buf.cap) return ATTUNER_OK;
  if (capturing(stream))
    return fail(ATTUNER_ERANGE, "the %s workspace must grow to %zu bytes (has %zu) while the stream is capturing a "
                                "graph: size it first with attuner_reserve", what, bytes, buf.cap);
  hipError_t e = buf.grow(bytes, c->retired);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(ATTUNER_ENOMEM, "%s workspace of %zu bytes: %s", what, bytes, hipGetErrorString(e));
  }
  return ATTUNER_OK;
}

// Host -> device upload of a small host array through the pinned staging
// slots; refused while the stream is capturing.
attuner_status upload_host(attuner_ctx* c, const void* src, size_t bytes, void* dst, hipStream_t stream,
                           const char* what) {
  if (bytes == 0) return ATTUNER_OK;
  if (capturing(stream))
    return fail(ATTUNER_EINVAL, "%s copies a host array to the device and cannot be captured into a graph", what);
  HIP_TRY(c->staging.upload(src, bytes, dst, stream));
  return ATTUNER_OK;
}

// Refuse a call that uploads a host array while `stream` is capturing,
// before anything else of the call happens.
attuner_status upload_check(attuner_ctx* c, hipStream_t stream, const char* what) {
  (void)c;
  if (capturing(stream))
    return fail(ATTUNER_EINVAL, "%s copies a host array to the device and cannot be captured into a graph", what);
  return ATTUNER_OK;
}

// (cos, sin) of pos * theta^(-2j/128) for pos < n, evaluated in double and
// stored fp32.  Growth builds the new table in pinned host memory and copies
// it on `stream` (no device wait); the old table stays alive for work
// already enqueued.  Refused while the stream is capturing.
attuner_status ensure_rope(attuner_ctx* c, int64_t n, hipStream_t stream) {
  if (n <= c->rope_pos) return ATTUNER_OK;
  if (capturing(stream))
    return fail(ATTUNER_ERANGE, "position %lld is past the RoPE table (%lld positions) while the stream is capturing a "
                                "graph: size it first with attuner_reserve", (long long)n - 1, (long long)c->rope_pos);
  int64_t want = std::max<int64_t>(kRopeInitPositions, c->rope_pos);
  while (want < n) want *= 2;
  const size_t bytes = (size_t)want * 64 * 2 * sizeof(float);
  float* tab = nullptr;
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&tab), bytes, hipHostMallocDefault);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(ATTUNER_ENOMEM, "pinned RoPE table of %zu bytes: %s", bytes, hipGetErrorString(e));
  }
  c->retired_host.push_back(tab);
  const double theta = c->cfg.rope_theta;
  for (int j = 0; j < 64; ++j) {
    const double inv_freq = std::pow(theta, -2.0 * j / 128.0);
    for (int64_t p = 0; p < want; ++p) {
      const double ang = (double)p * inv_freq;
      tab[((size_t)p * 64 + j) * 2] = (float)std::cos(ang);
      tab[((size_t)p * 64 + j) * 2 + 1] = (float)std::sin(ang);
    }
  }
  DeviceBuf fresh;
  e = fresh.grow(bytes, c->retired);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(ATTUNER_ENOMEM, "RoPE table of %zu bytes: %s", bytes, hipGetErrorString(e));
  }
  HIP_TRY(hipMemcpyAsync(fresh.ptr, tab, bytes, hipMemcpyHostToDevice, stream));
  if (c->rope.ptr) c->retired.push_back(c->rope.ptr);
  c->rope = fresh;
  c->rope_pos = want;
  return ATTUNER_OK;
}

// Wait for the device, then free what growth retired.
attuner_status free_retired(attuner_ctx* c) {
  if (c->retired.empty() && c->retired_host.empty()) return ATTUNER_OK;
  HIP_TRY(hipDeviceSynchronize());
  for (void* p : c->retired) (void)hipFree(p);
  for (void* p : c->retired_host) (void)hipHostFree(p);
  c->retired.clear();
  c->retired_host.clear();
  return ATTUNER_OK;
}

// One request of a norm+rope / attention batch, in host form.
struct ReqDesc {
  int32_t q_start, q_len, kv_start, art_len, pos0;
  int32_t span0 = 0, n_span = 0;  // packed online spans (attention only; see AttnReq)
};

// A packed online span for the attention pass: its first q row and offset.
struct SpanRow {
  int32_t row, off;
};

attuner_status run_norm_rope(attuner_ctx* c, const std::vector<ReqDesc>& reqs, int32_t total_q, const void* q_raw,
                             int64_t ld_q, const void* k_raw, const void* v_raw, int64_t ld_kv, const void* gamma_q,
                             const void* gamma_k, void* q_hat, uint16_t* k_plane, uint16_t* v_plane,
                             int64_t head_stride, hipStream_t stream) {
  int64_t max_pos = 0;
  for (const auto& r : reqs) max_pos = std::max<int64_t>(max_pos, (int64_t)r.pos0 + r.q_len);
  attuner_status st = ensure_rope(c, max_pos, stream);
  if (st != ATTUNER_OK) return st;
  NormRopeParams p;
  memset(&p, 0, sizeof p);
  p.q_raw = static_cast<const uint16_t*>(q_raw);
  p.k_raw = static_cast<const uint16_t*>(k_raw);
  p.v_raw = static_cast<const uint16_t*>(v_raw);
  p.ld_q = ld_q;
  p.ld_kv = ld_kv;
  p.gamma_q = static_cast<const uint16_t*>(gamma_q);
  p.gamma_k = static_cast<const uint16_t*>(gamma_k);
  p.rope = static_cast<const float2*>(c->rope.ptr);
  p.q_hat = static_cast<uint16_t*>(q_hat);
  p.k_cache = k_plane;
  p.v_cache = v_plane;
  p.kv_head_stride = head_stride;
  p.n_q_heads = c->cfg.n_q_heads;
  p.n_kv_heads = c->cfg.n_kv_heads;
  p.total_q = total_q;
  p.eps = c->cfg.rms_eps;
  p.n_req = (int32_t)reqs.size();
  for (size_t r = 0; r < reqs.size(); ++r) {
    p.req[r].q_start = reqs[r].q_start;
    p.req[r].q_len = reqs[r].q_len;
    p.req[r].kv_row0 = reqs[r].kv_start + reqs[r].art_len;
    p.req[r].pos0 = reqs[r].pos0;
  }
  HIP_TRY(launch_qk_norm_rope(p, stream));
  return ATTUNER_OK;
}

// Key splits per request for one attention launch, and the order in which
// the requests' workgroups are launched.  A workgroup serves one 64-token
// query block of one KV head (one per CU at a time) over a range of key
// tiles; workgroups start in launch order on whichever CU frees first.  The
// modelled finish time of a plan is that greedy schedule over 256 CUs, with
// a workgroup costing its tiles plus kWgOverhead tiles (loading Q and the
// first tile, the epilogue) and a plan with splits paying kMergeCost for the
// merge launch.  Candidates cut the longest request into k = 1 .. 16 splits
// (split size tau = its tiles / k) and every request into ceil(its tiles /
// tau); each is modelled with the requests in their own order and in order
// of decreasing workgroup length (longest first, which shortens the tail of
// a batch of unequal contexts); a candidate with more splits must be
// modelled 2% faster to win.  *order receives the launch order.
std::vector<int> plan_attention_splits(attuner_ctx* c, const std::vector<ReqDesc>& reqs, int64_t split_rows_max,
                                       std::vector<int>* order) {
  std::vector<int32_t> shape;
  shape.reserve(2 * reqs.size() + 1);
  shape.push_back((int32_t)split_rows_max);
  for (const auto& r : reqs) {
    shape.push_back(r.q_len);
    shape.push_back(r.art_len);
  }
  if (shape == c->split_shape) {
    if (order) *order = c->split_order;
    return c->split_plan;
  }
  constexpr double kWgOverhead = 4.0, kMergeCost = 3.0;
  constexpr int kCUs = 256;
  std::vector<int64_t> tiles(reqs.size(), 0);
  int64_t longest = 0;
  for (size_t r = 0; r < reqs.size(); ++r) {
    if (reqs[r].q_len <= 0) continue;
    tiles[r] = ((int64_t)reqs[r].art_len + reqs[r].q_len + 63) / 64;
    longest = std::max(longest, tiles[r]);
  }
  int64_t total_q = 0;
  for (const auto& r : reqs) total_q += std::max(0, r.q_len);
  std::vector<int> best(reqs.size(), 1), cand(reqs.size(), 1);
  std::vector<int> best_order(reqs.size()), in_order(reqs.size()), longest_first(reqs.size());
  for (size_t r = 0; r < reqs.size(); ++r) best_order[r] = in_order[r] = (int)r;
  double best_t = -1.0;
  int64_t prev_tau = -1;
  for (int k = 1; k <= kMaxAttnSplit && longest > 0; ++k) {
    const int64_t tau = std::max<int64_t>(4, (longest + k - 1) / k);
    if (tau == prev_tau) continue;
    prev_tau = tau;
    bool any_split = false;
    int max_ns = 1;
    for (size_t r = 0; r < reqs.size(); ++r) {
      cand[r] = (int)std::min<int64_t>(kMaxAttnSplit, std::max<int64_t>(1, (tiles[r] + tau - 1) / tau));
      any_split |= cand[r] > 1;
      max_ns = std::max(max_ns, cand[r]);
    }
    // the partials hold max_ns x total_q rows; plans past the cap are skipped
    if (any_split && (int64_t)max_ns * total_q > split_rows_max) continue;
    // longest workgroups first (ties: request order)
    longest_first = in_order;
    std::stable_sort(longest_first.begin(), longest_first.end(), [&](int a, int b) {
      return tiles[a] * cand[b] > tiles[b] * cand[a];  // tiles / splits, compared without division
    });
    for (const std::vector<int>* ord : {&in_order, &longest_first}) {
      std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
      for (int i = 0; i < kCUs; ++i) free_at.push(0.0);
      double finish = 0.0;
      for (int r : *ord) {
        const int nq = (reqs[r].q_len + 63) / 64;
        const int ns = cand[r];
        for (int u = 0; u < nq * ns; ++u) {
          const int split = u % ns, qb = nq - 1 - u / ns;
          const int64_t t0 = 64LL * qb;
          const int64_t n_t = ((int64_t)reqs[r].art_len + t0 + std::min<int64_t>(64, reqs[r].q_len - t0) + 63) / 64;
          const int64_t per = (n_t + ns - 1) / ns;
          const int64_t tb = std::min<int64_t>(n_t, split * per), te = std::min<int64_t>(n_t, tb + per);
          const double dur = (double)(te - tb) + kWgOverhead;
          for (int g = 0; g < c->cfg.n_kv_heads; ++g) {
            const double t = free_at.top() + dur;
            free_at.pop();
            free_at.push(t);
            finish = std::max(finish, t);
          }
        }
      }
      if (any_split) finish += kMergeCost;
      if (best_t < 0.0 || finish < 0.98 * best_t) {
        best_t = finish;
        best = cand;
        best_order = *ord;
      }
    }
  }
  c->split_shape = shape;
  c->split_plan = best;
  c->split_order = best_order;
  if (order) *order = best_order;
  return best;
}

// Key-split partials of one attention launch: n_split x total_q x Hq rows
// of a normalised bf16 O row and an fp32 (max, sum) pair.
size_t split_row_bytes(const attuner_ctx* c) {
  return (size_t)c->cfg.n_q_heads * (c->cfg.head_dim * sizeof(uint16_t) + 2 * sizeof(float));
}

// part_buf / part_bytes: a caller-provided buffer for the key-split
// partials (the plan is then limited to what fits); null: the context's
// workspace, grown as needed.
// A copy of one layer's pages that the attention launch carries (AttnParams
// g_*), or with `apart` a gather launch of its own before the attention.
struct GatherArgs {
  const int32_t* table;
  int64_t entries;
  int32_t layer;
  uint16_t* req_kv;
  int64_t cache_rows;
  bool apart;
};

hipError_t launch_gather_apart(attuner_ctx* c, const GatherArgs& g, hipStream_t stream) {
  return launch_gather(g.table, g.entries, c->pool, c->pool_pages, c->host_pool_dev, c->host_pages, c->stage_pool,
                       c->stage_pages, g.layer, 1, c->cfg.n_kv_heads, g.req_kv, g.cache_rows, stream);
}

attuner_status run_attention(attuner_ctx* c, const std::vector<ReqDesc>& reqs, int32_t total_q, const void* q,
                             const uint16_t* k_plane, const uint16_t* v_plane, int64_t head_stride, void* o,
                             float* lse, hipStream_t stream, const std::vector<SpanRow>* spans = nullptr,
                             void* part_buf = nullptr, size_t part_bytes = 0, const GatherArgs* gather = nullptr) {
  AttnParams p;
  memset(&p, 0, sizeof p);
  p.q = static_cast<const uint16_t*>(q);
  p.k = k_plane;
  p.v = v_plane;
  p.kv_head_stride = head_stride;
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.n_q_heads = c->cfg.n_q_heads;
  p.n_kv_heads = c->cfg.n_kv_heads;
  p.total_q = total_q;
  p.score_scale = (float)(1.4426950408889634 / std::sqrt((double)c->cfg.head_dim));
  p.n_req = (int32_t)reqs.size();

  const int64_t rows_max =
      part_buf ? std::min<int64_t>(kAttnSplitRowsMax, (int64_t)(part_bytes / split_row_bytes(c))) : kAttnSplitRowsMax;
  std::vector<int> order;
  const std::vector<int> ns_plan = plan_attention_splits(c, reqs, rows_max, &order);
  int n_split = 1;
  int32_t units = 0;
  // table entry i is request order[i]: the kernel needs only each entry's
  // workgroups to be contiguous, and every entry carries its own rows
  for (size_t i = 0; i < order.size(); ++i) {
    const int r = order[i];
    const int nq = (reqs[r].q_len + 63) / 64;
    const int ns = ns_plan[r];
    n_split = std::max(n_split, ns);
    p.req[i].q_start = reqs[r].q_start;
    p.req[i].q_len = reqs[r].q_len;
    p.req[i].kv_start = reqs[r].kv_start;
    p.req[i].art_len = reqs[r].art_len;
    p.req[i].n_qblk = nq;
    p.req[i].wg_start = units;
    p.req[i].n_split = ns;
    p.req[i].span0 = reqs[r].span0;
    p.req[i].n_span = reqs[r].n_span;
    units += nq * ns;
  }
  if (spans)
    for (size_t i = 0; i < spans->size(); ++i) {
      p.span_row[i] = (*spans)[i].row;
      p.span_off[i] = (*spans)[i].off;
    }
  p.n_split = n_split;
  p.n_units = units;
  if (gather != nullptr && gather->apart) {
    HIP_TRY(launch_gather_apart(c, *gather, stream));
    gather = nullptr;
  }
  if (gather != nullptr) {
    // Each workgroup takes an equal share of the copy's 1 KiB chunks, and
    // each of its 8 waves moves one chunk per key tile it passes; what the
    // tiles do not cover is copied after the tile loop, at a lower rate than
    // a gather launch of its own.  When that remainder would exceed half
    // the copy (short key ranges), the copy runs as its own launch instead.
    const int n_slab = 2 * c->cfg.n_kv_heads;
    const int64_t chunks = gather->entries * n_slab * 4;
    const int64_t wgs = (int64_t)units * c->cfg.n_kv_heads;
    const int64_t per_wg = (chunks + wgs - 1) / wgs;
    int64_t left = 0;
    for (size_t i = 0; i < order.size(); ++i) {
      const AttnReq& rq = p.req[i];
      for (int qb = 0; qb < rq.n_qblk; ++qb) {
        const int64_t kv_len = (int64_t)rq.art_len + std::min(rq.q_len, (qb + 1) * 64);
        const int64_t n_tiles = (kv_len + 63) / 64, per = (n_tiles + rq.n_split - 1) / rq.n_split;
        for (int sp = 0; sp < rq.n_split; ++sp) {
          const int64_t tb = std::min(n_tiles, sp * per), syncs = std::min(n_tiles, tb + per) - tb;
          left += c->cfg.n_kv_heads * std::max<int64_t>(0, per_wg - 8 * syncs);
        }
      }
    }
    if (2 * left > chunks) {
      HIP_TRY(launch_gather_apart(c, *gather, stream));
      gather = nullptr;
    }
  }
  if (gather != nullptr) {
    const int n_slab = 2 * c->cfg.n_kv_heads;
    const int64_t chunks = gather->entries * n_slab * 4;
    const int64_t wgs = (int64_t)units * c->cfg.n_kv_heads;
    p.g_table = gather->table;
    p.g_pool = c->pool;
    p.g_pool_pages = c->pool_pages;
    p.g_req_kv = gather->req_kv;
    p.g_cache_rows = gather->cache_rows;
    p.g_chunks = (int32_t)chunks;
    p.g_per_wg = (int32_t)((chunks + wgs - 1) / wgs);
    p.g_layer = gather->layer;
    int shift = 0;
    while ((1 << shift) < n_slab * 4) ++shift;
    p.g_shift = shift;
  }
  if (n_split > 1) {
    const size_t rows = (size_t)n_split * total_q * c->cfg.n_q_heads;
    const size_t po = rows * c->cfg.head_dim * sizeof(uint16_t);
    void* buf = part_buf;
    if (buf != nullptr) {
      if (po + rows * 2 * sizeof(float) > part_bytes)
        return fail(ATTUNER_ERANGE, "key-split partials of %zu bytes exceed the %zu-byte buffer",
                    po + rows * 2 * sizeof(float), part_bytes);
    } else {
      attuner_status st = grow(c, c->ws_part, po + rows * 2 * sizeof(float), stream, "key-split partials");
      if (st != ATTUNER_OK) return st;
      buf = c->ws_part.ptr;
    }
    p.part_o = static_cast<uint16_t*>(buf);
    p.part_ml = reinterpret_cast<float*>(static_cast<char*>(buf) + po);
  }
  HIP_TRY(launch_attention(p, stream));
  return ATTUNER_OK;
}

// One new token per request (reqs[r].q_len == 1, row r): attention over the
// request's art_len + 1 keys, cut into equal chunks.
attuner_status run_decode(attuner_ctx* c, const std::vector<ReqDesc>& reqs, const void* q_raw, int64_t ld_q,
                          const void* k_raw, const void* v_raw, int64_t ld_kv, const void* gamma_q,
                          const void* gamma_k, uint16_t* k_plane, uint16_t* v_plane, int64_t head_stride, void* o,
                          hipStream_t stream) {
  int64_t max_pos = 0;
  for (const auto& r : reqs) max_pos = std::max<int64_t>(max_pos, (int64_t)r.pos0 + 1);
  attuner_status st = ensure_rope(c, max_pos, stream);
  if (st != ATTUNER_OK) return st;
  DecodeParams p;
  memset(&p, 0, sizeof p);
  p.q_raw = static_cast<const uint16_t*>(q_raw);
  p.k_raw = static_cast<const uint16_t*>(k_raw);
  p.v_raw = static_cast<const uint16_t*>(v_raw);
  p.ld_q = ld_q;
  p.ld_kv = ld_kv;
  p.gamma_q = static_cast<const uint16_t*>(gamma_q);
  p.gamma_k = static_cast<const uint16_t*>(gamma_k);
  p.rope = static_cast<const float2*>(c->rope.ptr);
  p.eps = c->cfg.rms_eps;
  p.k = k_plane;
  p.v = v_plane;
  p.kv_head_stride = head_stride;
  p.o = static_cast<uint16_t*>(o);
  p.n_q_heads = c->cfg.n_q_heads;
  p.n_kv_heads = c->cfg.n_kv_heads;
  p.score_scale = (float)(1.4426950408889634 / std::sqrt((double)c->cfg.head_dim));
  p.n_req = (int32_t)reqs.size();
  // Chunks are a multiple of 64 keys (one step of the 32 key groups x 2),
  // at least two steps.  Two workgroups fit a CU (VGPRs and LDS).  Measured
  // on one request of 8.4k and 33.8k keys and on 16 requests of 128k keys in
  // all: the smallest chunk whose workgroups fit 256 (one per CU: longer
  // chunks amortise each workgroup's prologue and merge, and the chunk merge
  // has fewer slices); failing that within 2048 keys, the smallest whose
  // workgroups fit 512 (one round of two per CU); failing that, the smallest
  // whose workgroups fit 1024 (two full rounds, not one round and a thin
  // tail).
  auto wgs_for = [&](int32_t ch) {
    int64_t wgs = 0;
    for (const auto& r : reqs) wgs += ((int64_t)r.art_len + 1 + ch - 1) / ch;
    return wgs * c->cfg.n_kv_heads;
  };
  // (a chunk past the longest request's keys cannot lower the count further)
  int64_t max_keys = 1;
  for (const auto& r : reqs) max_keys = std::max<int64_t>(max_keys, (int64_t)r.art_len + 1);
  const int32_t whole = (int32_t)std::max<int64_t>(128, (max_keys + 63) / 64 * 64);
  auto smallest_fitting = [&](int64_t limit, int32_t max_chunk) {
    int32_t ch = 128;
    while (wgs_for(ch) > limit && ch < max_chunk) ch += 64;
    return ch;
  };
  int32_t chunk = smallest_fitting(256, std::min(2048, whole));
  if (wgs_for(chunk) > 256) chunk = smallest_fitting(512, std::min(2048, whole));
  if (wgs_for(chunk) > 512) chunk = smallest_fitting(1024, whole);
  p.chunk = chunk;
  int32_t splits = 0;
  for (size_t r = 0; r < reqs.size(); ++r) {
    const int32_t n_keys = reqs[r].art_len + 1;
    p.req[r].q_row = reqs[r].q_start;
    p.req[r].kv_start = reqs[r].kv_start;
    p.req[r].n_keys = n_keys;
    p.req[r].split0 = splits;
    p.req[r].n_split = (n_keys + p.chunk - 1) / p.chunk;
    p.req[r].pos = reqs[r].pos0;
    splits += p.req[r].n_split;
  }
  p.total_splits = splits;
  if (splits > (int32_t)reqs.size()) {
    const size_t rows = (size_t)splits * c->cfg.n_q_heads;
    const size_t po = rows * c->cfg.head_dim * sizeof(float);
    st = grow(c, c->ws_part, po + rows * 2 * sizeof(float), stream, "decode chunk partials");
    if (st != ATTUNER_OK) return st;
    p.part_o = static_cast<float*>(c->ws_part.ptr);
    p.part_ml = reinterpret_cast<float*>(static_cast<char*>(c->ws_part.ptr) + po);
  }
  HIP_TRY(launch_decode_attention(p, stream));
  return ATTUNER_OK;
}

// Validate the per-request host arrays of a norm/attention call against a cache.
attuner_status build_reqs(const attuner_ctx* c, int32_t n_req, const int32_t* cu_q, const int32_t* cu_ctx,
                          const int32_t* art_len, const int32_t* pos0, int64_t cache_rows,
                          std::vector<ReqDesc>* out, int32_t* total_q) {
  if (n_req < 0 || n_req > ATTUNER_MAX_REQUESTS)
    return fail(ATTUNER_ERANGE, "n_req %d outside [0, %d]", n_req, ATTUNER_MAX_REQUESTS);
  if (n_req > 0 && (!cu_q || !cu_ctx || !art_len)) return fail(ATTUNER_EINVAL, "null request array");
  (void)c;
  out->clear();
  if (n_req == 0) {
    *total_q = 0;
    return ATTUNER_OK;
  }
  if (cu_q[0] != 0 || cu_ctx[0] != 0) return fail(ATTUNER_EINVAL, "cu_q[0] and cu_ctx[0] must be 0");
  for (int r = 0; r < n_req; ++r) {
    ReqDesc d;
    d.q_start = cu_q[r];
    d.q_len = cu_q[r + 1] - cu_q[r];
    d.kv_start = cu_ctx[r];
    d.art_len = art_len[r];
    d.pos0 = pos0 ? pos0[r] : art_len[r];
    const int64_t rows = (int64_t)cu_ctx[r + 1] - cu_ctx[r];
    if (d.q_len < 0 || rows < 0 || d.art_len < 0 || d.pos0 < 0)
      return fail(ATTUNER_EINVAL, "request %d: negative length or position", r);
    if ((int64_t)d.art_len + d.q_len > rows)
      return fail(ATTUNER_EINVAL, "request %d: art_len %d + suffix %d exceeds its %lld cache rows", r, d.art_len,
                  d.q_len, (long long)rows);
    out->push_back(d);
  }
  if ((int64_t)cu_ctx[n_req] > cache_rows)
    return fail(ATTUNER_EINVAL, "cu_ctx[n_req] = %d exceeds cache_rows %lld", cu_ctx[n_req], (long long)cache_rows);
  *total_q = cu_q[n_req];
  return ATTUNER_OK;
}

attuner_status check_layer(const attuner_ctx* c, int32_t layer) {
  if (layer < 0 || layer >= c->cfg.n_layers)
    return fail(ATTUNER_EINVAL, "layer %d outside [0, %d)", layer, c->cfg.n_layers);
  return ATTUNER_OK;
}

uint16_t* cache_plane(void* req_kv, const attuner_ctx* c, int layer, int kv, int64_t cache_rows) {
  return static_cast<uint16_t*>(req_kv) +
         ((int64_t)layer * 2 + kv) * c->cfg.n_kv_heads * cache_rows * c->cfg.head_dim;
}

attuner_status qproj_impl(attuner_ctx* c, int32_t n_tok, const void* x, const void* w, int32_t n_out,
                          const void* a, const void* b, int32_t rank, float scale, int32_t lora_cols, void* out,
                          hipStream_t stream) {
  if (n_tok < 0) return fail(ATTUNER_EINVAL, "n_tok < 0");
  if (rank < 0 || rank > ATTUNER_MAX_RANK) return fail(ATTUNER_ERANGE, "rank %d outside [0, %d]", rank, ATTUNER_MAX_RANK);
  if (n_out <= 0 || n_out % 128 != 0) return fail(ATTUNER_EINVAL, "n_out %d must be a positive multiple of 128", n_out);
  if (rank > 0 && (lora_cols < 0 || lora_cols % 32 != 0 || lora_cols > n_out))
    return fail(ATTUNER_EINVAL, "lora_cols %d must be a multiple of 32 in [0, n_out]", lora_cols);
  if (n_tok == 0) return ATTUNER_OK;
  if (!x || !w || !out) return fail(ATTUNER_EINVAL, "null x, w or out");
  if (rank > 0 && (!a || !b)) return fail(ATTUNER_EINVAL, "rank %d needs a and b", rank);
  if (!aligned16(x) || !aligned16(w) || !aligned16(out) || (rank > 0 && !aligned16(a)))
    return fail(ATTUNER_EINVAL, "x, w, a and out must be 16-byte aligned");
  const int hidden = c->cfg.hidden;
  const int r_pad = rank > 0 && lora_cols > 0 ? (rank + 15) / 16 * 16 : 0;
  // ranks up to kGemmFusedLoraMaxRank: the GEMM computes t = scale * x A^T
  // itself where its tile hides the work; larger ranks, the GEMV of a few
  // tokens and the largest tile take a separate down-projection kernel first
  float* t_part = nullptr;
  if (r_pad > 0 && (r_pad > kGemmFusedLoraMaxRank || n_tok <= kGemvMaxTok || !gemm_fuses_lora(n_tok, n_out, hidden))) {
    const size_t part_bytes = (size_t)lora_down_slices(hidden, n_tok) * n_tok * r_pad * sizeof(float);
    attuner_status st = grow(c, c->ws_lora, part_bytes, stream, "LoRA down-projection");
    if (st != ATTUNER_OK) return st;
    t_part = static_cast<float*>(c->ws_lora.ptr);
    HIP_TRY(launch_lora_down(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(a), n_tok, hidden, rank,
                             r_pad, scale, t_part, stream));
  }
  HIP_TRY(launch_gemm_lora(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), n_tok, n_out, hidden,
                           static_cast<const uint16_t*>(a), scale, static_cast<const uint16_t*>(b), rank, r_pad,
                           lora_cols, t_part, static_cast<uint16_t*>(out), stream));
  return ATTUNER_OK;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================

extern "C" {

const char* attuner_last_error(void) { return g_last_error.c_str(); }

attuner_status attuner_create(const attuner_model_cfg* cfg, int64_t pool_pages, int32_t device, attuner_ctx** out) {
  g_last_error.clear();
  if (!cfg || !out) return fail(ATTUNER_EINVAL, "null cfg or out");
  *out = nullptr;
  if (cfg->head_dim != kHeadDim) return fail(ATTUNER_EINVAL, "head_dim %d: kernels are built for 128", cfg->head_dim);
  if (cfg->page_tokens != kPageTokens)
    return fail(ATTUNER_EINVAL, "page_tokens %d: kernels are built for 16", cfg->page_tokens);
  if (cfg->n_kv_heads <= 0 || cfg->n_q_heads != 4 * cfg->n_kv_heads)
    return fail(ATTUNER_EINVAL, "n_q_heads %d must be 4 * n_kv_heads (%d)", cfg->n_q_heads, cfg->n_kv_heads);
  if (cfg->hidden <= 0 || cfg->hidden % 64 != 0) return fail(ATTUNER_EINVAL, "hidden %d must be a multiple of 64", cfg->hidden);
  if (cfg->n_layers <= 0 || cfg->n_layers > 65535) return fail(ATTUNER_EINVAL, "n_layers %d outside [1, 65535]", cfg->n_layers);
  if (!(cfg->rope_theta > 1.0f) || !(cfg->rms_eps >= 0.0f)) return fail(ATTUNER_EINVAL, "bad rope_theta or rms_eps");
  if (pool_pages < 0 || pool_pages >= kStagePageFlag)
    return fail(ATTUNER_ERANGE, "pool_pages %lld outside [0, 2^29)", (long long)pool_pages);
  int n_dev = 0;
  HIP_TRY(hipGetDeviceCount(&n_dev));
  if (device < 0 || device >= n_dev) return fail(ATTUNER_EINVAL, "device %d of %d", device, n_dev);
  attuner_ctx* c = new (std::nothrow) attuner_ctx;
  if (!c) return fail(ATTUNER_ENOMEM, "host allocation");
  c->cfg = *cfg;
  c->device = device;
  c->pool_pages = pool_pages;
  c->page_bytes = (int64_t)cfg->n_layers * 2 * cfg->n_kv_heads * kPageTokens * kHeadDim * 2;
  DeviceGuard dg(device);
  if (pool_pages > 0) {
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&c->pool), (size_t)(pool_pages * c->page_bytes));
    if (e != hipSuccess) {
      const long long bytes = (long long)(pool_pages * c->page_bytes);
      delete c;
      return fail(ATTUNER_ENOMEM, "pool of %lld pages (%lld bytes): %s", (long long)pool_pages, bytes,
                  hipGetErrorString(e));
    }
  }
  for (int32_t p = 0; p < (int32_t)pool_pages; ++p) c->free_pages.insert(c->free_pages.end(), p);
  // the device address of the fixed scratch (attuner_suffix_attn_noalloc);
  // a failure is reported by that call only
  (void)locate_scratch(device);
  attuner_status st = ensure_rope(c, kRopeInitPositions, nullptr);
  if (st == ATTUNER_OK) st = free_retired(c);  // waits for the table's copy
  if (st != ATTUNER_OK) {
    attuner_destroy(c);
    return st;
  }
  *out = c;
  return ATTUNER_OK;
}

attuner_status attuner_reserve(attuner_ctx* c, const attuner_limits* lim) {
  if (!c || !lim) return fail(ATTUNER_EINVAL, "null ctx or limits");
  if (lim->max_tokens < 0 || lim->max_position < 0 || lim->max_rank < 0 || lim->max_out < 0 || lim->max_lm_rows < 0 ||
      lim->max_vocab < 0)
    return fail(ATTUNER_EINVAL, "negative limit");
  if (lim->max_rank > ATTUNER_MAX_RANK) return fail(ATTUNER_ERANGE, "max_rank %d > %d", lim->max_rank, ATTUNER_MAX_RANK);
  DeviceGuard dg(c->device);
  hipStream_t s = nullptr;
  attuner_status st = ensure_rope(c, lim->max_position, s);
  const int64_t T = lim->max_tokens, Hq = c->cfg.n_q_heads, d = c->cfg.head_dim;
  const int64_t nq = q_dim(c), nkv = kv_dim(c);
  // LoRA down-projection slice partials (ranks above the fused limit, or few tokens)
  if (st == ATTUNER_OK && lim->max_rank > 0 && T > 0) {
    const int64_t r_pad = (lim->max_rank + 15) / 16 * 16;
    st = grow(c, c->ws_lora, (size_t)lora_down_slices(c->cfg.hidden, 1) * T * r_pad * sizeof(float), s,
              "LoRA down-projection");
  }
  // key-split partials of attention (normalised bf16 O + fp32 max, sum) and
  // of decode (fp32 O + max, sum; at most 1024 workgroups of n_kv heads)
  if (st == ATTUNER_OK && T > 0) {
    const int64_t rows = std::min<int64_t>((int64_t)kMaxAttnSplit * T, kAttnSplitRowsMax) * Hq;
    const int64_t dec_rows = (1024 / c->cfg.n_kv_heads + ATTUNER_MAX_REQUESTS) * Hq;
    const size_t bytes = std::max((size_t)rows * (d * 2 + 2 * sizeof(float)), (size_t)dec_rows * (d + 2) * sizeof(float));
    st = grow(c, c->ws_part, bytes, s, "key-split partials");
  }
  if (st == ATTUNER_OK && T > 0)
    st = grow(c, c->ws_qkv, (size_t)T * (nq + 2 * nkv) * sizeof(uint16_t), s, "full-prefill projection");
  if (st == ATTUNER_OK && T > 0) st = grow(c, c->ws_rows, (size_t)T * sizeof(int32_t), s, "row list");
  const int64_t widest = std::max(lim->max_out, lim->max_vocab);
  if (st == ATTUNER_OK && T > 0 && widest > 0)
    st = grow(c, c->ws_split,
              (size_t)std::min<int64_t>(kGemmSplitWsMaxBytes, (int64_t)kMaxGemmSplit * T * widest * 4), s,
              "key-split product");
  if (st == ATTUNER_OK && lim->max_lm_rows > 0 && lim->max_vocab > 0)
    st = grow(c, c->ws_logits,
              (size_t)lim->max_lm_rows * lim->max_vocab * sizeof(float) + argmax_scratch_bytes(lim->max_lm_rows), s,
              "logits");
  if (st == ATTUNER_OK) st = free_retired(c);
  return st;
}

void attuner_destroy(attuner_ctx* c) {
  if (!c) return;
  DeviceGuard dg(c->device);
  (void)hipDeviceSynchronize();
  c->staging.release();
  c->ws_pages.release();
  c->ws_lora.release();
  c->ws_part.release();
  c->ws_qkv.release();
  c->ws_logits.release();
  c->ws_split.release();
  c->ws_rows.release();
  c->rope.release();
  for (void* p : c->retired) (void)hipFree(p);
  for (void* p : c->retired_host) (void)hipHostFree(p);
  c->retired.clear();
  c->retired_host.clear();
  if (g_tracer == &c->tracer) g_tracer = nullptr;
  c->tracer.release();
  if (c->pool) (void)hipFree(c->pool);
  if (c->host_pool) (void)hipHostFree(c->host_pool);
  if (c->stage_pool) (void)hipFree(c->stage_pool);
  delete c;
}

attuner_status attuner_pool_info(const attuner_ctx* c, int64_t* pool_pages, int64_t* free_pages, int64_t* page_bytes) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (pool_pages) *pool_pages = c->pool_pages;
  if (free_pages) *free_pages = (int64_t)c->free_pages.size();
  if (page_bytes) *page_bytes = c->page_bytes;
  return ATTUNER_OK;
}

static attuner_status store_impl(attuner_ctx* c, bool host, int32_t n_tokens, const void* k, const void* v,
                                 void* stream, int32_t* artifact_id) {
  if (!c || !artifact_id) return fail(ATTUNER_EINVAL, "null ctx or artifact_id");
  if (n_tokens <= 0) return fail(ATTUNER_EINVAL, "an artifact holds at least one token (got %d)", n_tokens);
  if (!k || !v) return fail(ATTUNER_EINVAL, "null k or v");
  if (!aligned16(k) || !aligned16(v)) return fail(ATTUNER_EINVAL, "k and v must be 16-byte aligned");
  if (host && !c->host_pool) return fail(ATTUNER_EINVAL, "no host pool (attuner_host_pool_create)");
  std::set<int32_t>& free_set = host ? c->host_free : c->free_pages;
  const int64_t need = (n_tokens + kPageTokens - 1) / kPageTokens;
  if (need > (int64_t)free_set.size())
    return fail(ATTUNER_ENOMEM, "%s pool full: artifact needs %lld pages, %zu free", host ? "host" : "HBM",
                (long long)need, free_set.size());
  DeviceGuard dg(c->device);
  try {
    hipStream_t s = static_cast<hipStream_t>(stream);
    attuner_status st = grow(c, c->ws_pages, (size_t)need * sizeof(int32_t), s, "page list");
    if (st != ATTUNER_OK) return st;
    Artifact art;
    art.n_tokens = n_tokens;
    art.host = host;
    auto it = free_set.begin();
    for (int64_t i = 0; i < need; ++i) art.pages.push_back(*it++);
    st = upload_host(c, art.pages.data(), art.pages.size() * sizeof(int32_t), c->ws_pages.ptr, s,
                     "attuner_store_artifact");
    if (st != ATTUNER_OK) return st;
    HIP_TRY(launch_store_pages(static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), n_tokens,
                               static_cast<const int32_t*>(c->ws_pages.ptr), (int)need,
                               host ? c->host_pool_dev : c->pool, host ? c->host_pages : c->pool_pages,
                               c->cfg.n_layers, c->cfg.n_kv_heads, s));
    for (int32_t pg : art.pages) free_set.erase(pg);
    const int32_t id = c->next_id++;
    c->artifacts.emplace(id, std::move(art));
    *artifact_id = id;
  } catch (const std::bad_alloc&) {
    return fail(ATTUNER_ENOMEM, "host allocation");
  }
  return ATTUNER_OK;
}

attuner_status attuner_store_artifact(attuner_ctx* c, int32_t n_tokens, const void* k, const void* v, void* stream,
                                      int32_t* artifact_id) {
  return store_impl(c, false, n_tokens, k, v, stream, artifact_id);
}

attuner_status attuner_host_pool_create(attuner_ctx* c, int64_t host_pages) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (c->host_pool) return fail(ATTUNER_EINVAL, "the context already has a host pool");
  if (host_pages <= 0 || host_pages >= kStagePageFlag)
    return fail(ATTUNER_ERANGE, "host_pages %lld outside [1, 2^29)", (long long)host_pages);
  DeviceGuard dg(c->device);
  void* h = nullptr;
  hipError_t e = hipHostMalloc(&h, (size_t)(host_pages * c->page_bytes), hipHostMallocMapped | hipHostMallocPortable);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(ATTUNER_ENOMEM, "host pool of %lld pages (%lld bytes): %s", (long long)host_pages,
                (long long)(host_pages * c->page_bytes), hipGetErrorString(e));
  }
  void* d = nullptr;
  e = hipHostGetDevicePointer(&d, h, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(h);
    return fail(ATTUNER_EDEVICE, "hipHostGetDevicePointer: %s", hipGetErrorString(e));
  }
  c->host_pool = static_cast<uint16_t*>(h);
  c->host_pool_dev = static_cast<uint16_t*>(d);
  c->host_pages = host_pages;
  for (int32_t p = 0; p < (int32_t)host_pages; ++p) c->host_free.insert(c->host_free.end(), p);
  return ATTUNER_OK;
}

attuner_status attuner_store_artifact_host(attuner_ctx* c, int32_t n_tokens, const void* k, const void* v,
                                           void* stream, int32_t* artifact_id) {
  return store_impl(c, true, n_tokens, k, v, stream, artifact_id);
}

attuner_status attuner_host_pool_info(const attuner_ctx* c, int64_t* host_pages, int64_t* free_pages) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (host_pages) *host_pages = c->host_pages;
  if (free_pages) *free_pages = (int64_t)c->host_free.size();
  return ATTUNER_OK;
}

attuner_status attuner_release_artifact(attuner_ctx* c, int32_t artifact_id) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  auto it = c->artifacts.find(artifact_id);
  if (it == c->artifacts.end()) return fail(ATTUNER_ENOENT, "unknown artifact id %d", artifact_id);
  std::set<int32_t>& free_set = it->second.host ? c->host_free : c->free_pages;
  for (int32_t pg : it->second.pages) free_set.insert(pg);
  c->artifacts.erase(it);
  return ATTUNER_OK;
}

attuner_status attuner_artifact_pages(const attuner_ctx* c, int32_t artifact_id, int32_t* pages_out, int32_t max_pages,
                                      int32_t* n_pages, int32_t* n_tokens) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  auto it = c->artifacts.find(artifact_id);
  if (it == c->artifacts.end()) return fail(ATTUNER_ENOENT, "unknown artifact id %d", artifact_id);
  const int32_t np = (int32_t)it->second.pages.size();
  if (n_pages) *n_pages = np;
  if (n_tokens) *n_tokens = it->second.n_tokens;
  if (pages_out) {
    if (max_pages < np) return fail(ATTUNER_ERANGE, "max_pages %d < %d pages", max_pages, np);
    for (int32_t i = 0; i < np; ++i) pages_out[i] = it->second.table_page(it->second.pages[i]);
  }
  return ATTUNER_OK;
}

static attuner_status plan_impl(const attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                const int32_t* artifact_ids, const int32_t* suffix_cap, int64_t* n_entries,
                                int64_t* cache_rows, std::vector<int32_t>* table, int32_t* cu_ctx,
                                int32_t* art_len) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_req < 0 || n_req > ATTUNER_MAX_REQUESTS)
    return fail(ATTUNER_ERANGE, "n_req %d outside [0, %d]", n_req, ATTUNER_MAX_REQUESTS);
  if (n_req > 0 && (!req_ptr || !suffix_cap)) return fail(ATTUNER_EINVAL, "null req_ptr or suffix_cap");
  if (n_req > 0 && req_ptr[0] != 0) return fail(ATTUNER_EINVAL, "req_ptr[0] must be 0");
  int64_t entries = 0, row = 0;
  if (cu_ctx) cu_ctx[0] = 0;
  for (int r = 0; r < n_req; ++r) {
    if (req_ptr[r + 1] < req_ptr[r]) return fail(ATTUNER_EINVAL, "req_ptr not monotone at %d", r);
    if (suffix_cap[r] < 0) return fail(ATTUNER_EINVAL, "suffix_cap[%d] < 0", r);
    if (req_ptr[r + 1] > req_ptr[r] && !artifact_ids) return fail(ATTUNER_EINVAL, "null artifact_ids");
    int64_t alen = 0;
    for (int32_t j = req_ptr[r]; j < req_ptr[r + 1]; ++j) {
      auto it = c->artifacts.find(artifact_ids[j]);
      if (it == c->artifacts.end()) return fail(ATTUNER_ENOENT, "request %d: unknown artifact id %d", r, artifact_ids[j]);
      const Artifact& a = it->second;
      if (table) {
        int32_t left = a.n_tokens;
        for (int32_t pg : a.pages) {
          const int32_t nv = std::min(left, kPageTokens);
          table->push_back(a.table_page(pg));
          table->push_back(nv);
          table->push_back((int32_t)(row + alen));
          table->push_back(r);
          alen += nv;
          left -= nv;
        }
      } else {
        alen += a.n_tokens;
      }
      entries += (int64_t)a.pages.size();
    }
    row += alen + suffix_cap[r];
    if (row > INT32_MAX) return fail(ATTUNER_ERANGE, "cache rows exceed 2^31");
    if (art_len) art_len[r] = (int32_t)alen;
    if (cu_ctx) cu_ctx[r + 1] = (int32_t)row;
  }
  if (n_entries) *n_entries = entries;
  if (cache_rows) *cache_rows = row;
  return ATTUNER_OK;
}

attuner_status attuner_assemble_plan(const attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                     const int32_t* artifact_ids, const int32_t* suffix_cap, int64_t* n_entries,
                                     int64_t* cache_rows) {
  return plan_impl(c, n_req, req_ptr, artifact_ids, suffix_cap, n_entries, cache_rows, nullptr, nullptr, nullptr);
}

static attuner_status assemble_table_impl(attuner_ctx* c, bool staged, int32_t n_req, const int32_t* req_ptr,
                                          const int32_t* artifact_ids, const int32_t* suffix_cap,
                                          int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                          int64_t cache_rows, int64_t* n_staged, void* stream);

attuner_status attuner_assemble_table(attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                      const int32_t* artifact_ids, const int32_t* suffix_cap, int32_t* block_table,
                                      int32_t* cu_ctx, int32_t* art_len, int64_t cache_rows, void* stream) {
  return assemble_table_impl(c, false, n_req, req_ptr, artifact_ids, suffix_cap, block_table, cu_ctx, art_len,
                             cache_rows, nullptr, stream);
}

// The staged form remaps every host page of the batch to a staging page:
// the distinct host pages, in ascending order, get staging pages 0, 1, ...,
// so that every maximal range of consecutive host pages is one copy run
// (artifacts stored one after another in the host pool then move in one copy
// per layer, whatever order the requests use them in).
static attuner_status stage_remap(attuner_ctx* c, std::vector<int32_t>& table, int64_t* n_staged) {
  c->stage_runs.clear();
  std::vector<int32_t> host;
  for (size_t e = 0; e < table.size(); e += 4)
    if (table[e] & kHostPageFlag) host.push_back(table[e] & kPageIdMask);
  std::sort(host.begin(), host.end());
  host.erase(std::unique(host.begin(), host.end()), host.end());
  if ((int64_t)host.size() > c->stage_pages)
    return fail(ATTUNER_ERANGE, "the batch uses %zu distinct host pages, the staging pool holds %lld", host.size(),
                (long long)c->stage_pages);
  for (size_t i = 0; i < host.size(); ++i) {
    if (i > 0 && host[i] == host[i - 1] + 1)
      ++c->stage_runs.back()[2];
    else
      c->stage_runs.push_back({host[i], (int32_t)i, 1});
  }
  for (size_t e = 0; e < table.size(); e += 4) {
    if (!(table[e] & kHostPageFlag)) continue;
    const auto it = std::lower_bound(host.begin(), host.end(), table[e] & kPageIdMask);
    table[e] = (int32_t)(it - host.begin()) | kStagePageFlag;
  }
  if (n_staged) *n_staged = (int64_t)host.size();
  return ATTUNER_OK;
}

static attuner_status assemble_table_impl(attuner_ctx* c, bool staged, int32_t n_req, const int32_t* req_ptr,
                                          const int32_t* artifact_ids, const int32_t* suffix_cap,
                                          int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                          int64_t cache_rows, int64_t* n_staged, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  c->last_table = nullptr;
  c->last_entries = c->last_rows = -1;
  c->last_staged = false;
  c->stage_runs.clear();
  if (staged && !c->stage_pool) return fail(ATTUNER_EINVAL, "no staging pool (attuner_stage_pool_create)");
  std::vector<int32_t> table;
  std::vector<int32_t> cu(n_req > 0 ? n_req + 1 : 1), al(n_req > 0 ? n_req : 1);
  int64_t entries = 0, rows = 0;
  try {
    attuner_status st = plan_impl(c, n_req, req_ptr, artifact_ids, suffix_cap, &entries, &rows, &table, cu.data(),
                                  al.data());
    if (st != ATTUNER_OK) return st;
    if (staged) {
      st = stage_remap(c, table, n_staged);
      if (st != ATTUNER_OK) {
        c->stage_runs.clear();
        return st;
      }
    }
  } catch (const std::bad_alloc&) {
    c->stage_runs.clear();
    return fail(ATTUNER_ENOMEM, "host allocation");
  }
  if (rows != cache_rows)
    return fail(ATTUNER_ERANGE, "cache_rows %lld does not match the plan (%lld)", (long long)cache_rows, (long long)rows);
  if (entries > 0 && !block_table) return fail(ATTUNER_EINVAL, "null block_table");
  if (entries > INT32_MAX) return fail(ATTUNER_ERANGE, "block table of %lld entries", (long long)entries);
  if (cu_ctx) memcpy(cu_ctx, cu.data(), (size_t)(n_req + 1) * sizeof(int32_t));
  if (art_len && n_req > 0) memcpy(art_len, al.data(), (size_t)n_req * sizeof(int32_t));
  if (entries > 0) {
    DeviceGuard dg(c->device);
    attuner_status st = upload_host(c, table.data(), table.size() * sizeof(int32_t), block_table,
                                    static_cast<hipStream_t>(stream),
                                    staged ? "attuner_assemble_table_staged" : "attuner_assemble_table");
    if (st != ATTUNER_OK) {
      c->stage_runs.clear();
      return st;
    }
  }
  c->last_table = block_table;
  c->last_entries = entries;
  c->last_rows = rows;
  c->last_staged = staged;
  c->last_hbm_only = true;
  for (size_t e = 0; e < table.size(); e += 4)
    if (table[e] & (kHostPageFlag | kStagePageFlag)) c->last_hbm_only = false;
  return ATTUNER_OK;
}

attuner_status attuner_assemble_table_staged(attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                             const int32_t* artifact_ids, const int32_t* suffix_cap,
                                             int32_t* block_table, int32_t* cu_ctx, int32_t* art_len,
                                             int64_t cache_rows, int64_t* staged_pages, void* stream) {
  return assemble_table_impl(c, true, n_req, req_ptr, artifact_ids, suffix_cap, block_table, cu_ctx, art_len,
                             cache_rows, staged_pages, stream);
}

attuner_status attuner_stage_pool_create(attuner_ctx* c, int64_t stage_pages) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (c->stage_pool) return fail(ATTUNER_EINVAL, "the context already has a staging pool");
  if (stage_pages <= 0 || stage_pages >= kStagePageFlag)
    return fail(ATTUNER_ERANGE, "stage_pages %lld outside [1, 2^29)", (long long)stage_pages);
  DeviceGuard dg(c->device);
  void* d = nullptr;
  hipError_t e = hipMalloc(&d, (size_t)(stage_pages * c->page_bytes));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(ATTUNER_ENOMEM, "staging pool of %lld pages (%lld bytes): %s", (long long)stage_pages,
                (long long)(stage_pages * c->page_bytes), hipGetErrorString(e));
  }
  c->stage_pool = static_cast<uint16_t*>(d);
  c->stage_pages = stage_pages;
  return ATTUNER_OK;
}

attuner_status attuner_stage_layers(attuner_ctx* c, int32_t layer_begin, int32_t n_layers, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (!c->last_staged) return fail(ATTUNER_EINVAL, "the last assembly was not attuner_assemble_table_staged");
  if (layer_begin < 0 || n_layers < 0 || layer_begin > c->cfg.n_layers || n_layers > c->cfg.n_layers - layer_begin)
    return fail(ATTUNER_ERANGE, "layers [%d, %d) outside [0, %d)", layer_begin, layer_begin + n_layers,
                c->cfg.n_layers);
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // one page of one layer: [2][n_kv][16][head_dim] bf16, contiguous in both pools
  const size_t layer_page = (size_t)(c->page_bytes / c->cfg.n_layers);
  const char* host = reinterpret_cast<const char*>(c->host_pool);
  char* stage = reinterpret_cast<char*>(c->stage_pool);
  for (int32_t l = layer_begin; l < layer_begin + n_layers; ++l)
    for (const auto& run : c->stage_runs)
      HIP_TRY(hipMemcpyAsync(stage + ((size_t)l * c->stage_pages + run[1]) * layer_page,
                             host + ((size_t)l * c->host_pages + run[0]) * layer_page, (size_t)run[2] * layer_page,
                             hipMemcpyHostToDevice, s));
  return ATTUNER_OK;
}

attuner_status attuner_stage_pool_info(const attuner_ctx* c, int64_t* stage_pages, int64_t* runs) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (stage_pages) *stage_pages = c->stage_pages;
  if (runs) *runs = c->last_staged ? (int64_t)c->stage_runs.size() : 0;
  return ATTUNER_OK;
}

attuner_status attuner_gather_layers(attuner_ctx* c, const int32_t* block_table, int64_t n_entries,
                                     int32_t layer_begin, int32_t n_layers, void* req_kv, int64_t cache_rows,
                                     void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (c->last_entries < 0 || block_table != c->last_table || n_entries != c->last_entries ||
      cache_rows != c->last_rows)
    return fail(ATTUNER_EINVAL, "block_table, n_entries and cache_rows must be those of the last "
                                "attuner_assemble_table call");
  if (layer_begin < 0 || n_layers < 0 || layer_begin > c->cfg.n_layers || n_layers > c->cfg.n_layers - layer_begin)
    return fail(ATTUNER_ERANGE, "layers [%d, %d) outside [0, %d)", layer_begin, layer_begin + n_layers,
                c->cfg.n_layers);
  if (n_entries == 0 || n_layers == 0) return ATTUNER_OK;
  if (!req_kv || !aligned16(req_kv)) return fail(ATTUNER_EINVAL, "req_kv must be non-null and 16-byte aligned");
  DeviceGuard dg(c->device);
  HIP_TRY(launch_gather(block_table, n_entries, c->pool, c->pool_pages, c->host_pool_dev, c->host_pages,
                        c->stage_pool, c->stage_pages, layer_begin, n_layers, c->cfg.n_kv_heads,
                        static_cast<uint16_t*>(req_kv), cache_rows, static_cast<hipStream_t>(stream)));
  return ATTUNER_OK;
}

attuner_status attuner_assemble_kv(attuner_ctx* c, int32_t n_req, const int32_t* req_ptr, const int32_t* artifact_ids,
                                   const int32_t* suffix_cap, int32_t* block_table, int32_t* cu_ctx,
                                   int32_t* art_len, void* req_kv, int64_t cache_rows, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  int64_t entries = 0, rows = 0;
  attuner_status st = plan_impl(c, n_req, req_ptr, artifact_ids, suffix_cap, &entries, &rows, nullptr, nullptr,
                                nullptr);
  if (st != ATTUNER_OK) return st;
  if (rows != cache_rows)
    return fail(ATTUNER_ERANGE, "cache_rows %lld does not match the plan (%lld)", (long long)cache_rows, (long long)rows);
  if (entries > 0 && (!block_table || !req_kv)) return fail(ATTUNER_EINVAL, "null block_table or req_kv");
  if (req_kv && !aligned16(req_kv)) return fail(ATTUNER_EINVAL, "req_kv must be 16-byte aligned");
  st = attuner_assemble_table(c, n_req, req_ptr, artifact_ids, suffix_cap, block_table, cu_ctx, art_len, cache_rows,
                              stream);
  if (st != ATTUNER_OK) return st;
  return attuner_gather_layers(c, block_table, entries, 0, c->cfg.n_layers, req_kv, cache_rows, stream);
}

// Prompts that interleave cached artifacts with online spans: segments[j]
// >= 0 is an artifact id, -n < 0 an online span of n tokens.  Request r
// owns rows [cu_ctx[r], cu_ctx[r+1]) holding its prompt in order; spans get
// (request, offset in the request, length).
static attuner_status plan_segments_impl(const attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                         const int32_t* segments, int64_t* n_entries, int64_t* cache_rows,
                                         int32_t* n_spans, std::vector<int32_t>* table, int32_t* cu_ctx,
                                         std::vector<int32_t>* spans) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_req < 0 || n_req > ATTUNER_MAX_REQUESTS)
    return fail(ATTUNER_ERANGE, "n_req %d outside [0, %d]", n_req, ATTUNER_MAX_REQUESTS);
  if (n_req > 0 && !req_ptr) return fail(ATTUNER_EINVAL, "null req_ptr");
  if (n_req > 0 && req_ptr[0] != 0) return fail(ATTUNER_EINVAL, "req_ptr[0] must be 0");
  int64_t entries = 0, row = 0;
  int32_t ns = 0;
  if (cu_ctx) cu_ctx[0] = 0;
  for (int r = 0; r < n_req; ++r) {
    if (req_ptr[r + 1] < req_ptr[r]) return fail(ATTUNER_EINVAL, "req_ptr not monotone at %d", r);
    if (req_ptr[r + 1] > req_ptr[r] && !segments) return fail(ATTUNER_EINVAL, "null segments");
    int64_t off = 0;
    for (int32_t j = req_ptr[r]; j < req_ptr[r + 1]; ++j) {
      const int32_t sg = segments[j];
      if (sg < 0) {
        if (sg == INT32_MIN) return fail(ATTUNER_EINVAL, "request %d: segment %d out of range", r, j);
        if (spans) {
          spans->push_back(r);
          spans->push_back((int32_t)off);
          spans->push_back(-sg);
        }
        off += -(int64_t)sg;
        ++ns;
        continue;
      }
      auto it = c->artifacts.find(sg);
      if (it == c->artifacts.end()) return fail(ATTUNER_ENOENT, "request %d: unknown artifact id %d", r, sg);
      const Artifact& a = it->second;
      if (table) {
        int32_t left = a.n_tokens;
        for (int32_t pg : a.pages) {
          const int32_t nv = std::min(left, kPageTokens);
          table->push_back(a.table_page(pg));
          table->push_back(nv);
          table->push_back((int32_t)(row + off));
          table->push_back(r);
          off += nv;
          left -= nv;
        }
      } else {
        off += a.n_tokens;
      }
      entries += (int64_t)a.pages.size();
      if (row + off > INT32_MAX) return fail(ATTUNER_ERANGE, "cache rows exceed 2^31");
    }
    row += off;
    if (row > INT32_MAX) return fail(ATTUNER_ERANGE, "cache rows exceed 2^31");
    if (cu_ctx) cu_ctx[r + 1] = (int32_t)row;
  }
  if (n_entries) *n_entries = entries;
  if (cache_rows) *cache_rows = row;
  if (n_spans) *n_spans = ns;
  return ATTUNER_OK;
}

attuner_status attuner_assemble_segments_plan(const attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                              const int32_t* segments, int64_t* n_entries, int64_t* cache_rows,
                                              int32_t* n_spans) {
  return plan_segments_impl(c, n_req, req_ptr, segments, n_entries, cache_rows, n_spans, nullptr, nullptr, nullptr);
}

attuner_status attuner_assemble_segments(attuner_ctx* c, int32_t n_req, const int32_t* req_ptr,
                                         const int32_t* segments, int32_t* block_table, int32_t* cu_ctx,
                                         int32_t* spans, void* req_kv, int64_t cache_rows, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  c->last_table = nullptr;
  c->last_entries = c->last_rows = -1;
  c->last_staged = false;
  c->stage_runs.clear();
  std::vector<int32_t> table, sp;
  std::vector<int32_t> cu(n_req > 0 ? n_req + 1 : 1);
  int64_t entries = 0, rows = 0;
  int32_t ns = 0;
  try {
    attuner_status st = plan_segments_impl(c, n_req, req_ptr, segments, &entries, &rows, &ns, &table, cu.data(), &sp);
    if (st != ATTUNER_OK) return st;
  } catch (const std::bad_alloc&) {
    return fail(ATTUNER_ENOMEM, "host allocation");
  }
  if (rows != cache_rows)
    return fail(ATTUNER_ERANGE, "cache_rows %lld does not match the plan (%lld)", (long long)cache_rows, (long long)rows);
  if (entries > 0 && !block_table) return fail(ATTUNER_EINVAL, "null block_table");
  if (entries > INT32_MAX) return fail(ATTUNER_ERANGE, "block table of %lld entries", (long long)entries);
  if (ns > 0 && !spans) return fail(ATTUNER_EINVAL, "null spans");
  if (entries > 0 && (!req_kv || !aligned16(req_kv))) return fail(ATTUNER_EINVAL, "null or unaligned req_kv");
  if (cu_ctx) memcpy(cu_ctx, cu.data(), (size_t)(n_req + 1) * sizeof(int32_t));
  if (ns > 0) memcpy(spans, sp.data(), sp.size() * sizeof(int32_t));
  if (entries > 0) {
    DeviceGuard dg(c->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    attuner_status st = upload_host(c, table.data(), table.size() * sizeof(int32_t), block_table, s,
                                    "attuner_assemble_segments");
    if (st != ATTUNER_OK) return st;
    HIP_TRY(launch_gather(block_table, entries, c->pool, c->pool_pages, c->host_pool_dev, c->host_pages, nullptr, 0,
                          0, c->cfg.n_layers, c->cfg.n_kv_heads,
                          static_cast<uint16_t*>(req_kv), cache_rows, s));
  }
  c->last_table = block_table;
  c->last_entries = entries;
  c->last_rows = rows;
  return ATTUNER_OK;
}

attuner_status attuner_rms_norm(attuner_ctx* c, const void* x, int64_t n_x_rows, int64_t ld_x, const int32_t* rows,
                                int32_t n_rows, const void* gamma, void* out, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  const int dim = c->cfg.hidden;
  if (n_rows < 0 || n_x_rows < 0) return fail(ATTUNER_EINVAL, "negative row count");
  if (rows == nullptr && n_rows > n_x_rows) return fail(ATTUNER_ERANGE, "n_rows %d > n_x_rows %lld", n_rows, (long long)n_x_rows);
  if (n_rows == 0) return ATTUNER_OK;
  if (!x || !gamma || !out) return fail(ATTUNER_EINVAL, "null x, gamma or out");
  if (ld_x < dim || ld_x % 8 != 0 || !aligned16(x) || !aligned16(gamma) || !aligned16(out))
    return fail(ATTUNER_EINVAL, "ld_x %lld must be >= hidden and a multiple of 8; x, gamma, out 16-byte aligned",
                (long long)ld_x);
  if (dim > 8192) return fail(ATTUNER_EINVAL, "hidden %d: the norm kernel takes at most 8192", dim);
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int32_t* rows_dev = nullptr;
  if (rows != nullptr) {
    for (int32_t i = 0; i < n_rows; ++i)
      if (rows[i] < 0 || rows[i] >= n_x_rows)
        return fail(ATTUNER_ERANGE, "rows[%d] = %d outside [0, %lld)", i, rows[i], (long long)n_x_rows);
    attuner_status st = upload_check(c, s, "attuner_rms_norm with a row list");
    if (st != ATTUNER_OK) return st;
    st = grow(c, c->ws_rows, (size_t)n_rows * sizeof(int32_t), s, "row list");
    if (st != ATTUNER_OK) return st;
    st = upload_host(c, rows, (size_t)n_rows * sizeof(int32_t), c->ws_rows.ptr, s, "attuner_rms_norm with a row list");
    if (st != ATTUNER_OK) return st;
    rows_dev = static_cast<const int32_t*>(c->ws_rows.ptr);
  }
  HIP_TRY(launch_rms_norm_rows(static_cast<const uint16_t*>(x), ld_x, rows_dev, n_rows, dim,
                               static_cast<const uint16_t*>(gamma), c->cfg.rms_eps, static_cast<uint16_t*>(out), s));
  return ATTUNER_OK;
}

attuner_status attuner_embed(attuner_ctx* c, int32_t n_tok, const int32_t* token_ids, const void* table,
                             int32_t vocab, void* out, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_tok < 0 || vocab <= 0) return fail(ATTUNER_EINVAL, "n_tok %d, vocab %d", n_tok, vocab);
  if (n_tok == 0) return ATTUNER_OK;
  if (!token_ids || !table || !out) return fail(ATTUNER_EINVAL, "null token_ids, table or out");
  const int dim = c->cfg.hidden;
  if (dim % 8 != 0 || !aligned16(table) || !aligned16(out))
    return fail(ATTUNER_EINVAL, "hidden %d must be a multiple of 8; table and out 16-byte aligned", dim);
  for (int32_t i = 0; i < n_tok; ++i)
    if (token_ids[i] < 0 || token_ids[i] >= vocab)
      return fail(ATTUNER_ERANGE, "token_ids[%d] = %d outside [0, %d)", i, token_ids[i], vocab);
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  attuner_status st = upload_check(c, s, "attuner_embed");
  if (st != ATTUNER_OK) return st;
  st = grow(c, c->ws_rows, (size_t)n_tok * sizeof(int32_t), s, "token id");
  if (st != ATTUNER_OK) return st;
  st = upload_host(c, token_ids, (size_t)n_tok * sizeof(int32_t), c->ws_rows.ptr, s, "attuner_embed");
  if (st != ATTUNER_OK) return st;
  HIP_TRY(launch_embed_rows(static_cast<const uint16_t*>(table), static_cast<const int32_t*>(c->ws_rows.ptr), n_tok,
                            dim, static_cast<uint16_t*>(out), s));
  return ATTUNER_OK;
}

static attuner_status check_gemm_args(int32_t n_tok, const void* x, int32_t k_dim, const void* w, int32_t n_out,
                                      const void* out) {
  if (n_tok < 0) return fail(ATTUNER_EINVAL, "n_tok < 0");
  if (k_dim <= 0 || k_dim % 64 != 0) return fail(ATTUNER_EINVAL, "k_dim %d must be a positive multiple of 64", k_dim);
  if (n_out <= 0 || n_out % 64 != 0) return fail(ATTUNER_EINVAL, "n_out %d must be a positive multiple of 64", n_out);
  if (n_tok > 0 && (!x || !w || !out)) return fail(ATTUNER_EINVAL, "null x, w or out");
  if (!aligned16(x) || !aligned16(w) || !aligned16(out)) return fail(ATTUNER_EINVAL, "x, w and out must be 16-byte aligned");
  return ATTUNER_OK;
}

// A plain product with epilogue epi: plans tile and key split, grows the
// split workspace when the plan splits the k range.
static attuner_status run_gemm(attuner_ctx* c, int32_t n_tok, const void* x, int32_t k_dim, const void* w,
                               int32_t n_out, GemmEpi epi, void* out, hipStream_t s) {
  const GemmPlan plan = plan_gemm(n_tok, n_out, k_dim, false);
  float* ws = nullptr;
  if (n_tok > kGemvMaxTok && plan.n_split > 1) {
    attuner_status st = grow(c, c->ws_split, (size_t)plan.n_split * n_tok * n_out * sizeof(float), s, "key-split product");
    if (st != ATTUNER_OK) return st;
    ws = static_cast<float*>(c->ws_split.ptr);
  }
  HIP_TRY(launch_gemm(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), n_tok, n_out, k_dim, epi,
                      static_cast<uint16_t*>(out), plan, ws, s));
  return ATTUNER_OK;
}

attuner_status attuner_linear(attuner_ctx* c, int32_t n_tok, const void* x, int32_t k_dim, const void* w,
                              int32_t n_out, const void* residual, void* out, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_gemm_args(n_tok, x, k_dim, w, n_out, out);
  if (st != ATTUNER_OK) return st;
  if (residual && !aligned16(residual)) return fail(ATTUNER_EINVAL, "residual must be 16-byte aligned");
  if (n_tok == 0) return ATTUNER_OK;
  DeviceGuard dg(c->device);
  const GemmEpi epi{residual ? kEpiResidual : kEpiBf16, static_cast<const uint16_t*>(residual), nullptr};
  return run_gemm(c, n_tok, x, k_dim, w, n_out, epi, out, static_cast<hipStream_t>(stream));
}

attuner_status attuner_gate_up_swiglu(attuner_ctx* c, int32_t n_tok, const void* x, int32_t k_dim, const void* w_gu,
                                      int32_t n_inter, void* out, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_inter <= 0 || n_inter % 32 != 0) return fail(ATTUNER_EINVAL, "n_inter %d must be a positive multiple of 32", n_inter);
  attuner_status st = check_gemm_args(n_tok, x, k_dim, w_gu, 2 * n_inter, out);
  if (st != ATTUNER_OK) return st;
  if (n_tok == 0) return ATTUNER_OK;
  DeviceGuard dg(c->device);
  return run_gemm(c, n_tok, x, k_dim, w_gu, 2 * n_inter, GemmEpi{kEpiSwiglu, nullptr, nullptr}, out,
                  static_cast<hipStream_t>(stream));
}

attuner_status attuner_lm_head_argmax(attuner_ctx* c, int32_t n_rows, const void* x, const void* w_lm, int32_t vocab,
                                      int32_t* ids, float* max_logit, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  const int H = c->cfg.hidden;
  if (vocab <= 0 || vocab % 64 != 0) return fail(ATTUNER_EINVAL, "vocab %d must be a positive multiple of 64", vocab);
  attuner_status st = check_gemm_args(n_rows, x, H, w_lm, vocab, x);
  if (st != ATTUNER_OK) return st;
  if (n_rows == 0) return ATTUNER_OK;
  if (!ids) return fail(ATTUNER_EINVAL, "null ids");
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t logit_bytes = (size_t)n_rows * vocab * sizeof(float);
  st = grow(c, c->ws_logits, logit_bytes + argmax_scratch_bytes(n_rows), s, "logits");
  if (st != ATTUNER_OK) return st;
  float* logits = static_cast<float*>(c->ws_logits.ptr);
  st = run_gemm(c, n_rows, x, H, w_lm, vocab, GemmEpi{kEpiF32, nullptr, logits}, nullptr, s);
  if (st != ATTUNER_OK) return st;
  HIP_TRY(launch_argmax_rows(logits, n_rows, vocab, ids, max_logit, static_cast<char*>(c->ws_logits.ptr) + logit_bytes,
                             s));
  return ATTUNER_OK;
}

attuner_status attuner_merge_lora(attuner_ctx* c, const void* w, int32_t n_out, int32_t k_dim, const void* a,
                                  const void* b, int32_t rank, float scale, int32_t lora_cols, void* w_out,
                                  void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_out < 0 || k_dim <= 0 || k_dim % 8 != 0)
    return fail(ATTUNER_EINVAL, "n_out %d, k_dim %d (a positive multiple of 8)", n_out, k_dim);
  if (rank < 0 || rank > ATTUNER_MAX_RANK) return fail(ATTUNER_ERANGE, "rank %d outside [0, %d]", rank, ATTUNER_MAX_RANK);
  if (lora_cols < 0 || lora_cols > n_out) return fail(ATTUNER_EINVAL, "lora_cols %d outside [0, n_out]", lora_cols);
  if (n_out == 0) return ATTUNER_OK;
  if (!w || !w_out || (rank > 0 && lora_cols > 0 && (!a || !b)))
    return fail(ATTUNER_EINVAL, "null w, w_out, a or b");
  if (!aligned16(w) || !aligned16(w_out) || (rank > 0 && !aligned16(a)))
    return fail(ATTUNER_EINVAL, "w, w_out and a must be 16-byte aligned");
  DeviceGuard dg(c->device);
  HIP_TRY(launch_merge_lora(static_cast<const uint16_t*>(w), n_out, k_dim, static_cast<const uint16_t*>(a),
                            static_cast<const uint16_t*>(b), rank, scale, rank > 0 ? lora_cols : 0,
                            static_cast<uint16_t*>(w_out), static_cast<hipStream_t>(stream)));
  return ATTUNER_OK;
}

attuner_status attuner_qproj_lora(attuner_ctx* c, int32_t n_tok, const void* x, const void* w, int32_t n_out,
                                  const void* a, const void* b, int32_t rank, float scale, int32_t lora_cols,
                                  void* out, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  DeviceGuard dg(c->device);
  return qproj_impl(c, n_tok, x, w, n_out, a, b, rank, scale, lora_cols, out, static_cast<hipStream_t>(stream));
}

static attuner_status check_norm_args(const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                      int64_t ld_kv, const void* gamma_q, const void* gamma_k, const attuner_ctx* c) {
  if (!q_raw || !k_raw || !v_raw || !gamma_q || !gamma_k) return fail(ATTUNER_EINVAL, "null q/k/v or gamma");
  if (ld_q < q_dim(c) || ld_kv < kv_dim(c)) return fail(ATTUNER_EINVAL, "ld_q %lld / ld_kv %lld too small", (long long)ld_q, (long long)ld_kv);
  if (ld_q % 8 != 0 || ld_kv % 8 != 0 || !aligned16(q_raw) || !aligned16(k_raw) || !aligned16(v_raw) ||
      !aligned16(gamma_q) || !aligned16(gamma_k))
    return fail(ATTUNER_EINVAL, "q/k/v rows (ld_q, ld_kv multiples of 8) and gamma must be 16-byte aligned");
  return ATTUNER_OK;
}

attuner_status attuner_qk_norm_rope(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                    const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                    const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                    int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* q_hat,
                                    void* req_kv, int64_t cache_rows, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_layer(c, layer);
  if (st != ATTUNER_OK) return st;
  std::vector<ReqDesc> reqs;
  int32_t total_q = 0;
  st = build_reqs(c, n_req, cu_q, cu_ctx, art_len, pos0, cache_rows, &reqs, &total_q);
  if (st != ATTUNER_OK) return st;
  if (total_q == 0) return ATTUNER_OK;
  st = check_norm_args(q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, c);
  if (st != ATTUNER_OK) return st;
  if (!q_hat || !req_kv || !aligned16(q_hat) || !aligned16(req_kv))
    return fail(ATTUNER_EINVAL, "q_hat and req_kv must be non-null and 16-byte aligned");
  DeviceGuard dg(c->device);
  const int64_t hs = cache_rows * c->cfg.head_dim;
  return run_norm_rope(c, reqs, total_q, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, q_hat,
                       cache_plane(req_kv, c, layer, 0, cache_rows), cache_plane(req_kv, c, layer, 1, cache_rows), hs,
                       static_cast<hipStream_t>(stream));
}

attuner_status attuner_attention(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                 const int32_t* cu_ctx, const int32_t* art_len, const void* q_hat,
                                 const void* req_kv, int64_t cache_rows, void* o, float* lse, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_layer(c, layer);
  if (st != ATTUNER_OK) return st;
  std::vector<ReqDesc> reqs;
  int32_t total_q = 0;
  st = build_reqs(c, n_req, cu_q, cu_ctx, art_len, nullptr, cache_rows, &reqs, &total_q);
  if (st != ATTUNER_OK) return st;
  if (total_q == 0) return ATTUNER_OK;
  if (!q_hat || !req_kv || !o || !aligned16(q_hat) || !aligned16(req_kv) || !aligned16(o))
    return fail(ATTUNER_EINVAL, "q_hat, req_kv and o must be non-null and 16-byte aligned");
  DeviceGuard dg(c->device);
  const int64_t hs = cache_rows * c->cfg.head_dim;
  return run_attention(c, reqs, total_q, q_hat, cache_plane(const_cast<void*>(req_kv), c, layer, 0, cache_rows),
                       cache_plane(const_cast<void*>(req_kv), c, layer, 1, cache_rows), hs, o, lse,
                       static_cast<hipStream_t>(stream));
}

static attuner_status suffix_attn_impl(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                       const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                       const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                       int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                       int64_t cache_rows, void* o, float* lse, void* stream, bool noalloc,
                                       const GatherArgs* gather = nullptr) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_layer(c, layer);
  if (st != ATTUNER_OK) return st;
  std::vector<ReqDesc> reqs;
  int32_t total_q = 0;
  st = build_reqs(c, n_req, cu_q, cu_ctx, art_len, pos0, cache_rows, &reqs, &total_q);
  if (st != ATTUNER_OK) return st;
  if (total_q == 0) {
    if (gather == nullptr) return ATTUNER_OK;
    DeviceGuard dg(c->device);
    HIP_TRY(launch_gather_apart(c, *gather, static_cast<hipStream_t>(stream)));
    return ATTUNER_OK;
  }
  st = check_norm_args(q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, c);
  if (st != ATTUNER_OK) return st;
  if (!req_kv || !o || !aligned16(req_kv) || !aligned16(o))
    return fail(ATTUNER_EINVAL, "req_kv and o must be non-null and 16-byte aligned");
  void* part = nullptr;
  if (noalloc) {
    part = scratch_ptr(c->device);
    if (part == nullptr)
      return fail(ATTUNER_EDEVICE, "the fixed scratch of device %d could not be located", c->device);
    int64_t max_pos = 0;
    for (const auto& r : reqs) max_pos = std::max<int64_t>(max_pos, (int64_t)r.pos0 + r.q_len);
    if (max_pos > c->rope_pos)
      return fail(ATTUNER_ERANGE, "position %lld is past the RoPE table (%lld positions); this call does not "
                                  "extend it (attuner_reserve does)", (long long)max_pos - 1, (long long)c->rope_pos);
  }
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t hs = cache_rows * c->cfg.head_dim;
  uint16_t* kp = cache_plane(req_kv, c, layer, 0, cache_rows);
  uint16_t* vp = cache_plane(req_kv, c, layer, 1, cache_rows);
  st = run_norm_rope(c, reqs, total_q, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, o, kp, vp, hs, s);
  if (st != ATTUNER_OK) return st;
  return run_attention(c, reqs, total_q, o, kp, vp, hs, o, lse, s, nullptr, part,
                       noalloc ? (size_t)ATTUNER_NOALLOC_SCRATCH_BYTES : 0, gather);
}

attuner_status attuner_suffix_attn(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                   const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                   const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                   int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                   int64_t cache_rows, void* o, float* lse, void* stream) {
  return suffix_attn_impl(c, layer, n_req, cu_q, cu_ctx, art_len, pos0, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q,
                          gamma_k, req_kv, cache_rows, o, lse, stream, false);
}

attuner_status attuner_suffix_attn_noalloc(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                           const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                           const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                           int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                           int64_t cache_rows, void* o, float* lse, void* stream) {
  return suffix_attn_impl(c, layer, n_req, cu_q, cu_ctx, art_len, pos0, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q,
                          gamma_k, req_kv, cache_rows, o, lse, stream, true);
}

attuner_status attuner_suffix_attn_gather(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_q,
                                          const int32_t* cu_ctx, const int32_t* art_len, const int32_t* pos0,
                                          const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                          int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                          int64_t cache_rows, void* o, float* lse, const int32_t* block_table,
                                          int64_t n_entries, int32_t gather_layer, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (c->last_entries < 0 || block_table != c->last_table || n_entries != c->last_entries ||
      cache_rows != c->last_rows)
    return fail(ATTUNER_EINVAL, "block_table, n_entries and cache_rows must be those of the last "
                                "attuner_assemble_table call");
  if (gather_layer < 0 || gather_layer >= c->cfg.n_layers)
    return fail(ATTUNER_ERANGE, "gather_layer %d outside [0, %d)", gather_layer, c->cfg.n_layers);
  if (gather_layer == layer)
    return fail(ATTUNER_EINVAL, "gather_layer must differ from layer (the attention reads that layer's rows)");
  if (!req_kv || !aligned16(req_kv)) return fail(ATTUNER_EINVAL, "req_kv must be non-null and 16-byte aligned");
  // the attention launch carries the copy when the table names HBM pages only
  // and one layer's offsets fit 32 bits; otherwise the copy is a launch of
  // its own, issued (like the carried one) only once every argument passed
  const int64_t n_slab = 2 * c->cfg.n_kv_heads;
  const bool pow2 = ((n_slab * 4) & (n_slab * 4 - 1)) == 0;
  const bool fits = n_entries * n_slab * 4 < INT32_MAX && c->pool_pages * n_slab * kPageTokens * 16 < (1LL << 32) &&
                    n_slab * cache_rows * 16 < (1LL << 32);
  const bool apart = !c->last_hbm_only || !pow2 || !fits || !c->pool;
  const GatherArgs g{block_table, n_entries, gather_layer, static_cast<uint16_t*>(req_kv), cache_rows, apart};
  return suffix_attn_impl(c, layer, n_req, cu_q, cu_ctx, art_len, pos0, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q,
                          gamma_k, req_kv, cache_rows, o, lse, stream, false, n_entries > 0 ? &g : nullptr);
}

attuner_status attuner_span_attn(attuner_ctx* c, int32_t layer, int32_t n_spans, const int32_t* cu_q,
                                 const int32_t* kv_start, const int32_t* offset, const int32_t* pos0,
                                 const void* q_raw, int64_t ld_q, const void* k_raw, const void* v_raw,
                                 int64_t ld_kv, const void* gamma_q, const void* gamma_k, void* req_kv,
                                 int64_t cache_rows, void* o, float* lse, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_layer(c, layer);
  if (st != ATTUNER_OK) return st;
  if (n_spans < 0 || n_spans > ATTUNER_MAX_REQUESTS)
    return fail(ATTUNER_ERANGE, "n_spans %d outside [0, %d]", n_spans, ATTUNER_MAX_REQUESTS);
  if (n_spans == 0) return ATTUNER_OK;
  if (!cu_q || !kv_start || !offset) return fail(ATTUNER_EINVAL, "null span array");
  if (cu_q[0] != 0) return fail(ATTUNER_EINVAL, "cu_q[0] must be 0");
  std::vector<ReqDesc> reqs;
  for (int s = 0; s < n_spans; ++s) {
    ReqDesc d;
    d.q_start = cu_q[s];
    d.q_len = cu_q[s + 1] - cu_q[s];
    d.kv_start = kv_start[s];
    d.art_len = offset[s];
    d.pos0 = pos0 ? pos0[s] : offset[s];
    if (d.q_len < 0 || d.kv_start < 0 || d.art_len < 0 || d.pos0 < 0)
      return fail(ATTUNER_EINVAL, "span %d: negative length, start, offset or position", s);
    if ((int64_t)d.kv_start + d.art_len + d.q_len > cache_rows)
      return fail(ATTUNER_EINVAL, "span %d: rows %d + %d + %d exceed cache_rows %lld", s, d.kv_start, d.art_len,
                  d.q_len, (long long)cache_rows);
    reqs.push_back(d);
  }
  const int32_t total_q = cu_q[n_spans];
  if (total_q == 0) return ATTUNER_OK;
  st = check_norm_args(q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, c);
  if (st != ATTUNER_OK) return st;
  if (!req_kv || !o || !aligned16(req_kv) || !aligned16(o))
    return fail(ATTUNER_EINVAL, "req_kv and o must be non-null and 16-byte aligned");
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t hs = cache_rows * c->cfg.head_dim;
  uint16_t* kp = cache_plane(req_kv, c, layer, 0, cache_rows);
  uint16_t* vp = cache_plane(req_kv, c, layer, 1, cache_rows);
  st = run_norm_rope(c, reqs, total_q, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, o, kp, vp, hs, s);
  if (st != ATTUNER_OK) return st;
  // Attention: consecutive spans of one request (same kv_start, rows back to
  // back) share one work-list entry, their rows packed into common 64-row
  // blocks, each row seeing the keys up to its own position.  A short span
  // then rides in a block with its neighbours instead of walking its whole
  // prefix of key tiles alone.
  std::vector<ReqDesc> packed;
  std::vector<SpanRow> table;
  for (size_t i = 0; i < reqs.size();) {
    if (reqs[i].q_len == 0) {
      ++i;
      continue;
    }
    // merge while the next span continues the rows and starts at or past the
    // end of the previous one (positions must grow from row to row)
    size_t j = i + 1;
    size_t last = i;  // last span with rows in the group
    while (j < reqs.size() && reqs[j].kv_start == reqs[i].kv_start &&
           (reqs[j].q_len == 0 ||
            (reqs[j].q_start == reqs[last].q_start + reqs[last].q_len &&
             reqs[j].art_len >= reqs[last].art_len + reqs[last].q_len))) {
      if (reqs[j].q_len > 0) last = j;
      ++j;
    }
    ReqDesc g = reqs[i];
    int32_t n_rows = 0, n_sp = 0;
    const int32_t span0 = (int32_t)table.size();
    for (size_t k = i; k < j; ++k) {
      if (reqs[k].q_len == 0) continue;
      table.push_back(SpanRow{reqs[k].q_start, reqs[k].art_len});
      n_rows += reqs[k].q_len;
      g.art_len = reqs[k].art_len + reqs[k].q_len - n_rows;  // art_len + q_len = last row's position + 1
      ++n_sp;
    }
    g.q_len = n_rows;
    if (n_sp > 1) {
      g.span0 = span0;
      g.n_span = n_sp;
    } else {
      table.pop_back();
      g.art_len = reqs[i].art_len;
    }
    packed.push_back(g);
    i = j;
  }
  return run_attention(c, packed, total_q, o, kp, vp, hs, o, lse, s, &table);
}

attuner_status attuner_decode_attn(attuner_ctx* c, int32_t layer, int32_t n_req, const int32_t* cu_ctx,
                                   const int32_t* ctx_len, const int32_t* pos, const void* q_raw, int64_t ld_q,
                                   const void* k_raw, const void* v_raw, int64_t ld_kv, const void* gamma_q,
                                   const void* gamma_k, void* req_kv, int64_t cache_rows, void* o, void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  attuner_status st = check_layer(c, layer);
  if (st != ATTUNER_OK) return st;
  if (n_req < 0 || n_req > ATTUNER_MAX_REQUESTS)
    return fail(ATTUNER_ERANGE, "n_req %d outside [0, %d]", n_req, ATTUNER_MAX_REQUESTS);
  if (n_req == 0) return ATTUNER_OK;
  if (c->cfg.n_q_heads != 4 * c->cfg.n_kv_heads)
    return fail(ATTUNER_EINVAL, "the decode kernel is built for 4 query heads per KV head");
  std::vector<int32_t> cu_q(n_req + 1);
  for (int32_t r = 0; r <= n_req; ++r) cu_q[r] = r;
  std::vector<ReqDesc> reqs;
  int32_t total_q = 0;
  st = build_reqs(c, n_req, cu_q.data(), cu_ctx, ctx_len, pos, cache_rows, &reqs, &total_q);
  if (st != ATTUNER_OK) return st;
  st = check_norm_args(q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, c);
  if (st != ATTUNER_OK) return st;
  if (!req_kv || !o || !aligned16(req_kv) || !aligned16(o))
    return fail(ATTUNER_EINVAL, "req_kv and o must be non-null and 16-byte aligned");
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t hs = cache_rows * c->cfg.head_dim;
  uint16_t* kp = cache_plane(req_kv, c, layer, 0, cache_rows);
  uint16_t* vp = cache_plane(req_kv, c, layer, 1, cache_rows);
  return run_decode(c, reqs, q_raw, ld_q, k_raw, v_raw, ld_kv, gamma_q, gamma_k, kp, vp, hs, o, s);
}

attuner_status attuner_full_prefill(attuner_ctx* c, int32_t n_tok, int32_t pos0, const void* x, const void* wqkv,
                                    const void* a, const void* b, int32_t rank, float scale, const void* gamma_q,
                                    const void* gamma_k, void* o, void* k_out, void* v_out, float* lse,
                                    void* stream) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (n_tok < 0 || pos0 < 0) return fail(ATTUNER_EINVAL, "negative n_tok or pos0");
  if (n_tok == 0) return ATTUNER_OK;
  if (!gamma_q || !gamma_k || !o || !k_out || !v_out) return fail(ATTUNER_EINVAL, "null gamma or output");
  if (!aligned16(o) || !aligned16(k_out) || !aligned16(v_out) || !aligned16(gamma_q) || !aligned16(gamma_k))
    return fail(ATTUNER_EINVAL, "outputs and gamma must be 16-byte aligned");
  DeviceGuard dg(c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nq = q_dim(c), nkv = kv_dim(c), n_out = nq + 2 * nkv;
  attuner_status st = grow(c, c->ws_qkv, (size_t)n_tok * n_out * sizeof(uint16_t), s, "full-prefill projection");
  if (st != ATTUNER_OK) return st;
  uint16_t* qkv = static_cast<uint16_t*>(c->ws_qkv.ptr);
  st = qproj_impl(c, n_tok, x, wqkv, n_out, a, b, rank, scale, nq, qkv, s);
  if (st != ATTUNER_OK) return st;
  std::vector<ReqDesc> reqs(1);
  reqs[0].q_start = 0;
  reqs[0].q_len = n_tok;
  reqs[0].kv_start = 0;
  reqs[0].art_len = 0;
  reqs[0].pos0 = pos0;
  const int64_t hs = (int64_t)n_tok * c->cfg.head_dim;
  st = run_norm_rope(c, reqs, n_tok, qkv, n_out, qkv + nq, qkv + nq + nkv, n_out, gamma_q, gamma_k, o,
                     static_cast<uint16_t*>(k_out), static_cast<uint16_t*>(v_out), hs, s);
  if (st != ATTUNER_OK) return st;
  return run_attention(c, reqs, n_tok, o, static_cast<const uint16_t*>(k_out), static_cast<const uint16_t*>(v_out), hs,
                       o, lse, s);
}

attuner_status attuner_trace_begin(attuner_ctx* c) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (g_tracer != nullptr && g_tracer != &c->tracer) return fail(ATTUNER_EINVAL, "another context is tracing on this thread");
  c->tracer.recs.clear();
  c->tracer.pool_used = 0;
  c->tracer.err = hipSuccess;
  g_tracer = &c->tracer;
  return ATTUNER_OK;
}

attuner_status attuner_trace_end(attuner_ctx* c, attuner_kernel_time* out, int32_t max_entries, int32_t* n_entries) {
  if (!c) return fail(ATTUNER_EINVAL, "null ctx");
  if (g_tracer != &c->tracer) return fail(ATTUNER_EINVAL, "this context is not tracing on this thread");
  g_tracer = nullptr;
  Tracer& t = c->tracer;
  if (t.err != hipSuccess) return fail(ATTUNER_EDEVICE, "trace event: %s", hipGetErrorString(t.err));
  DeviceGuard dg(c->device);
  std::vector<attuner_kernel_time> agg;
  for (const auto& r : t.recs) {
    HIP_TRY(hipEventSynchronize(r.stop));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.start, r.stop));
    auto it = std::find_if(agg.begin(), agg.end(), [&](const attuner_kernel_time& k) { return strcmp(k.kernel, r.name) == 0; });
    if (it == agg.end()) {
      attuner_kernel_time k;
      memset(&k, 0, sizeof k);
      snprintf(k.kernel, sizeof k.kernel, "%s", r.name);
      agg.push_back(k);
      it = agg.end() - 1;
    }
    it->launches += 1;
    it->total_ms += ms;
    it->max_ms = std::max(it->max_ms, (double)ms);
  }
  t.recs.clear();
  std::sort(agg.begin(), agg.end(),
            [](const attuner_kernel_time& a, const attuner_kernel_time& b) { return a.total_ms > b.total_ms; });
  if (n_entries) *n_entries = (int32_t)agg.size();
  if (out) {
    if (max_entries < (int32_t)agg.size()) return fail(ATTUNER_ERANGE, "max_entries %d < %zu kernels", max_entries, agg.size());
    memcpy(out, agg.data(), agg.size() * sizeof(attuner_kernel_time));
  }
  return ATTUNER_OK;
}

attuner_status attuner_bounds_checked(int32_t* checked) {
  if (!checked) return fail(ATTUNER_EINVAL, "null checked");
#ifdef ATTUNER_CHECKED
  *checked = 1;
#else
  *checked = 0;
#endif
  return ATTUNER_OK;
}

attuner_status attuner_bounds_violations(int32_t device, int32_t reset, uint32_t* bits) {
  if (!bits) return fail(ATTUNER_EINVAL, "null bits");
  *bits = 0;
#ifdef ATTUNER_CHECKED
  int n_dev = 0;
  HIP_TRY(hipGetDeviceCount(&n_dev));
  if (device < 0 || device >= n_dev) return fail(ATTUNER_EINVAL, "device %d of %d", device, n_dev);
  DeviceGuard dg(device);
  HIP_TRY(hipDeviceSynchronize());
  unsigned int v = 0;
  HIP_TRY(read_violations_gather(&v, reset != 0));
  HIP_TRY(read_violations_attention(&v, reset != 0));
  HIP_TRY(read_violations_decode(&v, reset != 0));
  *bits = v;
#else
  (void)device;
  (void)reset;
#endif
  return ATTUNER_OK;
}

}  // extern "C"
