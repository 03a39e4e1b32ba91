// Host runtime behind the C ABI of include/commitkv.h: context, workspace
// arena, pinned upload ring, page-table cache, argument validation and the
// launch sequence of each call.  Every argument error is caught here, before
// anything is enqueued, so no kernel ever sees an out-of-range page or a
// misaligned row.
#include "commitkv.h"
#include "ckv_host.h"
#include "ckv_kernels.h"
#include "ckv_trace.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

using namespace ckv;

namespace {

constexpr size_t kAlign = 256;
constexpr int kMaxDevices = 64;
constexpr int kPinnedSlots = 4;
constexpr int kPageCacheEntries = 16;
constexpr float kLog2eHost = 1.4426950408889634f;   // log2(e): natural-log LSE to log2 units
constexpr int kJointWindow = 32;       // candidates tested per joint round
constexpr int kJointRowsPerBlock = 64;
constexpr int kTargetBlocks = 256;     // one 8-wave workgroup per compute unit
// the fix-up recomputes a dominant page's whole split for one row, so long
// splits make it expensive: splits hold at most this many tokens
constexpr int kMaxSplitTokens = 8192;
// the token-mass kernel (64 VGPRs, 40 KB of LDS) keeps two workgroups per
// compute unit busy: 512 token chunks measured 31.7 us against 35.3 us with 256
constexpr int kMassBlocks = 512;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct PageEntry {
  std::vector<int32_t> key;   // start[0..n) then len[0..n)
  int32_t* dev = nullptr;
  size_t cap = 0;
  uint64_t used = 0;
};

struct PinnedSlot {
  char* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};

struct Plan {
  struct Item { void** dst; size_t bytes; };
  std::vector<Item> items;
  size_t total = 0;
  template <class T>
  void add(T** dst, size_t n) {
    items.push_back({reinterpret_cast<void**>(dst), n * sizeof(T)});
    total += round_up(std::max<size_t>(n * sizeof(T), 1), kAlign);
  }
};

}  // namespace

// Static device scratch of the allocation-free measurement call: every GPU
// the library runs on holds one copy for the life of the process.  In host
// code `scratch` names a host-side stand-in, not device memory: its device
// address (per device) comes from hipGetSymbolAddress at context creation,
// and only that address is ever handed to kernels or copies.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ckv_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  char* ws = nullptr;
  size_t ws_cap = 0;
  size_t ws_limit = 0;
  std::string err;
  PinnedSlot slots[kPinnedSlots];
  int next_slot = 0;
  std::vector<PageEntry> pages;
  uint64_t tick = 0;
  uint64_t call_tick = 0;   // first tick of the current call: entries used since are not evicted
  // grid selection state (zero between calls), sized for sel_seq sequences
  int32_t* sel_ctrl = nullptr;
  uint32_t* sel_hist = nullptr;
  int sel_seq = 0;
  int sel_resident = -1;     // workgroups of the grid selection resident at once
  uint32_t policy = 0;       // CKV_POLICY_* switches (Sec. 4.4 variants)
  long long barrier_ticks = ckv::kBarrierTicksDefault;   // grid-barrier wait bound
  // latched non-finite flag: a pinned, device-mapped host word the kernels
  // set; reported (and cleared) by the next call or by ckv_sync
  volatile uint32_t* nf_host = nullptr;
  uint32_t* nf_dev = nullptr;
  // the next word of the same block: the site of a failed device bounds
  // check (CKV_DEBUG builds only write it)
  volatile uint32_t* dbg_host = nullptr;
  uint32_t* dbg_dev = nullptr;
  void* scratch = nullptr;   // device address of the static scratch on this device
  std::string scratch_err;
  // kernel timing (events around every launch when enabled)
  bool timing = false;
  std::string timing_only;   // empty: every kernel
  struct Timed { int kid; hipEvent_t a, b; };
  std::vector<Timed> timed;
  std::vector<hipEvent_t> event_pool;
  std::vector<std::string> knames;
  std::vector<double> ktotal;
  std::vector<int64_t> kcount;
};

namespace {

int fail(ckv_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  return code;
}

int hip_fail(ckv_ctx* c, hipError_t e, const char* what) {
  return fail(c, CKV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define CKV_HIP(ctx, expr)                                  \
  do {                                                      \
    hipError_t e_ = (expr);                                 \
    if (e_ != hipSuccess) return hip_fail(ctx, e_, #expr);  \
  } while (0)

struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

}  // namespace

namespace ckv {
int ctx_fail(ckv_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  return code;
}
hipStream_t ctx_stream(const ckv_ctx* c) { return c->stream; }
int ctx_device(const ckv_ctx* c) { return c->device; }
}  // namespace ckv

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// start of an API call: clears the message and opens a new cache scope
void begin_call(ckv_ctx* c) {
  c->err.clear();
  c->call_tick = c->tick + 1;
}

// A non-finite value latched by an earlier call's kernels (visible once
// those kernels have finished) is reported once, then cleared.
int latched_nonfinite(ckv_ctx* c) {
  if (c->dbg_host && *c->dbg_host != 0u) {
    const uint32_t site = *c->dbg_host;
    *c->dbg_host = 0u;
    return fail(c, CKV_ERR_DEVICE_CHECK, "device bounds check %u failed in an earlier call on this context", site);
  }
  if (!c->nf_host || *c->nf_host == 0u) return CKV_OK;
  *c->nf_host = 0u;
  return fail(c, CKV_ERR_NONFINITE,
              "a NaN or infinite value reached the window outputs or log-sum-exp of an earlier call "
              "on this context (non-finite keys, values or queries, or recorded outputs)");
}

int ensure_ws(ckv_ctx* c, size_t need) {
  if (need <= c->ws_cap) return CKV_OK;
  if (c->ws_limit && need > c->ws_limit)
    return fail(c, CKV_ERR_NOMEM, "workspace of %zu bytes exceeds the limit of %zu", need, c->ws_limit);
  size_t want = std::max(need, c->ws_cap + c->ws_cap / 2);
  if (c->ws_limit) want = std::min(want, c->ws_limit);
  CKV_HIP(c, hipStreamSynchronize(c->stream));   // in-flight work may still use the old arena
  if (c->ws) {
    (void)hipFree(c->ws);
    c->ws = nullptr;
    c->ws_cap = 0;
  }
  void* p = nullptr;
  if (hipMalloc(&p, want) != hipSuccess) {
    (void)hipGetLastError();
    return fail(c, CKV_ERR_NOMEM, "hipMalloc of %zu workspace bytes failed", want);
  }
  c->ws = static_cast<char*>(p);
  c->ws_cap = want;
  return CKV_OK;
}

int realize(ckv_ctx* c, Plan& plan) {
  int rc = ensure_ws(c, plan.total);
  if (rc) return rc;
  size_t off = 0;
  for (auto& it : plan.items) {
    *it.dst = c->ws + off;
    off += round_up(std::max<size_t>(it.bytes, 1), kAlign);
  }
  return CKV_OK;
}

int kernel_id(ckv_ctx* c, const char* name) {
  for (size_t i = 0; i < c->knames.size(); ++i)
    if (c->knames[i] == name) return (int)i;
  c->knames.push_back(name);
  c->ktotal.push_back(0.0);
  c->kcount.push_back(0);
  return (int)c->knames.size() - 1;
}

hipError_t pooled_event(ckv_ctx* c, hipEvent_t* ev) {
  if (!c->event_pool.empty()) {
    *ev = c->event_pool.back();
    c->event_pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

// resolve recorded kernel timings (waits for the last recorded event)
int resolve_timings(ckv_ctx* c) {
  if (c->timed.empty()) return CKV_OK;
  CKV_HIP(c, hipEventSynchronize(c->timed.back().b));
  for (auto& t : c->timed) {
    float ms = 0.f;
    CKV_HIP(c, hipEventElapsedTime(&ms, t.a, t.b));
    c->ktotal[t.kid] += ms;
    c->kcount[t.kid] += 1;
    c->event_pool.push_back(t.a);
    c->event_pool.push_back(t.b);
  }
  c->timed.clear();
  return CKV_OK;
}

// launch a kernel (launcher expression), bracketed by events when timing is on
#define CKV_LAUNCH(ctx, name, expr)                                   \
  do {                                                                \
    hipEvent_t ea_ = nullptr, eb_ = nullptr;                          \
    const bool timed_ = (ctx)->timing &&                              \
        ((ctx)->timing_only.empty() || (ctx)->timing_only == (name)); \
    if (timed_) {                                                     \
      CKV_HIP(ctx, pooled_event(ctx, &ea_));                          \
      CKV_HIP(ctx, pooled_event(ctx, &eb_));                          \
      CKV_HIP(ctx, hipEventRecord(ea_, (ctx)->stream));               \
    }                                                                 \
    CKV_HIP(ctx, (expr));                                             \
    if (timed_) {                                                     \
      CKV_HIP(ctx, hipEventRecord(eb_, (ctx)->stream));               \
      (ctx)->timed.push_back({kernel_id(ctx, name), ea_, eb_});       \
    }                                                                 \
  } while (0)

// copy host bytes to device memory on the context stream via a pinned slot
int upload(ckv_ctx* c, const void* src, size_t bytes, void* dst) {
  if (bytes == 0) return CKV_OK;
  PinnedSlot& s = c->slots[c->next_slot];
  c->next_slot = (c->next_slot + 1) % kPinnedSlots;
  if (s.pending) {
    CKV_HIP(c, hipEventSynchronize(s.ev));
    s.pending = false;
  }
  if (s.cap < bytes) {
    if (s.host) (void)hipHostFree(s.host);
    s.host = nullptr;
    s.cap = 0;
    void* p = nullptr;
    const size_t want = std::max<size_t>(round_up(bytes, 4096), 1 << 16);
    CKV_HIP(c, hipHostMalloc(&p, want, hipHostMallocDefault));
    s.host = static_cast<char*>(p);
    s.cap = want;
  }
  if (!s.ev) CKV_HIP(c, hipEventCreateWithFlags(&s.ev, hipEventDisableTiming));
  std::memcpy(s.host, src, bytes);
  CKV_HIP(c, hipMemcpyAsync(dst, s.host, bytes, hipMemcpyHostToDevice, c->stream));
  CKV_HIP(c, hipEventRecord(s.ev, c->stream));
  s.pending = true;
  return CKV_OK;
}

// device copy of an int32 array, cached by content: an unchanged array is
// not copied again (the entries have their own allocations, so later calls'
// workspace never overwrites them)
//
// A call may take several copies (one per sequence, then the argument blob
// that points at them): an entry used since the call began (used >=
// call_tick) is never evicted, so the cache grows past kPageCacheEntries for
// such a call instead of overwriting or freeing a table the call's kernels
// are about to read.
int cached_copy(ckv_ctx* c, std::vector<int32_t>&& key, const int32_t** dev) {
  ++c->tick;
  for (auto& e : c->pages) {
    if (e.key == key) {
      e.used = c->tick;
      *dev = e.dev;
      return CKV_OK;
    }
  }
  PageEntry* e = nullptr;
  if ((int)c->pages.size() < kPageCacheEntries) {
    c->pages.emplace_back();
    e = &c->pages.back();
  } else {
    for (auto& x : c->pages)
      if (x.used < c->call_tick && (!e || x.used < e->used)) e = &x;
    if (!e) {
      c->pages.emplace_back();
      e = &c->pages.back();
    }
  }
  const size_t bytes = key.size() * sizeof(int32_t);
  if (e->cap < bytes) {
    if (e->dev) {
      CKV_HIP(c, hipStreamSynchronize(c->stream));
      (void)hipFree(e->dev);
      e->dev = nullptr;
      e->cap = 0;
    }
    void* p = nullptr;
    if (hipMalloc(&p, round_up(bytes, 4096)) != hipSuccess) {
      (void)hipGetLastError();
      e->key.clear();
      return fail(c, CKV_ERR_NOMEM, "device copy of %zu bytes failed", bytes);
    }
    e->dev = static_cast<int32_t*>(p);
    e->cap = round_up(bytes, 4096);
  }
  e->key.clear();
  int rc = upload(c, key.data(), bytes, e->dev);
  if (rc) return rc;
  e->key = std::move(key);
  e->used = c->tick;
  *dev = e->dev;
  return CKV_OK;
}

// device copy of a (validated) page list: start[0..n) then len[0..n)
int page_table(ckv_ctx* c, const ckv_page_list* pl, const int32_t** dstart, const int32_t** dlen) {
  CKV_RANGE("page table");
  const int n = pl->n_pages;
  *dstart = *dlen = nullptr;
  if (n == 0) return CKV_OK;
  std::vector<int32_t> key(2 * (size_t)n);
  std::memcpy(key.data(), pl->start, n * sizeof(int32_t));
  std::memcpy(key.data() + n, pl->len, n * sizeof(int32_t));
  const int32_t* d = nullptr;
  int rc = cached_copy(c, std::move(key), &d);
  if (rc) return rc;
  *dstart = d;
  *dlen = d + n;
  return CKV_OK;
}

int check_kv(ckv_ctx* c, const ckv_kv_view* kv) {
  if (!kv || !kv->k || !kv->v || !kv->pos) return fail(c, CKV_ERR_ARG, "kv view or one of its pointers is NULL");
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(c, CKV_ERR_SHAPE, "head_dim %d unsupported (64 or 128)", kv->head_dim);
  if (kv->n_tokens < 1 || kv->n_tokens > INT_MAX - 1024) return fail(c, CKV_ERR_SHAPE, "n_tokens %d out of range", kv->n_tokens);
  if (kv->n_kv_heads < 1) return fail(c, CKV_ERR_SHAPE, "n_kv_heads must be >= 1");
  if (!aligned16(kv->k) || !aligned16(kv->v) || kv->tok_stride % 8 || kv->head_stride % 8)
    return fail(c, CKV_ERR_ARG, "K/V rows must be 16-byte aligned (strides multiples of 8)");
  if (kv->tok_stride < kv->head_dim || kv->head_stride < 0)
    return fail(c, CKV_ERR_SHAPE, "K/V strides too small");
  if (kv->slot && (kv->pool_rows < 1 || (reinterpret_cast<uintptr_t>(kv->slot) & 3u)))
    return fail(c, CKV_ERR_ARG, "paged view: pool_rows must be >= 1 and slot 4-byte aligned");
  // the kernels address a token of one head with a 32-bit element offset
  // (24-bit multiply of row index and stride)
  const int64_t rows = kv->slot ? kv->pool_rows : kv->n_tokens;
  if (kv->tok_stride >= (1 << 24) || rows >= (1 << 24) || rows * kv->tok_stride >= ((int64_t)1 << 31))
    return fail(c, CKV_ERR_UNSUPPORTED, "rows * tok_stride must stay below 2^31 elements");
  return CKV_OK;
}

int check_win(ckv_ctx* c, const ckv_window_view* w, const ckv_kv_view* kv) {
  if (!w || !w->q || !w->qpos) return fail(c, CKV_ERR_ARG, "window view or one of its pointers is NULL");
  if (w->n_q_heads < 1 || w->n_q_heads % kv->n_kv_heads)
    return fail(c, CKV_ERR_SHAPE, "n_q_heads %d is not a multiple of n_kv_heads %d", w->n_q_heads, kv->n_kv_heads);
  if (w->n_rows < 1 || (int64_t)w->n_rows * w->n_q_heads > (1 << 20))
    return fail(c, CKV_ERR_SHAPE, "window rows %d out of range", w->n_rows);
  if (!aligned16(w->q) || w->row_stride % 8 || w->head_stride % 8)
    return fail(c, CKV_ERR_ARG, "query rows must be 16-byte aligned (strides multiples of 8)");
  if (w->row_stride < kv->head_dim) return fail(c, CKV_ERR_SHAPE, "query row stride too small");
  if (!(std::isfinite(w->scale))) return fail(c, CKV_ERR_ARG, "scale must be finite");
  return CKV_OK;
}

int check_pages(ckv_ctx* c, const ckv_page_list* pl, int n_tokens, const char* what) {
  if (!pl) return fail(c, CKV_ERR_ARG, "%s page list is NULL", what);
  if (pl->n_pages < 0) return fail(c, CKV_ERR_SHAPE, "%s: n_pages < 0", what);
  if (pl->n_pages == 0) return CKV_OK;
  if (!pl->start || !pl->len) return fail(c, CKV_ERR_ARG, "%s page arrays are NULL", what);
  int64_t prev_end = 0;
  for (int i = 0; i < pl->n_pages; ++i) {
    const int64_t s = pl->start[i], l = pl->len[i];
    if (l < 1 || l > CKV_MAX_PAGE_LEN) return fail(c, CKV_ERR_SHAPE, "%s page %d: length %lld not in [1, %d]", what, i, (long long)l, CKV_MAX_PAGE_LEN);
    if (s < 0 || s + l > n_tokens) return fail(c, CKV_ERR_SHAPE, "%s page %d: [%lld, %lld) outside [0, %d)", what, i, (long long)s, (long long)(s + l), n_tokens);
    if (s < prev_end) return fail(c, CKV_ERR_SHAPE, "%s page %d: pages must be sorted and disjoint", what, i);
    prev_end = s + l;
  }
  return CKV_OK;
}

AttnGeom make_geom(const ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* w) {
  AttnGeom a;
  a.dbg = c->dbg_dev;
  a.nonfinite = c->nf_dev;
  a.k = kv->k;
  a.v = kv->v;
  a.kv_head_stride = kv->head_stride;
  a.kv_tok_stride = kv->tok_stride;
  a.pos = kv->pos;
  a.S = kv->n_tokens;
  a.Hkv = kv->n_kv_heads;
  a.D = kv->head_dim;
  a.q = w->q;
  a.q_head_stride = w->head_stride;
  a.q_row_stride = w->row_stride;
  a.qpos = w->qpos;
  a.Hq = w->n_q_heads;
  a.W = w->n_rows;
  a.group = w->n_q_heads / kv->n_kv_heads;
  a.rows = a.group * a.W;
  const float scale = w->scale > 0.f ? w->scale : 1.0f / std::sqrt((float)kv->head_dim);
  a.sl2 = scale * 1.4426950408889634f;
  a.slot = kv->slot;
  a.pool_last = kv->slot ? (uint32_t)(kv->pool_rows - 1) : 0u;
  return a;
}

int max_page_len(const ckv_page_list* pl) {
  int m = 0;
  for (int i = 0; i < pl->n_pages; ++i) m = std::max(m, (int)pl->len[i]);
  return m;
}

// tokens per token-mass workgroup
int mass_chunk(const AttnGeom& a) {
  return (int)round_up(ceil_div(a.S, std::max(1, kMassBlocks / a.Hkv)), 64);
}

int items_per_block(int n_items, int other_blocks) {
  const int per = ceil_div(n_items * std::max(other_blocks, 1), kTargetBlocks);
  return std::min(ckv::kPageItemsMax, std::max(1, per));
}

}  // namespace

// ----------------------------------------------------------------- context

extern "C" int ckv_create(ckv_ctx** out, int device, void* hip_stream) {
  CKV_RANGE("ckv_create");
  if (!out) return CKV_ERR_ARG;
  *out = nullptr;
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) {
    (void)hipGetLastError();
    return CKV_ERR_HIP;
  }
  ckv_ctx* c = new (std::nothrow) ckv_ctx();
  if (!c) return CKV_ERR_NOMEM;
  c->device = device;
  c->stream = static_cast<hipStream_t>(hip_stream);
  {
    DeviceGuard g(device);
    void* h = nullptr;
    void* d = nullptr;
    if (!g.ok || hipHostMalloc(&h, 256, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
        hipHostGetDevicePointer(&d, h, 0) != hipSuccess) {
      (void)hipGetLastError();
      if (h) (void)hipHostFree(h);
      delete c;
      return CKV_ERR_HIP;
    }
    std::memset(h, 0, 256);
    c->nf_host = static_cast<volatile uint32_t*>(h);
    c->nf_dev = static_cast<uint32_t*>(d);
    c->dbg_host = c->nf_host + 1;
    c->dbg_dev = c->nf_dev + 1;
  }
  {
    // the static scratch's address on this device, looked up once per device
    // with the device current
    static std::mutex mu;
    static void* addr[kMaxDevices];
    static hipError_t err[kMaxDevices];
    static bool done[kMaxDevices];
    std::lock_guard<std::mutex> lock(mu);
    if (device < kMaxDevices) {
      if (!done[device]) {
        DeviceGuard g(device);
        void* p = nullptr;
        err[device] = g.ok ? hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) : hipErrorInvalidDevice;
        if (err[device] != hipSuccess) (void)hipGetLastError();
        addr[device] = err[device] == hipSuccess ? p : nullptr;
        done[device] = true;
      }
      c->scratch = addr[device];
      if (!c->scratch) c->scratch_err = hipGetErrorString(err[device]);
    } else {
      c->scratch_err = "device index beyond the scratch table";
    }
  }
  *out = c;
  return CKV_OK;
}

extern "C" int ckv_destroy(ckv_ctx* c) {
  CKV_RANGE("ckv_destroy");
  if (!c) return CKV_ERR_ARG;
  {
    DeviceGuard g(c->device);   // best effort: the context is freed whatever happens
    (void)hipStreamSynchronize(c->stream);
    if (c->ws) (void)hipFree(c->ws);
    if (c->sel_ctrl) (void)hipFree(c->sel_ctrl);
    if (c->sel_hist) (void)hipFree(c->sel_hist);
    for (auto& e : c->pages)
      if (e.dev) (void)hipFree(e.dev);
    for (auto& s : c->slots) {
      if (s.ev) (void)hipEventDestroy(s.ev);
      if (s.host) (void)hipHostFree(s.host);
    }
    if (c->nf_host) (void)hipHostFree(const_cast<uint32_t*>(c->nf_host));
    for (auto& t : c->timed) {
      (void)hipEventDestroy(t.a);
      (void)hipEventDestroy(t.b);
    }
    for (auto e : c->event_pool) (void)hipEventDestroy(e);
  }
  delete c;
  return CKV_OK;
}

extern "C" int ckv_set_stream(ckv_ctx* c, void* hip_stream) {
  if (!c) return CKV_ERR_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  CKV_HIP(c, hipStreamSynchronize(c->stream));
  c->stream = static_cast<hipStream_t>(hip_stream);
  return CKV_OK;
}

extern "C" int ckv_sync(ckv_ctx* c) {
  CKV_RANGE("ckv_sync");
  if (!c) return CKV_ERR_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  CKV_HIP(c, hipStreamSynchronize(c->stream));
  return latched_nonfinite(c);
}

extern "C" const char* ckv_last_error(const ckv_ctx* c) { return c ? c->err.c_str() : "NULL context"; }

extern "C" uint32_t ckv_build_flags(void) {
#ifdef CKV_DEBUG
  return CKV_BUILD_DEVICE_CHECKS;
#else
  return 0u;
#endif
}

extern "C" uint32_t ckv_version(void) {
  return (CKV_VERSION_MAJOR << 16) | (CKV_VERSION_MINOR << 8) | CKV_VERSION_PATCH;
}

extern "C" int ckv_set_workspace_limit(ckv_ctx* c, size_t bytes) {
  if (!c) return CKV_ERR_ARG;
  c->ws_limit = bytes;
  return CKV_OK;
}

extern "C" size_t ckv_workspace_bytes(const ckv_ctx* c) { return c ? c->ws_cap : 0; }

extern "C" int ckv_set_policy(ckv_ctx* c, uint32_t flags) {
  if (!c) return CKV_ERR_ARG;
  constexpr uint32_t known = CKV_POLICY_NO_PRECOMMIT | CKV_POLICY_NO_PERCENTILE | CKV_POLICY_NO_JOINT |
                             CKV_POLICY_NO_PROTECTION | CKV_POLICY_NO_LIFECYCLE;
  if (flags & ~known) return fail(c, CKV_ERR_ARG, "unknown policy bits 0x%x", flags & ~known);
  c->policy = flags;
  return CKV_OK;
}

extern "C" uint32_t ckv_get_policy(const ckv_ctx* c) { return c ? c->policy : 0u; }

extern "C" int ckv_set_barrier_timeout_us(ckv_ctx* c, int64_t us) {
  if (!c) return CKV_ERR_ARG;
  if (us < 0 || us > (int64_t)1 << 40) return fail(c, CKV_ERR_ARG, "barrier timeout %lld us out of range", (long long)us);
  c->barrier_ticks = us * 100;   // the device wall clock runs at 100 MHz
  return CKV_OK;
}

extern "C" int ckv_set_kernel_timing_only(ckv_ctx* c, const char* name) {
  if (!c) return CKV_ERR_ARG;
  c->timing_only = name ? name : "";
  return CKV_OK;
}

extern "C" int ckv_set_kernel_timing(ckv_ctx* c, int enable) {
  if (!c) return CKV_ERR_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  int rc = resolve_timings(c);
  if (rc) return rc;
  c->timing = enable != 0;
  return CKV_OK;
}

extern "C" int ckv_kernel_stats(ckv_ctx* c, int32_t idx, const char** name, double* total_ms,
                                int64_t* launches) {
  if (!c) return CKV_ERR_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  int rc = resolve_timings(c);
  if (rc) return rc;
  if (idx < 0 || idx >= (int32_t)c->knames.size()) return CKV_ERR_ARG;
  if (name) *name = c->knames[idx].c_str();
  if (total_ms) *total_ms = c->ktotal[idx];
  if (launches) *launches = c->kcount[idx];
  return CKV_OK;
}

extern "C" int ckv_reset_kernel_stats(ckv_ctx* c) {
  if (!c) return CKV_ERR_ARG;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  int rc = resolve_timings(c);
  if (rc) return rc;
  std::fill(c->ktotal.begin(), c->ktotal.end(), 0.0);
  std::fill(c->kcount.begin(), c->kcount.end(), 0);
  return CKV_OK;
}

// ------------------------------------------------------------- the calls

namespace {

// Workspace of one measurement call for a given number of token splits.
struct MeasureBufs {
  AttnSplit sp{};
  RowStats rs{};
  int* fix_list = nullptr;
  int* fix_count = nullptr;
  float* fpart = nullptr;
  int* arrive = nullptr;      // per listed pair: fix-up parts finished
};

void plan_measure(const AttnGeom& a, int n_splits, float* o, Plan& plan, MeasureBufs& b) {
  const int D = a.D, total_rows = a.Hq * a.W;
  const int rpb = rows_per_block_attention();
  const int nrb = ceil_div(a.rows, rpb);
  const int chunk = (int)round_up(ceil_div(a.S, n_splits), 64);
  n_splits = ceil_div(a.S, chunk);
  b.sp = AttnSplit{chunk, n_splits, nrb * rpb, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  b.rs = RowStats{o, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  const size_t nsr = (size_t)a.Hkv * n_splits * b.sp.rows_pad;
  plan.add(&b.sp.part_o, nsr * D);
  plan.add(&b.sp.part_m, nsr);
  plan.add(&b.sp.part_l, nsr);
  plan.add(&b.sp.part_c, nsr);
  plan.add(&b.sp.part_t, nsr);
  plan.add(&b.sp.part_p, nsr);
  if (!o) plan.add(&b.rs.o, (size_t)total_rows * D);
  plan.add(&b.rs.lse2, total_rows);
  plan.add(&b.rs.onorm, total_rows);
  plan.add(&b.rs.nvis, total_rows);
  plan.add(&b.rs.m2, total_rows);
  plan.add(&b.rs.m2t, total_rows);
  plan.add(&b.rs.m2p, total_rows);
  plan.add(&b.fix_list, 4 * (size_t)total_rows);
  plan.add(&b.fix_count, 1);
  plan.add(&b.fpart, (size_t)total_rows * ckv::kFixParts * (D + 1));
  plan.add(&b.arrive, total_rows);
}

// splits of the window pass: about one workgroup per compute unit, and at
// most kMaxSplitTokens tokens per split
int default_splits(const AttnGeom& a) {
  const int nrb = ceil_div(a.rows, rows_per_block_attention());
  return std::max(1, std::min(ceil_div(a.S, 64),
                              std::max(ceil_div(kTargetBlocks, a.Hkv * nrb), ceil_div(a.S, kMaxSplitTokens))));
}

int check_measure(ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* win, const ckv_page_list* pages,
                  const float* R, const float* token_mass) {
  int rc;
  if ((rc = check_kv(c, kv)) || (rc = check_win(c, win, kv)) || (rc = check_pages(c, pages, kv->n_tokens, "measured")))
    return rc;
  if (pages->n_pages > 0 && !R) return fail(c, CKV_ERR_ARG, "R is NULL");
  if (token_mass && (win->n_q_heads / kv->n_kv_heads) * win->n_rows > token_mass_max_rows())
    return fail(c, CKV_ERR_UNSUPPORTED, "token_mass supports at most %d window rows per KV head",
                token_mass_max_rows());
  return CKV_OK;
}

// the kernels of one measurement call, enqueued on the context's stream
int enqueue_measure(ckv_ctx* c, const AttnGeom& a, const MeasureBufs& b, const int32_t* dstart,
                    const int32_t* dlen, const ckv_page_list* pages, float* R, float* R_head, float* lse,
                    float* token_mass) {
  const int n = pages->n_pages, total_rows = a.Hq * a.W;
  CKV_LAUNCH(c, "window_attention", launch_window_attention(a, b.sp, c->stream));
  ZeroList zl{R, R ? (size_t)n : 0, R_head, R_head ? (size_t)n * a.Hq : 0, token_mass,
              token_mass ? (size_t)a.S : 0, b.fix_count, b.arrive, (size_t)total_rows, c->nf_dev};
  CKV_LAUNCH(c, "combine", launch_combine(a, b.sp, b.rs, lse, zl, c->stream));
  if (n > 0) {
    PageWork pw{};
    pw.start = dstart;
    pw.len = dlen;
    pw.n_items = n;
    pw.n_pages = n;
    pw.items_per_block = std::min(items_per_block(n, a.Hkv * ceil_div(a.rows, rows_per_block_page())),
                                  ckv::kPageRmaxCap / page_heads_per_block(a.W, a.group));
    pw.R = R;
    pw.R_head = R_head;
    pw.lse_scale = 1.f;
    pw.Hq = a.Hq;
    pw.total_rows = total_rows;
    pw.fix_list = b.fix_list;
    pw.fix_count = b.fix_count;
    pw.fix_cap = total_rows;
    pw.fix_a = ckv::kFixA;
    pw.fix_a_hi = ckv::kFixAHi;
    pw.split_tokens = b.sp.chunk;
    CKV_LAUNCH(c, "page_effect", launch_page_kernel(a, pw, b.rs, 0, max_page_len(pages), c->stream));
    if (token_mass && mass_fixup_applies(a)) {
      // the fix-up runs in the shadow of the token mass, in one launch
      CKV_LAUNCH(c, "token_mass_fixup", launch_mass_fixup(a, b.sp, b.rs, pw, b.fpart, b.arrive, ckv::kFixParts,
                                                          token_mass, mass_chunk(a), c->stream));
      return CKV_OK;
    }
    CKV_LAUNCH(c, "page_fixup", launch_page_fixup(a, b.sp, b.rs, pw, b.fpart, b.arrive, ckv::kFixParts, 0, c->stream));
  }
  if (token_mass) CKV_LAUNCH(c, "token_mass", launch_token_mass(a, b.rs, token_mass, mass_chunk(a), c->stream));
  return CKV_OK;
}

}  // namespace

extern "C" int ckv_measure_page_effects(ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* win,
                                        const ckv_page_list* pages, float* R, float* R_head, float* o,
                                        float* lse, float* token_mass) {
  CKV_RANGE("ckv_measure_page_effects");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  int rc;
  if ((rc = check_measure(c, kv, win, pages, R, token_mass))) return rc;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);

  const AttnGeom a = make_geom(c, kv, win);
  Plan plan;
  MeasureBufs b;
  plan_measure(a, default_splits(a), o, plan, b);
  const int32_t *dstart = nullptr, *dlen = nullptr;
  if ((rc = page_table(c, pages, &dstart, &dlen))) return rc;
  if ((rc = realize(c, plan))) return rc;
  return enqueue_measure(c, a, b, dstart, dlen, pages, R, R_head, lse, token_mass);
}

extern "C" int ckv_measure_page_effects_noalloc(ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* win,
                                                const ckv_page_list* pages, float* R, float* R_head, float* o,
                                                float* lse, float* token_mass) {
  CKV_RANGE("ckv_measure_page_effects_noalloc");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  int rc;
  if ((rc = check_measure(c, kv, win, pages, R, token_mass))) return rc;
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  if (!c->scratch) return fail(c, CKV_ERR_HIP, "the device's static scratch is unavailable: %s", c->scratch_err.c_str());

  const AttnGeom a = make_geom(c, kv, win);
  const int n = pages->n_pages;
  const size_t table = round_up(std::max<size_t>(2 * (size_t)n * sizeof(int32_t), 1), kAlign);
  // as many splits as the regular call uses, fewer if the split partials
  // would not fit the static scratch
  int splits = default_splits(a);
  Plan plan;
  MeasureBufs b;
  for (;; --splits) {
    plan = Plan();
    plan_measure(a, splits, o, plan, b);
    if (table + plan.total <= kScratchBytes || splits == 1) break;
  }
  if (table + plan.total > kScratchBytes)
    return fail(c, CKV_ERR_UNSUPPORTED,
                "the allocation-free call needs %zu bytes of scratch for this shape; it holds %zu",
                table + plan.total, (size_t)kScratchBytes);
  char* base = static_cast<char*>(c->scratch);
  int32_t* dtab = reinterpret_cast<int32_t*>(base);
  size_t off = table;
  for (auto& it : plan.items) {
    *it.dst = base + off;
    off += round_up(std::max<size_t>(it.bytes, 1), kAlign);
  }
  if (n > 0) {
    CKV_HIP(c, hipMemcpyAsync(dtab, pages->start, n * sizeof(int32_t), hipMemcpyHostToDevice, c->stream));
    CKV_HIP(c, hipMemcpyAsync(dtab + n, pages->len, n * sizeof(int32_t), hipMemcpyHostToDevice, c->stream));
  }
  // no kernel timing here: its events are created on demand
  const bool timing = c->timing;
  c->timing = false;
  rc = enqueue_measure(c, a, b, n > 0 ? dtab : nullptr, n > 0 ? dtab + n : nullptr, pages, R, R_head, lse,
                       token_mass);
  c->timing = timing;
  return rc;
}

extern "C" int ckv_measure_page_effects_batch(ckv_ctx* c, int32_t n, const ckv_kv_view* kv,
                                              const ckv_window_view* win, const ckv_page_list* pages,
                                              float* const* R, float* const* R_head, float* const* o,
                                              float* const* lse, float* const* token_mass) {
  CKV_RANGE("ckv_measure_page_effects_batch");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  if (n < 0 || (n > 0 && (!kv || !win || !pages || !R))) return fail(c, CKV_ERR_ARG, "batch: NULL arrays or n < 0");
  for (int i = 0; i < n; ++i) {
    int rc;
    if ((rc = check_kv(c, &kv[i])) || (rc = check_win(c, &win[i], &kv[i])) ||
        (rc = check_pages(c, &pages[i], kv[i].n_tokens, "measured"))) {
      const std::string m = c->err;
      return fail(c, rc, "batch problem %d: %s", i, m.c_str());
    }
    if (pages[i].n_pages > 0 && !R[i]) return fail(c, CKV_ERR_ARG, "batch problem %d: R is NULL", i);
    if (token_mass && token_mass[i] &&
        (win[i].n_q_heads / kv[i].n_kv_heads) * win[i].n_rows > token_mass_max_rows())
      return fail(c, CKV_ERR_UNSUPPORTED, "batch problem %d: too many window rows for token_mass", i);
  }
  for (int i = 0; i < n; ++i) {
    const int rc = ckv_measure_page_effects(c, &kv[i], &win[i], &pages[i], R[i], R_head ? R_head[i] : nullptr,
                                            o ? o[i] : nullptr, lse ? lse[i] : nullptr,
                                            token_mass ? token_mass[i] : nullptr);
    if (rc) {
      const std::string m = c->err;
      return fail(c, rc, "batch problem %d: %s", i, m.c_str());
    }
  }
  return CKV_OK;
}

extern "C" int ckv_measure_recorded(ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* win,
                                    const ckv_page_list* pages, const float* o, const float* lse, float* R,
                                    float* R_head, float* token_mass) {
  CKV_RANGE("ckv_measure_recorded");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  int rc;
  if ((rc = check_kv(c, kv)) || (rc = check_win(c, win, kv)) || (rc = check_pages(c, pages, kv->n_tokens, "measured")))
    return rc;
  if (!o || !lse) return fail(c, CKV_ERR_ARG, "recorded o or lse is NULL");
  if (!aligned16(o)) return fail(c, CKV_ERR_ARG, "recorded o must be 16-byte aligned");
  if (pages->n_pages > 0 && !R) return fail(c, CKV_ERR_ARG, "R is NULL");
  if (token_mass && (win->n_q_heads / kv->n_kv_heads) * win->n_rows > token_mass_max_rows())
    return fail(c, CKV_ERR_UNSUPPORTED, "token_mass supports at most %d window rows per KV head",
                token_mass_max_rows());
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);

  const AttnGeom a = make_geom(c, kv, win);
  const int n = pages->n_pages, total_rows = a.Hq * a.W;
  RowStats rs{const_cast<float*>(o), nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  Plan plan;
  plan.add(&rs.lse2, total_rows);
  plan.add(&rs.onorm, total_rows);
  plan.add(&rs.nvis, total_rows);
  int* nvis_part = nullptr;
  plan.add(&nvis_part, (size_t)a.W * recorded_slices(a.S));
  int *fix_list = nullptr, *fix_count = nullptr;
  plan.add(&fix_list, 4 * (size_t)total_rows);
  plan.add(&fix_count, 1);
  // pairs whose output without the page comes from the complement pass: a
  // row has at most one page with A > 0.5, so the list holds every row; the
  // pass spreads its pairs over a fixed number of (pair, part) items
  const int cap2 = total_rows;
  const int items2 = std::max(ckv::kFixComplementItems, total_rows);
  int *list2 = nullptr, *count2 = nullptr;
  plan.add(&list2, 4 * (size_t)cap2);
  plan.add(&count2, 1 + (size_t)cap2);   // the count, then the pairs' arrival counts
  float* fpart = nullptr;
  plan.add(&fpart, (size_t)items2 * (a.D + 1));
  const int32_t *dstart = nullptr, *dlen = nullptr;
  if ((rc = page_table(c, pages, &dstart, &dlen))) return rc;
  if ((rc = realize(c, plan))) return rc;

  ZeroList zl{R, R ? (size_t)n : 0, R_head, R_head ? (size_t)n * a.Hq : 0, token_mass,
              token_mass ? (size_t)a.S : 0, fix_count, count2, 1 + (size_t)cap2, c->nf_dev};
  // without pages the visible counts have no reader (the token mass latches
  // a non-finite sum itself), so the counting pass is skipped
  CKV_LAUNCH(c, "recorded_rows", launch_recorded_rows(a, o, lse, rs, n > 0 ? nvis_part : nullptr, zl, c->stream));
  if (n > 0) {
    PageWork pw{};
    pw.start = dstart;
    pw.len = dlen;
    pw.n_items = n;
    pw.n_pages = n;
    pw.items_per_block = std::min(items_per_block(n, a.Hkv * ceil_div(a.rows, rows_per_block_page())),
                                  ckv::kPageRmaxCap / page_heads_per_block(a.W, a.group));
    pw.R = R;
    pw.R_head = R_head;
    pw.lse_scale = 1.f;
    pw.Hq = a.Hq;
    pw.total_rows = total_rows;
    pw.fix_list = fix_list;
    pw.fix_count = fix_count;
    pw.fix_cap = total_rows;
    pw.fix_a = ckv::kFixARecorded;
    pw.fix_a_hi = ckv::kFixARecorded;
    CKV_LAUNCH(c, "page_effect", launch_page_kernel(a, pw, rs, 0, max_page_len(pages), c->stream));
    CKV_LAUNCH(c, "page_fixup_recorded", launch_page_fixup_recorded(a, rs, pw, list2, count2, cap2,
                                                                    ckv::kFixAComplement, c->stream));
    // the complement pass: one split covering the whole row, so the fix-up
    // recomputes every token of the row except the page's
    PageWork pw2 = pw;
    pw2.fix_list = list2;
    pw2.fix_count = count2;
    pw2.fix_cap = cap2;
    AttnSplit whole{(int)round_up(a.S, 64), 1, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
    CKV_LAUNCH(c, "page_fixup_complement",
               launch_page_fixup(a, whole, rs, pw2, fpart, count2 + 1, ckv::kFixPartsRow, items2, c->stream));
  }
  if (token_mass) {
    CKV_LAUNCH(c, "token_mass", launch_token_mass(a, rs, token_mass, mass_chunk(a), c->stream));
  }
  return CKV_OK;
}

extern "C" int ckv_classify_pages(ckv_ctx* c, int32_t n, const float* R_pre, const float* R_post,
                                  const ckv_thresholds* th, const uint8_t* force, int32_t max_cand,
                                  uint8_t* lambda, float* P_pre, float* P_post, int32_t* cand,
                                  int32_t* n_cand) {
  CKV_RANGE("ckv_classify_pages");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  if (n < 0) return fail(c, CKV_ERR_SHAPE, "n < 0");
  if (!n_cand) return fail(c, CKV_ERR_ARG, "n_cand is NULL");
  if (n > 0 && (!R_pre || !R_post || !lambda || !cand)) return fail(c, CKV_ERR_ARG, "NULL input or output array");
  ckv_thresholds t = th ? *th : ckv_thresholds{0.05f, 0.01f, 0.75f, 0.25f, 0.01f};
  if (!(t.tau_dead <= t.tau_use) || !(t.rho_dead <= t.rho_use))
    return fail(c, CKV_ERR_ARG, "thresholds must satisfy tau_dead <= tau_use and rho_dead <= rho_use");
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  ClassifyArgs a{};
  a.n = n;
  a.R_pre = R_pre;
  a.R_post = R_post;
  a.tau_use = t.tau_use;
  a.tau_dead = t.tau_dead;
  a.rho_use = t.rho_use;
  a.rho_dead = t.rho_dead;
  a.force = force;
  a.max_cand = max_cand;
  a.lambda = lambda;
  a.P_pre = P_pre;
  a.P_post = P_post;
  a.cand = cand;
  a.n_cand = n_cand;
  a.policy = c->policy;
  Plan plan;
  plan.add(&a.is_cand, std::max(n, 1));
  if (!P_pre) plan.add(&a.P_pre, std::max(n, 1));
  if (!P_post) plan.add(&a.P_post, std::max(n, 1));
  int rc = realize(c, plan);
  if (rc) return rc;
  CKV_LAUNCH(c, "classify", launch_classify(a, c->stream));
  return CKV_OK;
}

extern "C" int ckv_joint_test(ckv_ctx* c, const ckv_kv_view* kv, const ckv_window_view* win, const float* o,
                              const float* lse, const ckv_page_list* pages, const int32_t* cand,
                              const int32_t* n_cand, int32_t max_cand, float tau_joint, uint8_t* accepted,
                              float* union_R, int32_t* n_accepted) {
  CKV_RANGE("ckv_joint_test");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  int rc;
  if ((rc = check_kv(c, kv)) || (rc = check_win(c, win, kv)) || (rc = check_pages(c, pages, kv->n_tokens, "joint")))
    return rc;
  if (!o || !lse || !cand || !n_cand || !accepted || !n_accepted)
    return fail(c, CKV_ERR_ARG, "NULL input or output array");
  if (max_cand < 1) return fail(c, CKV_ERR_SHAPE, "max_cand must be >= 1");
  if (max_cand > (1 << 22)) return fail(c, CKV_ERR_UNSUPPORTED, "max_cand above 2^22 is not supported");
  if (!std::isfinite(tau_joint)) return fail(c, CKV_ERR_ARG, "tau_joint must be finite");
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  const AttnGeom a = make_geom(c, kv, win);
  const int total_rows = a.Hq * a.W, D = a.D;
  // the residual pass reads the caller's o and natural-log lse directly
  RowStats rs{const_cast<float*>(o), const_cast<float*>(lse), nullptr, nullptr, nullptr, nullptr, nullptr};
  JointArgs j{};
  j.total_rows = total_rows;
  j.D = D;
  j.max_cand = max_cand;
  j.W = a.W;
  j.n_cand = n_cand;
  j.window = kJointWindow;
  j.rows_per_block = kJointRowsPerBlock;
  j.tau = tau_joint;
  j.nonfinite = c->nf_dev;
  j.barrier_ticks = c->barrier_ticks;
  j.accept_all = (c->policy & CKV_POLICY_NO_JOINT) != 0;
  j.accepted = accepted;
  j.union_R = union_R;
  j.n_accepted = n_accepted;
  j.o = o;
  j.pos = a.pos;
  j.qpos = a.qpos;
  j.S = a.S;
  j.n_vis_slices = joint_vis_slices(a.S);
  j.test_cap = pages->n_pages > 0 ? max_cand : 0;
  j.geo = a;
  j.lse = lse;
  j.n_pages = pages->n_pages;
  j.cand = cand;
  float *resid, *resA, *Dst, *Ast;
  int *resC, *Cst;
  Plan plan;
  plan.add(&j.onorm, total_rows);
  plan.add(&j.nvis_part, (size_t)a.W * j.n_vis_slices);
  plan.add(&resid, (size_t)max_cand * total_rows * D);
  plan.add(&resA, (size_t)max_cand * total_rows);
  plan.add(&resC, (size_t)max_cand * total_rows);
  plan.add(&Dst, 2 * (size_t)total_rows * D);
  plan.add(&Ast, 2 * (size_t)total_rows);
  plan.add(&Cst, 2 * (size_t)total_rows);
  plan.add(&j.ctrl, 8);
  plan.add(&j.rbuf, kJointWindow);
  plan.add(&j.bmax, (size_t)kTargetBlocks * kJointWindow);
  plan.add(&j.in_acc, std::max(pages->n_pages, 1));
  plan.add(&j.fix_list, 2 * (size_t)kJointWindow * total_rows);
  plan.add(&j.fpart, (size_t)ckv::kJointFixItems * (D + 1));
  const int32_t *dstart = nullptr, *dlen = nullptr;
  if ((rc = page_table(c, pages, &dstart, &dlen))) return rc;
  if ((rc = realize(c, plan))) return rc;
  j.pstart = dstart;
  j.plen = dlen;
  j.resid = resid;
  j.resA = resA;
  j.resC = resC;
  j.Dstate = Dst;
  j.Astate = Ast;
  j.Cstate = Cst;

  // Nothing here reads the candidate count on the host: the kernels read
  // *n_cand and size their work from it (max_cand bounds the launches).
  // The residual pass also clears the joint kernel's control words.
  if (pages->n_pages > 0) {
    PageWork pw{};
    pw.start = dstart;
    pw.len = dlen;
    pw.n_items = max_cand;
    pw.n_pages = pages->n_pages;
    pw.items_per_block = items_per_block(std::min(max_cand, pages->n_pages),
                                         a.Hkv * ceil_div(a.rows, rows_per_block_page()));
    pw.cand = cand;
    pw.n_cand = n_cand;
    pw.Hq = a.Hq;
    pw.resid = resid;
    pw.resA = resA;
    pw.resC = resC;
    pw.total_rows = total_rows;
    pw.lse_scale = kLog2eHost;
    pw.clear = j.ctrl;
    pw.n_clear = 8;
    CKV_LAUNCH(c, "joint_residual", launch_page_kernel(a, pw, rs, 1, max_page_len(pages), c->stream));
  }
  // with no pages the joint kernel only writes the outputs
  CKV_LAUNCH(c, "joint_round", launch_joint_persistent(j, kTargetBlocks, c->stream));
  return CKV_OK;
}

extern "C" int ckv_pool_scores(ckv_ctx* c, const float* score, float* out, int32_t n_seq, int64_t seq_stride,
                               const int32_t* n_tokens, int32_t kernel, int32_t mode) {
  CKV_RANGE("ckv_pool_scores");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  if (n_seq < 0 || (n_seq > 0 && (!score || !out || !n_tokens)))
    return fail(c, CKV_ERR_ARG, "pool: NULL pointer or negative n_seq");
  if (kernel < 1 || kernel > 255 || kernel % 2 == 0) return fail(c, CKV_ERR_ARG, "pool: kernel must be odd, 1..255");
  if (mode != CKV_POOL_MAX && mode != CKV_POOL_MEAN) return fail(c, CKV_ERR_ARG, "pool: unknown mode %d", mode);
  int max_tokens = 0;
  for (int s = 0; s < n_seq; ++s) {
    if (n_tokens[s] < 0 || n_tokens[s] > seq_stride)
      return fail(c, CKV_ERR_SHAPE, "pool: n_tokens[%d] = %d outside [0, %lld]", s, n_tokens[s], (long long)seq_stride);
    max_tokens = std::max(max_tokens, (int)n_tokens[s]);
  }
  if (n_seq == 0 || max_tokens == 0) return CKV_OK;
  // the output may not overlap the input (each thread reads its neighbours)
  const char *a0 = reinterpret_cast<const char*>(score), *b0 = reinterpret_cast<const char*>(out);
  const int64_t bytes = ((int64_t)(n_seq - 1) * seq_stride + max_tokens) * 4;
  if (a0 < b0 + bytes && b0 < a0 + bytes) return fail(c, CKV_ERR_ARG, "pool: out overlaps score");
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);
  const int32_t* dn = nullptr;
  int rc = cached_copy(c, std::vector<int32_t>(n_tokens, n_tokens + n_seq), &dn);
  if (rc) return rc;
  CKV_LAUNCH(c, "pool", launch_pool(score, out, seq_stride, dn, n_seq, max_tokens, kernel, mode, c->stream));
  return CKV_OK;
}

extern "C" int ckv_select_and_compact(ckv_ctx* c, const ckv_cache_view* in, const int32_t* n_tokens,
                                      const float* score, int64_t score_seq_stride,
                                      const ckv_page_list* retired, const ckv_page_list* pending,
                                      const float* const* pending_r_pre,
                                      const ckv_accepted_pages* accepted, const ckv_budget* budget,
                                      const ckv_cache_view* out, int32_t* kept_idx, int32_t* n_kept,
                                      uint8_t* token_state) {
  CKV_RANGE("ckv_select_and_compact");
  if (!c) return CKV_ERR_ARG;
  begin_call(c);
  if (int rc0 = latched_nonfinite(c)) return rc0;
  if (!in || !n_tokens || !score || !retired || !pending || !budget || !kept_idx || !n_kept)
    return fail(c, CKV_ERR_ARG, "NULL argument");
  if (in->n_seq < 1 || in->capacity < 1) return fail(c, CKV_ERR_SHAPE, "empty cache shape");
  if (out) {
    if (!in->k || !in->v || !in->pos || !out->k || !out->v || !out->pos)
      return fail(c, CKV_ERR_ARG, "NULL cache pointer");
    if (in->n_layers < 1 || in->n_kv_heads < 1) return fail(c, CKV_ERR_SHAPE, "empty cache shape");
    if (in->head_dim != 64 && in->head_dim != 128)
      return fail(c, CKV_ERR_SHAPE, "head_dim %d unsupported", in->head_dim);
    if (out->n_seq != in->n_seq || out->n_layers != in->n_layers || out->n_kv_heads != in->n_kv_heads ||
        out->head_dim != in->head_dim)
      return fail(c, CKV_ERR_SHAPE, "input and output caches differ in shape");
    const ckv_cache_view* vv[2] = {in, out};
    for (const ckv_cache_view* v : vv) {
      if (!aligned16(v->k) || !aligned16(v->v) || v->tok_stride % 8 || v->head_stride % 8 || v->layer_stride % 8 ||
          v->seq_stride % 8)
        return fail(c, CKV_ERR_ARG, "cache rows must be 16-byte aligned (strides multiples of 8)");
      if (v->tok_stride < v->head_dim || v->capacity < 1) return fail(c, CKV_ERR_SHAPE, "cache strides or capacity");
    }
  }
  const int B = budget->budget;
  if (B < 1 || !(budget->eta >= 0.f && budget->eta <= 1.f) || budget->max_pending_pages < 0 || budget->keep_recent < 0)
    return fail(c, CKV_ERR_ARG, "invalid budget parameters");
  const int bn = (int)std::floor((double)budget->eta * (double)B);
  if ((int64_t)budget->keep_recent + bn > B)
    return fail(c, CKV_ERR_BUDGET, "keep_recent (%d) + B_N (%d) exceeds the budget %d", budget->keep_recent, bn, B);
  if (out && out->capacity < B) return fail(c, CKV_ERR_SHAPE, "output capacity %d < budget %d", out->capacity, B);
  const int ns = in->n_seq;
  for (int s = 0; s < ns; ++s) {
    if (n_tokens[s] < 1 || n_tokens[s] > in->capacity || n_tokens[s] > score_seq_stride)
      return fail(c, CKV_ERR_SHAPE, "sequence %d: n_tokens %d out of range", s, n_tokens[s]);
    int rc;
    if ((rc = check_pages(c, &retired[s], n_tokens[s], "retired")) ||
        (rc = check_pages(c, &pending[s], n_tokens[s], "pending")))
      return rc;
    if (pending[s].n_pages > 0 && (!pending_r_pre || !pending_r_pre[s]))
      return fail(c, CKV_ERR_ARG, "sequence %d: pending R_pre is NULL", s);
    if (accepted && accepted[s].cand) {
      if (!accepted[s].pages || !accepted[s].n_cand || !accepted[s].accepted || accepted[s].max_cand < 1)
        return fail(c, CKV_ERR_ARG, "sequence %d: incomplete accepted-page arguments", s);
      if ((rc = check_pages(c, accepted[s].pages, n_tokens[s], "accepted")) != 0) return rc;
    }
  }
  // the output must not overlap the input (bytes of K, V and positions)
  if (out) {
  auto extent = [](const ckv_cache_view* v) {
    return ((int64_t)(v->n_seq - 1) * v->seq_stride + (int64_t)(v->n_layers - 1) * v->layer_stride +
            (int64_t)(v->n_kv_heads - 1) * v->head_stride + (int64_t)(v->capacity - 1) * v->tok_stride +
            v->head_dim) * 2;
  };
  auto overlap = [](const void* a, int64_t na, const void* b, int64_t nb) {
    const char* x = static_cast<const char*>(a);
    const char* y = static_cast<const char*>(b);
    return x < y + nb && y < x + na;
  };
  const int64_t ei = extent(in), eo = extent(out);
  const int64_t pi = ((int64_t)(ns - 1) * in->pos_seq_stride + in->capacity) * 4;
  const int64_t po = ((int64_t)(ns - 1) * out->pos_seq_stride + out->capacity) * 4;
  const void* ins[3] = {in->k, in->v, in->pos};
  const int64_t inb[3] = {ei, ei, pi};
  const void* outs[3] = {out->k, out->v, out->pos};
  const int64_t outb[3] = {eo, eo, po};
  for (int x = 0; x < 3; ++x)
    for (int y = 0; y < 3; ++y)
      if (overlap(ins[x], inb[x], outs[y], outb[y])) return fail(c, CKV_ERR_ARG, "output cache overlaps the input");
  if (overlap(out->k, eo, out->v, eo)) return fail(c, CKV_ERR_ARG, "output K and V overlap");
  }
  DeviceGuard g(c->device);
  if (!g.ok) return fail(c, CKV_ERR_HIP, "cannot select device %d", c->device);

  // Sec. 4.4 variants: without transition protection no pending page is
  // protected; without the lifecycle mechanism nothing is retired either
  std::vector<ckv_page_list> no_pages(ns, ckv_page_list{nullptr, nullptr, 0});
  if (c->policy & (CKV_POLICY_NO_PROTECTION | CKV_POLICY_NO_LIFECYCLE)) pending = no_pages.data();
  if (c->policy & CKV_POLICY_NO_LIFECYCLE) {
    retired = no_pages.data();
    accepted = nullptr;
  }

  // accepted pages of this commit: device page tables (cached by content)
  std::vector<AccPages> acc(ns);
  bool any_acc = false;
  for (int s = 0; s < ns && accepted; ++s) {
    if (!accepted[s].cand) continue;
    AccPages& e = acc[s];
    int rc2 = page_table(c, accepted[s].pages, &e.start, &e.len);
    if (rc2) return rc2;
    e.cand = accepted[s].cand;
    e.n_cand = accepted[s].n_cand;
    e.accepted = accepted[s].accepted;
    e.max_cand = accepted[s].max_cand;
    e.n_pages = accepted[s].pages->n_pages;
    if (e.n_pages > 0) any_acc = true;
    else e.cand = nullptr;
  }

  // pack every host-side list into one blob: [accepted][pend_r ptrs][n_tokens][ret_off][pend_off][ret start,len][pend start,len]
  int tot_r = 0, tot_p = 0;
  for (int s = 0; s < ns; ++s) {
    tot_r += retired[s].n_pages;
    tot_p += pending[s].n_pages;
  }
  std::vector<uint64_t> blob64(ns);
  for (int s = 0; s < ns; ++s)
    blob64[s] = pending[s].n_pages > 0 ? reinterpret_cast<uint64_t>(pending_r_pre[s]) : 0;
  std::vector<int32_t> blob32;
  blob32.reserve(ns + 2 * (ns + 1) + 2 * (tot_r + tot_p));
  blob32.insert(blob32.end(), n_tokens, n_tokens + ns);
  int run = 0;
  for (int s = 0; s <= ns; ++s) { blob32.push_back(run); if (s < ns) run += retired[s].n_pages; }
  run = 0;
  for (int s = 0; s <= ns; ++s) { blob32.push_back(run); if (s < ns) run += pending[s].n_pages; }
  for (int s = 0; s < ns; ++s) blob32.insert(blob32.end(), retired[s].start, retired[s].start + retired[s].n_pages);
  for (int s = 0; s < ns; ++s) blob32.insert(blob32.end(), retired[s].len, retired[s].len + retired[s].n_pages);
  for (int s = 0; s < ns; ++s) blob32.insert(blob32.end(), pending[s].start, pending[s].start + pending[s].n_pages);
  for (int s = 0; s < ns; ++s) blob32.insert(blob32.end(), pending[s].len, pending[s].len + pending[s].n_pages);
  const size_t acc_bytes = any_acc ? acc.size() * sizeof(AccPages) : 0;
  std::vector<char> blob(acc_bytes + blob64.size() * 8 + blob32.size() * 4);
  if (acc_bytes) std::memcpy(blob.data(), acc.data(), acc_bytes);
  std::memcpy(blob.data() + acc_bytes, blob64.data(), blob64.size() * 8);
  std::memcpy(blob.data() + acc_bytes + blob64.size() * 8, blob32.data(), blob32.size() * 4);

  SelectArgs sa{};
  Plan plan;
  plan.add(&sa.pend_prot, std::max(tot_p, 1));
  plan.add(&sa.pend_ord, std::max(tot_p, 1));
  int max_s = 0;
  for (int s = 0; s < ns; ++s) max_s = std::max(max_s, n_tokens[s]);
  sa.n_chunks = (max_s + ckv::kSelChunk - 1) / ckv::kSelChunk;
  plan.add(&sa.kv, (size_t)ns * score_seq_stride);
  plan.add(&sa.ctrl, (size_t)ns * ckv::kSelCtrl);
  plan.add(&sa.hist, (size_t)ns * 3 * ckv::kSelBins);
  plan.add(&sa.wcnt, (size_t)ns * sa.n_chunks * 2);
  int rc = realize(c, plan);
  if (rc) return rc;
  // the argument blob, as 32-bit words, through the content cache (a step
  // that repeats the same lists uploads nothing)
  std::vector<int32_t> words((blob.size() + 3) / 4, 0);
  std::memcpy(words.data(), blob.data(), blob.size());
  const int32_t* dwords = nullptr;
  if ((rc = cached_copy(c, std::move(words), &dwords))) return rc;
  const char* dblob = reinterpret_cast<const char*>(dwords);
  const int32_t* d32 = reinterpret_cast<const int32_t*>(dblob + acc_bytes + blob64.size() * 8);
  sa.n_seq = ns;
  sa.acc = acc_bytes ? reinterpret_cast<const AccPages*>(dblob) : nullptr;
  sa.pend_r = reinterpret_cast<const uint64_t*>(dblob + acc_bytes);
  sa.n_tokens = d32;
  sa.ret_off = d32 + ns;
  sa.pend_off = d32 + ns + (ns + 1);
  sa.ret_start = d32 + ns + 2 * (ns + 1);
  sa.ret_len = sa.ret_start + tot_r;
  sa.pend_start = sa.ret_len + tot_r;
  sa.pend_len = sa.pend_start + tot_p;
  sa.score = score;
  sa.score_seq_stride = score_seq_stride;
  sa.budget = B;
  sa.bn = bn;
  sa.max_pages = budget->max_pending_pages;
  sa.keep_recent = budget->keep_recent;
  sa.state = token_state;
  sa.kept = kept_idx;
  sa.n_kept = n_kept;
  sa.barrier_ticks = c->barrier_ticks;
  int max_pend = 0;
  for (int s = 0; s < ns; ++s) max_pend = std::max(max_pend, pending[s].n_pages);
  if (c->sel_resident < 0) c->sel_resident = select_grid_resident();
  if (select_grid_fits(max_s, max_pend, ns, c->sel_resident)) {
    if (c->sel_seq < ns) {
      // grow the persistent state; it must start zeroed (the kernel keeps it so)
      CKV_HIP(c, hipStreamSynchronize(c->stream));
      if (c->sel_ctrl) (void)hipFree(c->sel_ctrl);
      if (c->sel_hist) (void)hipFree(c->sel_hist);
      c->sel_ctrl = nullptr;
      c->sel_hist = nullptr;
      c->sel_seq = 0;
      const size_t cb = (size_t)ns * ckv::kSelGridCtrl * sizeof(int32_t);
      const size_t hb = (size_t)ns * 3 * ckv::kSelBins * sizeof(uint32_t);
      void *pc = nullptr, *ph = nullptr;
      if (hipMalloc(&pc, cb) != hipSuccess || hipMalloc(&ph, hb) != hipSuccess) {
        (void)hipGetLastError();
        if (pc) (void)hipFree(pc);
        return fail(c, CKV_ERR_NOMEM, "selection state of %zu bytes failed", cb + hb);
      }
      CKV_HIP(c, hipMemset(pc, 0, cb));
      CKV_HIP(c, hipMemset(ph, 0, hb));
      CKV_HIP(c, hipDeviceSynchronize());
      c->sel_ctrl = static_cast<int32_t*>(pc);
      c->sel_hist = static_cast<uint32_t*>(ph);
      c->sel_seq = ns;
    }
    sa.gctrl = c->sel_ctrl;
    sa.ghist = c->sel_hist;
    CKV_LAUNCH(c, "select", launch_select_grid(sa, max_s, c->stream));
  } else {
    CKV_LAUNCH(c, "protect", launch_protect(sa, c->stream));
    CKV_LAUNCH(c, "select", launch_select(sa, c->stream));
  }

  if (!out) return CKV_OK;   // selection only: the caller applies I (e.g. to a paged block table)
  GatherArgs ga{};
  ga.k_in = in->k;
  ga.v_in = in->v;
  ga.in_seq = in->seq_stride;
  ga.in_layer = in->layer_stride;
  ga.in_head = in->head_stride;
  ga.in_tok = in->tok_stride;
  ga.k_out = out->k;
  ga.v_out = out->v;
  ga.out_seq = out->seq_stride;
  ga.out_layer = out->layer_stride;
  ga.out_head = out->head_stride;
  ga.out_tok = out->tok_stride;
  ga.pos_in = in->pos;
  ga.pos_in_seq = in->pos_seq_stride;
  ga.pos_out = out->pos;
  ga.pos_out_seq = out->pos_seq_stride;
  ga.n_seq = ns;
  ga.n_layers = in->n_layers;
  ga.Hkv = in->n_kv_heads;
  ga.D = in->head_dim;
  ga.kept = kept_idx;
  ga.n_kept = n_kept;
  ga.budget = B;
  ga.in_rows = in->capacity;
  ga.dbg = c->dbg_dev;
  CKV_LAUNCH(c, "gather", launch_gather(ga, c->stream));
  return CKV_OK;
}
