// Multi-commit lifecycle driver of CommitKV (Algorithm 1) behind
// include/commitkv_agent.h.  Host bookkeeping only: every measurement,
// classification, joint test and compaction is one of the calls of
// commitkv.h, on the context's stream.  The host keeps the resident
// positions, so pages (identified by absolute position) are mapped to
// resident index ranges without reading the device.
#include "commitkv_agent.h"
#include "ckv_host.h"
#include "ckv_trace.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

using ckv::ctx_fail;

namespace {

struct Page {
  int32_t start, len;          // first absolute position, token count
  bool operator==(const Page& o) const { return start == o.start && len == o.len; }
  bool operator<(const Page& o) const { return start < o.start || (start == o.start && len < o.len); }
};

struct Event {
  int32_t kind, start, n;      // positions start .. start + n - 1
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct DevGuard {
  int prev = -1;
  bool ok = true;
  explicit DevGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DevGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

bool pageable(int32_t kind) { return kind == CKV_EVENT_TOOL_CALL || kind == CKV_EVENT_OBSERVATION; }

}  // namespace

// paged agents: the slot table and the positions follow a checkpoint's
// index set, rows[j] = rows_in[I[j]], pos[j] = pos_in[I[j]]
__global__ void gather_rows_kernel(const int32_t* rows_in, const int32_t* pos_in, const int32_t* kept, int n,
                                   int32_t* rows_out, int32_t* pos_out) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n) {
    const int i = kept[j];
    rows_out[j] = rows_in[i];
    pos_out[j] = pos_in[i];
  }
}

struct ckv_agent {
  ckv_ctx* ctx = nullptr;
  ckv_cache_view buf[2];
  ckv_agent_config cfg;
  int cur = 0;
  int capacity = 0;                  // token slots
  bool paged = false;
  ckv_kv_view pool{};                // paged: the scoring layer's pool
  int32_t *d_rows[2] = {nullptr, nullptr}, *d_pos[2] = {nullptr, nullptr};   // paged, by resident index
  int32_t *up_pos = nullptr, *up_rows = nullptr;   // paged: pinned staging, by resident index
  std::vector<int32_t> rows;         // paged: pool row of each resident token
  std::vector<int32_t> freed;        // paged: rows released by the last checkpoint
  std::vector<int32_t> res;          // resident positions, ascending
  std::vector<Event> events;
  bool events_ordered = true;   // every event starts after the previous one ends
  int64_t decoded = 0;
  bool pending = false;
  size_t commit_events = 0;          // events seen when the pending commit was made
  std::vector<Page> pend;
  std::vector<float> pend_r;
  std::vector<Page> retired;         // D_c, sorted by start

  // device buffers (one allocation)
  char* dev = nullptr;
  float *d_r_pre = nullptr, *d_r_sub = nullptr, *d_r_post = nullptr, *d_union = nullptr;
  float *d_o = nullptr, *d_lse = nullptr, *d_score = nullptr, *d_pooled = nullptr;
  uint8_t *d_lambda = nullptr, *d_acc = nullptr;
  int32_t *d_cand = nullptr, *d_ncand = nullptr, *d_nacc = nullptr, *d_kept = nullptr, *d_nkept = nullptr;
  // pinned staging: uploads, then downloads
  char* pin = nullptr;
  float* up_r = nullptr;
  int32_t* dn_counts = nullptr;      // n_cand, n_accepted, n_kept
  int32_t* dn_cand = nullptr;
  uint8_t* dn_acc = nullptr;
  uint8_t* dn_lambda = nullptr;
  float *dn_r = nullptr, *dn_r_post = nullptr, *dn_union = nullptr, *dn_score = nullptr;
  int32_t* dn_kept = nullptr;

  // last report
  int32_t rep_op = 0, rep_ncand = 0, rep_nacc = 0, rep_compacted = 0, rep_before = 0, rep_nkept = 0;
  std::vector<int32_t> rep_start, rep_len, rep_cand, rep_kept;
  std::vector<float> rep_rpre, rep_rpost, rep_union, rep_score;
  std::vector<uint8_t> rep_lambda, rep_acc;

  int n_res() const { return (int)res.size(); }
  int max_pages() const { return cfg.max_scan_pages; }

  // resident index range of a page's positions
  void span(const Page& p, int* i0, int* i1) const {
    *i0 = (int)(std::lower_bound(res.begin(), res.end(), p.start) - res.begin());
    *i1 = (int)(std::lower_bound(res.begin(), res.end(), p.start + p.len) - res.begin());
  }
  bool resident(const Page& p) const {
    int a, b;
    span(p, &a, &b);
    return b - a == p.len;
  }

  ckv_kv_view layer_view() const {
    if (paged) {
      ckv_kv_view kv = pool;
      kv.pos = d_pos[cur];
      kv.n_tokens = n_res();
      kv.slot = d_rows[cur];
      return kv;
    }
    const ckv_cache_view& b = buf[cur];
    ckv_kv_view kv;
    kv.k = b.k + (int64_t)cfg.score_layer * b.layer_stride;
    kv.v = b.v + (int64_t)cfg.score_layer * b.layer_stride;
    kv.head_stride = b.head_stride;
    kv.tok_stride = b.tok_stride;
    kv.pos = b.pos;
    kv.n_tokens = n_res();
    kv.n_kv_heads = b.n_kv_heads;
    kv.head_dim = b.head_dim;
    kv.slot = nullptr;
    kv.pool_rows = 0;
    return kv;
  }

  // E_c: pages of tool calls and observations, fully resident, not in D_c,
  // the max_scan_pages of largest start
  std::vector<Page> eligible() const {
    CKV_RANGE("eligible pages");
    const size_t cap = (size_t)max_pages();
    std::vector<Page> out;
    if (events_ordered) {
      // Events hold disjoint, increasing positions, so their pages come in
      // increasing order and one forward walk over res (ascending, without
      // repeats) and retired (sorted) settles every page: a page is wholly
      // resident iff its first and last positions sit len - 1 entries apart.
      size_t ir = 0, it = 0;
      for (const Event& e : events) {
        if (!pageable(e.kind) || e.n <= 0) continue;
        ir = std::lower_bound(res.begin() + ir, res.end(), e.start) - res.begin();
        if (ir == res.size()) break;
        if (res[ir] >= e.start + e.n) continue;
        for (int off = (res[ir] - e.start) / cfg.page_size * cfg.page_size; off < e.n; off += cfg.page_size) {
          const Page p{e.start + off, std::min(cfg.page_size, e.n - off)};
          if (ir < res.size() && res[ir] < p.start)
            ir = std::lower_bound(res.begin() + ir, res.end(), p.start) - res.begin();
          if (res.size() - ir < (size_t)p.len) break;
          if (res[ir] != p.start || res[ir + p.len - 1] != p.start + p.len - 1) continue;
          ir += p.len;   // the next page, if resident, starts right here
          while (it < retired.size() && retired[it] < p) ++it;
          if (it < retired.size() && retired[it] == p) continue;
          out.push_back(p);
        }
      }
    } else {
      for (const Event& e : events) {
        if (!pageable(e.kind)) continue;
        for (int off = 0; off < e.n; off += cfg.page_size) {
          const Page p{e.start + off, std::min(cfg.page_size, e.n - off)};
          if (std::binary_search(retired.begin(), retired.end(), p)) continue;
          if (resident(p)) out.push_back(p);
        }
      }
      std::sort(out.begin(), out.end());
    }
    // the newest max_pages() pages are scored
    if (out.size() > cap) out.erase(out.begin(), out.end() - cap);
    return out;
  }

  void ranges(const std::vector<Page>& pages, std::vector<int32_t>* st, std::vector<int32_t>* ln) const {
    CKV_RANGE("page ranges");
    st->clear();
    ln->clear();
    for (const Page& p : pages) {
      int a, b;
      span(p, &a, &b);
      st->push_back(a);
      ln->push_back(b - a);
    }
  }

  int check_window(const ckv_window_view* w, const char* what) {
    if (!w) return ctx_fail(ctx, CKV_ERR_ARG, "%s window view is NULL", what);
    if (w->n_rows != cfg.window || w->n_q_heads != cfg.n_q_heads)
      return ctx_fail(ctx, CKV_ERR_SHAPE, "%s window: %d rows x %d heads, agent expects %d x %d", what,
                      w->n_rows, w->n_q_heads, cfg.window, cfg.n_q_heads);
    return CKV_OK;
  }

  int sync() {
    const hipError_t e = hipStreamSynchronize(ckv::ctx_stream(ctx));
    return e == hipSuccess ? CKV_OK : ctx_fail(ctx, CKV_ERR_HIP, "stream synchronisation: %s", hipGetErrorString(e));
  }

  int copy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind) {
    if (!bytes) return CKV_OK;
    const hipError_t e = hipMemcpyAsync(dst, src, bytes, kind, ckv::ctx_stream(ctx));
    return e == hipSuccess ? CKV_OK : ctx_fail(ctx, CKV_ERR_HIP, "agent copy: %s", hipGetErrorString(e));
  }

  void clear_report(int op) {
    rep_op = op;
    rep_ncand = rep_nacc = rep_compacted = rep_before = rep_nkept = 0;
    rep_start.clear();
    rep_len.clear();
    rep_cand.clear();
    rep_kept.clear();
    rep_rpre.clear();
    rep_rpost.clear();
    rep_union.clear();
    rep_score.clear();
    rep_lambda.clear();
    rep_acc.clear();
  }

  void report_pages(const std::vector<Page>& pages, const std::vector<float>& r) {
    for (const Page& p : pages) {
      rep_start.push_back(p.start);
      rep_len.push_back(p.len);
    }
    rep_rpre = r;
  }
};

namespace {

// configuration checks shared by both forms of the agent
int check_config(ckv_ctx* ctx, const ckv_agent_config* cfg, int n_kv_heads, int n_layers, int capacity) {
  const ckv_budget& bg = cfg->budget;
  if (cfg->page_size < 1 || cfg->page_size > CKV_MAX_PAGE_LEN)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: page_size %d not in [1, %d]", cfg->page_size, CKV_MAX_PAGE_LEN);
  if (cfg->window < 1 || cfg->n_q_heads < 1 || cfg->n_q_heads % n_kv_heads)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: bad window rows or query heads");
  if (cfg->max_scan_pages < 1 || cfg->max_scan_pages > 4096)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: max_scan_pages %d not in [1, 4096]", cfg->max_scan_pages);
  if (cfg->checkpoint_every < 1) return ctx_fail(ctx, CKV_ERR_ARG, "agent: checkpoint_every must be >= 1");
  if (cfg->score_layer < 0 || cfg->score_layer >= n_layers)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: score_layer %d outside [0, %d)", cfg->score_layer, n_layers);
  if (cfg->pool_kernel < 0 || cfg->pool_kernel > 255 || (cfg->pool_kernel > 1 && cfg->pool_kernel % 2 == 0) ||
      (cfg->pool_mode != CKV_POOL_MAX && cfg->pool_mode != CKV_POOL_MEAN))
    return ctx_fail(ctx, CKV_ERR_ARG, "agent: pool_kernel must be 0 or odd <= 255, pool_mode max or mean");
  if (bg.budget < 1 || bg.budget > capacity || !(bg.eta >= 0.f && bg.eta <= 1.f) || bg.keep_recent < 0 ||
      bg.max_pending_pages < 0)
    return ctx_fail(ctx, CKV_ERR_ARG, "agent: bad budget (B must fit the capacity)");
  if ((int64_t)std::floor((double)bg.eta * bg.budget) + bg.keep_recent > bg.budget)
    return ctx_fail(ctx, CKV_ERR_BUDGET, "agent: keep_recent + B_N exceeds B");
  return CKV_OK;
}

// device buffers and pinned staging (one allocation each)
int alloc_agent(ckv_agent* a, int head_dim) {
  ckv_ctx* ctx = a->ctx;
  const ckv_agent_config* cfg = &a->cfg;
  const size_t M = (size_t)cfg->max_scan_pages;
  const size_t rows = (size_t)cfg->n_q_heads * cfg->window;
  const size_t cap = (size_t)a->capacity, B = (size_t)cfg->budget.budget;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align256(std::max<size_t>(bytes, 1)); return o; };
  const size_t o_rpre = take(M * 4), o_rsub = take(M * 4), o_rpost = take(M * 4), o_union = take(M * 4);
  const size_t o_o = take(rows * head_dim * 4), o_lse = take(rows * 4), o_score = take(cap * 4);
  const size_t o_pooled = take(cap * 4);
  const size_t o_lam = take(M), o_acc = take(M), o_cand = take(M * 4), o_cnt = take(16), o_kept = take(B * 4);
  size_t o_tab[4] = {0, 0, 0, 0};
  if (a->paged)
    for (int i = 0; i < 4; ++i) o_tab[i] = take(cap * 4);
  DevGuard g(ckv::ctx_device(ctx));
  if (!g.ok) return ctx_fail(ctx, CKV_ERR_HIP, "agent: cannot select the context's device");
  if (hipMalloc((void**)&a->dev, off) != hipSuccess) {
    (void)hipGetLastError();
    a->dev = nullptr;
    return ctx_fail(ctx, CKV_ERR_NOMEM, "agent: device allocation of %zu bytes failed", off);
  }
  char* d = a->dev;
  a->d_r_pre = (float*)(d + o_rpre);
  a->d_r_sub = (float*)(d + o_rsub);
  a->d_r_post = (float*)(d + o_rpost);
  a->d_union = (float*)(d + o_union);
  a->d_o = (float*)(d + o_o);
  a->d_lse = (float*)(d + o_lse);
  a->d_score = (float*)(d + o_score);
  a->d_pooled = (float*)(d + o_pooled);
  a->d_lambda = (uint8_t*)(d + o_lam);
  a->d_acc = (uint8_t*)(d + o_acc);
  a->d_cand = (int32_t*)(d + o_cand);
  a->d_ncand = (int32_t*)(d + o_cnt);
  a->d_nacc = a->d_ncand + 1;
  a->d_nkept = a->d_ncand + 2;
  a->d_kept = (int32_t*)(d + o_kept);
  if (a->paged) {
    a->d_rows[0] = (int32_t*)(d + o_tab[0]);
    a->d_rows[1] = (int32_t*)(d + o_tab[1]);
    a->d_pos[0] = (int32_t*)(d + o_tab[2]);
    a->d_pos[1] = (int32_t*)(d + o_tab[3]);
  }
  size_t po = 0;
  auto ptake = [&](size_t bytes) { const size_t o = po; po += align256(std::max<size_t>(bytes, 1)); return o; };
  const size_t p_up = ptake(M * 4), p_cnt = ptake(16), p_cand = ptake(M * 4), p_acc = ptake(M), p_lam = ptake(M);
  const size_t p_r = ptake(M * 4), p_rpost = ptake(M * 4), p_union = ptake(M * 4), p_score = ptake(cap * 4);
  const size_t p_kept = ptake(B * 4);
  size_t p_tab[2] = {0, 0};
  if (a->paged) {
    p_tab[0] = ptake(cap * 4);
    p_tab[1] = ptake(cap * 4);
  }
  if (hipHostMalloc((void**)&a->pin, po, hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();
    a->pin = nullptr;
    return ctx_fail(ctx, CKV_ERR_NOMEM, "agent: pinned allocation of %zu bytes failed", po);
  }
  char* p = a->pin;
  a->up_r = (float*)(p + p_up);
  a->dn_counts = (int32_t*)(p + p_cnt);
  a->dn_cand = (int32_t*)(p + p_cand);
  a->dn_acc = (uint8_t*)(p + p_acc);
  a->dn_lambda = (uint8_t*)(p + p_lam);
  a->dn_r = (float*)(p + p_r);
  a->dn_r_post = (float*)(p + p_rpost);
  a->dn_union = (float*)(p + p_union);
  a->dn_score = (float*)(p + p_score);
  a->dn_kept = (int32_t*)(p + p_kept);
  if (a->paged) {
    a->up_pos = (int32_t*)(p + p_tab[0]);
    a->up_rows = (int32_t*)(p + p_tab[1]);
  }
  return CKV_OK;
}

void free_agent(ckv_agent* a) {
  DevGuard g(ckv::ctx_device(a->ctx));
  (void)hipStreamSynchronize(ckv::ctx_stream(a->ctx));
  if (a->dev) (void)hipFree(a->dev);
  if (a->pin) (void)hipHostFree(a->pin);
  delete a;
}

}  // namespace

extern "C" int ckv_agent_create(ckv_ctx* ctx, const ckv_cache_view* b0, const ckv_cache_view* b1,
                                const ckv_agent_config* cfg, ckv_agent** out) {
  CKV_RANGE("ckv_agent_create");
  if (!ctx) return CKV_ERR_ARG;
  if (!b0 || !b1 || !cfg || !out) return ctx_fail(ctx, CKV_ERR_ARG, "agent: NULL argument");
  *out = nullptr;
  for (const ckv_cache_view* b : {b0, b1})
    if (!b->k || !b->v || !b->pos) return ctx_fail(ctx, CKV_ERR_ARG, "agent: cache buffer with a NULL pointer");
  if (b0->n_seq != 1 || b1->n_seq != 1) return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: cache buffers hold one sequence");
  if (b0->n_layers != b1->n_layers || b0->n_kv_heads != b1->n_kv_heads || b0->head_dim != b1->head_dim ||
      b0->capacity != b1->capacity || b0->n_layers < 1)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: the two cache buffers differ in geometry");
  int rc;
  if ((rc = check_config(ctx, cfg, b0->n_kv_heads, b0->n_layers, b0->capacity))) return rc;
  ckv_agent* a = new (std::nothrow) ckv_agent();
  if (!a) return ctx_fail(ctx, CKV_ERR_NOMEM, "agent: host allocation failed");
  a->ctx = ctx;
  a->buf[0] = *b0;
  a->buf[1] = *b1;
  a->cfg = *cfg;
  a->capacity = b0->capacity;
  if ((rc = alloc_agent(a, b0->head_dim))) {
    free_agent(a);
    return rc;
  }
  *out = a;
  return CKV_OK;
}

extern "C" int ckv_agent_create_paged(ckv_ctx* ctx, const ckv_kv_view* pool, int32_t capacity,
                                      const ckv_agent_config* cfg, ckv_agent** out) {
  CKV_RANGE("ckv_agent_create_paged");
  if (!ctx) return CKV_ERR_ARG;
  if (!pool || !cfg || !out) return ctx_fail(ctx, CKV_ERR_ARG, "agent: NULL argument");
  *out = nullptr;
  if (!pool->k || !pool->v) return ctx_fail(ctx, CKV_ERR_ARG, "agent: pool with a NULL pointer");
  if (pool->head_dim != 64 && pool->head_dim != 128)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: head_dim %d unsupported", pool->head_dim);
  if (pool->n_kv_heads < 1 || pool->pool_rows < 1 || pool->tok_stride < pool->head_dim || pool->head_stride < 0)
    return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: bad pool geometry");
  if ((reinterpret_cast<uintptr_t>(pool->k) & 15u) || (reinterpret_cast<uintptr_t>(pool->v) & 15u) ||
      pool->tok_stride % 8 || pool->head_stride % 8)
    return ctx_fail(ctx, CKV_ERR_ARG, "agent: pool rows must be 16-byte aligned");
  if (capacity < 1 || capacity > pool->pool_rows) return ctx_fail(ctx, CKV_ERR_SHAPE, "agent: capacity outside [1, pool_rows]");
  // the measurement kernels form row offsets with a 24-bit multiply
  if (pool->tok_stride >= (1 << 24) || pool->pool_rows >= (1 << 24) ||
      (int64_t)pool->pool_rows * pool->tok_stride >= ((int64_t)1 << 31))
    return ctx_fail(ctx, CKV_ERR_UNSUPPORTED, "agent: pool_rows * tok_stride must stay below 2^31 elements");
  int rc;
  if ((rc = check_config(ctx, cfg, pool->n_kv_heads, cfg->score_layer + 1, capacity))) return rc;
  ckv_agent* a = new (std::nothrow) ckv_agent();
  if (!a) return ctx_fail(ctx, CKV_ERR_NOMEM, "agent: host allocation failed");
  a->ctx = ctx;
  a->cfg = *cfg;
  a->capacity = capacity;
  a->paged = true;
  a->pool = *pool;
  a->pool.pos = nullptr;
  a->pool.slot = nullptr;
  a->pool.n_tokens = 0;
  if ((rc = alloc_agent(a, pool->head_dim))) {
    free_agent(a);
    return rc;
  }
  *out = a;
  return CKV_OK;
}

extern "C" int ckv_agent_destroy(ckv_agent* a) {
  CKV_RANGE("ckv_agent_destroy");
  if (!a) return CKV_ERR_ARG;
  free_agent(a);
  return CKV_OK;
}

namespace {

// positions checks and event bookkeeping shared by both appends; rows (paged
// agents) are staged for the device before the host state changes
int record_tokens(ckv_agent* a, int32_t kind, const int32_t* pos, const int32_t* rows, int32_t n, int32_t decoded,
                  int32_t begins_event, int32_t* due) {
  ckv_ctx* c = a->ctx;
  if (kind < CKV_EVENT_REASONING || kind > CKV_EVENT_ANSWER) return ctx_fail(c, CKV_ERR_ARG, "append: unknown event kind %d", kind);
  if (n < 0 || (n > 0 && !pos)) return ctx_fail(c, CKV_ERR_ARG, "append: bad token count or NULL positions");
  if ((int64_t)a->n_res() + n > a->capacity)
    return ctx_fail(c, CKV_ERR_SHAPE, "append: %d resident + %d new tokens exceed the capacity %d", a->n_res(), n,
                    a->capacity);
  const bool fresh = begins_event || a->events.empty() || a->events.back().kind != kind;
  if (n > 0) {
    if (!a->res.empty() && pos[0] <= a->res.back()) return ctx_fail(c, CKV_ERR_ARG, "append: positions must increase");
    for (int i = 1; i < n; ++i)
      if (pos[i] != pos[i - 1] + 1) return ctx_fail(c, CKV_ERR_ARG, "append: positions inside an event must be consecutive");
    if (pos[n - 1] == INT_MAX) return ctx_fail(c, CKV_ERR_ARG, "append: position out of range");
    if (!fresh) {
      const Event& e = a->events.back();
      if (pos[0] != e.start + e.n) return ctx_fail(c, CKV_ERR_ARG, "append: an event's positions must be consecutive");
    }
  }
  if (a->paged && n > 0) {
    if (!rows) return ctx_fail(c, CKV_ERR_ARG, "append: NULL rows");
    for (int i = 0; i < n; ++i)
      if (rows[i] < 0 || rows[i] >= a->pool.pool_rows)
        return ctx_fail(c, CKV_ERR_ARG, "append: row %d outside the pool", rows[i]);
    // staging slots [n_res, n_res + n) are not reused before the next
    // checkpoint, which waits for the stream
    const int r0 = a->n_res();
    std::memcpy(a->up_pos + r0, pos, (size_t)n * 4);
    std::memcpy(a->up_rows + r0, rows, (size_t)n * 4);
    int rc;
    if ((rc = a->copy(a->d_pos[a->cur] + r0, a->up_pos + r0, (size_t)n * 4, hipMemcpyHostToDevice)) ||
        (rc = a->copy(a->d_rows[a->cur] + r0, a->up_rows + r0, (size_t)n * 4, hipMemcpyHostToDevice)))
      return rc;
    a->rows.insert(a->rows.end(), rows, rows + n);
  }
  if (n > 0 || fresh) {
    if (fresh) {
      const int st = n > 0 ? pos[0] : (a->res.empty() ? 0 : a->res.back() + 1);
      if (!a->events.empty() && st < a->events.back().start + a->events.back().n) a->events_ordered = false;
      a->events.push_back(Event{kind, st, 0});
    }
    a->events.back().n += n;
    a->res.insert(a->res.end(), pos, pos + n);
  }
  int flags = 0;
  if (decoded && n > 0) {
    const int64_t before = a->decoded;
    a->decoded += n;
    if (a->decoded / a->cfg.checkpoint_every > before / a->cfg.checkpoint_every) flags |= CKV_DUE_CHECKPOINT;
  }
  if (a->pending && a->events.size() > a->commit_events) {
    const Event& e = a->events.back();
    if (e.kind == CKV_EVENT_REASONING && e.n >= a->cfg.window) flags |= CKV_DUE_POST;
  }
  if (due) *due = flags;
  return CKV_OK;
}

}  // namespace

extern "C" int ckv_agent_append(ckv_agent* a, int32_t kind, const int32_t* pos, int32_t n, int32_t decoded,
                                int32_t begins_event, int32_t* due) {
  CKV_RANGE("ckv_agent_append");
  if (!a) return CKV_ERR_ARG;
  if (a->paged) return ctx_fail(a->ctx, CKV_ERR_ARG, "append: a paged agent takes ckv_agent_append_rows");
  return record_tokens(a, kind, pos, nullptr, n, decoded, begins_event, due);
}

extern "C" int ckv_agent_append_rows(ckv_agent* a, int32_t kind, const int32_t* pos, const int32_t* rows, int32_t n,
                                     int32_t decoded, int32_t begins_event, int32_t* due) {
  CKV_RANGE("ckv_agent_append_rows");
  if (!a) return CKV_ERR_ARG;
  if (!a->paged) return ctx_fail(a->ctx, CKV_ERR_ARG, "append_rows: the agent owns cache buffers (ckv_agent_append)");
  return record_tokens(a, kind, pos, rows, n, decoded, begins_event, due);
}

extern "C" int ckv_agent_commit(ckv_agent* a, const ckv_window_view* q_pre) {
  CKV_RANGE("ckv_agent_commit");
  if (!a) return CKV_ERR_ARG;
  int rc;
  if ((rc = a->check_window(q_pre, "commit"))) return rc;
  a->clear_report(1);
  std::vector<Page> E = a->eligible();
  std::vector<float> r(E.size(), 0.f);
  if (!E.empty()) {
    std::vector<int32_t> st, ln;
    a->ranges(E, &st, &ln);
    const ckv_page_list pl{st.data(), ln.data(), (int32_t)E.size()};
    const ckv_kv_view kv = a->layer_view();
    if ((rc = ckv_measure_page_effects(a->ctx, &kv, q_pre, &pl, a->d_r_pre, nullptr, nullptr, nullptr, nullptr)))
      return rc;
    CKV_RANGE("copy back and sync");
    if ((rc = a->copy(a->dn_r, a->d_r_pre, E.size() * 4, hipMemcpyDeviceToHost)) || (rc = a->sync())) return rc;
    std::memcpy(r.data(), a->dn_r, E.size() * 4);
  }
  a->pending = true;
  a->commit_events = a->events.size();
  a->pend = E;
  a->pend_r = r;
  a->report_pages(E, r);
  return CKV_OK;
}

extern "C" int ckv_agent_post(ckv_agent* a, const ckv_window_view* q_post) {
  CKV_RANGE("ckv_agent_post");
  if (!a) return CKV_ERR_ARG;
  int rc;
  if ((rc = a->check_window(q_post, "post"))) return rc;
  a->clear_report(2);
  if (!a->pending) return CKV_OK;
  std::vector<Page> P;
  std::vector<float> r;
  for (size_t i = 0; i < a->pend.size(); ++i)
    if (a->resident(a->pend[i])) {
      P.push_back(a->pend[i]);
      r.push_back(a->pend_r[i]);
    }
  a->report_pages(P, r);
  const int n = (int)P.size();
  if (n > 0) {
    std::vector<int32_t> st, ln;
    a->ranges(P, &st, &ln);
    const ckv_page_list pl{st.data(), ln.data(), n};
    const ckv_kv_view kv = a->layer_view();
    std::memcpy(a->up_r, r.data(), (size_t)n * 4);
    if ((rc = a->copy(a->d_r_sub, a->up_r, (size_t)n * 4, hipMemcpyHostToDevice))) return rc;
    if ((rc = ckv_measure_page_effects(a->ctx, &kv, q_post, &pl, a->d_r_post, nullptr, a->d_o, a->d_lse, nullptr)))
      return rc;
    if ((rc = ckv_classify_pages(a->ctx, n, a->d_r_sub, a->d_r_post, &a->cfg.thresholds, nullptr, 0, a->d_lambda,
                                 nullptr, nullptr, a->d_cand, a->d_ncand)))
      return rc;
    if ((rc = ckv_joint_test(a->ctx, &kv, q_post, a->d_o, a->d_lse, &pl, a->d_cand, a->d_ncand, n,
                             a->cfg.thresholds.tau_joint, a->d_acc, a->d_union, a->d_nacc)))
      return rc;
    if ((rc = a->copy(a->dn_counts, a->d_ncand, 8, hipMemcpyDeviceToHost)) ||
        (rc = a->copy(a->dn_cand, a->d_cand, (size_t)n * 4, hipMemcpyDeviceToHost)) ||
        (rc = a->copy(a->dn_acc, a->d_acc, (size_t)n, hipMemcpyDeviceToHost)))
      return rc;
    if (a->cfg.report_detail &&
        ((rc = a->copy(a->dn_r_post, a->d_r_post, (size_t)n * 4, hipMemcpyDeviceToHost)) ||
         (rc = a->copy(a->dn_lambda, a->d_lambda, (size_t)n, hipMemcpyDeviceToHost)) ||
         (rc = a->copy(a->dn_union, a->d_union, (size_t)n * 4, hipMemcpyDeviceToHost))))
      return rc;
    if ((rc = a->sync())) return rc;
    const int nc = a->dn_counts[0], na = a->dn_counts[1];
    if (na < 0)
      return ctx_fail(a->ctx, CKV_ERR_UNSUPPORTED,
                      "post: the joint test could not hold its workgroups resident at once (device busy)");
    if (nc < 0 || nc > n) return ctx_fail(a->ctx, CKV_ERR_HIP, "post: candidate count %d out of range", nc);
    a->rep_ncand = nc;
    a->rep_nacc = na;
    a->rep_cand.assign(a->dn_cand, a->dn_cand + nc);
    a->rep_acc.assign(a->dn_acc, a->dn_acc + nc);
    if (a->cfg.report_detail) {
      a->rep_rpost.assign(a->dn_r_post, a->dn_r_post + n);
      a->rep_lambda.assign(a->dn_lambda, a->dn_lambda + n);
      a->rep_union.assign(a->dn_union, a->dn_union + nc);
    }
    for (int i = 0; i < nc; ++i) {
      const int j = a->rep_cand[i];
      if (j < 0 || j >= n) return ctx_fail(a->ctx, CKV_ERR_HIP, "post: candidate index %d out of range", j);
      if (a->rep_acc[i] && !std::binary_search(a->retired.begin(), a->retired.end(), P[j]))
        a->retired.insert(std::upper_bound(a->retired.begin(), a->retired.end(), P[j]), P[j]);
    }
  }
  a->pending = false;
  a->pend.clear();
  a->pend_r.clear();
  return CKV_OK;
}

extern "C" int ckv_agent_checkpoint(ckv_agent* a, const ckv_window_view* q_score, int32_t* compacted) {
  CKV_RANGE("ckv_agent_checkpoint");
  if (!a) return CKV_ERR_ARG;
  int rc;
  if ((rc = a->check_window(q_score, "checkpoint"))) return rc;
  a->clear_report(3);
  if (compacted) *compacted = 0;
  a->freed.clear();
  const int S = a->n_res();
  a->rep_before = S;
  const uint32_t policy = ckv_get_policy(a->ctx);
  // resident parts of the retired pages (sorted, disjoint)
  std::vector<int32_t> rs, rl;
  for (const Page& p : a->retired) {
    int i0, i1;
    a->span(p, &i0, &i1);
    if (i1 > i0) {
      rs.push_back(i0);
      rl.push_back(i1 - i0);
    }
  }
  const bool ret_active = !rs.empty() && !(policy & CKV_POLICY_NO_LIFECYCLE);
  if (S <= a->cfg.budget.budget && !ret_active) return CKV_OK;
  // protectable pending pages
  std::vector<Page> P;
  std::vector<float> r;
  if (a->pending)
    for (size_t i = 0; i < a->pend.size(); ++i)
      if (a->resident(a->pend[i])) {
        P.push_back(a->pend[i]);
        r.push_back(a->pend_r[i]);
      }
  std::vector<int32_t> ps, pl;
  a->ranges(P, &ps, &pl);
  if (!P.empty()) {
    std::memcpy(a->up_r, r.data(), r.size() * 4);
    if ((rc = a->copy(a->d_r_sub, a->up_r, r.size() * 4, hipMemcpyHostToDevice))) return rc;
  }
  const ckv_kv_view kv = a->layer_view();
  const ckv_page_list none{nullptr, nullptr, 0};
  if ((rc = ckv_measure_page_effects(a->ctx, &kv, q_score, &none, nullptr, nullptr, nullptr, nullptr, a->d_score)))
    return rc;
  const float* score = a->d_score;
  if (a->cfg.pool_kernel > 1) {
    const int32_t nt = S;
    if ((rc = ckv_pool_scores(a->ctx, a->d_score, a->d_pooled, 1, a->capacity, &nt, a->cfg.pool_kernel,
                              a->cfg.pool_mode)))
      return rc;
    score = a->d_pooled;
  }
  const ckv_page_list ret_list{rs.data(), rl.data(), (int32_t)rs.size()};
  const ckv_page_list pend_list{ps.data(), pl.data(), (int32_t)ps.size()};
  const float* rptr = P.empty() ? nullptr : a->d_r_sub;
  const int32_t n_tok = S;
  ckv_cache_view index_only{};        // paged: selection only, the slot table follows below
  index_only.n_seq = 1;
  index_only.capacity = a->capacity;
  const ckv_cache_view* in = a->paged ? &index_only : &a->buf[a->cur];
  const ckv_cache_view* out = a->paged ? nullptr : &a->buf[1 - a->cur];
  if ((rc = ckv_select_and_compact(a->ctx, in, &n_tok, score, a->capacity, &ret_list, &pend_list, &rptr, nullptr,
                                   &a->cfg.budget, out, a->d_kept, a->d_nkept, nullptr)))
    return rc;
  const int B = a->cfg.budget.budget;
  if ((rc = a->copy(a->dn_counts + 2, a->d_nkept, 4, hipMemcpyDeviceToHost)) ||
      (rc = a->copy(a->dn_kept, a->d_kept, (size_t)B * 4, hipMemcpyDeviceToHost)))
    return rc;
  if (a->cfg.report_detail && (rc = a->copy(a->dn_score, score, (size_t)S * 4, hipMemcpyDeviceToHost)))
    return rc;
  if ((rc = a->sync())) return rc;
  const int nk = a->dn_counts[2];
  if (nk < 0) return ctx_fail(a->ctx, CKV_ERR_UNSUPPORTED, "checkpoint: the selection could not hold its workgroups resident at once");
  if (nk > B || nk > S) return ctx_fail(a->ctx, CKV_ERR_HIP, "checkpoint: kept count %d out of range", nk);
  std::vector<int32_t> kept(a->dn_kept, a->dn_kept + nk);
  std::vector<int32_t> npos(nk);
  for (int j = 0; j < nk; ++j) {
    if (kept[j] < 0 || kept[j] >= S || (j && kept[j] <= kept[j - 1]))
      return ctx_fail(a->ctx, CKV_ERR_HIP, "checkpoint: kept index list is not ascending inside the cache");
    npos[j] = a->res[kept[j]];
  }
  if (a->paged) {
    // the slot table and positions follow I; rows of the other tokens are free
    if (nk > 0) {
      hipLaunchKernelGGL(gather_rows_kernel, dim3((nk + 255) / 256), dim3(256), 0, ckv::ctx_stream(a->ctx),
                         a->d_rows[a->cur], a->d_pos[a->cur], a->d_kept, nk, a->d_rows[1 - a->cur],
                         a->d_pos[1 - a->cur]);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return ctx_fail(a->ctx, CKV_ERR_HIP, "checkpoint: row gather: %s", hipGetErrorString(e));
    }
    std::vector<uint8_t> keep(S, 0);
    for (int j = 0; j < nk; ++j) keep[kept[j]] = 1;
    std::vector<int32_t> nrows(nk);
    a->freed.clear();
    for (int i = 0, j = 0; i < S; ++i) {
      if (keep[i]) nrows[j++] = a->rows[i];
      else a->freed.push_back(a->rows[i]);
    }
    a->rows.swap(nrows);
  }
  a->res.swap(npos);
  a->cur = 1 - a->cur;
  std::vector<Page> keep_ret;
  for (const Page& p : a->retired) {
    int i0, i1;
    a->span(p, &i0, &i1);
    if (i1 > i0) keep_ret.push_back(p);
  }
  a->retired.swap(keep_ret);
  a->rep_compacted = 1;
  a->rep_nkept = nk;
  a->rep_kept.swap(kept);
  if (a->cfg.report_detail) a->rep_score.assign(a->dn_score, a->dn_score + S);
  if (compacted) *compacted = 1;
  return CKV_OK;
}

extern "C" int ckv_agent_state(const ckv_agent* a, int32_t* n_resident, int32_t* current, int64_t* decoded) {
  if (!a) return CKV_ERR_ARG;
  if (n_resident) *n_resident = a->n_res();
  if (current) *current = a->cur;
  if (decoded) *decoded = a->decoded;
  return CKV_OK;
}

extern "C" int ckv_agent_last_report(const ckv_agent* a, ckv_agent_report* o) {
  if (!a || !o) return CKV_ERR_ARG;
  std::memset(o, 0, sizeof *o);
  o->op = a->rep_op;
  o->n_pages = (int32_t)a->rep_start.size();
  o->page_start = a->rep_start.data();
  o->page_len = a->rep_len.data();
  o->r_pre = a->rep_rpre.data();
  o->r_post = a->rep_rpost.empty() ? nullptr : a->rep_rpost.data();
  o->lambda = a->rep_lambda.empty() ? nullptr : a->rep_lambda.data();
  o->n_cand = a->rep_ncand;
  o->cand = a->rep_cand.data();
  o->accepted = a->rep_acc.data();
  o->union_r = a->rep_union.empty() ? nullptr : a->rep_union.data();
  o->n_accepted = a->rep_nacc;
  o->compacted = a->rep_compacted;
  o->n_before = a->rep_before;
  o->n_kept = a->rep_nkept;
  o->kept = a->rep_kept.data();
  o->score = a->rep_score.empty() ? nullptr : a->rep_score.data();
  return CKV_OK;
}

extern "C" int ckv_agent_pages(const ckv_agent* a, int32_t which, int32_t* start, int32_t* len, float* value,
                               int32_t cap, int32_t* n) {
  if (!a || (which != 0 && which != 1) || cap < 0 || (cap > 0 && (!start || !len))) return CKV_ERR_ARG;
  const std::vector<Page>& L = which == 0 ? a->pend : a->retired;
  const int m = std::min<int>(cap, (int)L.size());
  for (int i = 0; i < m; ++i) {
    start[i] = L[i].start;
    len[i] = L[i].len;
    if (value) value[i] = which == 0 ? a->pend_r[i] : 0.f;
  }
  if (n) *n = (int32_t)L.size();
  return CKV_OK;
}

extern "C" int ckv_agent_rows(const ckv_agent* a, int32_t which, int32_t* rows, int32_t cap, int32_t* n) {
  if (!a || which < 0 || which > 2 || (which < 2 && !a->paged) || cap < 0 || (cap > 0 && !rows)) return CKV_ERR_ARG;
  const std::vector<int32_t>& L = which == 0 ? a->rows : which == 1 ? a->freed : a->res;
  const int m = std::min<int>(cap, (int)L.size());
  if (m > 0) std::memcpy(rows, L.data(), (size_t)m * 4);
  if (n) *n = (int32_t)L.size();
  return CKV_OK;
}
