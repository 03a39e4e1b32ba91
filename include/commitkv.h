/*
 * commitkv.h -- C ABI of the CommitKV hot path on MI355X (gfx950).
 *
 * The calls follow the paper's statement of the method (CommitKV,
 * "Lifecycle-Aware KV Cache Compression via Commit Transitions for Multi-Turn
 * Agents", Sec. 3):
 *
 *   ckv_measure_page_effects  Sec. 3.2, Eq. (5)-(8): window deletion effect
 *                             R(E;Q) of every event page, for one window.
 *   ckv_measure_recorded      the same from the window outputs the engine
 *                             recorded (per-page pass only).
 *   ckv_classify_pages        Sec. 3.2, Eq. (8)-(10): percentile ranks, high/low
 *                             indicators, lifecycle states; Sec. 3.3: ordered
 *                             completion candidates.
 *   ckv_joint_test            Sec. 3.3, Eq. (11), Algorithm 1: greedy joint
 *                             retirement test on the post-commit window.
 *   ckv_select_and_compact    Sec. 3.3, Eq. (12)-(13): pending protection and
 *                             the retained index set under budget B;
 *                             Sec. 3.1, Eq. (4): the same indices applied to
 *                             keys, values and absolute positions.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Tensor pointers are DEVICE pointers unless a field says "host".  The
 *    caller owns every tensor buffer; the library never frees or keeps them.
 *    Inputs are never written.
 *  - bf16 tensors are passed as uint16_t bit patterns.  The innermost (head
 *    width) axis is contiguous; other axes use element strides.  Key, value
 *    and query rows must start on 16-byte boundaries (base pointer 16-byte
 *    aligned, strides multiples of 8 elements).
 *  - Every call enqueues work on the context's HIP stream and returns without
 *    waiting.  Argument errors are detected on the host and returned at once
 *    (nothing is enqueued then).  Outputs are valid once the stream reaches
 *    the call's work (ckv_sync, or stream/event synchronisation).
 *  - Counts produced on the device (n_cand, n_accepted, n_kept) stay on the
 *    device so that calls can be chained without host round trips.
 *  - Errors found on the device: a NaN or infinite value that reaches a
 *    window row's output or log-sum-exp (non-finite keys, values or queries,
 *    or non-finite recorded outputs) latches a flag the context keeps in
 *    pinned host memory.  ckv_sync returns CKV_ERR_NONFINITE after the wait,
 *    and so does the first call that starts after the detecting kernel has
 *    finished (that call then enqueues nothing); either clears the flag.
 *    The outputs of the call whose inputs were non-finite are not valid.
 *  - Return value: CKV_OK (0) or a negative ckv_status.  No C++ exception
 *    crosses the ABI.  ckv_last_error() gives a message for the last failure
 *    on the context.
 *  - Thread safety: one context per host thread.  Calls on one context
 *    serialise on its stream.
 */
#ifndef COMMITKV_H
#define COMMITKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CKV_VERSION_MAJOR 0
#define CKV_VERSION_MINOR 1
#define CKV_VERSION_PATCH 0

/* Largest page length accepted (tokens).  Sec. 3.1: pages have |E| <= G. */
#define CKV_MAX_PAGE_LEN 64

typedef enum ckv_status {
  CKV_OK = 0,
  CKV_ERR_ARG = -1,         /* NULL pointer, misalignment, aliasing, bad scalar */
  CKV_ERR_SHAPE = -2,       /* head counts/width, page list, window size */
  CKV_ERR_BUDGET = -3,      /* protected tokens could exceed the budget B */
  CKV_ERR_UNSUPPORTED = -4, /* valid request outside what this build handles */
  CKV_ERR_NOMEM = -5,       /* workspace allocation failed or exceeds the limit */
  CKV_ERR_HIP = -6,         /* a HIP runtime call failed */
  CKV_ERR_NONFINITE = -7,   /* non-finite input detected on the device (latched) */
  CKV_ERR_DEVICE_CHECK = -8 /* a device bounds check failed (builds with device checks only; latched) */
} ckv_status;

/* Lifecycle states, Sec. 3.2 Eq. (10). */
typedef enum ckv_lifecycle {
  CKV_UNCERTAIN = 0,
  CKV_CANDIDATE = 1,     /* H^- and L^+ : high-to-low completion candidate */
  CKV_DORMANT = 2,       /* L^- and L^+ */
  CKV_NEWLY_ACTIVE = 3,  /* L^- and H^+ */
  CKV_STILL_ACTIVE = 4   /* H^- and H^+ */
} ckv_lifecycle;

/* Token states at a compression checkpoint (Sec. 3.3, Eq. (13)). */
typedef enum ckv_token_state {
  CKV_TOKEN_FREE = 0,
  CKV_TOKEN_PROTECTED = 1, /* in N_j (or among the keep_recent last tokens) */
  CKV_TOKEN_RETIRED = 2    /* in a page of the retirement set D_c */
} ckv_token_state;

typedef struct ckv_ctx ckv_ctx;

/* ---------------------------------------------------------------- context */

/* Create a context on HIP device `device`, enqueuing on `hip_stream`
 * (a hipStream_t; NULL = the device's null stream).  The context owns a
 * device workspace that grows on demand and is freed by ckv_destroy. */
int ckv_create(ckv_ctx** out, int device, void* hip_stream);

/* Wait for the context's stream, then free the context and its workspace. */
int ckv_destroy(ckv_ctx* ctx);

/* Switch the stream.  Work already enqueued on the old stream is waited for
 * first, so buffers the library owns are never shared by two streams. */
int ckv_set_stream(ckv_ctx* ctx, void* hip_stream);

/* Block until the context's stream is idle. */
int ckv_sync(ckv_ctx* ctx);

/* Message of the last failed call on `ctx` (empty string if none). */
const char* ckv_last_error(const ckv_ctx* ctx);

/* (major << 16) | (minor << 8) | patch */
uint32_t ckv_version(void);

/* Build switches of this library.  CKV_BUILD_DEVICE_CHECKS: compiled with
 * device bounds checks (-DCKV_DEBUG; libcommitkv_debug.so).  In such a build
 * a kernel index outside its buffer is clamped into it and the check's site
 * number latched in the context's pinned debug word; the next call on the
 * context (or ckv_sync, after its wait) returns CKV_ERR_DEVICE_CHECK, names
 * the site in ckv_last_error, and clears the word.  The sites cover the key
 * and value rows of staged tiles, split partials, window-row outputs, page
 * effects, residuals, fix-up entries, joint-test candidates and the
 * compaction's kept indices.  Release builds return 0 and check nothing. */
#define CKV_BUILD_DEVICE_CHECKS 1u
uint32_t ckv_build_flags(void);

/* Cap the workspace (bytes; 0 = no cap).  Calls that would need more fail
 * with CKV_ERR_NOMEM before enqueuing anything. */
int ckv_set_workspace_limit(ckv_ctx* ctx, size_t bytes);

/* Bytes of device workspace currently held by the context. */
size_t ckv_workspace_bytes(const ckv_ctx* ctx);

/* Kernel timing.  While enabled, every kernel the library launches is
 * bracketed by a pair of HIP events recorded on the context's stream, and
 * the elapsed times are summed per kernel name.  ckv_kernel_stats waits for
 * the recorded events, then reports kernel number idx (0-based, in order of
 * first launch): its name (owned by the context), total milliseconds and
 * launch count; idx past the last kernel returns CKV_ERR_ARG.
 * ckv_reset_kernel_stats zeroes the totals. */
int ckv_set_kernel_timing(ckv_ctx* ctx, int enable);
/* Restrict the timing to the kernel called `name` (as reported by
 * ckv_kernel_stats); NULL or "" times every kernel again.  Each timed launch
 * adds two event records to the stream, so a benchmark that times only its
 * dominant kernel perturbs the rest of the step least. */
int ckv_set_kernel_timing_only(ckv_ctx* ctx, const char* name);
int ckv_kernel_stats(ckv_ctx* ctx, int32_t idx, const char** name,
                     double* total_ms, int64_t* launches);
int ckv_reset_kernel_stats(ckv_ctx* ctx);

/* ------------------------------------------------------------------ views */

/* Resident KV cache of ONE layer of ONE sequence (Sec. 3.1, Eq. (3)):
 * key (g, t, e) is k[g*head_stride + row(t)*tok_stride + e] for KV head
 * g < n_kv_heads, token t < n_tokens, width e < head_dim; same for v.
 * row(t) = t for a contiguous cache.  For a paged pool (a block table with
 * one token per entry, as serving engines keep it) slot is a device
 * int32[n_tokens] and row(t) = slot[t], a row of the pool's pool_rows rows
 * (values outside [0, pool_rows) are clamped to the last row: wrong but in
 * bounds).  pos[t] is the token's absolute position p_t (Sec. 3.1), used for
 * causal visibility p_t <= p; it is indexed by token, not by row. */
typedef struct ckv_kv_view {
  const uint16_t* k;
  const uint16_t* v;
  int64_t head_stride;   /* elements */
  int64_t tok_stride;    /* elements */
  const int32_t* pos;    /* device int32[n_tokens] */
  int32_t n_tokens;      /* S >= 1 */
  int32_t n_kv_heads;    /* H_kv >= 1 */
  int32_t head_dim;      /* d: 64 or 128 */
  const int32_t* slot;   /* device int32[n_tokens], or NULL: contiguous */
  int32_t pool_rows;     /* rows of the pool when slot is given */
} ckv_kv_view;

/* Query window Q (Sec. 3.1, Eq. (5)): post-RoPE queries of the W window
 * positions for every query head.  Query (h, p, e) is
 * q[h*head_stride + p*row_stride + e]; qpos[p] is the absolute position of
 * window row p.  Query head h reads KV head h / (n_q_heads / n_kv_heads). */
typedef struct ckv_window_view {
  const uint16_t* q;
  int64_t head_stride;   /* elements */
  int64_t row_stride;    /* elements */
  const int32_t* qpos;   /* device int32[n_rows] */
  int32_t n_q_heads;     /* H_q, a multiple of n_kv_heads */
  int32_t n_rows;        /* W >= 1 */
  float scale;           /* softmax scale; <= 0 selects 1/sqrt(head_dim) */
} ckv_window_view;

/* Event pages (Sec. 3.1): page i covers tokens [start[i], start[i]+len[i]).
 * HOST arrays.  Requirements (else CKV_ERR_SHAPE): 1 <= len <= CKV_MAX_PAGE_LEN,
 * sorted by start, pairwise disjoint, inside [0, n_tokens).  Because pages are
 * sorted, "start ascending" and "page index ascending" are the same order. */
typedef struct ckv_page_list {
  const int32_t* start;
  const int32_t* len;
  int32_t n_pages;       /* >= 0 */
} ckv_page_list;

/* Thresholds of Eq. (9) and Eq. (11).  Paper defaults (Sec. 4.1):
 * tau_use 0.05, tau_dead 0.01, rho_use 0.75, rho_dead 0.25, tau_joint 0.01. */
typedef struct ckv_thresholds {
  float tau_use, tau_dead, rho_use, rho_dead, tau_joint;
} ckv_thresholds;

/* Budget of Eq. (12)-(13).  B_N = floor(eta * budget).  Paper: eta 0.125, at
 * most 16 protected pending pages (Sec. 4.1).  keep_recent protects the last
 * keep_recent resident tokens (counts against budget, not against B_N). */
typedef struct ckv_budget {
  int32_t budget;            /* B >= 1 */
  float eta;                 /* in [0, 1] */
  int32_t max_pending_pages; /* >= 0 */
  int32_t keep_recent;       /* >= 0 */
} ckv_budget;

/* Caches of several sequences and layers (Sec. 3.1, Eq. (3)-(4)):
 * key (s, l, g, t, e) is k[s*seq_stride + l*layer_stride + g*head_stride +
 * t*tok_stride + e]; same for v.  pos[s*pos_seq_stride + t]. */
typedef struct ckv_cache_view {
  uint16_t* k;
  uint16_t* v;
  int64_t seq_stride, layer_stride, head_stride, tok_stride;  /* elements */
  int32_t* pos;
  int64_t pos_seq_stride;
  int32_t n_seq, n_layers, n_kv_heads, head_dim;
  int32_t capacity;          /* token slots per (seq, layer, head) */
} ckv_cache_view;

/* Component switches of the method, for the ablation variants of Sec. 4.4
 * (Table 3).  A context-wide bit set, 0 (the default) being the complete
 * method; it applies to the calls enqueued after it is set.
 *   CKV_POLICY_NO_PRECOMMIT   ckv_classify_pages: every page with L+ is a
 *                             retirement candidate, whatever its pre-commit
 *                             state (instead of H- and L+ of Eq. (10))
 *   CKV_POLICY_NO_PERCENTILE  ckv_classify_pages: H and L of Eq. (9) from the
 *                             absolute thresholds tau_use / tau_dead alone
 *   CKV_POLICY_NO_JOINT       ckv_joint_test: every candidate is accepted
 *                             (no Eq. (11) gate); union_R still reports
 *                             R+(A u {E})
 *   CKV_POLICY_NO_PROTECTION  ckv_select_and_compact: no pending page is
 *                             protected (N_j empty)
 *   CKV_POLICY_NO_LIFECYCLE   no lifecycle operation: ckv_classify_pages
 *                             writes no candidate (n_cand = 0), and
 *                             ckv_select_and_compact retires nothing and
 *                             protects no pending page
 * Returns CKV_ERR_ARG for a NULL context or an unknown bit. */
typedef enum ckv_policy_flag {
  CKV_POLICY_NO_PRECOMMIT = 1,
  CKV_POLICY_NO_PERCENTILE = 2,
  CKV_POLICY_NO_JOINT = 4,
  CKV_POLICY_NO_PROTECTION = 8,
  CKV_POLICY_NO_LIFECYCLE = 16
} ckv_policy_flag;
int ckv_set_policy(ckv_ctx* ctx, uint32_t flags);
/* The context's current switches (0 for a NULL context). */
uint32_t ckv_get_policy(const ckv_ctx* ctx);

/*
 * Bound of one grid-wide wait (microseconds of the device wall clock) in the
 * one-launch kernels of ckv_joint_test (Algorithm 1's sequential rounds) and
 * of the grid selection in ckv_select_and_compact.  Their workgroups
 * synchronise through counters in device memory, which needs every
 * workgroup resident at once; on a device shared with other work that may
 * not hold, and a wait that passes the bound makes every workgroup of the
 * call leave, with *n_accepted = -1 or n_kept[s] = -1 as the result (the
 * outputs are then not valid; the lifecycle driver turns it into
 * CKV_ERR_UNSUPPORTED).  Default 1342177 us (about 1.3 s).  0 makes every
 * wait give up at once, which forces the failure path (for tests of the
 * caller's handling).  Returns
 * CKV_ERR_ARG for a negative or absurd value.
 */
int ckv_set_barrier_timeout_us(ckv_ctx* ctx, int64_t us);

/* ------------------------------------------------------------- the calls */

/*
 * Window deletion effect of every page (Sec. 3.2, Eq. (6)-(7)); called once
 * with the pre-commit window Q^- and once with the post-commit window Q^+
 * (Eq. (8)).
 *
 * For query head h and window row p: a_pi = softmax over visible tokens
 * (pos[i] <= qpos[p]) of scale * q_hp . k_i; o_p = sum_i a_pi v_i.  For page E:
 * A = sum_{i in E, visible} a_pi, u = sum_{i in E, visible} a_pi v_i and, by
 * Eq. (6), ||o_p - o_p^{\E}|| = ||u - A o_p|| / (1 - A).
 *   R_head[E, h] = max_p ||o_p - o_p^{\E}|| / ||o_p||   (0 if no row sees E;
 *                  +inf if a row sees only tokens of E)
 *   R[E]         = max_h R_head[E, h]
 *
 * Outputs (device, float32, written in full):
 *   R          [n_pages]                    required
 *   R_head     [n_pages * n_q_heads]        optional (NULL)
 *   o          [n_q_heads * n_rows * head_dim]  optional: window outputs o_p
 *   lse        [n_q_heads * n_rows]         optional: log-sum-exp of the
 *              scaled logits of each row (-inf for a row that sees nothing)
 *   token_mass [n_tokens]                   optional: max_h sum_p a_hpi, the
 *              window-attention mass of each token (a base score for
 *              ckv_select_and_compact)
 * Precision: bf16 inputs, float32 logits and accumulation, float16
 * attention weights and values inside the weighted sums (values must lie
 * within the float16 range).
 */
int ckv_measure_page_effects(ckv_ctx* ctx, const ckv_kv_view* kv,
                             const ckv_window_view* win,
                             const ckv_page_list* pages, float* R,
                             float* R_head, float* o, float* lse,
                             float* token_mass);

/*
 * ckv_measure_page_effects for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments, outputs and errors, but the call allocates
 * nothing -- no hipMalloc/hipFree, no pinned upload buffers, no events.  Its
 * working memory (split partial sums, row statistics, fix-up lists and the
 * page table, copied from the host arrays with hipMemcpyAsync) lives in one
 * static device array of 64 MiB that the library holds on every GPU it runs
 * on until the process ends.  When the split partials of the regular call
 * would not fit, the window pass uses fewer, longer token splits (results
 * then differ from the regular call's only by float32 summation order); a
 * shape whose working memory exceeds 64 MiB even with one split fails with
 * CKV_ERR_UNSUPPORTED before anything is enqueued.  Kernel timing is not
 * recorded for this call.
 *
 * Every call on one GPU shares that GPU's array, and the array keeps the
 * last call's contents (each call clears what it needs zeroed): two such
 * calls whose work overlaps on one GPU (two contexts on two streams without
 * ordering between them) race and give undefined results.
 */
int ckv_measure_page_effects_noalloc(ckv_ctx* ctx, const ckv_kv_view* kv,
                                     const ckv_window_view* win,
                                     const ckv_page_list* pages, float* R,
                                     float* R_head, float* o, float* lse,
                                     float* token_mass);

/*
 * Batched form of ckv_measure_page_effects for many (layer, sequence)
 * problems, such as every layer of every sequence in a batch: problem i
 * reads kv[i], win[i], pages[i] (arrays of n views) and writes R[i],
 * R_head[i], o[i], lse[i], token_mass[i] (host arrays of n device pointers;
 * an optional array may be NULL as a whole or hold NULL entries).  Every
 * problem is validated before anything is enqueued; the problems then run
 * in order on the context's stream, reusing one workspace.  A workspace or
 * HIP failure part-way returns the error with the earlier problems enqueued.
 */
int ckv_measure_page_effects_batch(ckv_ctx* ctx, int32_t n,
                                   const ckv_kv_view* kv,
                                   const ckv_window_view* win,
                                   const ckv_page_list* pages,
                                   float* const* R, float* const* R_head,
                                   float* const* o, float* const* lse,
                                   float* const* token_mass);

/*
 * Recorded-output variant of ckv_measure_page_effects (Sec. 3.2: the engine
 * records the window's attention outputs during its forward pass).  o
 * [n_q_heads * n_rows * head_dim] (16-byte aligned) and lse [n_q_heads *
 * n_rows] (natural log; -inf for a row that sees no token) are INPUTS: the
 * outputs and log-sum-exp of the window rows over this cache, as
 * ckv_measure_page_effects would return them.  Only the per-page pass (and
 * the token mass) runs; R, R_head and token_mass are as there.
 * Pages carrying between 0.5 and 0.99 of a row's mass are evaluated from
 * their own tokens in float32, with 1 - A taken against the recorded
 * log-sum-exp, so the rounding of lse and of the page's logits bounds their
 * relative error by a few ulp(lse)/(1 - A); above 0.99 the row's output
 * without the page is recomputed from all of its other tokens (every such
 * (page, row) pair, however many rows have one).
 */
int ckv_measure_recorded(ckv_ctx* ctx, const ckv_kv_view* kv,
                         const ckv_window_view* win,
                         const ckv_page_list* pages, const float* o,
                         const float* lse, float* R, float* R_head,
                         float* token_mass);

/*
 * Lifecycle classification of the n pages of E_c (Sec. 3.2, Eq. (8)-(10)).
 * R_pre, R_post: device float32[n] (outputs of the two measurements over the
 * same page list).  Percentile rank: P(E) = #{E' != E : R(E') < R(E)}/(n - 1),
 * 0.5 when n == 1.  Eq. (9) with inclusive comparisons as printed.
 *
 * Candidates (lambda == CKV_CANDIDATE, or force_candidate[i] != 0 when that
 * optional device uint8[n] mask is given) are written to cand in the order of
 * Sec. 3.3: R_post ascending, then R_pre descending, then page index
 * ascending; at most max_cand (<= 0: no cap) are written and *n_cand (device)
 * receives their count.
 *
 * Outputs (device): lambda uint8[n]; P_pre, P_post float32[n] (optional);
 * cand int32[n] (entries past *n_cand are -1); n_cand int32[1].
 */
int ckv_classify_pages(ckv_ctx* ctx, int32_t n, const float* R_pre,
                       const float* R_post, const ckv_thresholds* th,
                       const uint8_t* force_candidate, int32_t max_cand,
                       uint8_t* lambda, float* P_pre, float* P_post,
                       int32_t* cand, int32_t* n_cand);

/*
 * Greedy joint retirement test (Sec. 3.3, Eq. (11), Algorithm 1) on the
 * post-commit window.  Starting from A = {}, candidate cand[t] (t = 0, 1, ...
 * < min(*n_cand, max_cand)) is accepted iff R^+(A u {E}) <= tau_joint, where
 * R^+ of a page set deletes all of its tokens at once (Eq. (6)-(7) on the
 * union).  kv, win and pages must be those of the post-commit measurement;
 * o and lse are that measurement's outputs.  cand and n_cand are device
 * arrays (e.g. from ckv_classify_pages) indexing `pages`.
 *
 * Outputs (device): accepted uint8[max_cand] (1 = accepted); union_R
 * float32[max_cand] (optional): R^+(A u {E}) evaluated at step t;
 * n_accepted int32[1].  Entries at t >= *n_cand are 0 / NaN.
 * max_cand must be >= 1.
 * Like the other calls it only enqueues work: the kernels read *n_cand on
 * the device, and the sequential greedy loop runs as speculative rounds
 * inside one launch of at most as many workgroups as the device holds at
 * once, separated by grid barriers (each round decides at least one
 * candidate, so at most min(*n_cand, max_cand) rounds run).  A barrier wait
 * is bounded (about 1.3 s): if the workgroups cannot all run at once (the
 * device is shared with other work), every workgroup leaves and
 * *n_accepted is set to -1 (accepted and union_R are then incomplete).
 */
int ckv_joint_test(ckv_ctx* ctx, const ckv_kv_view* kv,
                   const ckv_window_view* win, const float* o,
                   const float* lse, const ckv_page_list* pages,
                   const int32_t* cand, const int32_t* n_cand,
                   int32_t max_cand, float tau_joint, uint8_t* accepted,
                   float* union_R, int32_t* n_accepted);

/*
 * Pooled base score, the SnapKV-style variant of the score that fills the
 * budget (the window mass smoothed over neighbouring tokens, so the tokens
 * around a heavily attended one are kept with it).  For sequence s and token
 * t < n_tokens[s]: out[s*seq_stride + t] = the max (CKV_POOL_MAX; NaN
 * entries are ignored, NaN only if the whole window is) or the mean
 * (CKV_POOL_MEAN, float32 sum in index order divided by the count) of
 * score[s*seq_stride + j] over the tokens j in [t - kernel/2, t + kernel/2]
 * inside [0, n_tokens[s]).
 * score, out: device float32[n_seq * seq_stride], not overlapping; n_tokens:
 * HOST int32[n_seq], each <= seq_stride; kernel odd in [1, 255].
 * Entries past n_tokens[s] are not written.
 */
#define CKV_POOL_MAX 0
#define CKV_POOL_MEAN 1
int ckv_pool_scores(ckv_ctx* ctx, const float* score, float* out, int32_t n_seq,
                    int64_t seq_stride, const int32_t* n_tokens, int32_t kernel,
                    int32_t mode);

/* Pages retired by the joint test of the current commit, resolved on the
 * device so that the checkpoint needs no host round trip (Algorithm 1: the
 * accepted set joins the retired set before the budget is applied).  Page
 * pages->start[cand[i]] .. + len[cand[i]] is retired when
 * i < min(*n_cand, max_cand) and accepted[i] != 0.  `pages` is a host page
 * list (the one given to ckv_joint_test); cand, n_cand and accepted are
 * device arrays as produced by ckv_classify_pages and ckv_joint_test. */
typedef struct ckv_accepted_pages {
  const ckv_page_list* pages;
  const int32_t* cand;       /* device int32[max_cand] */
  const int32_t* n_cand;     /* device int32[1] */
  const uint8_t* accepted;   /* device uint8[max_cand] */
  int32_t max_cand;
} ckv_accepted_pages;

/*
 * Compression checkpoint (Sec. 3.3, Eq. (12)-(13); Sec. 3.1, Eq. (4)) for
 * in->n_seq sequences.  For sequence s:
 *   1. Pending protection: pending[s] pages ordered by pending_r_pre[s]
 *      (device float32[pending[s].n_pages]) descending, then start
 *      ascending, are protected while fewer than max_pending_pages are taken
 *      and their token total stays <= B_N = floor(eta * B); the first page
 *      that does not fit ends the protection.
 *   2. Token state: retired (in a page of retired[s], or of accepted[s]
 *      when `accepted` is not NULL) > protected (protected page, or among
 *      the last keep_recent of n_tokens[s] tokens) > free.
 *   3. Retained set I: every protected token plus the
 *      min(B - #protected, #free) free tokens of highest score (float32
 *      score[s*score_seq_stride + t]; ties to the lower index; NaN ranks as
 *      -inf, -0.0 as +0.0), in ascending token order.
 *   4. Compaction: out key/value (s, l, g, j) = in (s, l, g, I[j]) for every
 *      layer and KV head, out pos[j] = in pos[I[j]]; bytes copied verbatim.
 *      Slots j >= |I| of `out` are left untouched.
 * Device inputs: score float32[n_seq * score_seq_stride] (whole rows may be
 * read; entries past n_tokens[s] are ignored).
 * Host arguments: n_tokens int32[n_seq]; retired, pending ckv_page_list[n_seq];
 * pending_r_pre: host array of n_seq device pointers (NULL allowed where
 * pending[s].n_pages == 0); accepted: ckv_accepted_pages[n_seq] or NULL
 * (an entry with cand == NULL adds nothing).  Device outputs: kept_idx int32[n_seq * B]
 * (row s holds I, entries past n_kept[s] are -1), n_kept int32[n_seq],
 * token_state uint8[n_seq * score_seq_stride] (optional).
 * `out` may be NULL: then only steps 1-3 run (kept_idx, n_kept, token_state)
 * and no byte is copied; only in->n_seq and in->capacity are read.  A
 * caller whose cache is a paged pool (ckv_kv_view.slot) applies I to its
 * block table instead, which moves no key or value.
 * Errors: CKV_ERR_BUDGET if keep_recent + B_N > B; CKV_ERR_ARG if `out`
 * overlaps `in`; CKV_ERR_SHAPE if out->capacity < B or shapes differ.
 */
int ckv_select_and_compact(ckv_ctx* ctx, const ckv_cache_view* in,
                           const int32_t* n_tokens, const float* score,
                           int64_t score_seq_stride,
                           const ckv_page_list* retired,
                           const ckv_page_list* pending,
                           const float* const* pending_r_pre,
                           const ckv_accepted_pages* accepted,
                           const ckv_budget* budget, const ckv_cache_view* out,
                           int32_t* kept_idx, int32_t* n_kept,
                           uint8_t* token_state);

#ifdef __cplusplus
}
#endif

#endif /* COMMITKV_H */
