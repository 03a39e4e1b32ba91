/*
 * commitkv_agent.h -- multi-commit lifecycle driver of CommitKV (Algorithm 1)
 * on top of the calls of commitkv.h.
 *
 * One agent holds the lifecycle state of ONE agent episode (one sequence)
 * across its turns (CommitKV, Sec. 3.1-3.3, Algorithm 1; operating point of
 * Sec. 4.1):
 *   - the resident cache, in one of two caller-owned cache buffers (a
 *     compression checkpoint compacts the current buffer into the other);
 *   - the events seen so far and their pages (tool calls and observations,
 *     cut into pages of at most G tokens from the event's first token,
 *     Sec. 3.1);
 *   - the pending commit: the pages measured before the last commit with
 *     their pre-commit effects R^-, until its post-commit window arrives;
 *   - the retirement set D_c (Sec. 3.3).
 *
 * The caller (the serving engine) writes every token's keys, values and
 * position into the current buffer, then reports it with ckv_agent_append;
 * it calls ckv_agent_commit when a tool call ends (window Q^- = the call's
 * last W tokens), ckv_agent_post once the first W reasoning tokens after the
 * observation exist (window Q^+), and ckv_agent_checkpoint after every
 * checkpoint_every decoded tokens (Sec. 4.1: 128); ckv_agent_append reports
 * when the last two are due.
 *
 * Driver rules (where the paper leaves the driver open):
 *   - E_c at a commit: the pages whose tokens are all resident and that are
 *     not in D_c; at most max_scan_pages of them, those of largest start
 *     position (Sec. 4.1: 64 pages per commit).
 *   - The post measurement covers the pending pages that are still fully
 *     resident; percentiles rank among them; their R^- is the stored value.
 *     Accepted candidates join D_c (Algorithm 1).
 *   - A checkpoint scores tokens with the token mass of its window on the
 *     scoring layer (pooled when pool_kernel > 1; one index set for every
 *     layer, Eq. (4)), protects the
 *     fully resident pending pages (Eq. (12)), excludes every resident token
 *     of D_c, and keeps at most B tokens (Eq. (13)).  With at most B resident
 *     tokens and no resident retired token it changes nothing.  A page of D_c
 *     with no resident token left leaves D_c.
 *   - The context's policy switches (ckv_set_policy, Sec. 4.4) apply to the
 *     calls the agent makes.
 *
 * Synchronisation: commit, post and checkpoint wait for the context's stream
 * before they return (the host needs R^-, the accepted pages and the kept
 * indices to update its state); append enqueues nothing.
 * Ownership: the agent owns its host state, a few device buffers (sized at
 * creation from max_scan_pages, the window and the cache capacity) and a
 * pinned staging area; the caller owns both cache buffers and every window
 * view.  One agent per sequence; an agent is used from one host thread.
 */
#ifndef COMMITKV_AGENT_H
#define COMMITKV_AGENT_H

#include "commitkv.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ckv_agent ckv_agent;

/* Event kinds of a ReAct trajectory (Sec. 3.1, Eq. (1)).  Tool calls and
 * observations are cut into pages; the other kinds are not. */
typedef enum ckv_event_kind {
  CKV_EVENT_REASONING = 0,
  CKV_EVENT_TOOL_CALL = 1,
  CKV_EVENT_OBSERVATION = 2,
  CKV_EVENT_PROMPT = 3,
  CKV_EVENT_ANSWER = 4
} ckv_event_kind;

typedef struct ckv_agent_config {
  int32_t page_size;         /* G: 1 .. CKV_MAX_PAGE_LEN */
  int32_t window;            /* W: rows of every window view passed in */
  int32_t n_q_heads;         /* query heads of every window view */
  int32_t max_scan_pages;    /* pages measured per commit: 1 .. 4096 */
  int32_t checkpoint_every;  /* decoded tokens between checkpoints: >= 1 */
  int32_t score_layer;       /* layer whose attention scores pages and tokens */
  int32_t report_detail;     /* 1: copy R^+, states, union effects and scores
                                to the host report as well */
  ckv_thresholds thresholds; /* Eq. (9), (11) */
  ckv_budget budget;         /* Eq. (12)-(13) */
  int32_t pool_kernel;       /* 0 or 1: the token mass is the base score; odd
                                k > 1: the token mass pooled over k tokens
                                (ckv_pool_scores) */
  int32_t pool_mode;         /* CKV_POOL_MAX or CKV_POOL_MEAN */
} ckv_agent_config;

/* Create an agent over two cache buffers of one sequence (n_seq == 1, the
 * same layers, heads, width and capacity, not overlapping; capacity >=
 * budget).  The cache starts empty in buffer 0.  Errors: CKV_ERR_ARG for
 * NULL or inconsistent arguments, CKV_ERR_SHAPE for geometry, CKV_ERR_NOMEM,
 * CKV_ERR_HIP. */
int ckv_agent_create(ckv_ctx* ctx, const ckv_cache_view* buf0, const ckv_cache_view* buf1,
                     const ckv_agent_config* cfg, ckv_agent** out);

/* Create an agent over a paged cache (vLLM-style block pool; CommitKV's
 * Eq. (4) index set then moves no key or value).  pool: the scoring layer's
 * pool, with k, v, n_kv_heads, head_dim, head_stride, tok_stride and
 * pool_rows set (pos, n_tokens and slot are ignored); the caller owns the
 * pool of every layer and writes each token's keys and values into the row
 * it reports with ckv_agent_append_rows.  capacity: the most tokens the
 * sequence holds at once (budget <= capacity <= pool_rows).  The agent keeps
 * the slot table (pool row of every resident token, in position order) and
 * the positions on the device, double-buffered; a checkpoint selects I_j
 * (Eq. (12)-(13)) and gathers both tables through I_j, and the rows of the
 * tokens it drops are returned by ckv_agent_rows(which = 1).  cfg's
 * score_layer is not used (the pool is the scoring layer's; it must be
 * >= 0).  Errors as ckv_agent_create, and CKV_ERR_UNSUPPORTED for a pool
 * whose pool_rows * tok_stride reaches 2^31 elements (the limit of
 * ckv_kv_view). */
int ckv_agent_create_paged(ckv_ctx* ctx, const ckv_kv_view* pool, int32_t capacity,
                           const ckv_agent_config* cfg, ckv_agent** out);

/* Free the agent's buffers (after waiting for the context's stream). */
int ckv_agent_destroy(ckv_agent* agent);

/* Due flags returned by ckv_agent_append. */
#define CKV_DUE_POST 1        /* the post-commit window of the pending commit is complete */
#define CKV_DUE_CHECKPOINT 2  /* checkpoint_every more decoded tokens since the last one */

/* Report n tokens that the caller has written at slots
 * [n_resident, n_resident + n) of the current buffer: keys and values of
 * every layer and their positions.  pos: HOST int32[n], the same positions,
 * strictly increasing past the last resident one and consecutive inside an
 * event.  kind: a ckv_event_kind; begins_event != 0 starts a new event (a
 * change of kind always does).  decoded != 0 counts the tokens towards the
 * checkpoint period.  *due (may be NULL) receives the CKV_DUE_* flags.
 * Errors: CKV_ERR_SHAPE if the buffer's capacity would be exceeded,
 * CKV_ERR_ARG for bad positions or kind. */
int ckv_agent_append(ckv_agent* agent, int32_t kind, const int32_t* pos, int32_t n,
                     int32_t decoded, int32_t begins_event, int32_t* due);

/* The paged form of ckv_agent_append: rows: HOST int32[n], the pool rows
 * holding the n tokens (in [0, pool_rows); the caller allocates them and
 * must not reuse a row before a checkpoint frees it).  The slot table and
 * positions are copied to the device on the context's stream.  Errors as
 * ckv_agent_append, and CKV_ERR_ARG for a row outside the pool or an agent
 * created with ckv_agent_create. */
int ckv_agent_append_rows(ckv_agent* agent, int32_t kind, const int32_t* pos, const int32_t* rows,
                          int32_t n, int32_t decoded, int32_t begins_event, int32_t* due);

/* Commit at the end of a tool call (Algorithm 1): E_c is formed and R^- is
 * measured over the window q_pre (Eq. (5)-(8)); the pages become pending. */
int ckv_agent_commit(ckv_agent* agent, const ckv_window_view* q_pre);

/* Post-commit step of the pending commit (Algorithm 1): R^+ over q_post,
 * classification (Eq. (9)-(10)), the greedy joint test (Eq. (11)); accepted
 * pages join D_c.  Without a pending commit it does nothing. */
int ckv_agent_post(ckv_agent* agent, const ckv_window_view* q_post);

/* Compression checkpoint (Eq. (12)-(13), Eq. (4)) with the base score from
 * the window q_score.  *compacted (may be NULL) is 1 if the cache moved to
 * the other buffer. */
int ckv_agent_checkpoint(ckv_agent* agent, const ckv_window_view* q_score, int32_t* compacted);

/* Resident token count, the buffer (0 or 1) holding the cache, and the
 * decoded-token counter. */
int ckv_agent_state(const ckv_agent* agent, int32_t* n_resident, int32_t* current,
                    int64_t* decoded);

/* Outcome of the last commit, post or checkpoint.  Every pointer is a HOST
 * array owned by the agent, valid until its next call.  Pages are given by
 * absolute position (first position, token count). */
typedef struct ckv_agent_report {
  int32_t op;                /* 0 none, 1 commit, 2 post, 3 checkpoint */
  int32_t n_pages;           /* commit: |E_c|; post: pending pages measured */
  const int32_t* page_start;
  const int32_t* page_len;
  const float* r_pre;        /* [n_pages] */
  const float* r_post;       /* post, report_detail: [n_pages] */
  const uint8_t* lambda;     /* post, report_detail: [n_pages] */
  int32_t n_cand;            /* post: candidates, in test order */
  const int32_t* cand;       /* post: [n_cand] indices into the page list */
  const uint8_t* accepted;   /* post: [n_cand] */
  const float* union_r;      /* post, report_detail: [n_cand] */
  int32_t n_accepted;
  int32_t compacted;         /* checkpoint */
  int32_t n_before;          /* checkpoint: resident tokens before it */
  int32_t n_kept;            /* checkpoint: |I_j| when compacted */
  const int32_t* kept;       /* checkpoint: I_j, indices before compaction */
  const float* score;        /* checkpoint, report_detail: [n_before] */
} ckv_agent_report;
int ckv_agent_last_report(const ckv_agent* agent, ckv_agent_report* out);

/* Host copies of the agent's page lists, by absolute position:
 * which = 0: the pending pages (value = R^-); which = 1: D_c (value = 0).
 * At most cap entries are written; *n receives the list's length. */
int ckv_agent_pages(const ckv_agent* agent, int32_t which, int32_t* start, int32_t* len,
                    float* value, int32_t cap, int32_t* n);

/* Host copies of per-token lists: which = 0, the pool rows of the resident
 * tokens in position order, and which = 1, the rows the last checkpoint
 * released (empty if it compacted nothing), both for paged agents only
 * (CKV_ERR_ARG otherwise); which = 2, the positions of the resident tokens
 * (any agent).  At most cap entries are written; *n receives the list's
 * length. */
int ckv_agent_rows(const ckv_agent* agent, int32_t which, int32_t* rows, int32_t cap, int32_t* n);

#ifdef __cplusplus
}
#endif

#endif /* COMMITKV_AGENT_H */
