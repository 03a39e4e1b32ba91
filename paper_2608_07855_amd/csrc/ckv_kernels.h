// Launch interface between the host runtime (api.cpp) and the HIP kernels.
// Plain structs of device pointers and sizes; no torch types anywhere.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ckv {

// one layer of one sequence and one query window
struct AttnGeom {
  const uint16_t* k;
  const uint16_t* v;
  int64_t kv_head_stride, kv_tok_stride;   // elements
  const int32_t* pos;
  int S, Hkv, D;
  const uint16_t* q;
  int64_t q_head_stride, q_row_stride;     // elements
  const int32_t* qpos;
  int Hq, W, group;                        // group = Hq / Hkv
  int rows;                                // window rows per KV head = group * W
  float sl2;                               // softmax scale * log2(e)
  const int32_t* slot;                     // paged pool: token t is row slot[t] of each head
                                           // (clamped to pool_last), or null: row t
  uint32_t pool_last;                      // last row of the pool
  uint32_t* dbg;                           // debug word of the context (CKV_DEBUG builds)
  uint32_t* nonfinite;                     // the context's latched non-finite flag (or null)
};

// split-sequence partials of pass A
struct AttnSplit {
  int chunk, n_splits, rows_pad;
  float* part_o;   // [Hkv][n_splits][rows_pad][D]
  float* part_m;   // [Hkv][n_splits][rows_pad]  (log2 units)
  float* part_l;
  int* part_c;     // visible-token counts
  int* part_t;     // start of the first tile of the split whose largest scaled logit
                   // equals the split's (the tile where the split's weight reference
                   // took its final value); -1 when the split shows the row no token
  float* part_p;   // the split's weight reference before that tile (log2 units; -inf
                   // when the reference grew only once)
};

// per window row (global row h*W + p): o [rows][D], lse2 (log2 units), ||o||, n_vis,
// and m2, the largest scaled logit of the row (log2 units): the reference the
// window pass's float16 weights were finally taken against, with m2t, the
// start of the tile where it entered that reference in the first split that
// holds it, and m2p, that split's reference before that tile (all null when
// the outputs were not computed by this library's window pass)
struct RowStats {
  float* o;
  float* lse2;
  float* onorm;
  int* nvis;
  float* m2;
  int* m2t;
  float* m2p;
};

// pages processed by pass B (MODE 0: item = page; MODE 1: item t = page cand[t])
constexpr int kPageItemsMax = 256;   // pages (or candidates) per page-kernel workgroup
constexpr int kPageRmaxCap = 4096;   // (page, head) maxima a MODE 0 workgroup keeps in LDS

struct PageWork {
  const int32_t* start;
  const int32_t* len;
  int n_items;            // MODE 0: pages; MODE 1: max_cand (capped by *n_cand)
  int n_pages;            // entries of start/len (MODE 1 ignores candidates outside)
  int items_per_block;
  const int32_t* cand;    // MODE 1
  const int32_t* n_cand;  // MODE 1 (device)
  float* R;               // MODE 0: [n_pages], zeroed before
  float* R_head;          // MODE 0: [n_pages][Hq] or null, zeroed before
  int Hq;
  int* fix_list;          // MODE 0: (page, global row, start, len) entries left to the fix-up kernel
  int* fix_count;         // MODE 0: entries in fix_list (zeroed before)
  int fix_cap;            // MODE 0: capacity of fix_list (window rows)
  float* resid;           // MODE 1: [total_rows][n_items][D] (a row's candidates together)
  float* resA;            // MODE 1: [total_rows][n_items]
  int* resC;              // MODE 1: [total_rows][n_items]
  int total_rows;         // Hq * W
  float lse_scale;        // rs.lse2 x lse_scale = log-sum-exp in log2 units (1, or log2 e
                          // when rs.lse2 holds natural-log values)
  int* clear;             // MODE 1: words set to zero by workgroup (0, 0, 0) (or null)
  int n_clear;
  float fix_a;            // MODE 0: pairs with A > fix_a (>= 0.5) go to the fix-up list ...
  float fix_a_hi;         // ... unless A <= fix_a_hi, the page holds its row's largest
                          // logit (rs.m2 set) and the window pass weighted all of it
                          // against that logit: then the closed form is kept
  int split_tokens;       // MODE 0: split length of the window pass (a multiple of 64;
                          // 0: unknown, and no page across a tile boundary keeps the
                          // closed form above fix_a; nor does one without rs.m2)
};

// Fix-up thresholds after this library's window pass.  A page that holds its
// row's largest logit and lies inside one 64-token tile of the window pass,
// or crosses into the next tile of the same split after that logit entered
// the split's reference (by the tile of the page's first part), was weighted
// against the same reference (that logit) in both passes, so
// its float16 weights are the very ones that formed o and Eq. (6) loses only
// the float32 digits of the row's log-sum-exp, amplified by 1/(1 - A): such
// pages keep the closed form up to kFixAHi.  Any other page's weights round
// differently in the two passes (by up to one float16 ulp, 2^-11 relative),
// and the residual u - A o inherits that rounding times A/(1 - A): 2e-3 of
// the effect at A = 0.8 if every token's rounding falls the same way, so
// those go above kFixA.
// A fix-up entry (page, row, start, length) whose length carries this flag
// has A <= kFixAHi after this library's window pass.  If its page lies in
// the first split holding the row's largest logit, from the tile before the
// one where that logit entered the split's reference on, the fix-up
// evaluates Eq. (6) with the window pass's own weights (tokens before that
// tile against the older reference, rescaled) instead of recomputing the
// split.  The length is the low byte.
constexpr int kFixRescaled = 1 << 16;
constexpr float kFixA = 0.8f;
constexpr float kFixAHi = 0.99f;
constexpr float kFixARecorded = 0.5f;   // with recorded window outputs (no shared weights)

struct ZeroList {
  float* p0; size_t n0;
  float* p1; size_t n1;
  float* p2; size_t n2;
  int* i0;               // one int set to zero (or null)
  int* i1; size_t n1i;   // ints set to zero
  uint32_t* nonfinite;   // latched flag (host memory), set when a window row's
                         // output or log-sum-exp is NaN or infinite (or null)
};

// Latch the non-finite flag: a plain system-scope store to the context's
// pinned host word (idempotent, so concurrent setters need no atomics).
__device__ __forceinline__ void latch_nonfinite(uint32_t* flag) {
  if (flag) __hip_atomic_store(flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

int rows_per_block_attention();
int rows_per_block_page();
int page_heads_per_block(int W, int group);   // bound on the query heads of one workgroup
int token_mass_max_rows();

hipError_t launch_window_attention(const AttnGeom& a, const AttnSplit& sp, hipStream_t s);
hipError_t launch_combine(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs, float* lse_out,
                          const ZeroList& zl, hipStream_t s);
hipError_t launch_page_kernel(const AttnGeom& a, const PageWork& pw, const RowStats& rs, int mode,
                              int max_len, hipStream_t s);
hipError_t launch_token_mass(const AttnGeom& a, const RowStats& rs, float* mass, int chunk,
                             hipStream_t s);
// fpart: workspace of [fix_cap][parts][D + 1] floats, or of [item_budget][D + 1]
// when item_budget > 0; each listed pair is spread over `parts` workgroups,
// or, with an item budget, over min(parts, item_budget / pairs) of them (at
// least 1, read from the device count), so every listed pair fits however
// many there are (item_budget >= fix_cap).  arrive: [fix_cap] ints, zero on
// entry: the last part of a pair to finish (counted there) adds the parts up
// and takes the ratio, so one launch does both steps.
constexpr int kFixParts = 8;        // after the window pass: the page's own split(s)
constexpr int kFixPartsRow = 32;    // recorded outputs: every other token of the row
hipError_t launch_page_fixup(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs,
                             const PageWork& pw, float* fpart, int* arrive, int parts, int item_budget,
                             hipStream_t s);

// The same fix-up fused with the token mass of the same pass (one launch):
// kMassFixBlocks blocks of 512 threads serve the listed pairs (grid-stride
// over (pair, part) items), the rest of the grid is launch_token_mass's.
// Applies unless the token mass needs its general kernel (window rows per KV
// head that do not fill whole workgroups); otherwise the launcher refuses.
constexpr int kMassFixBlocks = 256;
bool mass_fixup_applies(const AttnGeom& a);
hipError_t launch_mass_fixup(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs, const PageWork& pw,
                             float* fpart, int* arrive, int parts, float* mass, int chunk, hipStream_t s);

// recorded window outputs: row statistics from the caller's o and natural-log
// lse (nvis_part: workspace [W][recorded_slices(S)] ints, or null to skip the
// visible counts, which then read 0), and the fix-up of
// the listed pairs from the page's own tokens
int recorded_slices(int S);
hipError_t launch_recorded_rows(const AttnGeom& a, const float* o, const float* lse, const RowStats& rs,
                                int* nvis_part, const ZeroList& zl, hipStream_t s);
// pairs with A > a_hi go to list2 (int4 entries, count2 zeroed before, at most cap2)
hipError_t launch_page_fixup_recorded(const AttnGeom& a, const RowStats& rs, const PageWork& pw, int* list2,
                                      int* count2, int cap2, float a_hi, hipStream_t s);
constexpr float kFixAComplement = 0.99f;   // recorded outputs: above this, the complement pass
constexpr int kFixComplementItems = 32768; // (pair, part) items of the complement pass's workspace
                                           // (at least one per window row)

// classification (Eq. (8)-(10)) and candidate order
struct ClassifyArgs {
  int n;
  const float* R_pre;
  const float* R_post;
  float tau_use, tau_dead, rho_use, rho_dead;
  const uint8_t* force;   // optional
  int max_cand;           // <= 0: no cap
  uint8_t* lambda;
  float* P_pre;           // required (workspace if the caller passes none)
  float* P_post;
  uint8_t* is_cand;       // workspace [n]
  int32_t* cand;
  int32_t* n_cand;
  uint32_t policy;        // CKV_POLICY_* bits (Sec. 4.4 variants)
};
hipError_t launch_classify(const ClassifyArgs& c, hipStream_t s);

// joint test (Eq. (11))
struct JointArgs {
  int total_rows, D, max_cand, W;
  const int32_t* n_cand;
  const float* resid;     // [rows][max_cand][D]
  const float* resA;      // [rows][max_cand]
  const int* resC;
  float* onorm;           // [rows]: ||o_p|| (phase 0)
  int* nvis_part;         // [W][n_vis_slices]: visible tokens of window row p per slice (phase 0)
  int n_vis_slices;
  const float* o;         // [rows][D] window outputs
  const int32_t* pos;     // [S] token positions
  const int32_t* qpos;    // [W] window positions
  int S;
  int test_cap;           // candidates tested at most (0: none, e.g. no pages)
  float* Dstate;          // [rows][D] accumulated residual of accepted pages
  float* Astate;          // [rows]
  int* Cstate;            // [rows]
  int* ctrl;              // [8]: cursor, pending accepted item, barrier arrivals, error, parity
                          //      (zero before the launch: the residual pass clears them)
  unsigned int* rbuf;     // [window] per-candidate max ratio bits
  unsigned int* bmax;     // [workgroups][window] per-workgroup candidate maxima (owned-row form)
  int window;             // candidates evaluated per round
  int rows_per_block;
  float tau;
  long long barrier_ticks; // bound of a grid-barrier wait (100 MHz wall clock ticks)
  uint32_t* nonfinite;    // latched when an o or lse row is NaN or infinite (or null)
  int accept_all;         // no Eq. (11) gate: every candidate accepted
  uint8_t* accepted;
  float* union_R;
  int32_t* n_accepted;
  // recomputation by definition of (candidate, row) pairs whose union mass
  // exceeds kJointFixA (Eq. (6) is ill-conditioned there)
  AttnGeom geo;           // the post-commit cache and window
  const float* lse;       // [rows] natural-log log-sum-exp of each window row
  const int32_t* pstart;  // [n_pages] page table (sorted, disjoint)
  const int32_t* plen;
  int n_pages;
  const int32_t* cand;    // [max_cand] page of each candidate
  uint8_t* in_acc;        // [n_pages] accepted so far (phase 0 clears it)
  int* fix_list;          // [window * rows] (slot, row) pairs flagged in a round
  float* fpart;           // [kJointFixItems][D + 1] partial sums of the fix-up
};
constexpr float kJointFixA = 0.8f;      // union mass above which a pair is recomputed
constexpr int kJointFixItems = 32768;   // (pair, part) items of the fix-up workspace
constexpr int kJointFixParts = 16;      // parts a pair's row is split into at most
int joint_vis_slices(int S);
hipError_t launch_joint_persistent(const JointArgs& j, int max_blocks, hipStream_t s);

// checkpoint: protection, selection, compaction (Eq. (12)-(13), Eq. (4))
// pages retired on the device: page cand[i] (i < min(*n_cand, max_cand))
// of the table (start, len) when accepted[i] != 0
struct AccPages {
  const int32_t* cand;
  const int32_t* n_cand;
  const uint8_t* accepted;
  const int32_t* start;
  const int32_t* len;
  int32_t max_cand;
  int32_t n_pages;
};

struct SelectArgs {
  int n_seq;
  const AccPages* acc;           // [n_seq] or nullptr
  const int32_t* n_tokens;       // [n_seq]
  const float* score;
  int64_t score_seq_stride;
  const int32_t* ret_off;        // [n_seq+1] offsets into ret_start/ret_len
  const int32_t* ret_start;
  const int32_t* ret_len;
  const int32_t* pend_off;       // [n_seq+1]
  const int32_t* pend_start;
  const int32_t* pend_len;
  const uint64_t* pend_r;        // [n_seq] device pointers to R_pre arrays
  uint8_t* pend_prot;            // [total pending] workspace
  int32_t* pend_ord;             // [total pending] workspace
  int budget, bn, max_pages, keep_recent;
  uint8_t* state;                // [n_seq][score_seq_stride] or nullptr
  int32_t* kept;                 // [n_seq][budget]
  int32_t* n_kept;               // [n_seq]
  // workspace of the multi-workgroup selection
  int n_chunks;                  // token chunks of the longest sequence
  uint32_t* kv;                  // [n_seq][score_seq_stride] state-coded keys
  int32_t* ctrl;                 // [n_seq][kSelCtrl]
  uint32_t* hist;                // [n_seq][3][2048] digit histograms
  int32_t* wcnt;                 // [n_seq][n_chunks][2] per-chunk counts
  // persistent state of the grid selection (zero between calls)
  int32_t* gctrl;                // [n_seq][kSelGridCtrl]
  uint32_t* ghist;               // [n_seq][3][kSelBins]
  long long barrier_ticks;       // bound of a per-sequence barrier wait (100 MHz ticks)
};
constexpr long long kBarrierTicksDefault = 1ll << 27;   // ~1.34 s of the 100 MHz wall clock
constexpr int kSelChunk = 2048;  // tokens per selection workgroup
constexpr int kSelCtrl = 16;     // ints of per-sequence selection state
constexpr int kSelBins = 2048;   // radix digit bins (11-bit digits)
hipError_t launch_protect(const SelectArgs& a, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
constexpr int kSelGridChunk = 2048;       // tokens per grid-selection workgroup
constexpr int kSelGridMaxChunks = 64;     // longest sequence: 131072 tokens
constexpr int kSelGridPendMax = 256;      // pending pages per sequence the grid selection ranks
constexpr int kSelGridCtrl = 8 + 2 * kSelGridMaxChunks;   // control words per sequence
bool select_grid_fits(int max_tokens, int max_pending, int n_seq, int resident);
int select_grid_resident();
hipError_t launch_select_grid(const SelectArgs& a, int max_tokens, hipStream_t s);

struct GatherArgs {
  const uint16_t* k_in;
  const uint16_t* v_in;
  int64_t in_seq, in_layer, in_head, in_tok;
  uint16_t* k_out;
  uint16_t* v_out;
  int64_t out_seq, out_layer, out_head, out_tok;
  const int32_t* pos_in;
  int64_t pos_in_seq;
  int32_t* pos_out;
  int64_t pos_out_seq;
  int n_seq, n_layers, Hkv, D;
  const int32_t* kept;           // [n_seq][budget]
  const int32_t* n_kept;
  int budget;
  int64_t in_rows;               // token rows of an input sequence (capacity)
  uint32_t* dbg;                 // debug word of the context (CKV_DEBUG builds)
};
hipError_t launch_gather(const GatherArgs& g, hipStream_t s);

// pooled base score: n_tokens device int32[n_seq]; windows of `kernel` (odd) tokens
hipError_t launch_pool(const float* score, float* out, int64_t stride, const int32_t* n_tokens, int n_seq,
                       int max_tokens, int kernel, int mode, hipStream_t s);

}  // namespace ckv
