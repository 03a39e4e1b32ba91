// Window attention and per-page deletion effects (CommitKV, Sec. 3.2,
// Eq. (6)-(7)) on MFMA for gfx950.
//
// Two passes over the resident cache of one layer:
//   A. window_attention_kernel + combine_kernel: for every window row
//      (query head h, row p) the full attention output o_p, its log-sum-exp
//      and the number of visible tokens.  Split over the token axis, partial
//      (max, sum, unnormalised output) merged by the combine kernel.
//   B. page_kernel: for every page E and row p, with the page-local max
//      m_E = max_{i in E} x_i:
//        l^ = sum_{i in E} 2^(x_i - m_E),  U^ = sum_{i in E} 2^(x_i - m_E) v_i,
//        f  = 2^(m_E - lse_p),  A = f l^,
//        ||o_p - o_p^{\E}|| / ||o_p|| = f ||U^ - l^ o_p|| / ((1 - A) ||o_p||)
//      (Eq. (6) rescaled by the page maximum, so the float16 weights of the
//      page stay in (0, 1]).  MODE 0 reduces the ratio to max over rows and
//      heads (Eq. (7)); MODE 1 stores the residual f (U^ - l^ o_p), the mass
//      A and the visible count for the joint test.
//   C. token_mass_kernel: max_h sum_p a_hpi for every token.
// Logits are carried in log2 units: x = scale * log2(e) * q.k.
//
// Every kernel runs 8 waves of 32 window rows each (256 rows per workgroup),
// so a wave's registers (queries, one output block, one score block) fit in
// the 256 architectural VGPRs and two waves share each SIMD: one wave's
// softmax overlaps the other's MFMA.
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <algorithm>
#include <climits>

namespace ckv {

constexpr int kNW = 8;               // waves per workgroup
constexpr int kRowsWG = 32 * kNW;    // window rows per workgroup
// The running output is rescaled whenever a row's max grows (the wave skips
// the rescale when no row's max grew), so the float16 weight of a row's
// largest logit is exactly 1, as it is in the per-page pass (whose reference
// is the page's own max).  A page that carries most of a row's mass then
// enters o and its own sum with the same weight, which keeps the residual
// u - A o of Eq. (6) free of that token's rounding; a reference that lags
// the max (weights above 1) was measured to cost ~10x in score error on
// such pages.  It also keeps o itself exact in the weight of a row's
// dominant token, which recorded-output callers rely on: a reference
// allowed to lag the max by up to 15 (log2 units, which skipped most
// rescales) put a rounding of 2^-12 on that weight and about 4e-3 on the
// effects of dominant pages computed from such an o.
//
// A page that holds nearly all of a row's mass (A -> 1) is ill-conditioned
// for Eq. (6): o - u = (1 - A) o' keeps only the digits of o' that survive
// float32 accumulation of o, and every error of u - A o is amplified by
// 1/(1 - A).  How far the closed form holds depends on whether the window
// pass weighted all of the page against its row's largest logit, the
// reference the page kernel uses when the page holds that logit.  The
// window pass takes a tile's weights after the tile's own maximum has
// entered the reference (tiles start at multiples of 64 tokens, splits at
// multiples of the split length), so that holds for a page that holds the
// logit and lies inside one tile, and for a page that crosses into the next
// tile of the same split once the logit has entered that split's reference
// by the tile of the page's first part (the window pass records, per row,
// the tile where it did; the next tile keeps the reference).  Then the
// page's float16 weights are the very ones that formed o and cancel in
// u - A o; what is left is the
// float32 rounding of the log-sum-exp (through 1 - A), a few 1e-7 times
// 1/(1 - A), and such pairs keep the closed form up to A = kFixAHi.  Any
// other page's weights were rounded against different references in the
// two passes, and those roundings reach the residual amplified by
// 1/(1 - A): such pairs are listed above A = kFixA.  Listed rows are left
// out of the page kernel's maximum; the fix-up kernel recomputes the output
// without the page, o', directly (all other splits' partial sums as they
// are, the page's own split again with the page excluded) and takes
// ||o - o'|| / ||o|| by definition; a listed page across a tile boundary
// inside one split whose row maximum entered the reference with its second
// tile is instead evaluated with the window pass's own weights (older
// reference for the first part, then rescaled), which the window kernel's
// recorded references make known.  At most one page per row can exceed
// kFixA, so the list never holds more than one entry per window row.  With
// recorded outputs (computed without this pass's float16 weights) every
// pair above kFixARecorded is listed: the page pass's rounding is then no
// longer shared by o, and 1/(1 - A) would amplify it past the tolerance.

// ---------------------------------------------------------------------------
// staging of a 64-token tile made of two 32-token segments (slot 0: offsets
// 0..31, slot 1: offsets 32..63): K as [token][width] bf16, V^T as
// [width][slot] fp16 (slot = vt_slot(offset)), positions as int32 (INT_MAX
// for offsets past a segment's length, whose K and V rows are zero).
// ---------------------------------------------------------------------------
// PG: the cache is a paged pool, token t's key and value rows are row
// slot[t] (clamped to the pool) of each head's storage; positions stay by
// token.
template <int D, int NT, bool PG = false>
struct Stager {
  static constexpr int KP = D + 8;              // K tile row stride (elements)
  static constexpr int VP = kTile + 8;          // V^T tile row stride (halves)
  static constexpr int CPR = D / 8;             // 16-byte chunks per row
  static constexpr int KCH = kTile * CPR;       // chunks per K tile
  static constexpr int KPT = (KCH + NT - 1) / NT;
  static constexpr int VU = (kTile / 2) * CPR;  // (2 tokens x 8 widths) units of V
  static constexpr int VPT = (VU + NT - 1) / NT;

  u32x4 kr[KPT];
  u32x4 vr[VPT][2];
  int pr;        // loaded position (its use waits for the load: only in commit)
  bool pok;      // false: offset outside the segments, position INT_MAX

  // element offset of tile row r (0..63) inside the head; rows outside the
  // segments read token 0.  r depends only on the thread, so the slot test
  // is a per-thread constant.
  __device__ __forceinline__ static uint32_t row_off(int r, int s0, int n0, int s1, int n1, uint32_t ts,
                                                     const int32_t* slot, uint32_t last, int S, uint32_t* dbg,
                                                     bool& ok) {
    const bool hi = r >= 32;
    const int o = r & 31;
    ok = o < (hi ? n1 : n0);
    if constexpr (PG) {
      return __umul24(min((uint32_t)slot[ok ? CKV_IDX((hi ? s1 : s0) + o, S, dbg, 9) : 0], last), ts);
    } else {
      return ok ? __umul24((uint32_t)CKV_IDX((hi ? s1 : s0) + o, S, dbg, 9), ts) : 0u;
    }
  }

  // Loads are unconditional: a token outside the segments reads token 0,
  // which always exists.  Its key and value land in the tile as they are;
  // the offset's position is INT_MAX, so every row masks its score to -inf
  // and its weight is exactly 0 (values are finite).
  __device__ __forceinline__ void issue(const uint16_t* kh, const uint16_t* vh, uint32_t ts,
                                        const int32_t* slot, uint32_t last, const int32_t* pos, int s0,
                                        int n0, int s1, int n1, int tid, int S, uint32_t* dbg) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      bool ok;
      const uint32_t e = row_off((c / CPR) & (kTile - 1), s0, n0, s1, n1, ts, slot, last, S, dbg, ok);
      kr[i] = ldg_u4(kh + ((c < KCH ? e : 0u) + (c % CPR) * 8));
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      const int tp = (u / CPR) & (kTile / 2 - 1), cg = u % CPR;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        bool ok;
        const uint32_t e = row_off(2 * tp + j, s0, n0, s1, n1, ts, slot, last, S, dbg, ok);
        vr[i][j] = ldg_u4(vh + ((u < VU ? e : 0u) + cg * 8));
      }
    }
    const int r = tid & 63;
    const int t = (r >= 32 ? s1 : s0) + (r & 31);
    const bool ok = (r & 31) < (r >= 32 ? n1 : n0) && tid < kTile;
    pr = ldg_i32(pos + (ok ? CKV_IDX(t, S, dbg, 10) : 0));
    pok = ok;
  }

  // writes the tile; wave 0 also flags, per 32-token slot, whether every
  // position is <= minq (sFull[0], sFull[1])
  __device__ __forceinline__ void commit(uint16_t* sK, _Float16* sV, int* sP, int* sFull, int minq,
                                         int tid) const {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      if (c < KCH) *reinterpret_cast<u32x4*>(sK + (c / CPR) * KP + (c % CPR) * 8) = kr[i];
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      if (u < VU) {
        const int tp = u / CPR, cg = u % CPR;
        // rows cg*8 .. cg*8+7 share bits 4..6, hence one stored column
        const int col = vt_col(cg * 8, vt_slot(2 * tp));
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          const f32x2 w = {bf16_bits_to_float(chunk_elem(vr[i][0], e)),
                           bf16_bits_to_float(chunk_elem(vr[i][1], e))};
          *reinterpret_cast<f16x2*>(sV + (cg * 8 + e) * VP + col) = __builtin_convertvector(w, f16x2);
        }
      }
    }
    if (tid < kTile) {
      const int p = pok ? pr : INT_MAX;
      sP[tid] = p;
      const unsigned long long late = __ballot(p > minq);
      if (tid == 0) {
        sFull[0] = (late & 0xFFFFFFFFull) == 0ull;
        sFull[1] = (late >> 32) == 0ull;
      }
    }
  }
};

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ bf16x8 zero_bf16x8() {
  return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
}

// the window row a lane handles inside KV head g
struct RowInfo {
  int row;     // row inside the KV head (0 .. rows-1); padding rows are >= rows
  bool ok;
  int qp;      // absolute position of the window row
  int rg;      // global row index h*W + p
};

__device__ __forceinline__ RowInfo row_info(const AttnGeom& a, int g, int row) {
  RowInfo r;
  r.row = row;
  r.ok = row < a.rows;
  const int p = r.ok ? row % a.W : 0;
  r.qp = r.ok ? a.qpos[p] : INT_MIN;
  r.rg = g * a.rows + (r.ok ? row : 0);
  return r;
}

template <int D>
__device__ __forceinline__ void load_q(const AttnGeom& a, int g, const RowInfo& ri, int half,
                                       bf16x8 (&qf)[D / 16]) {
  const int h = g * a.group + (ri.ok ? ri.row / a.W : 0);
  const int p = ri.ok ? ri.row % a.W : 0;
  const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    qf[ks] = ri.ok ? load_bf16x8(qrow + 16 * ks + 8 * half) : zero_bf16x8();
}

// smallest window position among the valid rows of the workgroup
__device__ __forceinline__ int block_min_qpos(const RowInfo& ri, int* sMin) {
  if (threadIdx.x == 0) *sMin = INT_MAX;
  __syncthreads();
  int q = ri.ok ? ri.qp : INT_MAX;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) q = min(q, __shfl_xor(q, off, 64));
  if ((threadIdx.x & 63) == 0) atomicMin(sMin, q);
  __syncthreads();
  return *sMin;
}

// S^T block (32 tokens x 32 rows) of tile slot tb: K from LDS, Q^T in registers
template <int D, int KP>
__device__ __forceinline__ f32x16 scores(const uint16_t* sK, int tb, int col, int half,
                                         const bf16x8 (&qf)[D / 16]) {
  f32x16 acc = zero16();
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    acc = mfma_bf16(load_bf16x8(sK + (32 * tb + col) * KP + 16 * ks + 8 * half), qf[ks], acc);
  return acc;
}

// the same with the K fragments read kPFS steps ahead of the products
template <int D, int KP, int kPFS = 4>
__device__ __forceinline__ f32x16 scores_pf(const uint16_t* sK, int tb, int col, int half,
                                            const bf16x8 (&qf)[D / 16]) {
  constexpr int KS = D / 16;
  bf16x8 kf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) kf[ks] = load_bf16x8(sK + (32 * tb + col) * KP + 16 * ks + 8 * half);
  f32x16 acc = zero16();
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) acc = mfma_bf16(kf[ks], qf[ks], acc);
  __builtin_amdgcn_sched_group_barrier(0x100, kPFS, 0);
#pragma unroll
  for (int i = 0; i < KS - kPFS; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kPFS, 0);
  return acc;
}

// Rounds the 16 weights of a score block to float16 (the B operands of the
// two 16-token steps of O^T += V^T P^T) and adds the ROUNDED weights to sum.
// Normalising by the sum of exactly the weights that multiply V keeps the
// output a true weighted average; with unrounded sums, a page that carries
// nearly all of a row's mass would see its rounding error amplified by
// 1/(1 - A) in the residual u - A o.
__device__ __forceinline__ void to_f16(const f32x16& p, f16x8 (&h)[2], float& sum) {
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  const f16x2 one = {(_Float16)1.f, (_Float16)1.f};
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int e = 0; e < 8; ++e) h[u][e] = (_Float16)p[8 * u + e];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const f16x2 pr = {h[u][2 * e], h[u][2 * e + 1]};
      sum = __builtin_amdgcn_fdot2(pr, one, sum, false);
    }
  }
}

// O^T (+)= V^T P^T for one 32-token slot, P^T given as float16 operands
template <int D, int VP>
__device__ __forceinline__ void pv_slot(const _Float16* sV, int tb, int col, int half, const f16x8 (&h)[2],
                                        f32x16 (&acc)[D / 32]) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const f16x8 af =
          *reinterpret_cast<const f16x8*>(sV + vt_frag_lane<VP>(col, half) + vt_frag_const(VP, db, tb, u));
      acc[db] = mfma_f16(af, h[u], acc[db]);
    }
  }
}

// the same for the two width blocks db0, db0 + 1 only
template <int D, int VP>
__device__ __forceinline__ void pv_half(const _Float16* sV, int tb, int col, int half, const f16x8 (&h)[2],
                                        int db0, f32x16 (&acc)[2]) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const f16x8 af = *reinterpret_cast<const f16x8*>(sV + vt_frag_lane<VP>(col, half) +
                                                        vt_frag_const(VP, db0 + j, tb, u));
      acc[j] = mfma_f16(af, h[u], acc[j]);
    }
  }
}

// ---------------------------------------------------------------------------
// A. split window attention
// ---------------------------------------------------------------------------
template <int D, bool PG>
__global__ __launch_bounds__(kNW * 64, 1) void window_attention_kernel(AttnGeom a, AttnSplit sp) {
  constexpr int NT = kNW * 64, KS = D / 16, DB = D / 32;
  using St = Stager<D, NT, PG>;
  __shared__ __align__(16) uint16_t sK[2][kTile * St::KP];
  __shared__ __align__(16) _Float16 sV[2][D * St::VP];
  __shared__ __align__(16) int sP[2][kTile];
  __shared__ int sFull[2][2];
  __shared__ int sMin;

  const int g = blockIdx.z, split = blockIdx.x, rblk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int t_begin = split * sp.chunk;
  const int t_end = min(a.S, t_begin + sp.chunk);
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;

  const RowInfo ri = row_info(a, g, rblk * kRowsWG + wave * 32 + col);
  const bool wave_on = __ballot(ri.ok) != 0ull;
  const int minq = block_min_qpos(ri, &sMin);
  bf16x8 qf[KS];
  load_q<D>(a, g, ri, half, qf);

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = zero16();
  float mref = -INFINITY, l = 0.f;
  int cnt = 0;
  int mt = -1;          // start of the tile where mref last grew
  float mp = -INFINITY;  // mref before that tile

  const int n_tiles = t_end > t_begin ? (t_end - t_begin + kTile - 1) / kTile : 0;
  // Loads run two tiles ahead of the math: stager A holds even tiles, B odd
  // ones; a tile past the end is an empty segment (its loads read token 0).
  auto issue = [&](St& st, int it) {
    const int t0 = t_begin + it * kTile;
    const int n = it < n_tiles ? min(kTile, t_end - t0) : 0;
    st.issue(kh, vh, (uint32_t)a.kv_tok_stride, a.slot, a.pool_last, a.pos, t0, min(32, n), t0 + 32,
             max(0, n - 32), tid, a.S, a.dbg);
  };
  auto compute = [&](int b, int it) {
    if (wave_on) {
      f32x16 s[2];
      s[0] = scores<D, St::KP>(sK[b], 0, col, half, qf);
      s[1] = scores<D, St::KP>(sK[b], 1, col, half, qf);
      float mx = -INFINITY;
      if (sFull[b][0] && sFull[b][1]) {
        // every token of the tile is visible to every row of the workgroup
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[tb][r]);
        cnt += 32;
      } else {
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int4 pq = *reinterpret_cast<const int4*>(&sP[b][32 * tb + 8 * i + 4 * half]);
            const int pv[4] = {pq.x, pq.y, pq.z, pq.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const bool vis = ri.ok && pv[j] <= ri.qp;
              const float x = vis ? s[tb][4 * i + j] : -INFINITY;
              cnt += vis ? 1 : 0;
              s[tb][4 * i + j] = x;
              mx = fmaxf(mx, x);
            }
          }
      }
      mx = max32(mx) * a.sl2;
      // rescale the running output when a row max grew
      const bool need = mx > mref;
      if (__ballot(need) != 0ull) {
        const float nref = need ? mx : mref;
        const float alpha = need ? __builtin_amdgcn_exp2f(mref - nref) : 1.f;
        l *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        if (need) {
          mp = mref;
          mt = t_begin + it * kTile;
        }
        mref = nref;
      }
      const float base = mref == -INFINITY ? 0.f : mref;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[tb][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[tb][r], a.sl2, -base));
      f16x8 h[2][2];
      to_f16(s[0], h[0], l);
      to_f16(s[1], h[1], l);
      pv_slot<D, St::VP>(sV[b], 0, col, half, h[0], oacc);
      pv_slot<D, St::VP>(sV[b], 1, col, half, h[1], oacc);
    }
  };
  St stA, stB;
  issue(stA, 0);
  issue(stB, 1);
  if (n_tiles > 0) stA.commit(sK[0], sV[0], sP[0], sFull[0], minq, tid);
  __syncthreads();
  for (int it = 0; it < n_tiles; it += 2) {
    issue(stA, it + 2);
    compute(0, it);
    if (it + 1 < n_tiles) stB.commit(sK[1], sV[1], sP[1], sFull[1], minq, tid);
    __syncthreads();
    if (it + 1 >= n_tiles) break;
    issue(stB, it + 3);
    compute(1, it + 1);
    if (it + 2 < n_tiles) stA.commit(sK[0], sV[0], sP[0], sFull[0], minq, tid);
    __syncthreads();
  }

  // partial results of this split (m in log2 units, output relative to it)
  const float lt = sum32(l);
  const int ct = sum32i(cnt);
  if (!ri.ok) return;
  const size_t idx = CKV_IDX((size_t)(g * sp.n_splits + split) * sp.rows_pad + ri.row,
                             (int64_t)a.Hkv * sp.n_splits * sp.rows_pad, a.dbg, 1);
  if (half == 0) {
    sp.part_m[idx] = mref;
    sp.part_l[idx] = lt;
    sp.part_c[idx] = ct;
    sp.part_t[idx] = mt;
    sp.part_p[idx] = mp;
  }
  float* po = sp.part_o + idx * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 v4;
#pragma unroll
      for (int j = 0; j < 4; ++j) v4[j] = oacc[db][4 * i + j];
      *reinterpret_cast<f32x4*>(po + 32 * db + 8 * i + 4 * half) = v4;
    }
}

// Merge of the splits: D/4 lanes per window row (16 bytes of the partial
// output each), so a wave holds 256 / D rows.  Splits are read in batches of
// kCombBatch with every load of a batch in flight; the running maximum is
// updated once per batch (the weights of earlier batches are rescaled), and
// the batch order is fixed, so the result does not depend on scheduling.
// Writes o, lse, ||o||, the visible count and the row's largest logit.
constexpr int kCombBatch = 16;

template <int D>
__global__ __launch_bounds__(256) void combine_kernel(AttnGeom a, AttnSplit sp, RowStats rs,
                                                      float* lse_out, ZeroList zl) {
  constexpr int TPR = D / 4;          // lanes per row
  constexpr int RPW = 64 / TPR;       // rows per wave
  const int lane = threadIdx.x & 63, c = lane % TPR;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  // zero the outputs that later kernels reduce into with atomic max
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  for (size_t i = gid; i < zl.n0; i += gsz) zl.p0[i] = 0.f;
  for (size_t i = gid; i < zl.n1; i += gsz) zl.p1[i] = 0.f;
  for (size_t i = gid; i < zl.n2; i += gsz) zl.p2[i] = 0.f;
  if (zl.i0 && gid == 0) *zl.i0 = 0;
  for (size_t i = gid; i < zl.n1i; i += gsz) zl.i1[i] = 0;
  const int total = a.Hkv * a.rows;
  const int rw = wid * RPW + lane / TPR;     // this lane's (KV head, row) pair
  if (wid * RPW >= total) return;
  const bool ok = rw < total;
  const int g = ok ? rw / a.rows : 0, row = ok ? rw % a.rows : 0;
  const int rg = g * a.rows + row;
  const size_t base = (size_t)g * sp.n_splits * sp.rows_pad + row;
  float M = -INFINITY, wsum = 0.f;
  int nv = 0, mt = -1;   // mt: tile where M entered the first split that holds it
  float mp = -INFINITY;  // that split's reference before the tile
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < sp.n_splits; s0 += kCombBatch) {
    float ms[kCombBatch], ls[kCombBatch];
    int cs[kCombBatch], ts[kCombBatch];
    float ps[kCombBatch];
    f32x4 os[kCombBatch];
#pragma unroll
    for (int u = 0; u < kCombBatch; ++u) {
      const bool in = s0 + u < sp.n_splits;
      const size_t idx = CKV_IDX(base + (size_t)min(s0 + u, sp.n_splits - 1) * sp.rows_pad,
                                 (int64_t)a.Hkv * sp.n_splits * sp.rows_pad, a.dbg, 2);
      ms[u] = in ? sp.part_m[idx] : -INFINITY;
      ls[u] = sp.part_l[idx];
      cs[u] = in ? sp.part_c[idx] : 0;
      ts[u] = sp.part_t[idx];
      ps[u] = sp.part_p[idx];
      os[u] = *reinterpret_cast<const f32x4*>(sp.part_o + idx * D + 4 * c);
    }
    float mb = M;
#pragma unroll
    for (int u = 0; u < kCombBatch; ++u) {
      mt = ms[u] > mb ? ts[u] : mt;   // the first split wins a tie
      mp = ms[u] > mb ? ps[u] : mp;
      mb = fmaxf(mb, ms[u]);
    }
    if (mb != -INFINITY) {
      if (mb > M) {
        const float r = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(M - mb);
        wsum *= r;
        acc *= r;
        M = mb;
      }
#pragma unroll
      for (int u = 0; u < kCombBatch; ++u) {
        const float w = ms[u] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms[u] - M);
        wsum += ls[u] * w;
        acc += os[u] * w;
      }
    }
#pragma unroll
    for (int u = 0; u < kCombBatch; ++u) nv += cs[u];
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const f32x4 ov = acc * inv;
  float n2 = ov[0] * ov[0] + ov[1] * ov[1] + ov[2] * ov[2] + ov[3] * ov[3];
#pragma unroll
  for (int off = TPR / 2; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
  if (!ok) return;
  *reinterpret_cast<f32x4*>(rs.o + (size_t)CKV_IDX(rg, a.Hq * a.W, a.dbg, 3) * D + 4 * c) = ov;
  if (c == 0) {
    const float l2 = wsum > 0.f ? M + __log2f(wsum) : -INFINITY;
    rs.lse2[rg] = l2;
    rs.onorm[rg] = sqrtf(n2);
    rs.nvis[rg] = nv;
    if (rs.m2) rs.m2[rg] = M;
    if (rs.m2t) rs.m2t[rg] = mt;
    if (rs.m2p) rs.m2p[rg] = mp;
    if (lse_out) lse_out[rg] = l2 * kLn2;
    // a NaN or infinite key, query or value reaches the row's output or its
    // log-sum-exp (a row that sees no token has lse -inf and o = 0)
    if (!(n2 <= 3.4e38f) || (nv > 0 && !(l2 > -INFINITY && l2 < INFINITY))) latch_nonfinite(zl.nonfinite);
  }
}

// ---------------------------------------------------------------------------
// B. per-page deletion effect (MODE 0) or per-candidate residual (MODE 1)
//
// A staged 64-token tile holds either two pages of at most 32 tokens (one per
// 32-token slot) or one page of 33..64 tokens (both slots).  Every thread
// derives the same tile sequence from the page lengths.
// ---------------------------------------------------------------------------
// NB: 32-token slots a page may span (1 when every page has <= 32 tokens).
constexpr int kAcrossSplit = 0x7f;   // page class: across a split boundary of the window pass
template <int D, int MODE, int NB, bool PG>
__global__ __launch_bounds__(kNW * 64, 1) void page_kernel(AttnGeom a, PageWork pw, RowStats rs) {
  constexpr int NT = kNW * 64, KS = D / 16, DB = D / 32;
  using St = Stager<D, NT, PG>;
  __shared__ __align__(16) uint16_t sK[2][kTile * St::KP];
  __shared__ __align__(16) _Float16 sV[2][D * St::VP];
  __shared__ __align__(16) int sP[2][kTile];
  __shared__ int sFull[2][2];
  // MODE 0: per (page of the block, local head) maximum ratio, flushed to
  // global memory once after the last tile, so the tile loop issues no
  // global atomics (a wave that waits on them stalls the whole workgroup at
  // the tile barrier); the host bounds pages x heads by kPageRmaxCap
  __shared__ unsigned int sRm[MODE == 0 ? kPageRmaxCap : 1];
  // MODE 0: rows left to the fix-up kernel, published after the last tile
  // (a row has at most one page with A > fix_a >= 0.5, so kRowsWG entries suffice
  // unless the inputs hold NaN; an overflow appends to the global list)
  __shared__ int4 sFix[MODE == 0 ? kRowsWG : 1];
  __shared__ int sFixN, sFixBase;
  __shared__ int sMin;
  __shared__ int sItStart[kPageItemsMax], sItLen[kPageItemsMax];   // this block's pages
  __shared__ int sItLo[MODE == 0 ? kPageItemsMax : 1];   // start of the split of a page's first part
  __shared__ int4 sTileSeg[kPageItemsMax];    // per tile: segments (s0, n0, s1, n1)
  __shared__ int sTileIt[kPageItemsMax + 1];  // per tile: first item; entry n_tiles = i_end
  __shared__ int sNTiles;

  const int g = blockIdx.z, rblk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  int n_items = pw.n_items;
  if (MODE == 1) n_items = min(*pw.n_cand, pw.n_items);
  if (MODE == 1 && pw.clear && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && tid < pw.n_clear)
    pw.clear[tid] = 0;
  const int i_begin = blockIdx.x * pw.items_per_block;
  const int i_end = min(n_items, i_begin + pw.items_per_block);
  if (i_begin >= i_end) return;
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;

  // the block's page spans go to LDS once, so the tile sequence never waits
  // on a global load inside the loop (a wait there would also drain the
  // loads issued ahead); an invalid candidate index is an empty page
  for (int i = tid; i < i_end - i_begin; i += NT) {
    const int item = i_begin + i;
    const int pg = MODE == 0 ? item : pw.cand[item];
    const bool ok = pg >= 0 && pg < pw.n_pages;
    sItStart[i] = ok ? pw.start[pg] : 0;
    // the length, and above bit 8 (MODE 0) where the page meets the window
    // pass's tiles: 0 inside one tile, n < 64 across a tile boundary after
    // n tokens inside one split, kAcrossSplit across a split boundary (or
    // with the split length unknown)
    int lw = ok ? pw.len[pg] : 0;
    if (MODE == 0 && ok) {
      const int s0 = pw.start[pg], nf = (s0 / kTile + 1) * kTile - s0;
      if (nf < lw) lw |= (pw.split_tokens > 0 && (s0 + nf) % pw.split_tokens != 0 ? nf : kAcrossSplit) << 8;
      if (pw.split_tokens > 0) sItLo[i] = s0 - s0 % pw.split_tokens;
    }
    sItLen[i] = lw;
  }
  const RowInfo ri = row_info(a, g, rblk * kRowsWG + wave * 32 + col);
  const bool wave_on = __ballot(ri.ok) != 0ull;
  const int minq = block_min_qpos(ri, &sMin);    // its barriers also publish the page spans
  bf16x8 qf[KS];
  load_q<D>(a, g, ri, half, qf);
  // o_p in accumulator layout: register r of block db holds width 32db + 8(r/4) + 4h + r%4
  f32x16 of[DB];
  {
    const float* orow = rs.o + (size_t)CKV_IDX(ri.rg, a.Hq * a.W, a.dbg, 4) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 v4 = ri.ok ? *reinterpret_cast<const f32x4*>(orow + 32 * db + 8 * i + 4 * half)
                               : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) of[db][4 * i + j] = v4[j];
      }
  }
  const float lse2 = ri.ok ? rs.lse2[ri.rg] * pw.lse_scale : -INFINITY;   // -inf stays -inf
  const float onorm = (MODE == 0 && ri.ok) ? rs.onorm[ri.rg] : 0.f;   // read by MODE 0 only
  const float inv_onorm = onorm > 0.f ? 1.f / onorm : 0.f;
  const int nvis = (MODE == 0 && ri.ok) ? rs.nvis[ri.rg] : 0;   // read by MODE 0 only
  // the row's largest scaled logit, the window pass's final weight reference
  // (NaN when unknown: no page then counts as holding it)
  const float m2row = (MODE == 0 && rs.m2 && ri.ok) ? rs.m2[ri.rg] : __builtin_nanf("");
  // where that logit entered the window pass's reference (first split holding it)
  const int m2trow = (MODE == 0 && rs.m2t && ri.ok) ? rs.m2t[ri.rg] : -1;
  const int row0 = rblk * kRowsWG;
  const int head0 = row0 / a.W;
  const int n_heads_blk = min(a.group, (min(a.rows, row0 + kRowsWG) - 1) / a.W + 1) - head0;
  const bool wave_one_head = (a.W % 32) == 0;   // the 32 rows of a wave share one head
  const int my_hl = ri.ok ? ri.row / a.W - head0 : 0;   // this row's head inside the block
  if (MODE == 0) {
    for (int i = tid; i < (i_end - i_begin) * n_heads_blk; i += NT) sRm[i] = 0u;
    if (tid == 0) sFixN = 0;
  }

  auto pstart = [&](int item) { return sItStart[item - i_begin]; };
  auto plen = [&](int item) { return sItLen[item - i_begin] & 0xff; };
  // pages in the tile that starts at item `it`: two short pages share a tile
  auto tile_items = [&](int it) {
    return (it + 1 < i_end && plen(it) <= 32 && plen(it + 1) <= 32) ? 2 : 1;
  };
  // the block's tile sequence, built once (thread 0) into LDS
  if (tid == 0) {
    int k = 0;
    for (int it = i_begin; it < i_end; ++k) {
      const int m = tile_items(it);
      const int s0 = pstart(it), l0 = plen(it);
      sTileIt[k] = it;
      sTileSeg[k] = m == 2 ? make_int4(s0, l0, pstart(it + 1), plen(it + 1))
                           : make_int4(s0, min(l0, 32), s0 + 32, max(0, l0 - 32));
      it += m;
    }
    sTileIt[k] = i_end;
    sNTiles = k;
  }
  __syncthreads();
  const int n_tiles = sNTiles;
  // The next tile's loads are issued before the current tile's math; a tile
  // index past the end is an empty segment (its loads read token 0).
  auto issue_tile = [&](St& st, int k) {
    const int4 sg = k < n_tiles ? sTileSeg[k] : make_int4(0, 0, 0, 0);
    st.issue(kh, vh, (uint32_t)a.kv_tok_stride, a.slot, a.pool_last, a.pos, sg.x, sg.y, sg.z, sg.w, tid, a.S,
             a.dbg);
  };
  // A row sees at least nvis tokens; a page (at most kMaxPage tokens) can
  // hold all of them only if nvis <= kMaxPage, so most waves skip the count.
  const bool need_count = MODE == 1 || __ballot(ri.ok && nvis <= kMaxPage) != 0ull;

  // the pages of the tile in buffer b
  // page `item` of the tile in buffer b, at slot ps (a constant at each call,
  // so the slot's LDS offsets fold into the instructions)
  auto page = [&](int b, int item, int m, const int ps) {
    {
      const int lw = sItLen[item - i_begin];
      const int len = lw & 0xff, cross = lw >> 8;
      // a short page occupies slot ps; a long one both slots from slot 0
      const int nblk = (NB == 1 || m == 2) ? 1 : (len > 32 ? 2 : 1);
      const int slot0 = ps;
      f32x16 s[2];
      s[0] = scores<D, St::KP>(sK[b], slot0, col, half, qf);
      if (NB == 2) s[1] = nblk == 2 ? scores<D, St::KP>(sK[b], 1, col, half, qf) : zero16();
      // Offsets past the page's length carry position INT_MAX, so the
      // position test alone masks them (window positions are < INT_MAX).
      // A slot whose every position is <= the workgroup's smallest window
      // position (a whole page, all visible) needs no test at all.
      float mx = -INFINITY;
      int c = 0;
      if (sFull[b][slot0] && (nblk == 1 || sFull[b][1])) {
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
          if (tb < nblk) {
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[tb][r]);
          }
        c = 32 * nblk;
      } else {
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        if (tb < nblk) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int4 pq = *reinterpret_cast<const int4*>(&sP[b][32 * (slot0 + tb) + 8 * i + 4 * half]);
            const int pv[4] = {pq.x, pq.y, pq.z, pq.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const bool vis = pv[j] <= ri.qp;
              const float x = vis ? s[tb][4 * i + j] : -INFINITY;
              if (need_count) c += vis ? 1 : 0;
              s[tb][4 * i + j] = x;
              mx = fmaxf(mx, x);
            }
          }
        }
      }
      if (need_count) c = sum32i(c);
      }
      mx = max32(mx);
      const bool touched = mx != -INFINITY;
      const float base = touched ? mx * a.sl2 : 0.f;
      const bool holds_max = base == m2row;   // the row's largest logit is in the page
#pragma unroll
      for (int r = 0; r < 16; ++r) s[0][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[0][r], a.sl2, -base));
      float ls = 0.f;
      f16x8 h0[2], h1[2];
      to_f16(s[0], h0, ls);
      if (NB == 2 && nblk == 2) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[1][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[1][r], a.sl2, -base));
        to_f16(s[1], h1, ls);
      }
      const float lhat = sum32(ls);
      const float f = touched ? __builtin_amdgcn_exp2f(base - lse2) : 0.f;
      const float A = f * lhat;
      // r^ = U^ - l^ o in two halves of the width (32 accumulator registers
      // each): the accumulators start at -l^ o, so the MFMAs leave r^.
      float n2 = 0.f;
#pragma unroll
      for (int hh = 0; hh < DB / 2; ++hh) {
        f32x16 u[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) u[j] = of[2 * hh + j] * (-lhat);
        pv_half<D, St::VP>(sV[b], slot0, col, half, h0, 2 * hh, u);
        if (NB == 2 && nblk == 2) pv_half<D, St::VP>(sV[b], 1, col, half, h1, 2 * hh, u);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) n2 = __builtin_fmaf(u[j][r], u[j][r], n2);
        if (MODE == 1 && ri.ok) {
          float* rrow = pw.resid + (size_t)CKV_IDX((size_t)ri.rg * pw.n_items + item,
                                                   (int64_t)pw.total_rows * pw.n_items, a.dbg, 6) * D;
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              f32x4 v4;
#pragma unroll
              for (int e = 0; e < 4; ++e) v4[e] = f * u[j][4 * i + e];
              *reinterpret_cast<f32x4*>(rrow + 32 * (2 * hh + j) + 8 * i + 4 * half) = v4;
            }
        }
      }
      n2 = sum32(n2);
      // Past fix_a the closed form is kept only where the window pass
      // weighted all of the page against the row's largest logit.  For a
      // page across a tile boundary inside one split, that logit must have
      // entered the split's reference by the tile of the page's first part
      // (lanes without a row have m2row NaN, so holds_max is false there).
      bool form_ok = MODE == 0 && holds_max && A <= pw.fix_a_hi;
      // the fix-up may evaluate a listed pair with the window pass's own weights
      const bool cand = MODE == 0 && rs.m2t != nullptr && A <= pw.fix_a_hi;
      if (MODE == 0 && cross != 0) {
        if (cross == kAcrossSplit) {
          form_ok = false;
        } else {
          const int hi = pstart(item) + cross - kTile, lo = sItLo[item - i_begin];
          form_ok = form_ok && m2trow >= lo && m2trow <= hi;
        }
      }
      // the ratio of Eq. (6)-(7)
      if (MODE == 0) {
        float ratio = 0.f;
        if (touched) {
          const float keep = 1.f - A;
          if (need_count && c >= nvis) {
            ratio = INFINITY;                 // the page holds every visible token
          } else if ((A > pw.fix_a && !form_ok) || !(keep > 0.f)) {
            if (ri.ok && half == 0) {         // ill-conditioned: recomputed by the fix-up
              const int4 ent = make_int4(item, ri.rg, pstart(item), len | (cand ? kFixRescaled : 0));
              const int ls = atomicAdd(&sFixN, 1);
              if (ls < kRowsWG) {
                sFix[ls] = ent;
              } else {
                const int slot = atomicAdd(pw.fix_count, 1);
                if (slot < pw.fix_cap) reinterpret_cast<int4*>(pw.fix_list)[slot] = ent;
              }
            }
          } else if (onorm > 0.f) {
            // hardware square root and reciprocal (about 1 ulp each): the
            // ratio's tolerance is four orders of magnitude looser, and the
            // IEEE sequences cost some 35 instructions per page
            ratio = f * __builtin_amdgcn_sqrtf(n2) * inv_onorm * __builtin_amdgcn_rcpf(keep);
          } else {
            ratio = n2 > 0.f ? INFINITY : 0.f;
          }
        }
        if (!ri.ok) ratio = 0.f;
        unsigned int* rm = &sRm[(item - i_begin) * n_heads_blk + my_hl];
        if (wave_one_head) {
          float wm = ratio;
#pragma unroll
          for (int off = 16; off >= 1; off >>= 1) wm = fmaxf(wm, __shfl_xor(wm, off, 64));
          if (lane == 0 && ri.ok) atomicMax(rm, __float_as_uint(wm));
        } else if (ri.ok && half == 0) {
          atomicMax(rm, __float_as_uint(ratio));
        }
      } else if (ri.ok) {
        const size_t base_i = (size_t)ri.rg * pw.n_items + item;
        if (half == 0) {
          pw.resA[base_i] = A;
          pw.resC[base_i] = c;
        }
      }
    }
  };
  auto process = [&](int b, int it, int m) {
    if (!wave_on) return;
    page(b, it, m, 0);
    if (m == 2) page(b, it + 1, m, 1);
  };

  St st;
  issue_tile(st, 0);
  st.commit(sK[0], sV[0], sP[0], sFull[0], minq, tid);
  __syncthreads();
  for (int k = 0; k < n_tiles; ++k) {
    const int b = k & 1;
    const int t_cur = sTileIt[k], m = sTileIt[k + 1] - t_cur;
    issue_tile(st, k + 1);
    process(b, t_cur, m);
    // unconditional: after the last tile an empty tile goes to the idle
    // buffer, so no path leaves a load outstanding into the next iteration
    st.commit(sK[b ^ 1], sV[b ^ 1], sP[b ^ 1], sFull[b ^ 1], minq, tid);
    __syncthreads();
  }
  if (MODE == 0) {
    // Eq. (7): maxima over the block's rows, per head and over heads
    const int n_it = i_end - i_begin;
    for (int i = tid; i < n_it; i += NT) {
      const int page = i_begin + i;
      unsigned int mx = 0u;
      for (int hl = 0; hl < n_heads_blk; ++hl) {
        const unsigned int v = sRm[i * n_heads_blk + hl];
        mx = max(mx, v);
        if (pw.R_head)
          atomic_max_nonneg(&pw.R_head[CKV_IDX((size_t)page * pw.Hq + g * a.group + head0 + hl,
                                               (int64_t)pw.n_pages * pw.Hq, a.dbg, 5)],
                            __uint_as_float(v));
      }
      atomic_max_nonneg(&pw.R[CKV_IDX(page, pw.n_pages, a.dbg, 5)], __uint_as_float(mx));
    }
    const int nf = min(sFixN, kRowsWG);
    if (nf > 0) {
      if (tid == 0) sFixBase = atomicAdd(pw.fix_count, nf);
      __syncthreads();
      for (int i = tid; i < nf; i += NT) {
        const int slot = sFixBase + i;
        if (slot < pw.fix_cap) reinterpret_cast<int4*>(pw.fix_list)[slot] = sFix[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// B'. fix-up of ill-conditioned (page, row) pairs: o' = output without the
// page from the other splits' partial sums plus the page's own split(s)
// recomputed in float32 with the page excluded; ratio = ||o - o'|| / ||o||.
//
// Each listed pair is spread over kFixParts workgroups: part j takes the
// other splits s = j (mod kFixParts) and the j-th segment of the page's own
// split(s), with every load of a 128-token round in flight at once, and
// stores its partial sums (fixed order inside the part).  The part that
// finishes last (an arrival count per pair) adds the parts in order (so the
// result does not depend on scheduling) and takes the ratio.  The sums cross
// workgroups through agent-scope atomic stores and loads, which bypass the
// per-XCD L2, so no cache-wide fence is needed; the workgroup barrier before
// the arrival waits for the stores.  Weights are taken relative to the row's
// log-sum-exp (every weight <= 1).
// ---------------------------------------------------------------------------
constexpr int kFixT = 256;        // threads of a fix-up workgroup
constexpr int kFixGrid = 1024;    // (pair, part) items in flight

constexpr int kFixMinSeg = 256;   // tokens of the page's split per part, at least, when parts grow
constexpr int kFixPartsMax = 32;

// parts per listed pair: within an item budget for n pairs; or, without one,
// at least `parts`, and more while the n pairs leave fix-up blocks idle and
// each part still takes kFixMinSeg tokens of a split of `chunk` (the partial
// sums buffer holds cap x parts entries)
__device__ __forceinline__ int fix_parts(int parts, int item_budget, int n, int nb, int chunk, int cap) {
  const int m = max(n, 1);
  if (item_budget > 0) return max(1, min(parts, item_budget / m));
  const int grow = min(min(nb / m, chunk / kFixMinSeg), kFixPartsMax);
  return max(parts, min(grow, cap * parts / m));
}

// ratio of listed pair e from its parts' sums (one wave)
template <int D>
__device__ void fixup_ratio(const AttnGeom& a, const RowStats& rs, const PageWork& pw, const float* fpart, int e,
                            int parts, int lane) {
  const int4 ent = reinterpret_cast<const int4*>(pw.fix_list)[e];
  const int page = (int)CKV_IDX(ent.x, pw.n_pages, a.dbg, 8), rg = (int)CKV_IDX(ent.y, a.Hq * a.W, a.dbg, 7);
  const int h = rg / a.W;
  const float* fp = fpart + (size_t)e * parts * (D + 1);
  auto ld = [](const float* p) {
    return __uint_as_float(__hip_atomic_load(reinterpret_cast<const unsigned*>(p), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT));
  };
  float num[D / 64], den = 0.f;
#pragma unroll
  for (int j = 0; j < D / 64; ++j) num[j] = 0.f;
#pragma unroll 8
  for (int part = 0; part < parts; ++part) {
#pragma unroll
    for (int j = 0; j < D / 64; ++j) num[j] += ld(fp + part * (D + 1) + lane + 64 * j);
    den += ld(fp + part * (D + 1) + D);
  }
  float dd = 0.f, oo = 0.f;
#pragma unroll
  for (int j = 0; j < D / 64; ++j) {
    const float ov = rs.o[(size_t)rg * D + lane + 64 * j];
    const float od = den > 0.f ? num[j] / den : 0.f;
    dd += (ov - od) * (ov - od);
    oo += ov * ov;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    dd += __shfl_xor(dd, off, 64);
    oo += __shfl_xor(oo, off, 64);
  }
  if (lane == 0) {
    float ratio;
    if (!(den > 0.f)) ratio = INFINITY;
    else if (oo > 0.f) ratio = sqrtf(dd) / sqrtf(oo);
    else ratio = dd > 0.f ? INFINITY : 0.f;
    if (pw.R_head) atomic_max_nonneg(&pw.R_head[(size_t)page * pw.Hq + h], ratio);
    atomic_max_nonneg(&pw.R[page], ratio);
  }
}

// Eq. (6)-(7) for a listed pair whose page lies in tiles with known window
// references (see rescaled_entry): its first nf tokens were weighted in
// float16 against the split's older reference, and the running output was
// rescaled by 2^(older - largest) when the largest logit arrived; the rest
// against the largest.  One wave takes the same weights (the key fragments
// and the query in the layout and product chain of the window pass, so the
// scores are bit-identical), rescales the first part's sums the same way and
// evaluates the closed form; the cancellation in u - A o then loses only
// float32 digits.
template <int D, bool PG>
__device__ void rescaled_pair(const AttnGeom& a, const RowStats& rs, const PageWork& pw, const int4 ent,
                              int nf, int lane) {
  constexpr int KS = D / 16;
  const int half = lane >> 5, col = lane & 31;
  const int page = (int)CKV_IDX(ent.x, pw.n_pages, a.dbg, 8), rg = (int)CKV_IDX(ent.y, a.Hq * a.W, a.dbg, 7);
  const int st = ent.z, ln = ent.w & 0xFF;
  const int h = rg / a.W, p = rg % a.W, g = h / a.group;
  const int qp = a.qpos[p];
  const float M = rs.m2[rg], mprev = rs.m2p[rg];
  const float alpha = __builtin_amdgcn_exp2f(mprev - M);
  __shared__ float sW[32];   // one block's weights
  const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride;
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;
  auto krow = [&](int t) -> int64_t { return PG ? (int64_t)min((uint32_t)a.slot[t], a.pool_last) : t; };
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = load_bf16x8(qrow + 16 * ks + 8 * half);
  constexpr int DPL = D / 64;   // widths per lane: lane * DPL .. lane * DPL + DPL - 1
  float l1 = 0.f, l2 = 0.f;      // weight sums of the first and the second part
  float u1[DPL], u2[DPL];        // U over each part, at this lane's widths
#pragma unroll
  for (int j = 0; j < DPL; ++j) u1[j] = u2[j] = 0.f;
  // one 32-token block at a time (every column of the product is the same row)
#pragma unroll 1
  for (int tb = 0; tb < 2 && 32 * tb < ln; ++tb) {
    const int nb = min(32, ln - 32 * tb);
    // the block's value rows, loaded before its products (this lane's widths)
    uint32_t vraw[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const uint16_t* vr = vh + krow(st + min(32 * tb + i, ln - 1)) * a.kv_tok_stride + lane * DPL;
      vraw[i] = DPL == 2 ? *reinterpret_cast<const uint32_t*>(vr) : (uint32_t)vr[0];
    }
    const int ok_tok = 32 * tb + col < ln;
    const uint16_t* kr = kh + krow(ok_tok ? st + 32 * tb + col : st) * a.kv_tok_stride;
    f32x16 acc = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = mfma_bf16(ok_tok ? load_bf16x8(kr + 16 * ks + 8 * half) : zero_bf16x8(), qf[ks], acc);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int o = 32 * tb + 8 * (r >> 2) + 4 * half + (r & 3);
      const bool vis = o < ln && a.pos[st + min(o, ln - 1)] <= qp;
      const float ref = o < nf ? mprev : M;
      const float x = vis ? __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r], a.sl2, -ref)) : 0.f;
      acc[r] = (float)(_Float16)x;
      if (o < nf) l1 += acc[r];
      else l2 += acc[r];
    }
    // the block's weights through LDS (lanes 0 and 32 hold the two halves)
    if (col == 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sW[8 * (r >> 2) + 4 * half + (r & 3)] = acc[r];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      if (i < nb) {
        const int o = 32 * tb + i;
        const float wt = sW[i];
#pragma unroll
        for (int j = 0; j < DPL; ++j) {
          // through float16, as the window pass converted the values
          const float v = (float)(_Float16)bf16_bits_to_float((vraw[i] >> (16 * j)) & 0xFFFFu);
          if (o < nf) u1[j] = __builtin_fmaf(wt, v, u1[j]);
          else u2[j] = __builtin_fmaf(wt, v, u2[j]);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
  // token sums over both halves (lanes l and l ^ 32 hold the two halves)
  l1 += __shfl_xor(l1, 32, 64);
  l2 += __shfl_xor(l2, 32, 64);
  const float lhat = alpha * l1 + l2;
  float n2 = 0.f;
#pragma unroll
  for (int j = 0; j < DPL; ++j) {
    const float ov = rs.o[(size_t)rg * D + lane * DPL + j];
    const float uj = __builtin_fmaf(alpha, u1[j], u2[j]) - lhat * ov;
    n2 = __builtin_fmaf(uj, uj, n2);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
  if (lane == 0) {
    const float f = __builtin_amdgcn_exp2f(M - rs.lse2[rg] * pw.lse_scale);
    const float keep = 1.f - f * lhat;
    const float onorm = rs.onorm[rg];
    float ratio;
    if (onorm > 0.f) ratio = keep > 0.f ? f * sqrtf(n2) / (onorm * keep) : INFINITY;
    else ratio = n2 > 0.f ? INFINITY : 0.f;
    if (pw.R_head) atomic_max_nonneg(&pw.R_head[(size_t)page * pw.Hq + h], ratio);
    atomic_max_nonneg(&pw.R[page], ratio);
  }
}

// A listed pair with A <= fix_a_hi (flagged by the page kernel) whose page
// lies in tiles whose window-pass references are known: in the first split
// that holds the row's largest logit, the tile before the one where it
// entered (reference m2p, rescaled when it entered) and every tile from that
// one on (reference m2).  Returns the page's tokens before that tile (the
// ones weighted against m2p), or -1 if the pair is not such a pair; every
// part of the pair takes the same decision.
__device__ __forceinline__ int rescaled_entry(const AttnSplit& sp, const RowStats& rs, const int4 ent) {
  if (!(ent.w & kFixRescaled) || !rs.m2t || !rs.m2p) return -1;
  const int st = ent.z, ln = ent.w & 0xFF, mt = rs.m2t[ent.y];
  if (mt < 0) return -1;
  const int first = st / kTile * kTile, last = (st + ln - 1) / kTile * kTile;
  const int s_lo = mt / sp.chunk * sp.chunk, s_hi = s_lo + sp.chunk;
  if (first < mt - kTile || first < s_lo || last >= s_hi) return -1;
  return min(max(mt - st, 0), ln);
}

// the fix-up of block bx of nb fix-up blocks, each of T threads
template <int D, bool PG, int T>
__device__ __forceinline__ void page_fixup_body(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs,
                                                const PageWork& pw, float* fpart, int* arrive, int parts,
                                                int item_budget, int bx, int nb) {
  constexpr int TPR = D / 8;                  // threads per token row (16 bytes each)
  constexpr int RPR = T / TPR;                // token rows per round
  constexpr int UNR = 128 / RPR;              // rounds whose loads are in flight together
  __shared__ float sacc[RPR][D + 1];
  __shared__ int sLast;
  const int tid = threadIdx.x, c = tid % TPR, r = tid / TPR;
  const int n = min(*pw.fix_count, pw.fix_cap);
  parts = fix_parts(parts, item_budget, n, nb, sp.chunk, pw.fix_cap);
  for (int item = bx; item < n * parts; item += nb) {
    const int e = item / parts, part = item % parts;
    // entry: page, global row, page start, page length
    const int4 ent = reinterpret_cast<const int4*>(pw.fix_list)[e];
    const int nf_resc = rescaled_entry(sp, rs, ent);
    if (nf_resc >= 0) {   // evaluated with the window pass's own weights, by one wave
      if (part == 0 && tid < 64) rescaled_pair<D, PG>(a, rs, pw, ent, nf_resc, tid);
      continue;
    }
    const int rg = (int)CKV_IDX(ent.y, a.Hq * a.W, a.dbg, 7), st = ent.z, ln = ent.w & 0xFF;
    const int h = rg / a.W, p = rg % a.W, g = h / a.group, row = rg - g * a.rows;
    const int qp = a.qpos[p];
    const float ref = rs.lse2[rg];
    const int s0 = st / sp.chunk, s1 = (st + ln - 1) / sp.chunk;
    // this part's segment of the page's split(s): its first round of loads
    // is issued before the other splits' partial sums are read
    const int t_lo = s0 * sp.chunk, t_hi = min(a.S, (s1 + 1) * sp.chunk);
    const int seg = (((t_hi - t_lo + parts - 1) / parts) + RPR - 1) / RPR * RPR;
    const int a0 = t_lo + part * seg, a1 = min(t_hi, a0 + seg);
    const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
    const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;
    const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride;
    const u32x4 qc = ldg_u4(qrow + 8 * c);
    u32x4 kc[UNR], vc[UNR];
    int pv[UNR];
    auto load_round = [&](int b0) {
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int t = max(a0, min(b0 + u * RPR + r, a1 - 1));
        const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[t], a.pool_last) : t;
        kc[u] = ldg_u4(kh + row * a.kv_tok_stride + 8 * c);
        vc[u] = ldg_u4(vh + row * a.kv_tok_stride + 8 * c);
        pv[u] = ldg_i32(a.pos + t);
      }
    };
    if (a0 < a1) load_round(a0);
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    float lacc = 0.f;
    // other splits' partial sums as they are: this part's splits, one per row group
    for (int s = part + parts * r; s < sp.n_splits; s += parts * RPR) {
      if (s >= s0 && s <= s1) continue;
      const size_t idx = (size_t)(g * sp.n_splits + s) * sp.rows_pad + row;
      const float ms = sp.part_m[idx];
      const float w = ms == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms - ref);
      const u32x4 o0 = ldg_u4(sp.part_o + idx * D + 8 * c);
      const u32x4 o1 = ldg_u4(sp.part_o + idx * D + 8 * c + 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[j] = __builtin_fmaf(w, __uint_as_float(o0[j]), acc[j]);
        acc[4 + j] = __builtin_fmaf(w, __uint_as_float(o1[j]), acc[4 + j]);
      }
      if (c == 0) lacc = __builtin_fmaf(w, sp.part_l[idx], lacc);
    }
    // the segment without the page, in float32
    if (a0 < a1) {
      float qv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) qv[j] = bf16_bits_to_float(chunk_elem(qc, j));
      for (int b0 = a0; b0 < a1; b0 += UNR * RPR) {
        if (b0 != a0) load_round(b0);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int t = b0 + u * RPR + r;
          float x = 0.f;
#pragma unroll
          for (int j = 0; j < 8; ++j) x = __builtin_fmaf(qv[j], bf16_bits_to_float(chunk_elem(kc[u], j)), x);
#pragma unroll
          for (int off = TPR / 2; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
          const bool keep = t < a1 && pv[u] <= qp && !(t >= st && t < st + ln);
          const float w = keep ? __builtin_amdgcn_exp2f(__builtin_fmaf(x, a.sl2, -ref)) : 0.f;
#pragma unroll
          for (int j = 0; j < 8; ++j)
            acc[j] = __builtin_fmaf(w, bf16_bits_to_float(chunk_elem(vc[u], j)), acc[j]);
          if (c == 0) lacc += w;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) sacc[r][8 * c + j] = acc[j];
    if (c == 0) sacc[r][D] = lacc;
    __syncthreads();
    // the part's sums: row groups added in order
    float* out = fpart + ((size_t)e * parts + part) * (D + 1);
    for (int i = tid; i <= D; i += T) {
      float v = 0.f;
      for (int k = 0; k < RPR; ++k) v += sacc[k][i];
      __hip_atomic_store(reinterpret_cast<unsigned*>(out + i), __float_as_uint(v), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (tid == 0)
      sLast = __hip_atomic_fetch_add(&arrive[e], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == parts - 1;
    __syncthreads();
    if (sLast && tid < 64) fixup_ratio<D>(a, rs, pw, fpart, e, parts, tid);
  }
}

template <int D, bool PG>
__global__ __launch_bounds__(kFixT) void page_fixup_kernel(AttnGeom a, AttnSplit sp, RowStats rs, PageWork pw,
                                                           float* fpart, int* arrive, int parts, int item_budget) {
  page_fixup_body<D, PG, kFixT>(a, sp, rs, pw, fpart, arrive, parts, item_budget, blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
// C. window-attention mass of every token: max_h sum_p a_hpi
//
// Workgroup (token chunk, KV head g).  A (query head, 32-row block) pair is
// one wave's unit of work: its scores use the C = Q K^T orientation (tokens
// on lanes, rows in registers), so the sum over the block's rows is
// lane-local.  Pair sums go to LDS; a query head's rows are then added in a
// fixed block order (deterministic) and the max over heads is taken.
// ---------------------------------------------------------------------------
constexpr int kMassMaxRows = 2048;   // window rows per KV head the mass kernel supports
constexpr int kMassMaxPairs = kMassMaxRows / 32;

template <int D, bool PG>
__global__ __launch_bounds__(kNW * 64) void token_mass_kernel(AttnGeom a, RowStats rs, float* mass,
                                                              int chunk) {
  constexpr int NT = kNW * 64, KS = D / 16;
  constexpr int KP = D + 8, CPR = D / 8, KCH = kTile * CPR, KPT = (KCH + NT - 1) / NT;
  __shared__ __align__(16) uint16_t sK[2][kTile * KP];
  __shared__ int sP[2][kTile];
  __shared__ float sPart[kMassMaxPairs][kTile];
  __shared__ float sL2[kMassMaxRows];
  __shared__ int sQP[kMassMaxRows];
  const int g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int t_begin = blockIdx.x * chunk;
  const int t_end = min(a.S, t_begin + chunk);
  if (t_begin >= t_end) return;
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const int nrb = (a.W + 31) / 32;
  const int n_pairs = a.group * nrb;
  for (int r = tid; r < a.rows; r += NT) {
    sL2[r] = rs.lse2[g * a.rows + r];
    sQP[r] = a.qpos[r % a.W];
  }
  u32x4 kr[KPT];
  int pr = INT_MAX;
  auto issue = [&](int t0) {
    const int nv = min(kTile, t_end - t0);
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      const int tr = (c / CPR) & (kTile - 1);
      const bool ok = c < KCH && tr < nv;
      const int tk = ok ? t0 + tr : 0;
      const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[tk], a.pool_last) : tk;
      const u32x4 v = ldg_u4(kh + row * a.kv_tok_stride + (c % CPR) * 8);
      kr[i] = ok ? v : u32x4{0u, 0u, 0u, 0u};
    }
    const bool okp = tid < nv;
    const int pv = ldg_i32(a.pos + (okp ? t0 + tid : 0));
    pr = okp ? pv : INT_MAX;
  };
  auto commit = [&](int b) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      if (c < KCH) *reinterpret_cast<u32x4*>(&sK[b][(c / CPR) * KP + (c % CPR) * 8]) = kr[i];
    }
    if (tid < kTile) sP[b][tid] = pr;
  };
  const int n_tiles = (t_end - t_begin + kTile - 1) / kTile;
  issue(t_begin);
  commit(0);
  __syncthreads();
  for (int it = 0; it < n_tiles; ++it) {
    const int b = it & 1;
    const int t0 = t_begin + it * kTile;
    if (it + 1 < n_tiles) issue(t0 + kTile);
    for (int pi = wave; pi < n_pairs; pi += kNW) {
      const int hl = pi / nrb, rb = pi % nrb;
      const int h = g * a.group + hl;
      const int prow = 32 * rb + col;          // A operand row of this lane
      const bool aok = prow < a.W;
      const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)(aok ? prow : 0) * a.q_row_stride;
      bf16x8 qa[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qa[ks] = aok ? load_bf16x8(qrow + 16 * ks + 8 * half) : zero_bf16x8();
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        f32x16 acc = zero16();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          acc = mfma_bf16(qa[ks], load_bf16x8(&sK[b][(32 * tb + col) * KP + 16 * ks + 8 * half]), acc);
        const int pt = sP[b][32 * tb + col];
        float msum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int p = 32 * rb + 8 * (r >> 2) + 4 * half + (r & 3);
          if (p < a.W) {
            const int row = hl * a.W + p;
            const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r], a.sl2, -sL2[row]));
            msum += pt <= sQP[row] ? e : 0.f;
          }
        }
        msum += xor32(msum);
        if (half == 0) sPart[pi][32 * tb + col] = msum;
      }
    }
    if (it + 1 < n_tiles) commit(b ^ 1);
    __syncthreads();
    if (tid < kTile && t0 + tid < t_end) {
      float best = 0.f;
      bool bad = false;
      for (int hl = 0; hl < a.group; ++hl) {
        float sum = 0.f;
        for (int rb = 0; rb < nrb; ++rb) sum += sPart[hl * nrb + rb][tid];
        bad |= !(sum <= 3.4e38f);   // a NaN or infinite weight (e.g. a row's lse of -inf)
        best = fmaxf(best, sum);
      }
      if (bad) latch_nonfinite(a.nonfinite);
      atomic_max_nonneg(&mass[t0 + tid], best);
    }
    __syncthreads();
  }
}

// The same with every (query head, 32-row block) pair of the workgroup owned
// by one wave for the whole launch (PPW pairs per wave): the wave's query
// fragments, log-sum-exp and window positions stay in registers, keys are
// loaded two tiles ahead, and a tile whose positions are all <= the smallest
// window position skips the visibility test.  Workgroup z takes pairs
// [8 PPW z, 8 PPW (z+1)), whole heads only (8 PPW is a multiple of the row
// blocks per head); heads of other z-slices meet in the atomic max.
template <int D, int PPW, bool PG>
__device__ __forceinline__ void token_mass_body(const AttnGeom& a, const RowStats& rs, float* mass, int chunk,
                                                int bx, int by, int bz) {
  constexpr int NT = kNW * 64, KS = D / 16;
  constexpr int KP = D + 8, CPR = D / 8, KCH = kTile * CPR, KPT = (KCH + NT - 1) / NT;
  constexpr int NP = kNW * PPW;                 // pairs per workgroup
  __shared__ __align__(16) uint16_t sK[2][kTile * KP];
  __shared__ int sP[2][kTile];
  __shared__ int sFull[2];
  __shared__ float sPart[2][NP][kTile];
  __shared__ int sMin;
  const int g = by;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int t_begin = bx * chunk;
  const int t_end = min(a.S, t_begin + chunk);
  if (t_begin >= t_end) return;
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const int nrb = (a.W + 31) / 32;
  const int n_pairs = a.group * nrb;
  const int p0 = bz * NP;
  const int np_blk = min(NP, n_pairs - p0);
  // smallest window position (every head has the same window rows)
  if (tid == 0) sMin = INT_MAX;
  __syncthreads();
  {
    int q = INT_MAX;
    for (int p = tid; p < a.W; p += NT) q = min(q, a.qpos[p]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) q = min(q, __shfl_xor(q, off, 64));
    if (lane == 0) atomicMin(&sMin, q);
  }
  __syncthreads();
  const int minq = sMin;

  bf16x8 qa[PPW][KS];
  float l2[PPW][16];
  int qp[PPW][16];
  bool pon[PPW];
#pragma unroll
  for (int j = 0; j < PPW; ++j) {
    const int pl = wave + kNW * j;               // pair inside the workgroup
    const int pi = p0 + pl;
    pon[j] = pl < np_blk;
    const int hl = pon[j] ? pi / nrb : 0, rb = pon[j] ? pi % nrb : 0;
    const int h = g * a.group + hl;
    const int prow = 32 * rb + col;            // A operand row of this lane
    const bool aok = pon[j] && prow < a.W;
    const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)(aok ? prow : 0) * a.q_row_stride;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qa[j][ks] = aok ? load_bf16x8(qrow + 16 * ks + 8 * half) : zero_bf16x8();
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int p = 32 * rb + 8 * (r >> 2) + 4 * half + (r & 3);
      const bool ok = pon[j] && p < a.W;
      // rows outside the window get weight 0: -inf log-sum-exp offset
      l2[j][r] = ok ? rs.lse2[g * a.rows + hl * a.W + p] : INFINITY;
      qp[j][r] = ok ? a.qpos[p] : INT_MIN;
    }
  }

  struct KStage { u32x4 kr[KPT]; int pr; bool pok; };   // position used only in commit
  KStage sa, sb;
  const int n_tiles = (t_end - t_begin + kTile - 1) / kTile;
  auto issue = [&](KStage& st, int it) {
    const int t0 = t_begin + it * kTile;
    const int nv = it < n_tiles ? min(kTile, t_end - t0) : 0;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      const int tr = (c / CPR) & (kTile - 1);
      const bool ok = c < KCH && tr < nv;
      const int tk = ok ? t0 + tr : 0;
      const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[tk], a.pool_last) : tk;
      st.kr[i] = ldg_u4(kh + row * a.kv_tok_stride + (c % CPR) * 8);
    }
    st.pok = tid < nv;
    st.pr = ldg_i32(a.pos + (st.pok ? t0 + tid : 0));
  };
  auto commit = [&](const KStage& st, int b) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      if (c < KCH) *reinterpret_cast<u32x4*>(&sK[b][(c / CPR) * KP + (c % CPR) * 8]) = st.kr[i];
    }
    if (tid < kTile) {
      const int p = st.pok ? st.pr : INT_MAX;
      sP[b][tid] = p;
      const unsigned long long late = __ballot(p > minq);
      if (tid == 0) sFull[b] = late == 0ull;
    }
  };
  auto compute = [&](int b, int it) {
    const bool full = sFull[b];
#pragma unroll
    for (int j = 0; j < PPW; ++j) {
      if (!pon[j]) continue;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        f32x16 acc = zero16();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          acc = mfma_bf16(qa[j][ks], load_bf16x8(&sK[b][(32 * tb + col) * KP + 16 * ks + 8 * half]), acc);
        float msum = 0.f;
        if (full) {
#pragma unroll
          for (int r = 0; r < 16; ++r) msum += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r], a.sl2, -l2[j][r]));
        } else {
          const int pt = sP[b][32 * tb + col];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r], a.sl2, -l2[j][r]));
            msum += pt <= qp[j][r] ? e : 0.f;
          }
        }
        msum = sum32(msum);
        if (half == 0) sPart[it & 1][wave + kNW * j][32 * tb + col] = msum;
      }
    }
  };
  // threads 0..63: sum a head's row blocks, max over the heads of the workgroup
  auto reduce = [&](int it) {
    const int t0 = t_begin + it * kTile;
    if (tid < kTile && t0 + tid < t_end) {
      float best = 0.f;
      bool bad = false;
      for (int hp = 0; hp < np_blk; hp += nrb) {
        float sum = 0.f;
        for (int rb = 0; rb < nrb; ++rb) sum += sPart[it & 1][hp + rb][tid];
        bad |= !(sum <= 3.4e38f);   // a NaN or infinite weight (e.g. a row's lse of -inf)
        best = fmaxf(best, sum);
      }
      if (bad) latch_nonfinite(a.nonfinite);
      atomic_max_nonneg(&mass[t0 + tid], best);
    }
  };
  issue(sa, 0);
  issue(sb, 1);
  commit(sa, 0);
  __syncthreads();
  for (int it = 0; it < n_tiles; it += 2) {
    issue(sa, it + 2);
    compute(0, it);
    if (it + 1 < n_tiles) commit(sb, 1);
    __syncthreads();
    reduce(it);
    if (it + 1 >= n_tiles) break;
    issue(sb, it + 3);
    compute(1, it + 1);
    if (it + 2 < n_tiles) commit(sa, 0);
    __syncthreads();
    reduce(it + 1);
  }
}

template <int D, int PPW, bool PG>
__global__ __launch_bounds__(kNW * 64) void token_mass_fast(AttnGeom a, RowStats rs, float* mass, int chunk) {
  token_mass_body<D, PPW, PG>(a, rs, mass, chunk, blockIdx.x, blockIdx.y, blockIdx.z);
}

// The fix-up of the listed pairs and the token mass in one launch (the post
// pass runs both after the page kernel): blocks [0, nfix) are fix-up
// blocks, the rest the token-mass grid (mx x my x mz) in x-fastest order.
// The fix-up is a short chain of dependent latencies; here it runs in the
// shadow of the token mass instead of taking a launch of its own.
template <int D, int PPW, bool PG>
__global__ __launch_bounds__(kNW * 64) void mass_fixup_kernel(AttnGeom a, AttnSplit sp, RowStats rs, PageWork pw,
                                                              float* fpart, int* arrive, int parts, float* mass,
                                                              int chunk, int nfix, int mx, int my) {
  if ((int)blockIdx.x < nfix) {
    page_fixup_body<D, PG, kNW * 64>(a, sp, rs, pw, fpart, arrive, parts, 0, blockIdx.x, nfix);
    return;
  }
  const int b = blockIdx.x - nfix;
  token_mass_body<D, PPW, PG>(a, rs, mass, chunk, b % mx, (b / mx) % my, b / (mx * my));
}


// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
int rows_per_block_attention() { return kRowsWG; }
int rows_per_block_page() { return kRowsWG; }
int page_heads_per_block(int W, int group) { return std::min(group, (kRowsWG - 1) / W + 2); }
int token_mass_max_rows() { return kMassMaxRows; }

hipError_t launch_window_attention(const AttnGeom& a, const AttnSplit& sp, hipStream_t s) {
  const int nrb = (a.rows + kRowsWG - 1) / kRowsWG;
  dim3 grid(sp.n_splits, nrb, a.Hkv), block(kNW * 64);
  const bool pg = a.slot != nullptr;
  if (a.D == 128) {
    if (pg) hipLaunchKernelGGL((window_attention_kernel<128, true>), grid, block, 0, s, a, sp);
    else hipLaunchKernelGGL((window_attention_kernel<128, false>), grid, block, 0, s, a, sp);
  } else {
    if (pg) hipLaunchKernelGGL((window_attention_kernel<64, true>), grid, block, 0, s, a, sp);
    else hipLaunchKernelGGL((window_attention_kernel<64, false>), grid, block, 0, s, a, sp);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs, float* lse_out,
                          const ZeroList& zl, hipStream_t s) {
  const int waves = (a.Hkv * a.rows * a.D + 255) / 256;   // 256 / D rows per wave
  dim3 grid((waves + 3) / 4), block(256);
  if (a.D == 128) hipLaunchKernelGGL((combine_kernel<128>), grid, block, 0, s, a, sp, rs, lse_out, zl);
  else hipLaunchKernelGGL((combine_kernel<64>), grid, block, 0, s, a, sp, rs, lse_out, zl);
  return hipGetLastError();
}

hipError_t launch_page_kernel(const AttnGeom& a, const PageWork& pw, const RowStats& rs, int mode,
                              int max_len, hipStream_t s) {
  const int nrb = (a.rows + kRowsWG - 1) / kRowsWG;
  const int nblk = (pw.n_items + pw.items_per_block - 1) / pw.items_per_block;
  if (nblk == 0) return hipSuccess;
  dim3 grid(nblk, nrb, a.Hkv), block(kNW * 64);
  const bool two = max_len > 32, pg = a.slot != nullptr;
#define CKV_PAGE_LAUNCH(DD, MM)                                                                   \
  do {                                                                                            \
    if (pg) {                                                                                     \
      if (two) hipLaunchKernelGGL((page_kernel<DD, MM, 2, true>), grid, block, 0, s, a, pw, rs);  \
      else hipLaunchKernelGGL((page_kernel<DD, MM, 1, true>), grid, block, 0, s, a, pw, rs);      \
    } else {                                                                                      \
      if (two) hipLaunchKernelGGL((page_kernel<DD, MM, 2, false>), grid, block, 0, s, a, pw, rs); \
      else hipLaunchKernelGGL((page_kernel<DD, MM, 1, false>), grid, block, 0, s, a, pw, rs);     \
    }                                                                                             \
  } while (0)
  if (a.D == 128) {
    if (mode == 0) CKV_PAGE_LAUNCH(128, 0);
    else CKV_PAGE_LAUNCH(128, 1);
  } else {
    if (mode == 0) CKV_PAGE_LAUNCH(64, 0);
    else CKV_PAGE_LAUNCH(64, 1);
  }
#undef CKV_PAGE_LAUNCH
  return hipGetLastError();
}

hipError_t launch_page_fixup(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs,
                             const PageWork& pw, float* fpart, int* arrive, int parts, int item_budget,
                             hipStream_t s) {
  dim3 grid(std::max(1, std::min(pw.fix_cap * parts, kFixGrid))), block(kFixT);
  const bool pg = a.slot != nullptr;
  const int ib = item_budget;
  if (a.D == 128) {
    if (pg) hipLaunchKernelGGL((page_fixup_kernel<128, true>), grid, block, 0, s, a, sp, rs, pw, fpart, arrive, parts, ib);
    else hipLaunchKernelGGL((page_fixup_kernel<128, false>), grid, block, 0, s, a, sp, rs, pw, fpart, arrive, parts, ib);
  } else {
    if (pg) hipLaunchKernelGGL((page_fixup_kernel<64, true>), grid, block, 0, s, a, sp, rs, pw, fpart, arrive, parts, ib);
    else hipLaunchKernelGGL((page_fixup_kernel<64, false>), grid, block, 0, s, a, sp, rs, pw, fpart, arrive, parts, ib);
  }
  return hipGetLastError();
}

bool mass_fixup_applies(const AttnGeom& a) {
  const int nrb = (a.W + 31) / 32, n_pairs = a.group * nrb;
  const int ppw = n_pairs <= kNW ? 1 : 2;
  return (kNW * ppw) % nrb == 0;
}

hipError_t launch_mass_fixup(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs, const PageWork& pw,
                             float* fpart, int* arrive, int parts, float* mass, int chunk, hipStream_t s) {
  if (!mass_fixup_applies(a)) return hipErrorInvalidValue;
  const int nrb = (a.W + 31) / 32, n_pairs = a.group * nrb;
  const int ppw = n_pairs <= kNW ? 1 : 2;
  const int nz = (n_pairs + kNW * ppw - 1) / (kNW * ppw);
  const int mx = (a.S + chunk - 1) / chunk, my = a.Hkv;
  const int nfix = kMassFixBlocks;
  dim3 grid(nfix + mx * my * nz), block(kNW * 64);
  const bool pg = a.slot != nullptr;
#define CKV_MF_LAUNCH(DD, PP)                                                                             \
  do {                                                                                                    \
    if (pg) hipLaunchKernelGGL((mass_fixup_kernel<DD, PP, true>), grid, block, 0, s, a, sp, rs, pw, fpart,  \
                               arrive, parts, mass, chunk, nfix, mx, my);                                 \
    else hipLaunchKernelGGL((mass_fixup_kernel<DD, PP, false>), grid, block, 0, s, a, sp, rs, pw, fpart,    \
                            arrive, parts, mass, chunk, nfix, mx, my);                                    \
  } while (0)
  if (a.D == 128) {
    if (ppw == 1) CKV_MF_LAUNCH(128, 1);
    else CKV_MF_LAUNCH(128, 2);
  } else {
    if (ppw == 1) CKV_MF_LAUNCH(64, 1);
    else CKV_MF_LAUNCH(64, 2);
  }
#undef CKV_MF_LAUNCH
  return hipGetLastError();
}

hipError_t launch_token_mass(const AttnGeom& a, const RowStats& rs, float* mass, int chunk,
                             hipStream_t s) {
  const int nrb = (a.W + 31) / 32, n_pairs = a.group * nrb;
  const int ppw = n_pairs <= kNW ? 1 : 2;
  const bool pg = a.slot != nullptr;
  if ((kNW * ppw) % nrb == 0) {
    const int nz = (n_pairs + kNW * ppw - 1) / (kNW * ppw);
    dim3 grid((a.S + chunk - 1) / chunk, a.Hkv, nz), block(kNW * 64);
#define CKV_MASS_LAUNCH(DD, PP)                                                                       \
  do {                                                                                                \
    if (pg) hipLaunchKernelGGL((token_mass_fast<DD, PP, true>), grid, block, 0, s, a, rs, mass, chunk); \
    else hipLaunchKernelGGL((token_mass_fast<DD, PP, false>), grid, block, 0, s, a, rs, mass, chunk);   \
  } while (0)
    if (a.D == 128) {
      if (ppw == 1) CKV_MASS_LAUNCH(128, 1);
      else CKV_MASS_LAUNCH(128, 2);
    } else {
      if (ppw == 1) CKV_MASS_LAUNCH(64, 1);
      else CKV_MASS_LAUNCH(64, 2);
    }
#undef CKV_MASS_LAUNCH
    return hipGetLastError();
  }
  dim3 grid((a.S + chunk - 1) / chunk, a.Hkv), block(kNW * 64);
  if (a.D == 128) {
    if (pg) hipLaunchKernelGGL((token_mass_kernel<128, true>), grid, block, 0, s, a, rs, mass, chunk);
    else hipLaunchKernelGGL((token_mass_kernel<128, false>), grid, block, 0, s, a, rs, mass, chunk);
  } else {
    if (pg) hipLaunchKernelGGL((token_mass_kernel<64, true>), grid, block, 0, s, a, rs, mass, chunk);
    else hipLaunchKernelGGL((token_mass_kernel<64, false>), grid, block, 0, s, a, rs, mass, chunk);
  }
  return hipGetLastError();
}

}  // namespace ckv
