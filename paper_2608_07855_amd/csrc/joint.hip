// Greedy joint retirement test (CommitKV, Sec. 3.3, Eq. (11), Algorithm 1).
//
// For a page set X deleted at once, Eq. (6) gives, per window row,
//   o - o^{\X} = (sum_{E in X} r_E) / (1 - sum_{E in X} A_E),
//   r_E = sum_{i in E} a_i v_i - A_E o,
// so the union effect follows from per-page residuals r_E (computed once per
// candidate by the page kernel in residual mode) and the running sums
// D = sum_{E in A} r_E, A_A = sum_{E in A} A_E over the accepted set A.
//
// The greedy loop is evaluated in speculative rounds: a round tests the next
// `window` candidates against the same accepted set (each test is exact,
// because all earlier candidates are decided); the first one that passes is
// accepted, the ones before it are rejected, and the ones after it are
// tested again in the next round.  The accepted candidate's residual is
// folded into the state by the next round while it copies the state into
// the other buffer (double buffering, so no block reads a row another block
// is writing).
//
// All rounds run in one launch of at most as many workgroups as the device
// holds at once: phase 0 clears the state and computes ||o_p|| and the
// visible-token counts, then a grid barrier ends each round's tests, block 0
// takes the decision, and a second barrier publishes it.  The candidate count
// is read on the device, so the call needs no host round trip; each round
// decides at least one candidate, so the loop ends within max_cand rounds.
// A barrier wait is bounded: if the workgroups cannot all run at once (a
// device shared with other work), every block leaves and *n_accepted = -1.
//
// A union that holds nearly all of a row's attention mass makes Eq. (6)
// ill-conditioned: o - o^{\X} = D / (1 - A_X) divides float32 cancellation
// by a small 1 - A_X.  A (candidate, row) pair whose union mass exceeds
// kJointFixA is therefore left out of the closed form and listed; after the
// round's tests every workgroup recomputes the listed pairs by definition --
// the row's output over the tokens outside the union, o', in float32 from
// the keys and values -- and the ratio ||o - o'|| / ||o|| joins the
// candidate's maximum before the decision.
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <algorithm>
#include <climits>

namespace ckv {

// control words (cleared by the residual pass before this kernel starts)
enum { kCursor = 0, kPending = 1, kBarrier = 2, kError = 3, kParity = 4, kFixN = 5 };
constexpr int kVisSlice = 8192;                         // tokens per visible-count item

// Grid barrier: thread 0 of every block publishes the block's writes, adds
// one arrival and waits until the arrivals reach `target`.  Returns false
// (in every thread) if the wait timed out or another block gave up.
__device__ bool grid_barrier(int* ctrl, int target, long long timeout, int* s_ok) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    atomicAdd(&ctrl[kBarrier], 1);
    const long long t0 = wall_clock64();
    int ok = 1;
    if (timeout <= 0) {   // a zero bound gives up at once: the failure path, forced
      __hip_atomic_store(&ctrl[kError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ok = 0;
    }
    while (ok && __hip_atomic_load(&ctrl[kBarrier], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(&ctrl[kError], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
          wall_clock64() - t0 >= timeout) {
        __hip_atomic_store(&ctrl[kError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    __threadfence();
    *s_ok = ok;
  }
  __syncthreads();
  return *s_ok != 0;
}

// The same barrier without the fences: for phases whose cross-workgroup
// data moves only through agent-scope atomics (a fence writes back and
// invalidates the whole L2 of the workgroup's XCD, which costs more than
// a round's work).  __syncthreads() first waits for the workgroup's own
// memory operations, so its atomics are performed before the arrival.
__device__ bool grid_barrier_nofence(int* ctrl, int target, long long timeout, int* s_ok) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(&ctrl[kBarrier], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long t0 = wall_clock64();
    int ok = 1;
    if (timeout <= 0) {   // a zero bound gives up at once: the failure path, forced
      __hip_atomic_store(&ctrl[kError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ok = 0;
    }
    while (ok && __hip_atomic_load(&ctrl[kBarrier], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(&ctrl[kError], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
          wall_clock64() - t0 >= timeout) {
        __hip_atomic_store(&ctrl[kError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *s_ok = ok;
  }
  __syncthreads();
  return *s_ok != 0;
}

__device__ __forceinline__ void store_pair(int* p, int2 v) {
  __hip_atomic_store(p, v.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(p + 1, v.y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int2 load_pair(const int* p) {
  return make_int2(__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                   __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// One candidate x row-block test item of a round (the body of a round):
// item (jx, rb) tests candidate cursor + jx on the rows of block rb and
// raises rbuf[jx] to its largest ratio; items with jx == 0 also copy the
// state (with the pending accepted residual folded in) into the other buffer.
__device__ void joint_item(const JointArgs& j, const RowStats& rs, int jx, int rb, int cursor, int pend,
                           int par, int n_eff, unsigned int* smax) {
  const int t = cursor + jx;
  const bool valid = t < n_eff;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = rb * j.rows_per_block;
  const int r1 = min(j.total_rows, r0 + j.rows_per_block);
  const size_t RD = (size_t)j.total_rows * j.D;
  const float* Din = j.Dstate + (size_t)par * RD;
  float* Dout = j.Dstate + (size_t)(par ^ 1) * RD;
  const float* Ain = j.Astate + (size_t)par * j.total_rows;
  float* Aout = j.Astate + (size_t)(par ^ 1) * j.total_rows;
  const int* Cin = j.Cstate + (size_t)par * j.total_rows;
  int* Cout = j.Cstate + (size_t)(par ^ 1) * j.total_rows;
  if (threadIdx.x == 0) *smax = 0u;
  __syncthreads();
  float wmax = 0.f;
  // a wave takes RB rows at a time (rows w, w + 4, ...) and issues every
  // load of the RB rows before the first use, so the rows' memory
  // latencies overlap instead of adding up
  constexpr int RB = 4, KD = 4;   // rows in flight per wave; width chunks of 64 (D <= 256)
  for (int base = r0 + wave; base < r1; base += 4 * RB) {
    float dv[RB][KD], rv[RB][KD], tv[RB][KD];
    float Acur[RB], At[RB], on[RB];
    int Ccur[RB], Ct[RB], nv[RB];
#pragma unroll
    for (int q = 0; q < RB; ++q) {
      const int row = base + 4 * q;
      const bool ok = row < r1;
      const int rr = ok ? row : r0;
      const float* rp =
          pend >= 0 ? j.resid + (size_t)CKV_IDX((size_t)rr * j.max_cand + pend, (int64_t)j.total_rows * j.max_cand,
                                                j.geo.dbg, 11) * j.D
                    : nullptr;
      const float* rt =
          valid ? j.resid + (size_t)CKV_IDX((size_t)rr * j.max_cand + t, (int64_t)j.total_rows * j.max_cand,
                                            j.geo.dbg, 11) * j.D
                : nullptr;
#pragma unroll
      for (int k = 0; k < KD; ++k) {
        const int d = lane + 64 * k;
        const bool dk = d < j.D;
        dv[q][k] = dk ? Din[(size_t)rr * j.D + d] : 0.f;
        rv[q][k] = (dk && rp) ? rp[d] : 0.f;
        tv[q][k] = (dk && rt) ? rt[d] : 0.f;
      }
      Acur[q] = Ain[rr];
      Ccur[q] = Cin[rr];
      if (pend >= 0) {
        Acur[q] += j.resA[(size_t)rr * j.max_cand + pend];
        Ccur[q] += j.resC[(size_t)rr * j.max_cand + pend];
      }
      At[q] = valid ? j.resA[(size_t)rr * j.max_cand + t] : 0.f;
      Ct[q] = valid ? j.resC[(size_t)rr * j.max_cand + t] : 0;
      on[q] = rs.onorm[rr];
      int c = 0;
      for (int sl = 0; sl < j.n_vis_slices; ++sl) c += j.nvis_part[(rr % j.W) * j.n_vis_slices + sl];
      nv[q] = c;
    }
#pragma unroll
    for (int q = 0; q < RB; ++q) {
      const int row = base + 4 * q;
      if (row >= r1) continue;
      float n2 = 0.f;
#pragma unroll
      for (int k = 0; k < KD; ++k) {
        const int d = lane + 64 * k;
        if (d < j.D) {
          const float x = dv[q][k] + rv[q][k];
          if (jx == 0) Dout[(size_t)row * j.D + d] = x;
          const float y = x + tv[q][k];
          n2 += y * y;
        }
      }
      if (jx == 0 && lane == 0) { Aout[row] = Acur[q]; Cout[row] = Ccur[q]; }
      if (!valid) continue;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
      const float Au = Acur[q] + At[q];
      const int Cu = Ccur[q] + Ct[q];
      float ratio = 0.f;
      if (Cu > 0) {
        const float keep = 1.f - Au;
        if (Cu >= nv[q]) {
          ratio = INFINITY;
        } else if (Au > kJointFixA) {
          // recomputed by definition after the round's tests
          if (lane == 0) {
            const int slot = atomicAdd(&j.ctrl[kFixN], 1);
            if (slot < j.window * j.total_rows) store_pair(j.fix_list + 2 * slot, make_int2(jx, row));
          }
        } else if (on[q] > 0.f) {
          ratio = sqrtf(n2) / (keep * on[q]);
        } else {
          ratio = n2 > 0.f ? INFINITY : 0.f;
        }
      }
      wmax = fmaxf(wmax, ratio);
    }
  }
  if (valid && lane == 0) atomicMax(smax, __float_as_uint(wmax));
  __syncthreads();
  if (threadIdx.x == 0 && valid) atomicMax(&j.rbuf[jx], *smax);
  __syncthreads();
}

// Block 0, thread 0, after a round's tests: the first candidate in order
// whose union maximum passes is accepted, the ones before it are rejected;
// the cursor moves past the decided candidates and the accepted one becomes
// the pending residual that the next round folds into the state.
__device__ void decide_round(const JointArgs& j, int cursor, int n_eff) {
  int cur = cursor, acc = -1;
  for (int k = 0; k < j.window; ++k) {
    const int tt = cursor + k;
    if (tt >= n_eff) break;
    const float r = __uint_as_float(__hip_atomic_load(&j.rbuf[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    if (j.union_R) j.union_R[tt] = r;
    cur = tt + 1;
    if (r <= j.tau || j.accept_all) {
      j.accepted[tt] = 1;
      acc = tt;
      *j.n_accepted += 1;
      const int ap = j.cand[tt];
      if (ap >= 0 && ap < j.n_pages) __hip_atomic_store(&j.in_acc[ap], (uint8_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
  }
  for (int k = 0; k < j.window; ++k) __hip_atomic_store(&j.rbuf[k], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kFixN], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kCursor], cur, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kPending], acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The decision of decide_round from per-candidate maxima held in LDS (the
// owned-row form); the global maxima are cleared for the next round.
constexpr int kTargetBlocksMax = 256;   // workgroups of the owned-row form at most
__device__ void decide_round_lds(const JointArgs& j, const unsigned int* sMax, int cursor, int n_eff) {
  int cur = cursor, acc = -1;
  for (int k = 0; k < j.window; ++k) {
    const int tt = cursor + k;
    if (tt >= n_eff) break;
    const float r = __uint_as_float(sMax[k]);
    if (j.union_R) j.union_R[tt] = r;
    cur = tt + 1;
    if (r <= j.tau || j.accept_all) {
      j.accepted[tt] = 1;
      acc = tt;
      *j.n_accepted += 1;
      const int ap = j.cand[tt];
      if (ap >= 0 && ap < j.n_pages) __hip_atomic_store(&j.in_acc[ap], (uint8_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
  }
  for (int k = 0; k < j.window; ++k) __hip_atomic_store(&j.rbuf[k], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kFixN], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kCursor], cur, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&j.ctrl[kPending], acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fix-up of listed pairs e0 .. e0 + np - 1, `parts` items per pair: item
// (e, part) sums w_i and w_i v_i over its slice of the row's tokens that are
// visible and outside the union (accepted pages and the candidate's page),
// with w_i = 2^(x_i - lse) <= 1, and writes the (D + 1) sums to fpart.
// Thread layout: D / 8 threads per token (16 bytes of its key and value
// each), 256 / (D / 8) tokens per round.
template <int D, bool PG>
__device__ void joint_fix_partial(const JointArgs& j, int cursor, int e0, int np, int parts, float* sacc) {
  constexpr int TPR = D / 8, RPR = 256 / TPR;
  const AttnGeom& a = j.geo;
  const int tid = threadIdx.x, c = tid % TPR, r = tid / TPR;
  for (int item = blockIdx.x; item < np * parts; item += gridDim.x) {
    const int e = e0 + item / parts, part = item % parts;
    const int2 ent = load_pair(j.fix_list + 2 * e);
    const int rg = (int)CKV_IDX(ent.y, j.total_rows, j.geo.dbg, 12);
    const int cp = j.cand[CKV_IDX(cursor + ent.x, j.max_cand, j.geo.dbg, 13)];   // the candidate's page
    const int h = rg / a.W, p = rg % a.W, g = h / a.group;
    const int qp = a.qpos[p];
    const float ref = j.lse[rg] * kLog2e;
    const int seg = ((a.S + parts - 1) / parts + RPR - 1) / RPR * RPR;
    const int a0 = part * seg, a1 = min(a.S, a0 + seg);
    const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
    const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;
    const u32x4 qc = ldg_u4(a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride + 8 * c);
    float qv[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) qv[m] = bf16_bits_to_float(chunk_elem(qc, m));
    float acc[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) acc[m] = 0.f;
    float lacc = 0.f;
    // first page whose end lies past this thread's first token
    int pp = 0;
    {
      int lo = 0, hi = j.n_pages;
      const int t0 = a0 + r;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (j.pstart[mid] + j.plen[mid] <= t0) lo = mid + 1;
        else hi = mid;
      }
      pp = lo;
    }
    for (int b0 = a0; b0 < a1; b0 += RPR) {
      const int t = b0 + r;
      const int tt = min(t, a1 - 1);
      const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[tt], a.pool_last) : tt;
      const u32x4 kc = ldg_u4(kh + row * a.kv_tok_stride + 8 * c);
      const u32x4 vc = ldg_u4(vh + row * a.kv_tok_stride + 8 * c);
      float x = 0.f;
#pragma unroll
      for (int m = 0; m < 8; ++m) x = __builtin_fmaf(qv[m], bf16_bits_to_float(chunk_elem(kc, m)), x);
#pragma unroll
      for (int off = TPR / 2; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
      while (pp < j.n_pages && j.pstart[pp] + j.plen[pp] <= tt) ++pp;
      const bool in_union = pp < j.n_pages && j.pstart[pp] <= tt && (pp == cp || __hip_atomic_load(&j.in_acc[pp], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0);
      const bool keep = t < a1 && ldg_i32(a.pos + tt) <= qp && !in_union;
      const float w = keep ? __builtin_amdgcn_exp2f(__builtin_fmaf(x, a.sl2, -ref)) : 0.f;
#pragma unroll
      for (int m = 0; m < 8; ++m) acc[m] = __builtin_fmaf(w, bf16_bits_to_float(chunk_elem(vc, m)), acc[m]);
      if (c == 0) lacc += w;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) sacc[r * (D + 1) + 8 * c + m] = acc[m];
    if (c == 0) sacc[r * (D + 1) + D] = lacc;
    __syncthreads();
    // the item's sums: token rows added in order
    float* out = j.fpart + ((size_t)(e - e0) * parts + part) * (D + 1);
    for (int i = tid; i <= D; i += 256) {
      float v = 0.f;
      for (int k = 0; k < RPR; ++k) v += sacc[k * (D + 1) + i];
      out[i] = v;
    }
    __syncthreads();
  }
}

// One wave per listed pair: parts added in order, o' = sum w v / sum w and
// ||o - o'|| / ||o|| raised into the candidate's round maximum.
template <int D>
__device__ void joint_fix_final(const JointArgs& j, int e0, int np, int parts) {
  const int lane = threadIdx.x & 63;
  for (int e = e0 + blockIdx.x * 4 + (threadIdx.x >> 6); e < e0 + np; e += gridDim.x * 4) {
    const int2 ent = load_pair(j.fix_list + 2 * e);
    const int rg = ent.y;
    const float* fp = j.fpart + (size_t)(e - e0) * parts * (D + 1);
    float num[D / 64], den = 0.f;
#pragma unroll
    for (int m = 0; m < D / 64; ++m) num[m] = 0.f;
    for (int part = 0; part < parts; ++part) {
#pragma unroll
      for (int m = 0; m < D / 64; ++m) num[m] += fp[part * (D + 1) + lane + 64 * m];
      den += fp[part * (D + 1) + D];
    }
    float dd = 0.f, oo = 0.f;
#pragma unroll
    for (int m = 0; m < D / 64; ++m) {
      const float ov = j.o[(size_t)rg * D + lane + 64 * m];
      const float od = den > 0.f ? num[m] / den : 0.f;
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
      atomicMax(&j.rbuf[ent.x], __float_as_uint(ratio));
    }
  }
}

__global__ __launch_bounds__(256) void joint_persistent(JointArgs j, RowStats rs) {
  __shared__ unsigned int smax;
  __shared__ int s_ok, s_part[4];
  __shared__ float sacc[32 * 65];    // fix-up: RPR token rows x (D + 1) sums (16 x 129 for D = 128)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  const int n_eff = min(min(*j.n_cand, j.max_cand), j.test_cap);
  // phase 0: outputs, state, ||o_p|| and visible-token counts
  for (size_t i = gid; i < (size_t)j.max_cand; i += gsz) {
    j.accepted[i] = 0;
    if (j.union_R) j.union_R[i] = __builtin_nanf("");
  }
  if (gid == 0) *j.n_accepted = 0;
  if (n_eff <= 0) return;              // nothing to test: the same in every block
  for (size_t i = gid; i < (size_t)j.total_rows * j.D; i += gsz) j.Dstate[i] = 0.f;
  for (size_t i = gid; i < (size_t)j.total_rows; i += gsz) { j.Astate[i] = 0.f; j.Cstate[i] = 0; }
  for (size_t i = gid; i < (size_t)j.window; i += gsz) j.rbuf[i] = 0u;
  for (size_t i = gid; i < (size_t)j.n_pages; i += gsz) j.in_acc[i] = 0;
  if (gid == 0) {
    j.ctrl[kCursor] = 0;
    j.ctrl[kPending] = -1;
    j.ctrl[kParity] = 0;
  }
  for (int row = blockIdx.x * 4 + wave; row < j.total_rows; row += gridDim.x * 4) {
    float n2 = 0.f;
    for (int d = lane; d < j.D; d += 64) {
      const float v = j.o[(size_t)row * j.D + d];
      n2 += v * v;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
    if (lane == 0) {
      rs.onorm[row] = sqrtf(n2);
      if (!(n2 <= 3.4e38f) || !(j.lse[row] < INFINITY)) latch_nonfinite(j.nonfinite);
    }
  }
  // n_vis of window row p (shared by every query head): #{i : pos[i] <= qpos[p]},
  // one partial count per (row, token slice)
  for (int it = blockIdx.x; it < j.W * j.n_vis_slices; it += gridDim.x) {
    const int p = it / j.n_vis_slices, sl = it % j.n_vis_slices;
    const int qp = j.qpos[p];
    const int t0 = sl * kVisSlice, t1 = min(j.S, t0 + kVisSlice);
    int c = 0;
    for (int i = t0 + (int)threadIdx.x; i < t1; i += 256) c += j.pos[i] <= qp ? 1 : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off, 64);
    if (lane == 0) s_part[wave] = c;
    __syncthreads();
    if (threadIdx.x == 0) j.nvis_part[it] = s_part[0] + s_part[1] + s_part[2] + s_part[3];
    __syncthreads();
  }
  int target = gridDim.x;
  if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
    if (threadIdx.x == 0) *j.n_accepted = -1;
    return;
  }
  const int n_rb = (j.total_rows + j.rows_per_block - 1) / j.rows_per_block;
  const int items = j.window * n_rb;
  // every round decides at least one candidate: n_eff rounds suffice
  for (int round = 0; round < n_eff; ++round) {
    const int cursor = __hip_atomic_load(&j.ctrl[kCursor], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int pend = __hip_atomic_load(&j.ctrl[kPending], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int par = __hip_atomic_load(&j.ctrl[kParity], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cursor >= n_eff) break;               // the same decision in every block
    for (int it = blockIdx.x; it < items; it += gridDim.x)
      joint_item(j, rs, it / n_rb, it % n_rb, cursor, pend, par, n_eff, &smax);
    target += gridDim.x;
    if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
    // listed pairs, recomputed by definition in chunks that fit the
    // workspace (the same count and chunks in every block)
    const int nfix = min(__hip_atomic_load(&j.ctrl[kFixN], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                         j.window * j.total_rows);
    for (int e0 = 0; e0 < nfix; e0 += kJointFixItems) {
      const int np = min(nfix - e0, kJointFixItems);
      const int parts = max(1, min(kJointFixParts, kJointFixItems / np));
      const bool pg = j.geo.slot != nullptr;
      if (j.D == 128) {
        if (pg) joint_fix_partial<128, true>(j, cursor, e0, np, parts, sacc);
        else joint_fix_partial<128, false>(j, cursor, e0, np, parts, sacc);
      } else {
        if (pg) joint_fix_partial<64, true>(j, cursor, e0, np, parts, sacc);
        else joint_fix_partial<64, false>(j, cursor, e0, np, parts, sacc);
      }
      target += gridDim.x;
      if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
        if (threadIdx.x == 0) *j.n_accepted = -1;
        return;
      }
      if (j.D == 128) joint_fix_final<128>(j, e0, np, parts);
      else joint_fix_final<64>(j, e0, np, parts);
      target += gridDim.x;
      if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
        if (threadIdx.x == 0) *j.n_accepted = -1;
        return;
      }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      decide_round(j, cursor, n_eff);
      __hip_atomic_store(&j.ctrl[kParity], par ^ 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    target += gridDim.x;
    if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
  }
}

// Rows owned by workgroups: the fast form of the rounds.  Workgroup b owns
// window rows [b * rpb, (b + 1) * rpb) for the whole call and keeps their
// accumulated state (D, A_A, visible counts) in LDS, so a round touches
// global memory only to read the tested candidates' residual rows and to
// publish one maximum per candidate; nothing written to global memory has
// to be made visible across workgroups except through atomics.  A wave
// tests a row against up to 16 candidates with every load issued first.
constexpr int kRowsOwnedMax = 64;   // rows a workgroup owns at most (host checks)
constexpr int kCandBatch = 16;      // candidates whose residual rows are loaded together

template <int D>
__device__ void owned_round_tests(const JointArgs& j, float* sD, const float* sA, const int* sC,
                                  const float* sOn, const int* sNv, unsigned int* sMax, int rb0, int nr,
                                  int cursor, int n_eff) {
  constexpr int KD = D / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int r = wave; r < nr; r += 4) {
    const int row = rb0 + r;
    float dv[KD];
#pragma unroll
    for (int k = 0; k < KD; ++k) dv[k] = sD[r * D + lane + 64 * k];
    const float Acur = sA[r], on = sOn[r];
    const int Ccur = sC[r], nv = sNv[r];
    for (int jb = 0; jb < j.window; jb += kCandBatch) {
      float tv[kCandBatch][KD], tA[kCandBatch];
      int tC[kCandBatch];
      // this row's candidates sit together: 32-bit offsets from the row's base
      const float* rrow = j.resid + (size_t)row * j.max_cand * D;
      const float* arow = j.resA + (size_t)row * j.max_cand;
      const int* crow = j.resC + (size_t)row * j.max_cand;
#pragma unroll
      for (int q = 0; q < kCandBatch; ++q) {
        const int t = cursor + jb + q;
        const bool valid = jb + q < j.window && t < n_eff;
        const int tt = valid ? t : cursor;
#pragma unroll
        for (int k = 0; k < KD; ++k) tv[q][k] = rrow[tt * D + lane + 64 * k];
        tA[q] = arow[tt];
        tC[q] = crow[tt];
        if (!valid) {
#pragma unroll
          for (int k = 0; k < KD; ++k) tv[q][k] = 0.f;
          tA[q] = 0.f;
          tC[q] = 0;
        }
      }
      // squared norms of the batch's unions, reduced across the wave
      // together (the batch's exchanges overlap instead of chaining)
      float n2v[kCandBatch];
#pragma unroll
      for (int q = 0; q < kCandBatch; ++q) {
        float n2 = 0.f;
#pragma unroll
        for (int k = 0; k < KD; ++k) {
          const float y = dv[k] + tv[q][k];
          n2 += y * y;
        }
        n2v[q] = n2;
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
        for (int q = 0; q < kCandBatch; ++q) n2v[q] += __shfl_xor(n2v[q], off, 64);
#pragma unroll
      for (int q = 0; q < kCandBatch; ++q) {
        const int jx = jb + q;
        if (jx >= j.window || cursor + jx >= n_eff) break;
        const float n2 = n2v[q];
        const float Au = Acur + tA[q];
        const int Cu = Ccur + tC[q];
        float ratio = 0.f;
        if (Cu > 0) {
          if (Cu >= nv) {
            ratio = INFINITY;
          } else if (Au > kJointFixA) {
            // recomputed by definition after the round's tests
            if (lane == 0) {
              const int slot = atomicAdd(&j.ctrl[kFixN], 1);
              if (slot < j.window * j.total_rows) store_pair(j.fix_list + 2 * slot, make_int2(jx, row));
            }
          } else if (on > 0.f) {
            ratio = sqrtf(n2) / ((1.f - Au) * on);
          } else {
            ratio = n2 > 0.f ? INFINITY : 0.f;
          }
        }
        if (lane == 0 && ratio > 0.f) atomicMax(&sMax[jx], __float_as_uint(ratio));
      }
    }
  }
}

__global__ __launch_bounds__(256) void joint_owned(JointArgs j, RowStats rs) {
  __shared__ float sD[kRowsOwnedMax * 128];
  __shared__ float sA[kRowsOwnedMax], sOn[kRowsOwnedMax];
  __shared__ int sC[kRowsOwnedMax], sNv[kRowsOwnedMax];
  __shared__ unsigned int sMax[64];
  __shared__ int s_ok, s_part[4];
  __shared__ float sacc[32 * 65];    // fix-up: RPR token rows x (D + 1) sums
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  const int n_eff = min(min(*j.n_cand, j.max_cand), j.test_cap);
  // phase 0: outputs, ||o_p|| and visible-token counts
  for (size_t i = gid; i < (size_t)j.max_cand; i += gsz) {
    j.accepted[i] = 0;
    if (j.union_R) j.union_R[i] = __builtin_nanf("");
  }
  if (gid == 0) *j.n_accepted = 0;
  if (n_eff <= 0) return;              // nothing to test: the same in every block
  for (size_t i = gid; i < (size_t)j.window; i += gsz) j.rbuf[i] = 0u;
  for (size_t i = gid; i < (size_t)j.n_pages; i += gsz) j.in_acc[i] = 0;
  if (gid == 0) {
    j.ctrl[kCursor] = 0;
    j.ctrl[kPending] = -1;
  }
  for (int row = blockIdx.x * 4 + wave; row < j.total_rows; row += gridDim.x * 4) {
    float n2 = 0.f;
    for (int d = lane; d < j.D; d += 64) {
      const float v = j.o[(size_t)row * j.D + d];
      n2 += v * v;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
    if (lane == 0) {
      rs.onorm[row] = sqrtf(n2);
      if (!(n2 <= 3.4e38f) || !(j.lse[row] < INFINITY)) latch_nonfinite(j.nonfinite);
    }
  }
  for (int it = blockIdx.x; it < j.W * j.n_vis_slices; it += gridDim.x) {
    const int p = it / j.n_vis_slices, sl = it % j.n_vis_slices;
    const int qp = j.qpos[p];
    const int t0 = sl * kVisSlice, t1 = min(j.S, t0 + kVisSlice);
    int c = 0;
    for (int i = t0 + (int)threadIdx.x; i < t1; i += 256) c += j.pos[i] <= qp ? 1 : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off, 64);
    if (lane == 0) s_part[wave] = c;
    __syncthreads();
    if (threadIdx.x == 0) j.nvis_part[it] = s_part[0] + s_part[1] + s_part[2] + s_part[3];
    __syncthreads();
  }
  int target = gridDim.x;
  if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
    if (threadIdx.x == 0) *j.n_accepted = -1;
    return;
  }
  // this workgroup's rows and their state
  const int rpb = (j.total_rows + gridDim.x - 1) / gridDim.x;
  const int rb0 = blockIdx.x * rpb;
  const int nr = max(0, min(rpb, j.total_rows - rb0));
  for (int i = threadIdx.x; i < nr * j.D; i += 256) sD[i] = 0.f;
  for (int r = threadIdx.x; r < nr; r += 256) {
    const int row = rb0 + r;
    sA[r] = 0.f;
    sC[r] = 0;
    sOn[r] = rs.onorm[row];
    int c = 0;
    for (int q = 0; q < j.n_vis_slices; ++q) c += j.nvis_part[(row % j.W) * j.n_vis_slices + q];
    sNv[r] = c;
  }
  // every round decides at least one candidate: n_eff rounds suffice
  for (int round = 0; round < n_eff; ++round) {
    const int cursor = __hip_atomic_load(&j.ctrl[kCursor], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int pend = __hip_atomic_load(&j.ctrl[kPending], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cursor >= n_eff) break;               // the same decision in every block
    // the candidate accepted last round joins this workgroup's rows' state
    if (pend >= 0) {
      // every load of the fold issued before the first add
      constexpr int kFold = kRowsOwnedMax * 128 / 256;
      float add[kFold];
      const float* pbase = j.resid + ((size_t)rb0 * j.max_cand + pend) * j.D;
      const int rstride = j.max_cand * j.D;
#pragma unroll
      for (int q = 0; q < kFold; ++q) {
        const int i = threadIdx.x + 256 * q;
        add[q] = i < nr * j.D ? pbase[(i / j.D) * rstride + i % j.D] : 0.f;
      }
      float aA = 0.f;
      int aC = 0;
      if ((int)threadIdx.x < nr) {
        aA = j.resA[(size_t)(rb0 + threadIdx.x) * j.max_cand + pend];
        aC = j.resC[(size_t)(rb0 + threadIdx.x) * j.max_cand + pend];
      }
#pragma unroll
      for (int q = 0; q < kFold; ++q) {
        const int i = threadIdx.x + 256 * q;
        if (i < nr * j.D) sD[i] += add[q];
      }
      if ((int)threadIdx.x < nr) {
        sA[threadIdx.x] += aA;
        sC[threadIdx.x] += aC;
      }
    }
    for (int i = threadIdx.x; i < j.window; i += 256) sMax[i] = 0u;
    __syncthreads();
    if (j.D == 128) owned_round_tests<128>(j, sD, sA, sC, sOn, sNv, sMax, rb0, nr, cursor, n_eff);
    else owned_round_tests<64>(j, sD, sA, sC, sOn, sNv, sMax, rb0, nr, cursor, n_eff);
    __syncthreads();
    // this workgroup's maxima go to its own slots (no contended atomics);
    // workgroup 0 reduces them after the barrier
    for (int i = threadIdx.x; i < j.window; i += 256)
      __hip_atomic_store(&j.bmax[(size_t)blockIdx.x * j.window + i], sMax[i], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    target += gridDim.x;
    if (!grid_barrier_nofence(j.ctrl, target, j.barrier_ticks, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
    // listed pairs, recomputed by definition in chunks that fit the
    // workspace (the same count and chunks in every block)
    const int nfix = min(__hip_atomic_load(&j.ctrl[kFixN], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                         j.window * j.total_rows);
    for (int e0 = 0; e0 < nfix; e0 += kJointFixItems) {
      const int np = min(nfix - e0, kJointFixItems);
      const int parts = max(1, min(kJointFixParts, kJointFixItems / np));
      const bool pg = j.geo.slot != nullptr;
      if (j.D == 128) {
        if (pg) joint_fix_partial<128, true>(j, cursor, e0, np, parts, sacc);
        else joint_fix_partial<128, false>(j, cursor, e0, np, parts, sacc);
      } else {
        if (pg) joint_fix_partial<64, true>(j, cursor, e0, np, parts, sacc);
        else joint_fix_partial<64, false>(j, cursor, e0, np, parts, sacc);
      }
      target += gridDim.x;
      if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
        if (threadIdx.x == 0) *j.n_accepted = -1;
        return;
      }
      if (j.D == 128) joint_fix_final<128>(j, e0, np, parts);
      else joint_fix_final<64>(j, e0, np, parts);
      target += gridDim.x;
      if (!grid_barrier(j.ctrl, target, j.barrier_ticks, &s_ok)) {
        if (threadIdx.x == 0) *j.n_accepted = -1;
        return;
      }
    }
    if (blockIdx.x == 0) {
      // maxima over the workgroups' slots and the fix-up's maxima, every
      // load issued at once; then the decision from LDS
      for (int i = threadIdx.x; i < j.window; i += 256) sMax[i] = 0u;
      __syncthreads();
      {
        constexpr int kPer = kTargetBlocksMax / 8;   // slots per thread: 8 threads per candidate
        const int jx = threadIdx.x % 32, b0 = threadIdx.x / 32;
        unsigned int v[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
          const int b = b0 + 8 * q;
          v[q] = (jx < j.window && b < (int)gridDim.x)
                     ? __hip_atomic_load(&j.bmax[(size_t)b * j.window + jx], __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT)
                     : 0u;
        }
        unsigned int m = 0u;
#pragma unroll
        for (int q = 0; q < kPer; ++q) m = max(m, v[q]);
        if (jx < j.window && b0 == 0)
          m = max(m, __hip_atomic_load(&j.rbuf[jx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        if (jx < j.window) atomicMax(&sMax[jx], m);
      }
      __syncthreads();
      if (threadIdx.x == 0) decide_round_lds(j, sMax, cursor, n_eff);
    }
    target += gridDim.x;
    if (!grid_barrier_nofence(j.ctrl, target, j.barrier_ticks, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
  }
}

int joint_vis_slices(int S) { return (S + kVisSlice - 1) / kVisSlice; }

hipError_t launch_joint_persistent(const JointArgs& j, int max_blocks, hipStream_t s) {
  RowStats rs{nullptr, nullptr, const_cast<float*>(j.onorm), nullptr, nullptr, nullptr, nullptr};
  const int n_rb = (j.total_rows + j.rows_per_block - 1) / j.rows_per_block;
  // workgroups of each form that fit on the device at once (queried once per device)
  static int resident[64][2];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (resident[dev][0] <= 0) {
    int per_cu = 0, per_cu2 = 0, cus = 0;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, joint_persistent, 256, 0)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu2, joint_owned, 256, 0)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    resident[dev][0] = std::max(1, per_cu * cus);
    resident[dev][1] = std::max(1, per_cu2 * cus);
  }
  // rows owned by workgroups: about 8 rows each, at most kRowsOwnedMax
  const int nb_owned = std::max(1, std::min({(j.total_rows + 7) / 8, resident[dev][1], max_blocks, kTargetBlocksMax}));
  if (j.window <= 64 && j.D <= 128 && (j.total_rows + nb_owned - 1) / nb_owned <= kRowsOwnedMax) {
    hipLaunchKernelGGL(joint_owned, dim3(nb_owned), dim3(256), 0, s, j, rs);
    return hipGetLastError();
  }
  const int nb = std::max(1, std::min({j.window * n_rb, resident[dev][0], max_blocks}));
  hipLaunchKernelGGL(joint_persistent, dim3(nb), dim3(256), 0, s, j, rs);
  return hipGetLastError();
}

}  // namespace ckv
