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
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <algorithm>
#include <climits>

namespace ckv {

// control words (cleared by the residual pass before this kernel starts)
enum { kCursor = 0, kPending = 1, kBarrier = 2, kError = 3, kParity = 4 };
constexpr long long kBarrierTimeoutTicks = 1ll << 27;   // ~1.3 s of the 100 MHz wall clock
constexpr int kVisSlice = 8192;                         // tokens per visible-count item

// Grid barrier: thread 0 of every block publishes the block's writes, adds
// one arrival and waits until the arrivals reach `target`.  Returns false
// (in every thread) if the wait timed out or another block gave up.
__device__ bool grid_barrier(int* ctrl, int target, int* s_ok) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    atomicAdd(&ctrl[kBarrier], 1);
    const long long t0 = wall_clock64();
    int ok = 1;
    while (__hip_atomic_load(&ctrl[kBarrier], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(&ctrl[kError], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
          wall_clock64() - t0 > kBarrierTimeoutTicks) {
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
  for (int row = r0 + wave; row < r1; row += 4) {
    float n2 = 0.f;
    const float* rp = pend >= 0 ? j.resid + ((size_t)pend * j.total_rows + row) * j.D : nullptr;
    const float* rt = valid ? j.resid + ((size_t)t * j.total_rows + row) * j.D : nullptr;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int d = lane + 64 * k;
      if (d < j.D) {
        float dv = Din[(size_t)row * j.D + d];
        if (rp) dv += rp[d];
        if (jx == 0) Dout[(size_t)row * j.D + d] = dv;
        if (rt) {
          const float x = dv + rt[d];
          n2 += x * x;
        }
      }
    }
    float Acur = Ain[row];
    int Ccur = Cin[row];
    if (pend >= 0) {
      Acur += j.resA[(size_t)pend * j.total_rows + row];
      Ccur += j.resC[(size_t)pend * j.total_rows + row];
    }
    if (jx == 0 && lane == 0) { Aout[row] = Acur; Cout[row] = Ccur; }
    if (!valid) continue;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
    const float At = Acur + j.resA[(size_t)t * j.total_rows + row];
    const int Ct = Ccur + j.resC[(size_t)t * j.total_rows + row];
    float ratio = 0.f;
    if (Ct > 0) {
      const float keep = 1.f - At;
      const float on = rs.onorm[row];
      int nv = 0;
      for (int q = 0; q < j.n_vis_slices; ++q) nv += j.nvis_part[(row % j.W) * j.n_vis_slices + q];
      if (Ct >= nv || !(keep > 0.f)) ratio = INFINITY;
      else if (on > 0.f) ratio = sqrtf(n2) / (keep * on);
      else ratio = n2 > 0.f ? INFINITY : 0.f;
    }
    wmax = fmaxf(wmax, ratio);
  }
  if (valid && lane == 0) atomicMax(smax, __float_as_uint(wmax));
  __syncthreads();
  if (threadIdx.x == 0 && valid) atomicMax(&j.rbuf[jx], *smax);
  __syncthreads();
}

__global__ __launch_bounds__(256) void joint_persistent(JointArgs j, RowStats rs) {
  __shared__ unsigned int smax;
  __shared__ int s_ok, s_part[4];
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
    if (lane == 0) rs.onorm[row] = sqrtf(n2);
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
  if (!grid_barrier(j.ctrl, target, &s_ok)) {
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
    if (!grid_barrier(j.ctrl, target, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      // the first passer in order is accepted, the ones before it rejected
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
          break;
        }
      }
      for (int k = 0; k < j.window; ++k) __hip_atomic_store(&j.rbuf[k], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&j.ctrl[kCursor], cur, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&j.ctrl[kPending], acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&j.ctrl[kParity], par ^ 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    target += gridDim.x;
    if (!grid_barrier(j.ctrl, target, &s_ok)) {
      if (threadIdx.x == 0) *j.n_accepted = -1;
      return;
    }
  }
}

int joint_vis_slices(int S) { return (S + kVisSlice - 1) / kVisSlice; }

hipError_t launch_joint_persistent(const JointArgs& j, int max_blocks, hipStream_t s) {
  RowStats rs{nullptr, nullptr, const_cast<float*>(j.onorm), nullptr};
  const int n_rb = (j.total_rows + j.rows_per_block - 1) / j.rows_per_block;
  // workgroups that fit on the device at once (queried once per device)
  static int resident[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (resident[dev] <= 0) {
    int per_cu = 0, cus = 0;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, joint_persistent, 256, 0)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    resident[dev] = std::max(1, per_cu * cus);
  }
  const int nb = std::max(1, std::min({j.window * n_rb, resident[dev], max_blocks}));
  hipLaunchKernelGGL(joint_persistent, dim3(nb), dim3(256), 0, s, j, rs);
  return hipGetLastError();
}

}  // namespace ckv
