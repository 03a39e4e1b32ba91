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
// tested again in the next round.  One launch per round: the last block of a
// round to finish takes the decision; the accepted candidate's residual is
// folded into the state by the next round while it copies the state into
// the other buffer (double buffering, so no block reads a row another block
// is writing).
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <climits>

namespace ckv {

enum { kCursor = 0, kPending = 1, kDone = 2, kCounter = 3, kParity = 4 };

// per row: ||o||, n_vis, lse in log2 units; clear the joint state and outputs
__global__ __launch_bounds__(256) void joint_prep_rows(AttnGeom a, const float* o, const float* lse,
                                                      RowStats rs, JointArgs j) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  for (size_t i = gid; i < (size_t)j.total_rows * j.D; i += gsz) j.Dstate[i] = 0.f;
  for (size_t i = gid; i < (size_t)j.total_rows; i += gsz) { j.Astate[i] = 0.f; j.Cstate[i] = 0; }
  for (size_t i = gid; i < (size_t)j.max_cand; i += gsz) {
    j.accepted[i] = 0;
    if (j.union_R) j.union_R[i] = __builtin_nanf("");
  }
  for (size_t i = gid; i < (size_t)j.window; i += gsz) j.rbuf[i] = 0u;
  for (size_t i = gid; i < (size_t)j.W; i += gsz) rs.nvis[i] = 0;
  if (gid == 0) {
    j.ctrl[kCursor] = 0;
    j.ctrl[kPending] = -1;
    j.ctrl[kDone] = 0;
    j.ctrl[kCounter] = 0;
    j.ctrl[kParity] = 0;
    *j.n_accepted = 0;
  }
  if (row >= j.total_rows) return;
  float n2 = 0.f;
  for (int d = lane; d < j.D; d += 64) {
    const float v = o[(size_t)row * j.D + d];
    n2 += v * v;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
  if (lane == 0) {
    rs.onorm[row] = sqrtf(n2);
    const float l = lse[row];
    rs.lse2[row] = l == -INFINITY ? -INFINITY : l * kLog2e;
  }
}

// n_vis of window row p (shared by every query head): #{i : pos[i] <= qpos[p]},
// counted over a (row, token slice) grid; rs.nvis holds one count per row p
// and is zeroed by joint_prep_rows.
constexpr int kVisSlice = 8192;

__global__ __launch_bounds__(256) void joint_prep_vis(AttnGeom a, RowStats rs) {
  __shared__ int part[4];
  const int p = blockIdx.x;
  const int qp = a.qpos[p];
  const int t0 = blockIdx.y * kVisSlice, t1 = min(a.S, t0 + kVisSlice);
  int c = 0;
  for (int i = t0 + threadIdx.x; i < t1; i += 256) c += a.pos[i] <= qp ? 1 : 0;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(&rs.nvis[p], part[0] + part[1] + part[2] + part[3]);
}

// outputs when there is no candidate to test
__global__ __launch_bounds__(256) void joint_init_outputs(JointArgs j) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < j.max_cand; i += gridDim.x * 256) {
    j.accepted[i] = 0;
    if (j.union_R) j.union_R[i] = __builtin_nanf("");
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *j.n_accepted = 0;
}

hipError_t launch_joint_prepare(const AttnGeom& a, const float* o, const float* lse, RowStats rs,
                                const JointArgs& j, hipStream_t s) {
  hipLaunchKernelGGL(joint_prep_rows, dim3((j.total_rows + 3) / 4), dim3(256), 0, s, a, o, lse, rs, j);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(joint_prep_vis, dim3(a.W, (a.S + kVisSlice - 1) / kVisSlice), dim3(256), 0, s, a, rs);
  return hipGetLastError();
}

hipError_t launch_joint_init(const JointArgs& j, hipStream_t s) {
  hipLaunchKernelGGL(joint_init_outputs, dim3((j.max_cand + 255) / 256), dim3(256), 0, s, j);
  return hipGetLastError();
}

// one round: block (jx, rb) tests candidate cursor + jx on rows of block rb
__global__ __launch_bounds__(256) void joint_round_kernel(JointArgs j, RowStats rs) {
  __shared__ unsigned int smax;
  __shared__ int is_last;
  if (j.ctrl[kDone]) return;
  const int cursor = j.ctrl[kCursor];
  const int pend = j.ctrl[kPending];
  const int par = j.ctrl[kParity];
  const int n_eff = min(*j.n_cand, j.max_cand);
  const int jx = blockIdx.x;
  const int t = cursor + jx;
  const bool valid = t < n_eff;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.y * j.rows_per_block;
  const int r1 = min(j.total_rows, r0 + j.rows_per_block);
  const size_t RD = (size_t)j.total_rows * j.D;
  const float* Din = j.Dstate + (size_t)par * RD;
  float* Dout = j.Dstate + (size_t)(par ^ 1) * RD;
  const float* Ain = j.Astate + (size_t)par * j.total_rows;
  float* Aout = j.Astate + (size_t)(par ^ 1) * j.total_rows;
  const int* Cin = j.Cstate + (size_t)par * j.total_rows;
  int* Cout = j.Cstate + (size_t)(par ^ 1) * j.total_rows;
  if (threadIdx.x == 0) smax = 0u;
  __syncthreads();
  float wmax = 0.f;
  for (int row = r0 + wave; row < r1; row += 4) {
    // current state of this row = stored state + residual of the pending accept
    float dcur[4];
    float n2 = 0.f;
    const float* rp = pend >= 0 ? j.resid + ((size_t)pend * j.total_rows + row) * j.D : nullptr;
    const float* rt = valid ? j.resid + ((size_t)t * j.total_rows + row) * j.D : nullptr;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int d = lane + 64 * k;
      float dv = 0.f;
      if (d < j.D) {
        dv = Din[(size_t)row * j.D + d];
        if (rp) dv += rp[d];
        if (jx == 0) Dout[(size_t)row * j.D + d] = dv;
        if (rt) {
          const float x = dv + rt[d];
          n2 += x * x;
        }
      }
      dcur[k] = dv;
    }
    (void)dcur;
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
      if (Ct >= rs.nvis[row % j.W] || !(keep > 0.f)) ratio = INFINITY;
      else if (on > 0.f) ratio = sqrtf(n2) / (keep * on);
      else ratio = n2 > 0.f ? INFINITY : 0.f;
    }
    wmax = fmaxf(wmax, ratio);
  }
  if (valid && lane == 0) atomicMax(&smax, __float_as_uint(wmax));
  __syncthreads();
  if (threadIdx.x == 0) {
    if (valid) atomicMax(&j.rbuf[jx], smax);
    __threadfence();
    const int total = gridDim.x * gridDim.y;
    const int prev = atomicAdd(&j.ctrl[kCounter], 1);
    is_last = (prev == total - 1);
  }
  __syncthreads();
  if (!is_last || threadIdx.x != 0) return;
  // decision: the first passer in order is accepted, the ones before it rejected
  __threadfence();
  int cur = cursor;
  int acc = -1;
  for (int k = 0; k < (int)gridDim.x; ++k) {
    const int tt = cursor + k;
    if (tt >= n_eff) break;
    const unsigned int bits = __hip_atomic_load(&j.rbuf[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const float r = __uint_as_float(bits);
    if (j.union_R) j.union_R[tt] = r;
    cur = tt + 1;
    if (r <= j.tau) {
      j.accepted[tt] = 1;
      acc = tt;
      *j.n_accepted += 1;
      break;
    }
  }
  for (int k = 0; k < (int)gridDim.x; ++k) j.rbuf[k] = 0u;
  j.ctrl[kCursor] = cur;
  j.ctrl[kPending] = acc;
  j.ctrl[kParity] = par ^ 1;
  j.ctrl[kDone] = cur >= n_eff ? 1 : 0;
  j.ctrl[kCounter] = 0;
}

hipError_t launch_joint_round(const JointArgs& j, hipStream_t s) {
  RowStats rs{nullptr, nullptr, const_cast<float*>(j.onorm), const_cast<int*>(j.nvis)};
  dim3 grid(j.window, (j.total_rows + j.rows_per_block - 1) / j.rows_per_block);
  hipLaunchKernelGGL(joint_round_kernel, grid, dim3(256), 0, s, j, rs);
  return hipGetLastError();
}


}  // namespace ckv
