// Lifecycle classification of event pages (CommitKV, Sec. 3.2, Eq. (8)-(10))
// and the candidate order of Sec. 3.3.
//
// rank_kernel: 16 lanes per page.  Percentile P(E) = (number of other pages
// with a strictly smaller effect) / (n - 1), 0.5 for n = 1; counted exactly
// against every page (values staged through LDS in chunks, so the count loop
// never waits on a global load), so ties share the lower rank.  The comparison P >= rho is made in double precision on the integer
// count.  Then H/L of Eq. (9) and the state of Eq. (10).
// order_kernel: 16 lanes per page, the same staging.  A candidate's slot in the ordered list
// is the number of candidates that precede it under (R+ ascending, R-
// descending, index ascending); the keys are unique so the slots form a
// permutation without any sort.
#include "ckv_device.h"
#include "ckv_kernels.h"
#include "commitkv.h"

namespace ckv {

namespace {
constexpr int kCT = 256;
}

// 16 lanes cooperate on one page: lane j of the group compares against pages
// j, j + 16, ...; the counts are summed with shuffles.
constexpr int kLanes = 16;
constexpr int kPagesPerBlock = kCT / kLanes;
constexpr int kStage = 2048;   // pages staged in LDS per chunk

__global__ __launch_bounds__(kCT) void rank_kernel(ClassifyArgs c) {
  const int i = blockIdx.x * kPagesPerBlock + threadIdx.x / kLanes;
  const int sub = threadIdx.x % kLanes;
  const bool act = i < c.n;
  const float rp = act ? c.R_pre[i] : 0.f;
  const float rq = act ? c.R_post[i] : 0.f;
  __shared__ float sPre[kStage], sPost[kStage];
  int less_pre = 0, less_post = 0;
  for (int base = 0; base < c.n; base += kStage) {
    const int m = min(kStage, c.n - base);
    __syncthreads();
    for (int j = threadIdx.x; j < m; j += kCT) {
      sPre[j] = c.R_pre[base + j];
      sPost[j] = c.R_post[base + j];
    }
    __syncthreads();
    for (int j = sub; j < m; j += kLanes) {
      less_pre += sPre[j] < rp ? 1 : 0;
      less_post += sPost[j] < rq ? 1 : 0;
    }
  }
#pragma unroll
  for (int off = kLanes / 2; off >= 1; off >>= 1) {
    less_pre += __shfl_xor(less_pre, off, 64);
    less_post += __shfl_xor(less_post, off, 64);
  }
  if (!act || sub != 0) return;
  const double den = c.n > 1 ? (double)(c.n - 1) : 1.0;
  const double Pm = c.n > 1 ? less_pre / den : 0.5;
  const double Pp = c.n > 1 ? less_post / den : 0.5;
  // Eq. (9), inclusive comparisons (absolute thresholds alone without the
  // percentile calibration, Sec. 4.4)
  const bool pct = !(c.policy & CKV_POLICY_NO_PERCENTILE);
  const bool H_pre = rp >= c.tau_use && (!pct || Pm >= (double)c.rho_use);
  const bool L_pre = rp <= c.tau_dead && (!pct || Pm <= (double)c.rho_dead);
  const bool H_post = rq >= c.tau_use && (!pct || Pp >= (double)c.rho_use);
  const bool L_post = rq <= c.tau_dead && (!pct || Pp <= (double)c.rho_dead);
  // Eq. (10); without the pre-commit state (Sec. 4.4) L+ alone makes a candidate
  uint8_t lam = 0;
  if (c.policy & CKV_POLICY_NO_PRECOMMIT) {
    if (L_post) lam = 1;
    else if (L_pre && H_post) lam = 3;
    else if (H_pre && H_post) lam = 4;
  } else {
    if (H_pre && L_post) lam = 1;
    else if (L_pre && L_post) lam = 2;
    else if (L_pre && H_post) lam = 3;
    else if (H_pre && H_post) lam = 4;
  }
  c.lambda[i] = lam;
  c.P_pre[i] = (float)Pm;
  c.P_post[i] = (float)Pp;
  const bool none = (c.policy & CKV_POLICY_NO_LIFECYCLE) != 0;
  c.is_cand[i] = (!none && (lam == 1 || (c.force && c.force[i]))) ? 1 : 0;
  c.cand[i] = -1;
}

__device__ __forceinline__ bool precedes(float qj, float pj, int j, float qi, float pi, int i) {
  if (qj != qi) return qj < qi;          // R+ ascending
  if (pj != pi) return pj > pi;          // then R- descending
  return j < i;                          // then page order
}

__global__ __launch_bounds__(kCT) void order_kernel(ClassifyArgs c) {
  const int i = blockIdx.x * kPagesPerBlock + threadIdx.x / kLanes;
  const int sub = threadIdx.x % kLanes;
  const bool act = i < c.n;
  const bool me = act && c.is_cand[i];
  const float rp = act ? c.R_pre[i] : 0.f;
  const float rq = act ? c.R_post[i] : 0.f;
  __shared__ float sPre[kStage], sPost[kStage];
  __shared__ uint8_t sCand[kStage];
  int before = 0, total = 0;
  for (int base = 0; base < c.n; base += kStage) {
    const int m = min(kStage, c.n - base);
    __syncthreads();
    for (int j = threadIdx.x; j < m; j += kCT) {
      sPre[j] = c.R_pre[base + j];
      sPost[j] = c.R_post[base + j];
      sCand[j] = c.is_cand[base + j];
    }
    __syncthreads();
    for (int j = sub; j < m; j += kLanes) {
      if (!sCand[j]) continue;
      ++total;
      before += precedes(sPost[j], sPre[j], base + j, rq, rp, i) ? 1 : 0;
    }
  }
#pragma unroll
  for (int off = kLanes / 2; off >= 1; off >>= 1) {
    before += __shfl_xor(before, off, 64);
    total += __shfl_xor(total, off, 64);
  }
  const int cap = c.max_cand > 0 ? min(c.max_cand, c.n) : c.n;
  if (me && sub == 0 && before < cap) c.cand[before] = i;
  if (blockIdx.x == 0 && threadIdx.x == 0) *c.n_cand = min(total, cap);
}

hipError_t launch_classify(const ClassifyArgs& c, hipStream_t s) {
  const int nb = c.n > 0 ? (c.n + kPagesPerBlock - 1) / kPagesPerBlock : 1;
  hipLaunchKernelGGL(rank_kernel, dim3(nb), dim3(kCT), 0, s, c);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(order_kernel, dim3(nb), dim3(kCT), 0, s, c);
  return hipGetLastError();
}

}  // namespace ckv
