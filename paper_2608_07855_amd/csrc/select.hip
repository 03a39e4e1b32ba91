// Compression checkpoint (CommitKV, Sec. 3.3, Eq. (12)-(13); Sec. 3.1, Eq. (4)).
//
// protect_kernel (one block per sequence): pending pages are ranked by
//   (R- descending, page order ascending) by counting, and protected in that
//   order while fewer than max_pages are taken and the token total stays
//   within B_N; the first page that does not fit stops the protection.
// Selection, on token chunks of kSelChunk tokens (grid: chunks x sequences):
//   sel_keys   token states (retired > protected > free) in LDS, one coded
//              key per token (0 retired, ~0 protected, else the order-
//              preserving image of the score, NaN as -inf and -0.0 as +0.0),
//              counts, and the histogram of the first 11-bit digit;
//   sel_pass   the histograms of digits 2 and 3 among the keys that share
//              the digits chosen so far (radix select of the k-th largest);
//   sel_count  per chunk: tokens kept outright, free tokens tied at the
//              threshold key;
//   sel_write  kept indices in ascending order; ties at the threshold go to
//              the lowest indices.
//   k = min(B - #protected, #free).  The last workgroup of each histogram
//   launch (atomic arrival counter) chooses the digit for every sequence.
// select_grid (sequences of at most kSelGridMaxChunks chunks and
//   kSelGridPendMax pending pages, every workgroup resident at once): all of
//   the above in one launch of one workgroup per 2048-token chunk, phases
//   separated by a per-sequence grid barrier.
// gather_kernel: K'[s,l,g,j] = K[s,l,g,I[j]], the same for V, and
//   pos'[s,j] = pos[s,I[j]], 16-byte vector copies of whole rows.
#include "ckv_device.h"
#include "ckv_kernels.h"

namespace ckv {

namespace {
constexpr uint8_t kFree = 0, kProt = 1, kRet = 2;
}  // namespace

// larger key <=> larger score; NaN ranks as -inf, -0.0 as +0.0
__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) f = -INFINITY;
  if (f == 0.f) f = 0.f;
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float pend_key(float f) { return f != f ? -INFINITY : f; }

constexpr int kProtLds = 1024;   // pending pages ranked from LDS (more: from global memory)

__global__ __launch_bounds__(256) void protect_kernel(SelectArgs a) {
  __shared__ float sR[kProtLds];
  __shared__ int sLen[kProtLds], sOrd[kProtLds];
  const int s = blockIdx.x;
  const int off = a.pend_off[s];
  const int n = a.pend_off[s + 1] - off;
  const float* R = reinterpret_cast<const float*>(a.pend_r[s]);
  const int32_t* len = a.pend_len + off;
  uint8_t* prot = a.pend_prot + off;
  int32_t* ord = a.pend_ord + off;
  const bool lds = n <= kProtLds;
  // clear the selection state of this sequence for the kernels that follow
  for (int i = threadIdx.x; i < kSelCtrl; i += 256) a.ctrl[(size_t)s * kSelCtrl + i] = 0;
  for (int i = threadIdx.x; i < 3 * kSelBins; i += 256) a.hist[(size_t)s * 3 * kSelBins + i] = 0u;
  if (lds)
    for (int i = threadIdx.x; i < n; i += 256) {
      sR[i] = pend_key(R[i]);
      sLen[i] = len[i];
    }
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += 256) {
    const float ri = lds ? sR[i] : pend_key(R[i]);
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const float rj = lds ? sR[j] : pend_key(R[j]);
      rank += (rj > ri || (rj == ri && j < i)) ? 1 : 0;
    }
    if (lds) sOrd[rank] = i;
    else ord[rank] = i;
    prot[i] = 0;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int taken = 0, tok = 0;
    for (int r = 0; r < n; ++r) {
      const int i = lds ? sOrd[r] : ord[r];
      const int li = lds ? sLen[i] : len[i];
      if (taken >= a.max_pages || tok + li > a.bn) break;
      prot[i] = 1;
      ++taken;
      tok += li;
    }
  }
}

// Histogram increment with lanes of a wave that share a bin combined into
// one atomic: the leading key bytes of float scores take few values, and
// plain LDS atomics on one address serialise.  After a few combining rounds
// the remaining (spread) bins use plain atomics.
__device__ __forceinline__ void hist_add(unsigned int* hist, uint32_t bin, bool act) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int round = 0; round < 4; ++round) {
    const unsigned long long m = __ballot(act);
    if (m == 0ull) return;
    const int leader = __ffsll((long long)m) - 1;
    const uint32_t lb = __shfl((int)bin, leader, 64);
    const bool same = act && bin == lb;
    const unsigned long long sm = __ballot(same);
    if (lane == leader) atomicAdd(&hist[lb], (unsigned int)__popcll(sm));
    if (same) act = false;
  }
  if (act) atomicAdd(&hist[bin], 1u);
}

namespace {
constexpr int kSelT = 256;                       // threads per selection workgroup
constexpr int kPerT = kSelChunk / kSelT;         // tokens per thread
constexpr uint32_t kKeyRet = 0u, kKeyProt = 0xFFFFFFFFu;
// control block of one sequence
enum { cNP = 0, cNF = 1, cArr0 = 2, cArr1 = 3, cArr2 = 4, cK = 5, cMode = 6, cPrefix = 7,
       cMask = 8, cNeed = 9, cT = 10, cNeedEq = 11 };
enum { kModeRadix = 0, kModeAll = 1, kModeNone = 2 };
constexpr int kShift[3] = {21, 10, 0};
constexpr uint32_t kDigit[3] = {0x7FFu, 0x7FFu, 0x3FFu};

__device__ __forceinline__ bool key_free(uint32_t k) { return k != kKeyRet && k != kKeyProt; }
}  // namespace

// exclusive scan of one int per thread over a block of NT threads
template <int NT>
__device__ int block_scan(int v, int* tmp, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) tmp[w] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    const int t = tmp[i];
    base += i < w ? t : 0;
    tot += t;
  }
  total = tot;
  __syncthreads();
  return base + x - v;
}

// Last workgroup of a histogram launch, for sequence s: choose the digit of
// pass p that holds the need-th largest matching key.  Thread i owns bins
// [8(255-i), 8(255-i)+8), so an exclusive scan in thread order counts the
// keys in higher bins.
__device__ void choose_digit(const SelectArgs& a, int s, int p, int* tmp) {
  int32_t* ctrl = a.ctrl + (size_t)s * kSelCtrl;
  const uint32_t* hg = a.hist + ((size_t)s * 3 + p) * kSelBins;
  const int g = kSelT - 1 - (int)threadIdx.x;
  int h[8], sum = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    h[j] = (int)__hip_atomic_load(&hg[8 * g + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sum += h[j];
  }
  int total;
  int above = block_scan<kSelT>(sum, tmp, total);
  const int need = ctrl[cNeed];
  __syncthreads();
#pragma unroll
  for (int j = 7; j >= 0; --j) {
    if (above < need && above + h[j] >= need) {
      const uint32_t d = (uint32_t)(8 * g + j);
      const uint32_t prefix = (uint32_t)ctrl[cPrefix] | (d << kShift[p]);
      ctrl[cPrefix] = (int)prefix;
      ctrl[cMask] = (int)((uint32_t)ctrl[cMask] | (kDigit[p] << kShift[p]));
      ctrl[cNeed] = need - above;
      if (p == 2) {
        ctrl[cT] = (int)prefix;
        ctrl[cNeedEq] = need - above;
      }
    }
    above += h[j];
  }
}

// arrival at the end of a histogram launch; true in the last workgroup of
// sequence s (all threads)
__device__ bool arrive_last(int32_t* counter, int n_blocks, int* s_flag) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    *s_flag = atomicAdd(counter, 1) == n_blocks - 1;
  }
  __syncthreads();
  const bool last = *s_flag;
  if (last) __threadfence();
  return last;
}

__device__ __forceinline__ void bins_to_global(uint32_t* hg, const unsigned int* hl) {
  for (int i = threadIdx.x; i < kSelBins; i += kSelT)
    if (hl[i]) atomicAdd(&hg[i], hl[i]);
}

// token states, coded keys, counts and the first digit's histogram
__global__ __launch_bounds__(kSelT) void sel_keys(SelectArgs a) {
  __shared__ uint8_t st[kSelChunk];
  __shared__ unsigned int hl[kSelBins];
  __shared__ int tmp[kSelT / 64];
  __shared__ int s_flag;
  const int s = blockIdx.y;
  const int S = a.n_tokens[s];
  const int t0 = blockIdx.x * kSelChunk;
  if (t0 >= S) return;
  const int t1 = min(S, t0 + kSelChunk);
  const int tid = threadIdx.x;
  for (int i = tid; i < kSelBins; i += kSelT) hl[i] = 0u;
  for (int i = tid; i < kSelChunk; i += kSelT) st[i] = (t0 + i >= S - a.keep_recent) ? kProt : kFree;
  __syncthreads();
  // protected pending pages, then retired pages (retired wins)
  {
    const int off = a.pend_off[s], n = a.pend_off[s + 1] - off;
    for (int idx = tid; idx < n * kMaxPage; idx += kSelT) {
      const int i = idx / kMaxPage, e = idx % kMaxPage;
      const int t = a.pend_start[off + i] + e;
      if (a.pend_prot[off + i] && e < a.pend_len[off + i] && t >= t0 && t < t1) st[t - t0] = kProt;
    }
  }
  __syncthreads();
  {
    const int off = a.ret_off[s], n = a.ret_off[s + 1] - off;
    for (int idx = tid; idx < n * kMaxPage; idx += kSelT) {
      const int i = idx / kMaxPage, e = idx % kMaxPage;
      const int t = a.ret_start[off + i] + e;
      if (e < a.ret_len[off + i] && t >= t0 && t < t1) st[t - t0] = kRet;
    }
    if (a.acc && a.acc[s].cand) {
      const AccPages ap = a.acc[s];
      const int nc = min(*ap.n_cand, ap.max_cand);
      for (int idx = tid; idx < nc * kMaxPage; idx += kSelT) {
        const int i = idx / kMaxPage, e = idx % kMaxPage;
        if (!ap.accepted[i]) continue;
        const int pg = ap.cand[i];
        if (pg < 0 || pg >= ap.n_pages || e >= ap.len[pg]) continue;
        const int t = ap.start[pg] + e;
        if (t >= t0 && t < t1) st[t - t0] = kRet;
      }
    }
  }
  __syncthreads();
  const float* sc = a.score + (size_t)s * a.score_seq_stride;
  uint32_t* kv = a.kv + (size_t)s * a.score_seq_stride;
  uint8_t* sto = a.state ? a.state + (size_t)s * a.score_seq_stride : nullptr;
  float f[kPerT];
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int t = t0 + u * kSelT + tid;
    f[u] = t < t1 ? sc[t] : 0.f;
  }
  int np = 0, nf = 0;
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int i = u * kSelT + tid, t = t0 + i;
    const bool in = t < t1;
    const uint8_t x = in ? st[i] : kRet;
    const uint32_t key = x == kProt ? kKeyProt : (x == kRet ? kKeyRet : score_key(f[u]));
    if (in) {
      kv[t] = key;
      if (sto) sto[t] = x;
    }
    np += x == kProt && in;
    nf += x == kFree && in;
    hist_add(hl, key >> kShift[0], in && x == kFree);
  }
  int tot;
  block_scan<kSelT>(np, tmp, tot);
  np = tot;
  block_scan<kSelT>(nf, tmp, tot);
  nf = tot;
  int32_t* ctrl = a.ctrl + (size_t)s * kSelCtrl;
  if (tid == 0) {
    atomicAdd(&ctrl[cNP], np);
    atomicAdd(&ctrl[cNF], nf);
  }
  bins_to_global(a.hist + (size_t)s * 3 * kSelBins, hl);
  const int nb = (S + kSelChunk - 1) / kSelChunk;
  if (!arrive_last(&ctrl[cArr0], nb, &s_flag)) return;
  // last workgroup of the sequence: k, the mode, and the first digit
  const int NP = __hip_atomic_load(&ctrl[cNP], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int NF = __hip_atomic_load(&ctrl[cNF], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int k = max(0, min(a.budget - NP, NF));
  const int mode = k == 0 ? kModeNone : (k == NF ? kModeAll : kModeRadix);
  __syncthreads();
  if (tid == 0) {
    ctrl[cK] = k;
    ctrl[cMode] = mode;
    ctrl[cPrefix] = 0;
    ctrl[cMask] = 0;
    ctrl[cNeed] = k;
    // all free tokens: every free key is > 0; none: no free key is >= ~0 - 1
    ctrl[cT] = mode == kModeAll ? 0 : (int)(kKeyProt - 1u);
    ctrl[cNeedEq] = 0;
  }
  __syncthreads();
  if (mode == kModeRadix) choose_digit(a, s, 0, tmp);
}

// histogram of digit p (1 or 2) among free keys matching the chosen prefix
__global__ __launch_bounds__(kSelT) void sel_pass(SelectArgs a, int p) {
  __shared__ unsigned int hl[kSelBins];
  __shared__ int tmp[kSelT / 64];
  __shared__ int s_flag;
  const int s = blockIdx.y;
  const int S = a.n_tokens[s];
  const int t0 = blockIdx.x * kSelChunk;
  int32_t* ctrl = a.ctrl + (size_t)s * kSelCtrl;
  if (t0 >= S || ctrl[cMode] != kModeRadix) return;
  const int t1 = min(S, t0 + kSelChunk);
  const int tid = threadIdx.x;
  for (int i = tid; i < kSelBins; i += kSelT) hl[i] = 0u;
  const uint32_t prefix = (uint32_t)ctrl[cPrefix], mask = (uint32_t)ctrl[cMask];
  const uint32_t* kv = a.kv + (size_t)s * a.score_seq_stride;
  uint32_t key[kPerT];
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int t = t0 + u * kSelT + tid;
    key[u] = t < t1 ? kv[t] : kKeyRet;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const bool act = key_free(key[u]) && (key[u] & mask) == prefix;
    hist_add(hl, (key[u] >> kShift[p]) & kDigit[p], act);
  }
  __syncthreads();
  bins_to_global(a.hist + ((size_t)s * 3 + p) * kSelBins, hl);
  const int nb = (S + kSelChunk - 1) / kSelChunk;
  if (!arrive_last(&ctrl[cArr0 + p], nb, &s_flag)) return;
  choose_digit(a, s, p, tmp);
}

// per chunk: tokens kept outright (protected, or free above the threshold
// key T) and free tokens with key == T
__global__ __launch_bounds__(kSelT) void sel_count(SelectArgs a) {
  __shared__ int tmp[kSelT / 64];
  const int s = blockIdx.y;
  const int S = a.n_tokens[s];
  const int t0 = blockIdx.x * kSelChunk;
  if (t0 >= S) return;
  const int t1 = min(S, t0 + kSelChunk);
  const int32_t* ctrl = a.ctrl + (size_t)s * kSelCtrl;
  const uint32_t T = (uint32_t)ctrl[cT];
  const uint32_t* kv = a.kv + (size_t)s * a.score_seq_stride;
  int nk = 0, ne = 0;
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int t = t0 + u * kSelT + threadIdx.x;
    const uint32_t key = t < t1 ? kv[t] : kKeyRet;
    nk += (key == kKeyProt || (key_free(key) && key > T)) ? 1 : 0;
    ne += (key_free(key) && key == T) ? 1 : 0;
  }
  int tk, te;
  block_scan<kSelT>(nk, tmp, tk);
  block_scan<kSelT>(ne, tmp, te);
  if (threadIdx.x == 0) {
    int32_t* w = a.wcnt + ((size_t)s * a.n_chunks + blockIdx.x) * 2;
    w[0] = tk;
    w[1] = te;
  }
}

// kept indices of the chunk, in order, at the chunk's offset
__global__ __launch_bounds__(kSelT) void sel_write(SelectArgs a) {
  __shared__ int tmp[kSelT / 64];
  const int s = blockIdx.y;
  const int S = a.n_tokens[s];
  const int t0 = blockIdx.x * kSelChunk;
  const int32_t* ctrl = a.ctrl + (size_t)s * kSelCtrl;
  const int n_kept = ctrl[cNP] + ctrl[cK];
  int32_t* kept = a.kept + (size_t)s * a.budget;
  // pad the tail of the index list
  for (int j = n_kept + blockIdx.x * kSelT + (int)threadIdx.x; j < a.budget; j += gridDim.x * kSelT) kept[j] = -1;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.n_kept[s] = n_kept;
  if (t0 >= S) return;
  const int t1 = min(S, t0 + kSelChunk);
  const uint32_t T = (uint32_t)ctrl[cT];
  const int need_eq = ctrl[cNeedEq];
  // offsets from the chunks before this one
  int out = 0, eq_before = 0;
  const int32_t* wc = a.wcnt + (size_t)s * a.n_chunks * 2;
  for (int w = 0; w < (int)blockIdx.x; ++w) {
    const int nk = wc[2 * w], ne = wc[2 * w + 1];
    out += nk + max(0, min(ne, need_eq - eq_before));
    eq_before += ne;
  }
  const uint32_t* kv = a.kv + (size_t)s * a.score_seq_stride;
  uint32_t key[kPerT];
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int t = t0 + u * kSelT + threadIdx.x;
    key[u] = t < t1 ? kv[t] : kKeyRet;
  }
  // rounds of kSelT consecutive tokens: ranks from an exclusive scan
#pragma unroll
  for (int u = 0; u < kPerT; ++u) {
    const int t = t0 + u * kSelT + threadIdx.x;
    const bool eq = key_free(key[u]) && key[u] == T;
    int te;
    const int eq_rank = eq_before + block_scan<kSelT>(eq ? 1 : 0, tmp, te);
    eq_before += te;
    const bool keep = key[u] == kKeyProt || (key_free(key[u]) && key[u] > T) || (eq && eq_rank < need_eq);
    int tk;
    const int pos = out + block_scan<kSelT>(keep ? 1 : 0, tmp, tk);
    if (keep && pos < a.budget) kept[pos] = t;
    out += tk;
  }
}

hipError_t launch_protect(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(protect_kernel, dim3(a.n_seq), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const dim3 grid(a.n_chunks, a.n_seq), block(kSelT);
  hipLaunchKernelGGL(sel_keys, grid, block, 0, s, a);
  hipError_t e = hipGetLastError();
  for (int p = 1; p <= 2 && e == hipSuccess; ++p) {
    hipLaunchKernelGGL(sel_pass, grid, block, 0, s, a, p);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sel_count, grid, block, 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(sel_write, grid, block, 0, s, a);
  return hipGetLastError();
}

// wave-level helpers of the grid selection
namespace {
__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// one combining round for the most common bin of the wave, then plain atomics
__device__ __forceinline__ void hist_add1(unsigned int* hist, uint32_t bin, bool act) {
  const unsigned long long m = __ballot(act);
  if (m == 0ull) return;
  const int leader = __ffsll((long long)m) - 1;      // uniform: a scalar read of its bin
  const uint32_t lb = (uint32_t)__builtin_amdgcn_readlane((int)bin, leader);
  const bool same = act && bin == lb;
  const unsigned long long sm = __ballot(same);
  if ((int)(threadIdx.x & 63) == leader) atomicAdd(&hist[lb], (unsigned int)__popcll(sm));
  if (act && !same) atomicAdd(&hist[bin], 1u);
}
}  // namespace

// ---------------------------------------------------------------------------
// Grid selection: one kQT-thread workgroup per kSelGridChunk tokens of a
// sequence (grid: chunks x sequences), every workgroup resident at once.
// Phases are separated by a per-sequence grid barrier with a bounded wait:
//   0. scores, protection (every workgroup ranks the pending pages itself),
//      token states and keys of the chunk; #protected, #free and the range
//      of the free keys go to the sequence's control words;
//   1. up to three narrowings of the threshold range: chunk histograms are
//      added into a global histogram, then every workgroup makes the same
//      choice from it;
//   2. per-chunk counts of kept tokens and of ties at the threshold, then
//      the ordered write at the chunk's offset.
// The control words and histograms start at zero (allocated zeroed); the
// last workgroup of a sequence to finish clears them again for the next
// call, and marks a call whose barrier timed out with n_kept = -1.  Every
// word that crosses workgroups (control words, histograms, the candidate
// list, chunk counts, n_kept) moves through agent-scope atomics, so the
// barrier needs no fence (one writes back and invalidates the whole L2 of
// the workgroup's XCD); the workgroup barrier before an arrival waits for
// the workgroup's own memory operations.
// ---------------------------------------------------------------------------
namespace {
constexpr int kQT = 256;
constexpr int kQW = kQT / 64;
constexpr int kQKPT = kSelGridChunk / kQT;   // keys per thread
static_assert(kSelGridPendMax <= kQT, "one pending page per thread");
enum { qArrive = 0, qDone = 1, qNP = 2, qNF = 3, qNotLo = 4, qHi = 5, qError = 6, qCand = 7, qCounts = 8 };
// when the threshold bin of the first pass holds at most this many free
// keys, they are listed (in the histogram rows of the later passes) and every
// workgroup finishes the selection on the list in LDS: no further grid pass
constexpr int kCandMax = kSelBins;

__device__ bool seq_barrier(int* ctrl, int target, long long timeout, int* s_ok) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(&ctrl[qArrive], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long t0 = wall_clock64();
    int ok = 1;
    if (timeout <= 0) {   // a zero bound gives up at once: the failure path, forced
      __hip_atomic_store(&ctrl[qError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ok = 0;
    }
    while (ok && __hip_atomic_load(&ctrl[qArrive], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(&ctrl[qError], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
          wall_clock64() - t0 >= timeout) {
        __hip_atomic_store(&ctrl[qError], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

__device__ __forceinline__ int ld_agent(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// sum of the chunk counts (which = 0: kept, 1: ties) of the chunks before
// chunk cb (< 64): lane q reads chunk q, the same sum in every wave
__device__ __forceinline__ int counts_before(const int* ctrl, int cb, int which) {
  const int q = threadIdx.x & 63;
  return wave_sum(q < cb ? ld_agent(&ctrl[qCounts + 2 * q + which]) : 0);
}
}  // namespace

__global__ __launch_bounds__(kQT) void select_grid(SelectArgs a) {
  __shared__ uint8_t sRet[kSelGridChunk], sPro[kSelGridChunk];
  __shared__ unsigned int hist[kSelBins];
  __shared__ float sR[kSelGridPendMax];
  __shared__ int sLen[kSelGridPendMax], sStart[kSelGridPendMax], sOrd[kSelGridPendMax];
  __shared__ uint8_t sProt[kSelGridPendMax];
  __shared__ int tmp[kQW], wa[kQW], wb[kQW];
  __shared__ uint32_t wlo[kQW], whi[kQW];
  __shared__ uint32_t s_lo, s_hi;
  __shared__ int s_need, s_ok, s_m;
  __shared__ uint32_t sCk[kCandMax];
  __shared__ int sCi[kCandMax];
  const int s = blockIdx.y, cb = blockIdx.x, C = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int* ctrl = a.gctrl + (size_t)s * kSelGridCtrl;
  uint32_t* gh = a.ghist + (size_t)s * 3 * kSelBins;
  const int c0 = cb * kSelGridChunk;
  // the scores first: their loads overlap everything up to the keys
  const float* sc = a.score + (size_t)s * a.score_seq_stride;
  const int t_base = c0 + wave * 64 * kQKPT + lane;
  float f[kQKPT];
#pragma unroll
  for (int u = 0; u < kQKPT; ++u) {
    const int t = t_base + 64 * u;
    f[u] = t < a.score_seq_stride ? sc[t] : 0.f;
  }
  const int S = a.n_tokens[s];
  const int c1 = min(S, c0 + kSelGridChunk);          // chunk [c0, c1), empty if c0 >= S
  const int poff = a.pend_off[s], n = a.pend_off[s + 1] - poff;   // n <= kSelGridPendMax
  const int roff = a.ret_off[s], nr = a.ret_off[s + 1] - roff;
  const float* R = reinterpret_cast<const float*>(a.pend_r[s]);
  const AccPages ap = a.acc ? a.acc[s] : AccPages{};
  // The loads of each thread's first pending page, retired page and accepted
  // candidate (with its page span) are issued before the LDS is cleared, so
  // their latencies overlap one another and the barrier; a candidate's flag
  // and page index do not wait for the candidate count.
  float pr = 0.f;
  int pln = 0, pst = 0, rst = 0, rln = 0, ast = 0, aln = 0;
  if (tid < n) {
    pr = pend_key(R[tid]);
    pln = a.pend_len[poff + tid];
    pst = a.pend_start[poff + tid];
  }
  if (tid < nr) {
    rst = a.ret_start[roff + tid];
    rln = a.ret_len[roff + tid];
  }
  int nc = 0;
  if (ap.cand) {
    nc = min(*ap.n_cand, ap.max_cand);
    if (tid < ap.max_cand) {
      const uint8_t acc = ap.accepted[tid];
      const int pg = ap.cand[tid];
      if (acc && pg >= 0 && pg < ap.n_pages) {
        ast = ap.start[pg];
        aln = ap.len[pg];
      }
    }
  }
  for (int i = tid; i < kSelGridChunk / 4; i += kQT) {
    reinterpret_cast<uint32_t*>(sRet)[i] = 0u;
    reinterpret_cast<uint32_t*>(sPro)[i] = 0u;
  }
  __syncthreads();
  // pending pages to LDS; retired and accepted pages that overlap the chunk
  // marked meanwhile
  if (tid < n) {
    sR[tid] = pr;
    sLen[tid] = pln;
    sStart[tid] = pst;
    sProt[tid] = 0;
  }
  if (tid < nr)
    for (int t = max(rst, c0); t < min(rst + rln, c1); ++t) sRet[t - c0] = 1;
  for (int i = tid + kQT; i < nr; i += kQT) {
    const int st = a.ret_start[roff + i], ln = a.ret_len[roff + i];
    for (int t = max(st, c0); t < min(st + ln, c1); ++t) sRet[t - c0] = 1;
  }
  if (tid < nc)
    for (int t = max(ast, c0); t < min(ast + aln, c1); ++t) sRet[t - c0] = 1;
  for (int i = tid + kQT; i < nc; i += kQT) {
    if (!ap.accepted[i]) continue;
    const int pg = ap.cand[i];
    if (pg < 0 || pg >= ap.n_pages) continue;
    const int st = ap.start[pg], ln = ap.len[pg];
    for (int t = max(st, c0); t < min(st + ln, c1); ++t) sRet[t - c0] = 1;
  }
  __syncthreads();
  // Eq. (12): pending pages ranked by (R- descending, page order), protected
  // in that order while fewer than max_pages are taken and the tokens fit B_N
  {
    int G = 64;
    while (G > 1 && G * n > kQT) G >>= 1;
    for (int i = tid / G; i < n; i += kQT / G) {
      const float ri = sR[i];
      int rank = 0;
      for (int j = tid % G; j < n; j += G) {
        const float rj = sR[j];
        rank += (rj > ri || (rj == ri && j < i)) ? 1 : 0;
      }
      for (int off = G / 2; off >= 1; off >>= 1) rank += __shfl_xor(rank, off, 64);
      if (tid % G == 0) sOrd[rank] = i;
    }
  }
  __syncthreads();
  {
    // thread r takes rank r (n <= kQT): protected while r < max_pages and
    // the running token total in rank order, this page included, fits B_N;
    // the total only grows, so this is the prefix the rule above takes
    const int li = tid < n ? sLen[sOrd[tid]] : 0;
    int total;
    const int before = block_scan<kQT>(li, tmp, total);
    if (tid < n && tid < a.max_pages && before + li <= a.bn) sProt[sOrd[tid]] = 1;
  }
  __syncthreads();
  for (int i = tid; i < n; i += kQT) {
    if (!sProt[i]) continue;
    for (int t = max(sStart[i], c0); t < min(sStart[i] + sLen[i], c1); ++t) sPro[t - c0] = 1;
  }
  __syncthreads();

  // token states (retired wins over protected) and coded keys
  uint32_t key[kQKPT];
  int np = 0, nf = 0;
  uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
  for (int u = 0; u < kQKPT; ++u) {
    const int t = t_base + 64 * u, i = t - c0;
    const bool in = t < c1;
    const uint8_t x = !in || sRet[i] ? kRet : ((sPro[i] || t >= S - a.keep_recent) ? kProt : kFree);
    key[u] = x == kProt ? kKeyProt : (x == kRet ? kKeyRet : score_key(f[u]));
    np += x == kProt ? 1 : 0;
    nf += x == kFree ? 1 : 0;
    if (x == kFree) {
      lo = min(lo, key[u]);
      hi = max(hi, key[u]);
    }
  }
  if (a.state) {
    uint8_t* sto = a.state + (size_t)s * a.score_seq_stride;
    for (int t = c0 + tid; t < c1; t += kQT)
      sto[t] = sRet[t - c0] ? kRet : ((sPro[t - c0] || t >= S - a.keep_recent) ? kProt : kFree);
  }
  np = wave_sum(np);
  nf = wave_sum(nf);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, off, 64));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, off, 64));
  }
  if (lane == 0) { wa[wave] = np; wb[wave] = nf; wlo[wave] = lo; whi[wave] = hi; }
  __syncthreads();
  if (tid == 0) {
    int NPc = 0, NFc = 0;
    uint32_t l = 0xFFFFFFFFu, h = 0u;
    for (int w = 0; w < kQW; ++w) { NPc += wa[w]; NFc += wb[w]; l = min(l, wlo[w]); h = max(h, whi[w]); }
    if (NPc) atomicAdd(&ctrl[qNP], NPc);
    if (NFc) {
      atomicAdd(&ctrl[qNF], NFc);
      atomicMax(reinterpret_cast<unsigned int*>(&ctrl[qNotLo]), ~l);   // the minimum, as a maximum of ~key
      atomicMax(reinterpret_cast<unsigned int*>(&ctrl[qHi]), h);
    }
  }
  int target = C;
  bool ok = seq_barrier(ctrl, target, a.barrier_ticks, &s_ok);
  int32_t* kept = a.kept + (size_t)s * a.budget;
  if (ok) {
    const int NP = ld_agent(&ctrl[qNP]), NF = ld_agent(&ctrl[qNF]);
    lo = ~(uint32_t)ld_agent(&ctrl[qNotLo]);
    hi = (uint32_t)ld_agent(&ctrl[qHi]);
    // Eq. (13): the k = min(B - #protected, #free) largest free keys
    const int k = max(0, min(a.budget - NP, NF));
    uint32_t T;
    int need_eq = 0;
    bool listed = false;                 // threshold decided from the candidate list
    int k_before = 0, e_before = 0;      // kept tokens and ties at T in the chunks before this one
    if (k == 0) {
      T = kKeyProt - 1u;                 // no free key reaches it
    } else if (k == NF) {
      T = 0u;                            // every free key is above it
    } else {
      int need = k;
      for (int pass = 0; pass < 3 && lo != hi; ++pass) {
        const uint32_t range = hi - lo;
        const int shift = max(0, 32 - __clz((int)range) - 11);
        for (int i = tid; i < kSelBins; i += kQT) hist[i] = 0u;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kQKPT; ++u) {
          const uint32_t kk = key[u];
          const bool act = key_free(kk) && kk >= lo && kk <= hi;
          hist_add1(hist, (kk - lo) >> shift, act);
        }
        __syncthreads();
        for (int i = tid; i < kSelBins; i += kQT)
          if (hist[i]) atomicAdd(&gh[pass * kSelBins + i], hist[i]);
        target += C;
        if (!seq_barrier(ctrl, target, a.barrier_ticks, &s_ok)) { ok = false; break; }
        // thread g owns bins 8(kQT-1-g) .. 8(kQT-1-g)+7: an exclusive scan in
        // thread order counts the keys in higher bins
        const int g = kQT - 1 - tid;
        int h[8], sum = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          h[j] = (int)__hip_atomic_load(&gh[pass * kSelBins + 8 * g + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          sum += h[j];
        }
        int total;
        int above = block_scan<kQT>(sum, tmp, total);
#pragma unroll
        for (int j = 7; j >= 0; --j) {
          if (above < need && above + h[j] >= need) {
            const uint32_t nlo = lo + ((uint32_t)(8 * g + j) << shift);
            const uint32_t width = (1u << shift) - 1u;
            s_lo = nlo;
            s_hi = min(hi, nlo + min(width, 0xFFFFFFFFu - nlo));
            s_need = need - above;
            s_m = h[j];
          }
          above += h[j];
        }
        __syncthreads();
        lo = s_lo;
        hi = s_hi;
        need = s_need;
        // few keys left in the bin: list them instead of narrowing further
        if (pass == 0 && lo != hi && s_m <= kCandMax) {
          listed = true;
          break;
        }
      }
      if (ok && listed) {
        // every free key in [lo, hi] goes to the sequence's candidate list
        // (the histogram rows of the later passes, unused on this path);
        // the chunk publishes how many of its tokens are kept outright
        uint32_t* gc = gh + kSelBins;
        int nk = 0, nin = 0;
        unsigned long long inm[kQKPT];
#pragma unroll
        for (int u = 0; u < kQKPT; ++u) {
          const uint32_t kk = key[u];
          nk += (kk == kKeyProt || (key_free(kk) && kk > hi)) ? 1 : 0;
          inm[u] = __ballot(key_free(kk) && kk >= lo && kk <= hi);
          nin += __popcll(inm[u]);
        }
        // one slot reservation per wave for all of its keys in the bin
        int base = 0;
        if (nin && lane == 0) base = atomicAdd(&ctrl[qCand], nin);
        base = __shfl(base, 0, 64);
#pragma unroll
        for (int u = 0; u < kQKPT; ++u) {
          const int slot = base + lanes_below(inm[u]);
          base += __popcll(inm[u]);
          if (((inm[u] >> lane) & 1ull) && slot < kCandMax) {
            st_agent(&gc[2 * slot], key[u]);
            st_agent(&gc[2 * slot + 1], (uint32_t)(t_base + 64 * u));
          }
        }
        nk = wave_sum(nk);
        __syncthreads();
        if (lane == 0) wa[wave] = nk;
        __syncthreads();
        if (tid == 0) {
          int tk = 0;
          for (int w = 0; w < kQW; ++w) tk += wa[w];
          st_agent(&ctrl[qCounts + 2 * cb], tk);
        }
        target += C;
        ok = seq_barrier(ctrl, target, a.barrier_ticks, &s_ok);
        if (ok) {
          const int M = min(ld_agent(&ctrl[qCand]), kCandMax);
          {
            // every load of the list in flight before the first LDS store
            constexpr int kCPT = kCandMax / kQT;
            uint32_t ck[kCPT], ci[kCPT];
#pragma unroll
            for (int j = 0; j < kCPT; ++j) {
              const int i = tid + j * kQT;
              ck[j] = i < M ? __hip_atomic_load(&gc[2 * i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
              ci[j] = i < M ? __hip_atomic_load(&gc[2 * i + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
            }
#pragma unroll
            for (int j = 0; j < kCPT; ++j) {
              const int i = tid + j * kQT;
              if (i < M) {
                sCk[i] = ck[j];
                sCi[i] = (int)ci[j];
              }
            }
          }
          // the same narrowing as the grid passes, on the list in LDS
          while (lo != hi) {
            const uint32_t range = hi - lo;
            const int shift = max(0, 32 - __clz((int)range) - 11);
            for (int i = tid; i < kSelBins; i += kQT) hist[i] = 0u;
            __syncthreads();
            for (int i = tid; i < M; i += kQT) {
              const uint32_t kk = sCk[i];
              if (kk >= lo && kk <= hi) atomicAdd(&hist[(kk - lo) >> shift], 1u);
            }
            __syncthreads();
            const int g = kQT - 1 - tid;
            int h[8], sum = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              h[j] = (int)hist[8 * g + j];
              sum += h[j];
            }
            int total;
            int above = block_scan<kQT>(sum, tmp, total);
#pragma unroll
            for (int j = 7; j >= 0; --j) {
              if (above < need && above + h[j] >= need) {
                const uint32_t nlo = lo + ((uint32_t)(8 * g + j) << shift);
                const uint32_t width = (1u << shift) - 1u;
                s_lo = nlo;
                s_hi = min(hi, nlo + min(width, 0xFFFFFFFFu - nlo));
                s_need = need - above;
              }
              above += h[j];
            }
            __syncthreads();
            lo = s_lo;
            hi = s_hi;
            need = s_need;
          }
          T = lo;                        // the need-th largest key; need ties at T are kept
          need_eq = need;
          // what the chunks before this one hold of the listed keys: counted
          // per thread, then added over the block (LDS atomics on two words
          // would serialise over the whole list)
          int gt = 0, eq = 0;
          for (int i = tid; i < M; i += kQT) {
            if (sCi[i] >= c0) continue;
            gt += sCk[i] > T ? 1 : 0;
            eq += sCk[i] == T ? 1 : 0;
          }
          gt = wave_sum(gt);
          eq = wave_sum(eq);
          if (lane == 0) { wa[wave] = gt; wb[wave] = eq; }
          __syncthreads();
#pragma unroll
          for (int w = 0; w < kQW; ++w) { k_before += wa[w]; e_before += wb[w]; }
          __syncthreads();
          k_before += counts_before(ctrl, cb, 0);
        }
      } else {
        T = lo;                          // lo == hi: the need-th largest key
        need_eq = need;
      }
    }
    if (ok) {
      // per-wave counts of kept tokens and of ties at T
      int nk = 0, ne = 0;
#pragma unroll
      for (int u = 0; u < kQKPT; ++u) {
        const uint32_t kk = key[u];
        nk += (kk == kKeyProt || (key_free(kk) && kk > T)) ? 1 : 0;
        ne += (key_free(kk) && kk == T) ? 1 : 0;
      }
      nk = wave_sum(nk);
      ne = wave_sum(ne);
      __syncthreads();
      if (lane == 0) { wa[wave] = nk; wb[wave] = ne; }
      __syncthreads();
      if (!listed) {
        // the chunks' totals, exchanged through the control words
        if (tid == 0) {
          int tk = 0, te = 0;
          for (int w = 0; w < kQW; ++w) { tk += wa[w]; te += wb[w]; }
          st_agent(&ctrl[qCounts + 2 * cb], tk);
          st_agent(&ctrl[qCounts + 2 * cb + 1], te);
        }
        target += C;
        ok = seq_barrier(ctrl, target, a.barrier_ticks, &s_ok);
        if (ok)
          {
            k_before += counts_before(ctrl, cb, 0);
            e_before += counts_before(ctrl, cb, 1);
          }
      }
    }
    if (ok) {
      // offsets from the chunks before this one and the waves before this one
      for (int w = 0; w < wave; ++w) { k_before += wa[w]; e_before += wb[w]; }
      int out = k_before + min(need_eq, e_before), eq_run = e_before;
#pragma unroll
      for (int u = 0; u < kQKPT; ++u) {
        const int t = t_base + 64 * u;
        const uint32_t kk = key[u];
        const bool eq = key_free(kk) && kk == T;
        const unsigned long long em = __ballot(eq);
        const int eq_rank = eq_run + lanes_below(em);
        eq_run += __popcll(em);
        const bool keep = kk == kKeyProt || (key_free(kk) && kk > T) || (eq && eq_rank < need_eq);
        const unsigned long long km = __ballot(keep);
        const int pos = out + lanes_below(km);
        out += __popcll(km);
        if (keep && pos < a.budget) kept[pos] = t;
      }
      const int n_kept = min(a.budget, NP + k);
      for (int j = n_kept + cb * kQT + tid; j < a.budget; j += C * kQT) kept[j] = -1;
      if (cb == 0 && tid == 0) st_agent(&a.n_kept[s], n_kept);   // ordered before a give-up's -1
    }
  }
  // the last workgroup of the sequence clears the control words and the
  // histograms for the next call (every other workgroup is done with them)
  __syncthreads();
  if (tid == 0) s_ok = __hip_atomic_fetch_add(&ctrl[qDone], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == C - 1;
  __syncthreads();
  if (s_ok) {
    if (tid == 0 && ld_agent(&ctrl[qError]) != 0) st_agent(&a.n_kept[s], -1);
    for (int i = tid; i < 3 * kSelBins; i += kQT) st_agent(&gh[i], 0u);
    for (int i = tid; i < kSelGridCtrl; i += kQT) st_agent(&ctrl[i], 0);
  }
}

bool select_grid_fits(int max_tokens, int max_pending, int n_seq, int resident) {
  const int C = (max_tokens + kSelGridChunk - 1) / kSelGridChunk;
  return max_pending <= kSelGridPendMax && C <= kSelGridMaxChunks && (int64_t)C * n_seq <= resident;
}

int select_grid_resident() {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, select_grid, kQT, 0) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return per_cu * cus;
}

hipError_t launch_select_grid(const SelectArgs& a, int max_tokens, hipStream_t s) {
  const int C = (max_tokens + kSelGridChunk - 1) / kSelGridChunk;
  hipLaunchKernelGGL(select_grid, dim3(C, a.n_seq), dim3(kQT), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// gather: grid (row chunks, seq*layer*head); 16 bytes per lane per row chunk
// ---------------------------------------------------------------------------
namespace {
constexpr int kGT = 256;
constexpr int kGRows = 128;   // rows per block
}

template <int D>
__global__ __launch_bounds__(kGT) void gather_kernel(GatherArgs g) {
  constexpr int CPR = D / 8;               // 16-byte chunks per row
  constexpr int RPI = kGT / CPR;           // rows per iteration
  const int combo = blockIdx.y;
  const int s = combo / (g.n_layers * g.Hkv);
  const int rem = combo % (g.n_layers * g.Hkv);
  const int l = rem / g.Hkv, h = rem % g.Hkv;
  const int nk0 = g.n_kept[s];   // -1: the selection gave up
  const int nk = nk0 < 0 ? nk0 : (int)CKV_IDX(nk0, g.budget + 1, g.dbg, 15);
  const int j0 = blockIdx.x * kGRows;
  if (j0 >= nk) return;
  const int32_t* kept = g.kept + (size_t)s * g.budget;
  const uint16_t* kin = g.k_in + s * g.in_seq + l * g.in_layer + h * g.in_head;
  const uint16_t* vin = g.v_in + s * g.in_seq + l * g.in_layer + h * g.in_head;
  uint16_t* kout = g.k_out + s * g.out_seq + l * g.out_layer + h * g.out_head;
  uint16_t* vout = g.v_out + s * g.out_seq + l * g.out_layer + h * g.out_head;
  const int cc = threadIdx.x % CPR;
  const int j1 = min(nk, j0 + kGRows);
#pragma unroll 4
  for (int j = j0 + threadIdx.x / CPR; j < j1; j += RPI) {
    const int src = (int)CKV_IDX(kept[j], g.in_rows, g.dbg, 14);
    const uint4 kv = *reinterpret_cast<const uint4*>(kin + (int64_t)src * g.in_tok + cc * 8);
    const uint4 vv = *reinterpret_cast<const uint4*>(vin + (int64_t)src * g.in_tok + cc * 8);
    *reinterpret_cast<uint4*>(kout + (int64_t)j * g.out_tok + cc * 8) = kv;
    *reinterpret_cast<uint4*>(vout + (int64_t)j * g.out_tok + cc * 8) = vv;
  }
  if (l == 0 && h == 0) {
    for (int j = j0 + threadIdx.x; j < j1; j += kGT)
      g.pos_out[s * g.pos_out_seq + j] = g.pos_in[s * g.pos_in_seq + CKV_IDX(kept[j], g.in_rows, g.dbg, 14)];
  }
}

hipError_t launch_gather(const GatherArgs& g, hipStream_t s) {
  dim3 grid((g.budget + kGRows - 1) / kGRows, g.n_seq * g.n_layers * g.Hkv);
  if (grid.y == 0 || grid.x == 0) return hipSuccess;
  if (g.D == 128) hipLaunchKernelGGL((gather_kernel<128>), grid, dim3(kGT), 0, s, g);
  else hipLaunchKernelGGL((gather_kernel<64>), grid, dim3(kGT), 0, s, g);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Pooled base score (the SnapKV-style variant of the score that fills the
// budget): out[t] = max (mode 0) or mean (mode 1) of score[j] over the tokens
// j in [t - h, t + h] that lie inside [0, n_tokens), h = kernel / 2.  The max
// ignores NaN entries (NaN only if the whole window is); the mean adds the
// window in index order in float32.  One thread per token;
// grid: (token blocks, sequences).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pool_kernel(const float* score, float* out, int64_t stride,
                                                   const int32_t* n_tokens, int half, int mode) {
  const int s = blockIdx.y;
  const int n = n_tokens[s];
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= n) return;
  const float* x = score + (int64_t)s * stride;
  const int j0 = max(0, t - half), j1 = min(n - 1, t + half);
  float acc = mode == 0 ? -INFINITY : 0.f;
  bool any = false;   // max: a window of NaN only gives NaN
  for (int j = j0; j <= j1; ++j) {
    const float v = x[j];
    any = any || v == v;
    acc = mode == 0 ? fmaxf(acc, v) : acc + v;
  }
  out[(int64_t)s * stride + t] = mode == 0 ? (any ? acc : NAN) : acc / (float)(j1 - j0 + 1);
}

hipError_t launch_pool(const float* score, float* out, int64_t stride, const int32_t* n_tokens, int n_seq,
                       int max_tokens, int kernel, int mode, hipStream_t s) {
  if (max_tokens <= 0 || n_seq <= 0) return hipSuccess;
  dim3 grid((max_tokens + 255) / 256, n_seq), block(256);
  hipLaunchKernelGGL(pool_kernel, grid, block, 0, s, score, out, stride, n_tokens, kernel / 2, mode);
  return hipGetLastError();
}

}  // namespace ckv
