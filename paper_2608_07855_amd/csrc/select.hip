// Compression checkpoint (CommitKV, Sec. 3.3, Eq. (12)-(13); Sec. 3.1, Eq. (4)).
//
// protect_kernel (one block per sequence): pending pages are ranked by
//   (R- descending, page order ascending) by counting, and protected in that
//   order while fewer than max_pages are taken and the token total stays
//   within B_N; the first page that does not fit stops the protection.
// select_kernel (one block per sequence): token states (retired > protected >
//   free), then the k = min(B - #protected, #free) free tokens with the
//   largest score are found by a 4-pass 8-bit radix select on an order-
//   preserving 32-bit image of the score; ties at the threshold go to the
//   lowest indices.  Kept indices are written in ascending order.
// gather_kernel: K'[s,l,g,j] = K[s,l,g,I[j]], the same for V, and
//   pos'[s,j] = pos[s,I[j]], 16-byte vector copies of whole rows.
#include "ckv_device.h"
#include "ckv_kernels.h"

namespace ckv {

namespace {
constexpr int kST = 1024;   // threads of the selection block
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

__global__ __launch_bounds__(256) void protect_kernel(SelectArgs a) {
  const int s = blockIdx.x;
  const int off = a.pend_off[s];
  const int n = a.pend_off[s + 1] - off;
  const float* R = reinterpret_cast<const float*>(a.pend_r[s]);
  const int32_t* len = a.pend_len + off;
  uint8_t* prot = a.pend_prot + off;
  int32_t* ord = a.pend_ord + off;
  for (int i = threadIdx.x; i < n; i += 256) {
    const float ri = pend_key(R[i]);
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const float rj = pend_key(R[j]);
      rank += (rj > ri || (rj == ri && j < i)) ? 1 : 0;
    }
    ord[rank] = i;
    prot[i] = 0;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int taken = 0, tok = 0;
    for (int r = 0; r < n; ++r) {
      const int i = ord[r];
      if (taken >= a.max_pages || tok + len[i] > a.bn) break;
      prot[i] = 1;
      ++taken;
      tok += len[i];
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

// block-wide exclusive scan of one int per thread (kST threads)
__device__ int block_exclusive_scan(int v, int* tmp, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) tmp[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < kST / 64; ++i) {
      const int t = tmp[i];
      tmp[i] = run;
      run += t;
    }
    tmp[kST / 64] = run;
  }
  __syncthreads();
  const int res = tmp[w] + x - v;
  total = tmp[kST / 64];
  __syncthreads();
  return res;
}

__global__ __launch_bounds__(kST) void select_kernel(SelectArgs a) {
  __shared__ unsigned int hist[256];
  __shared__ int tmp[kST / 64 + 1];
  __shared__ unsigned int s_prefix, s_mask;
  __shared__ int s_need;
  const int s = blockIdx.x;
  const int S = a.n_tokens[s];
  uint8_t* st = a.state + (size_t)s * a.score_seq_stride;
  const float* sc = a.score + (size_t)s * a.score_seq_stride;
  const int tid = threadIdx.x;

  // token states: recent -> protected; protected pending pages; retired pages
  for (int t = tid; t < S; t += kST) st[t] = (t >= S - a.keep_recent) ? kProt : kFree;
  __syncthreads();
  {
    const int off = a.pend_off[s], n = a.pend_off[s + 1] - off;
    for (int idx = tid; idx < n * kMaxPage; idx += kST) {
      const int i = idx / kMaxPage, e = idx % kMaxPage;
      if (a.pend_prot[off + i] && e < a.pend_len[off + i]) st[a.pend_start[off + i] + e] = kProt;
    }
  }
  __syncthreads();
  {
    const int off = a.ret_off[s], n = a.ret_off[s + 1] - off;
    for (int idx = tid; idx < n * kMaxPage; idx += kST) {
      const int i = idx / kMaxPage, e = idx % kMaxPage;
      if (e < a.ret_len[off + i]) st[a.ret_start[off + i] + e] = kRet;
    }
  }
  __syncthreads();

  // counts
  int np = 0, nf = 0;
  for (int t = tid; t < S; t += kST) {
    const uint8_t x = st[t];
    np += x == kProt;
    nf += x == kFree;
  }
  int tot_p, tot_f;
  block_exclusive_scan(np, tmp, tot_p);
  block_exclusive_scan(nf, tmp, tot_f);
  const int k = max(0, min(a.budget - tot_p, tot_f));

  // radix select of the k-th largest key among free tokens
  bool take_all = (k == tot_f);
  if (tid == 0) { s_prefix = 0u; s_mask = 0u; s_need = k; }
  __syncthreads();
  if (k > 0 && !take_all) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      for (int i = tid; i < 256; i += kST) hist[i] = 0u;
      __syncthreads();
      const unsigned int prefix = s_prefix, mask = s_mask;
      for (int t0 = 0; t0 < S; t0 += kST) {
        const int t = t0 + tid;
        bool act = false;
        uint32_t bin = 0;
        if (t < S && st[t] == kFree) {
          const uint32_t key = score_key(sc[t]);
          act = (key & mask) == prefix;
          bin = (key >> shift) & 255u;
        }
        hist_add(hist, bin, act);
      }
      __syncthreads();
      if (tid == 0) {
        int need = s_need;
        int d = 255;
        for (; d > 0; --d) {
          if ((int)hist[d] >= need) break;
          need -= (int)hist[d];
        }
        s_prefix = prefix | ((unsigned int)d << shift);
        s_mask = mask | (255u << shift);
        s_need = need;
      }
      __syncthreads();
    }
  }
  const uint32_t T = s_prefix;
  const int need_eq = s_need;     // how many tokens with key == T to keep

  // One ordered sweep in blocks of kST tokens (one per thread, coalesced):
  // a free token with key == T is kept while fewer than need_eq such tokens
  // precede it; kept tokens are written in ascending order.  Prefix counts
  // inside a wave come from ballots, across the 16 waves from LDS.
  int32_t* kept = a.kept + (size_t)s * a.budget;
  const int lane = tid & 63, w = tid >> 6;
  const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int eq_run = 0, out_run = 0;
  for (int t0 = 0; t0 < S; t0 += kST) {
    const int t = t0 + tid;
    bool prot = false, free_gt = false, free_eq = false;
    if (t < S) {
      const uint8_t x = st[t];
      prot = x == kProt;
      if (x == kFree && k > 0) {
        if (take_all) free_gt = true;
        else {
          const uint32_t key = score_key(sc[t]);
          free_gt = key > T;
          free_eq = key == T;
        }
      }
    }
    // rank of this token among the block's key == T tokens
    const unsigned long long me = __ballot(free_eq);
    if (lane == 0) tmp[w] = __popcll(me);
    __syncthreads();
    int wbase = 0, btot = 0;
    for (int i = 0; i < kST / 64; ++i) {
      const int c = tmp[i];
      wbase += i < w ? c : 0;
      btot += c;
    }
    const int eq_rank = eq_run + wbase + __popcll(me & lt_mask);
    eq_run += btot;
    const bool keep = prot || free_gt || (free_eq && eq_rank < need_eq);
    __syncthreads();
    const unsigned long long km = __ballot(keep);
    if (lane == 0) tmp[w] = __popcll(km);
    __syncthreads();
    int kbase = 0, ktot = 0;
    for (int i = 0; i < kST / 64; ++i) {
      const int c = tmp[i];
      kbase += i < w ? c : 0;
      ktot += c;
    }
    if (keep) kept[out_run + kbase + __popcll(km & lt_mask)] = t;
    out_run += ktot;
    __syncthreads();
  }
  for (int j = out_run + tid; j < a.budget; j += kST) kept[j] = -1;
  if (tid == 0) a.n_kept[s] = out_run;
}

hipError_t launch_protect(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(protect_kernel, dim3(a.n_seq), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(select_kernel, dim3(a.n_seq), dim3(kST), 0, s, a);
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
  const int nk = g.n_kept[s];
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
    const int src = kept[j];
    const uint4 kv = *reinterpret_cast<const uint4*>(kin + (int64_t)src * g.in_tok + cc * 8);
    const uint4 vv = *reinterpret_cast<const uint4*>(vin + (int64_t)src * g.in_tok + cc * 8);
    *reinterpret_cast<uint4*>(kout + (int64_t)j * g.out_tok + cc * 8) = kv;
    *reinterpret_cast<uint4*>(vout + (int64_t)j * g.out_tok + cc * 8) = vv;
  }
  if (l == 0 && h == 0) {
    for (int j = j0 + threadIdx.x; j < j1; j += kGT)
      g.pos_out[s * g.pos_out_seq + j] = g.pos_in[s * g.pos_in_seq + kept[j]];
  }
}

hipError_t launch_gather(const GatherArgs& g, hipStream_t s) {
  dim3 grid((g.budget + kGRows - 1) / kGRows, g.n_seq * g.n_layers * g.Hkv);
  if (grid.y == 0 || grid.x == 0) return hipSuccess;
  if (g.D == 128) hipLaunchKernelGGL((gather_kernel<128>), grid, dim3(kGT), 0, s, g);
  else hipLaunchKernelGGL((gather_kernel<64>), grid, dim3(kGT), 0, s, g);
  return hipGetLastError();
}

}  // namespace ckv
