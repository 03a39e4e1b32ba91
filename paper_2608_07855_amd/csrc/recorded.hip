// Page deletion effects from recorded window outputs (CommitKV, Sec. 3.2:
// the engine records the window's attention outputs during its forward
// pass, so the window-attention pass of measure.hip is not needed).
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <algorithm>
#include <climits>

namespace ckv {

// ---------------------------------------------------------------------------
// Recorded window outputs.  The engine records o_p and the log-sum-exp of
// every window row during its forward pass; given those, only the per-page
// pass (and the token mass) has to run.  Two small kernels supply what the
// page kernel reads per row (log-sum-exp in log2 units, ||o_p||, visible
// token count), and the fix-up recomputes the ill-conditioned pairs from the
// page's own tokens.
// ---------------------------------------------------------------------------
constexpr int kVisSlices = 64;        // cache slices counted per window row

// block (window row p, slice): tokens of the slice visible to row p
__global__ __launch_bounds__(256) void recorded_count_kernel(AttnGeom a, int* nvis_part, int n_slices) {
  __shared__ int red[4];
  const int p = blockIdx.x / n_slices, slice = blockIdx.x % n_slices;
  const int per = (a.S + n_slices - 1) / n_slices;
  const int t0 = slice * per, t1 = min(a.S, t0 + per);
  const int qp = a.qpos[p];
  int c = 0;
  for (int t = t0 + (int)threadIdx.x; t < t1; t += 256) c += a.pos[t] <= qp ? 1 : 0;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) nvis_part[p * n_slices + slice] = red[0] + red[1] + red[2] + red[3];
}

// one wave per window row: lse2 = lse log2(e), ||o_p||, n_vis; also zeroes
// the outputs later kernels reduce into (as the combine kernel does)
template <int D>
__global__ __launch_bounds__(256) void recorded_rows_kernel(AttnGeom a, const float* o, const float* lse,
                                                            RowStats rs, const int* nvis_part, int n_slices,
                                                            ZeroList zl) {
  const int lane = threadIdx.x & 63;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t gsz = (size_t)gridDim.x * blockDim.x;
  for (size_t i = gid; i < zl.n0; i += gsz) zl.p0[i] = 0.f;
  for (size_t i = gid; i < zl.n1; i += gsz) zl.p1[i] = 0.f;
  for (size_t i = gid; i < zl.n2; i += gsz) zl.p2[i] = 0.f;
  if (zl.i0 && gid == 0) *zl.i0 = 0;
  for (size_t i = gid; i < zl.n1i; i += gsz) zl.i1[i] = 0;
  const int rg = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (rg >= a.Hq * a.W) return;
  const int p = rg % a.W;
  float n2 = 0.f;
#pragma unroll
  for (int j = 0; j < D / 64; ++j) {
    const float ov = o[(size_t)rg * D + lane + 64 * j];
    n2 += ov * ov;
  }
  int nv = lane < n_slices ? nvis_part[p * n_slices + lane] : 0;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    n2 += __shfl_xor(n2, off, 64);
    nv += __shfl_xor(nv, off, 64);
  }
  if (lane == 0) {
    const float l = lse[rg];
    rs.lse2[rg] = l == -INFINITY ? -INFINITY : l * kLog2e;
    rs.onorm[rg] = sqrtf(n2);
    rs.nvis[rg] = nv;
    // recorded o or lse NaN or infinite (lse -inf only for a row that sees nothing)
    if (!(n2 <= 3.4e38f) || !(l < INFINITY) || (nv > 0 && !(l > -INFINITY))) latch_nonfinite(zl.nonfinite);
  }
}

// One wave per listed pair (page E, window row): with weights relative to
// the recorded log-sum-exp, A = sum_{i in E} w_i and u = sum_{i in E} w_i v_i
// in float32 from the page's tokens, and Eq. (6):
// ratio = ||u - A o|| / ((1 - A) ||o||); +inf when E holds every visible token.
// 1 - A is then known to a few ulp of the log-sum-exp only, so a pair with
// A > a_hi is appended to list2 instead (while it has room): the
// complement pass computes its output without the page from every other
// token of the row.
// Scores: four lanes per token (a quarter of the width each), 16 tokens per
// pass; every key, position and query load of the pair is issued before the
// first product, and the values of a pass's 16 tokens are loaded together.
template <int D, bool PG>
__global__ __launch_bounds__(256) void page_fixup_recorded(AttnGeom a, RowStats rs, PageWork pw, int4* list2,
                                                           int* count2, int cap2, float a_hi) {
  constexpr int J = D / 64;            // widths lane + 64 j of u
  constexpr int QC = D / 32;           // 16-byte chunks of a lane's quarter row
  constexpr int NP = kMaxPage / 16;    // passes of 16 tokens
  const int lane = threadIdx.x & 63, sub = lane & 3, tk = lane >> 2;
  const int n = min(*pw.fix_count, pw.fix_cap);
  for (int e = blockIdx.x * 4 + (threadIdx.x >> 6); e < n; e += gridDim.x * 4) {
    const int4 ent = reinterpret_cast<const int4*>(pw.fix_list)[e];
    const int page = ent.x, rg = ent.y, st = ent.z, ln = ent.w & 0xFF;
    const int h = rg / a.W, p = rg % a.W, g = h / a.group;
    const int qp = a.qpos[p];
    const float ref = rs.lse2[rg];
    const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
    const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;
    const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride;
    u32x4 qc[QC], kc[NP][QC];
    int pv[NP];
#pragma unroll
    for (int c = 0; c < QC; ++c) qc[c] = ldg_u4(qrow + 8 * (sub * QC + c));
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
      const int i = ps * 16 + tk;
      const int t = st + min(i, ln - 1);           // in-range address for every lane
      const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[t], a.pool_last) : t;
#pragma unroll
      for (int c = 0; c < QC; ++c) kc[ps][c] = ldg_u4(kh + row * a.kv_tok_stride + 8 * (sub * QC + c));
      pv[ps] = i < ln ? ldg_i32(a.pos + t) : INT_MAX;
    }
    float ov[J];
#pragma unroll
    for (int j = 0; j < J; ++j) ov[j] = rs.o[(size_t)CKV_IDX(rg, a.Hq * a.W, a.dbg, 4) * D + lane + 64 * j];
    // weights of the pass's tokens (0 for tokens the row does not see)
    float w[NP];
    float Al = 0.f;
    int cl = 0;
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
      float x = 0.f;
#pragma unroll
      for (int c = 0; c < QC; ++c)
#pragma unroll
        for (int m = 0; m < 8; ++m)
          x = __builtin_fmaf(bf16_bits_to_float(chunk_elem(qc[c], m)), bf16_bits_to_float(chunk_elem(kc[ps][c], m)), x);
      x += __shfl_xor(x, 1, 64);
      x += __shfl_xor(x, 2, 64);
      const bool vis = pv[ps] <= qp;
      w[ps] = vis ? __builtin_amdgcn_exp2f(__builtin_fmaf(x, a.sl2, -ref)) : 0.f;
      if (sub == 0) {
        Al += w[ps];
        cl += vis ? 1 : 0;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      Al += __shfl_xor(Al, off, 64);
      cl += __shfl_xor(cl, off, 64);
    }
    const float A = Al;
    const int cnt = cl;
    float u[J];
#pragma unroll
    for (int j = 0; j < J; ++j) u[j] = 0.f;
#pragma unroll
    for (int ps = 0; ps < NP; ++ps) {
      if (ps * 16 >= ln) break;
      float vv[16][J];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = st + min(ps * 16 + i, ln - 1);
        const int64_t row = PG ? (int64_t)min((uint32_t)a.slot[t], a.pool_last) : t;
#pragma unroll
        for (int j = 0; j < J; ++j) vv[i][j] = bf16_bits_to_float(vh[row * a.kv_tok_stride + lane + 64 * j]);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float wt = __shfl(w[ps], 4 * i, 64);   // zero past the page's end
#pragma unroll
        for (int j = 0; j < J; ++j) u[j] = __builtin_fmaf(wt, vv[i][j], u[j]);
      }
    }
    float rr = 0.f, oo = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const float r = __builtin_fmaf(-A, ov[j], u[j]);
      rr += r * r;
      oo += ov[j] * ov[j];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      rr += __shfl_xor(rr, off, 64);
      oo += __shfl_xor(oo, off, 64);
    }
    if (cnt > 0 && cnt < rs.nvis[rg] && A > a_hi) {
      int slot = 0;
      if (lane == 0) slot = atomicAdd(count2, 1);
      slot = __shfl(slot, 0, 64);
      if (slot < cap2) {
        if (lane == 0) list2[slot] = ent;
        continue;
      }
    }
    if (lane == 0 && cnt > 0) {
      const float den = 1.f - A;
      float ratio;
      if (cnt >= rs.nvis[rg] || !(den > 0.f)) ratio = INFINITY;
      else if (oo > 0.f) ratio = sqrtf(rr) / (den * sqrtf(oo));
      else ratio = rr > 0.f ? INFINITY : 0.f;
      if (pw.R_head)
        atomic_max_nonneg(&pw.R_head[CKV_IDX((size_t)page * pw.Hq + h, (int64_t)pw.n_pages * pw.Hq, a.dbg, 5)], ratio);
      atomic_max_nonneg(&pw.R[CKV_IDX(page, pw.n_pages, a.dbg, 5)], ratio);
    }
  }
}

int recorded_slices(int S) { return std::max(1, std::min(kVisSlices, (S + 1023) / 1024)); }

hipError_t launch_recorded_rows(const AttnGeom& a, const float* o, const float* lse, const RowStats& rs,
                                int* nvis_part, const ZeroList& zl, hipStream_t s) {
  const int ns = nvis_part ? recorded_slices(a.S) : 0;   // no counts: every row's count reads 0
  if (ns > 0) {
    hipLaunchKernelGGL(recorded_count_kernel, dim3(a.W * ns), dim3(256), 0, s, a, nvis_part, ns);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  dim3 grid((a.Hq * a.W + 3) / 4), block(256);
  if (a.D == 128)
    hipLaunchKernelGGL((recorded_rows_kernel<128>), grid, block, 0, s, a, o, lse, rs, nvis_part, ns, zl);
  else
    hipLaunchKernelGGL((recorded_rows_kernel<64>), grid, block, 0, s, a, o, lse, rs, nvis_part, ns, zl);
  return hipGetLastError();
}

hipError_t launch_page_fixup_recorded(const AttnGeom& a, const RowStats& rs, const PageWork& pw, int* list2,
                                      int* count2, int cap2, float a_hi, hipStream_t s) {
  dim3 grid(std::max(1, std::min((pw.fix_cap + 3) / 4, 256))), block(256);
  int4* l2 = reinterpret_cast<int4*>(list2);
  const bool pg = a.slot != nullptr;
  if (a.D == 128) {
    if (pg) hipLaunchKernelGGL((page_fixup_recorded<128, true>), grid, block, 0, s, a, rs, pw, l2, count2, cap2, a_hi);
    else hipLaunchKernelGGL((page_fixup_recorded<128, false>), grid, block, 0, s, a, rs, pw, l2, count2, cap2, a_hi);
  } else {
    if (pg) hipLaunchKernelGGL((page_fixup_recorded<64, true>), grid, block, 0, s, a, rs, pw, l2, count2, cap2, a_hi);
    else hipLaunchKernelGGL((page_fixup_recorded<64, false>), grid, block, 0, s, a, rs, pw, l2, count2, cap2, a_hi);
  }
  return hipGetLastError();
}

}  // namespace ckv
