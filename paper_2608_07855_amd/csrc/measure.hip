// Window attention and per-page deletion effects (CommitKV, Sec. 3.2,
// Eq. (6)-(7)) on MFMA for gfx950.
//
// Two passes over the resident cache of one layer:
//   A. window_attention_kernel + combine_kernel: for every window row
//      (query head h, row p) the full attention output o_p, its log-sum-exp
//      and the number of visible tokens.  Split over the token axis, partial
//      (max, sum, unnormalised output) merged by the combine kernel.
//   B. page_kernel: for every page E and row p, with a page-local max m_E:
//        l^ = sum_{i in E} 2^(x_i - m_E),  U^ = sum_{i in E} 2^(x_i - m_E) v_i,
//        f  = 2^(m_E - lse_p),  A = f l^,
//        ||o_p - o_p^{\E}|| / ||o_p|| = f ||U^ - l^ o_p|| / ((1 - A) ||o_p||)
//      (Eq. (6) rescaled by the page maximum, so the float16 weights of the
//      page stay in (0, 1]).  MODE 0 reduces the ratio to max over rows and
//      heads (Eq. (7)); MODE 1 stores the residual f (U^ - l^ o_p), the mass
//      A and the visible count for the joint test.
//   C. token_mass_kernel: max_h sum_p a_hpi for every token.
// Logits are carried in log2 units: x = scale * log2(e) * q.k.
#include "ckv_device.h"
#include "ckv_kernels.h"

#include <climits>

namespace ckv {

// ---------------------------------------------------------------------------
// staging of a 64-token tile: K as [token][width] bf16, V^T as
// [width][slot] fp16 (slot = vt_slot(token)), positions as int32.
// ---------------------------------------------------------------------------
template <int D, int NT>
struct Stager {
  static constexpr int KP = D + 8;          // K tile row stride (elements)
  static constexpr int VP = kTile + 8;      // V^T tile row stride (halves)
  static constexpr int CPR = D / 8;         // 16-byte chunks per row
  static constexpr int KCH = kTile * CPR;   // chunks per K tile
  static constexpr int KPT = (KCH + NT - 1) / NT;
  static constexpr int VQ = (kTile / 4) * CPR;   // (4 tokens x 8 widths) quads
  static constexpr int VPT = (VQ + NT - 1) / NT;

  uint4 kr[KPT];
  uint4 vr[VPT][4];
  int pr;

  // load tokens t0 .. t0+63 of one head; tokens at offset >= n_valid are zero
  __device__ __forceinline__ void issue(const uint16_t* kh, const uint16_t* vh,
                                        int64_t ts, const int32_t* pos, int t0,
                                        int n_valid, int tid) {
    const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      const int tr = c / CPR, cc = c % CPR;
      kr[i] = (c < KCH && tr < n_valid)
                  ? *reinterpret_cast<const uint4*>(kh + (int64_t)(t0 + tr) * ts + cc * 8)
                  : z;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int qd = tid + i * NT;
      const int tq = qd / CPR, cg = qd % CPR;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int tr = 4 * tq + j;
        vr[i][j] = (qd < VQ && tr < n_valid)
                       ? *reinterpret_cast<const uint4*>(vh + (int64_t)(t0 + tr) * ts + cg * 8)
                       : z;
      }
    }
    pr = (tid < kTile && tid < n_valid) ? pos[t0 + tid] : INT_MAX;
  }

  __device__ __forceinline__ void commit(uint16_t* sK, _Float16* sV, int* sP, int tid) const {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      if (c < KCH) {
        const int tr = c / CPR, cc = c % CPR;
        *reinterpret_cast<uint4*>(sK + tr * KP + cc * 8) = kr[i];
      }
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int qd = tid + i * NT;
      if (qd < VQ) {
        const int tq = qd / CPR, cg = qd % CPR;
        const int slot = vt_slot(4 * tq);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          f16x4 w;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            w[j] = (_Float16)bf16_bits_to_float(chunk_elem(vr[i][j], e));
          *reinterpret_cast<f16x4*>(sV + (cg * 8 + e) * VP + slot) = w;
        }
      }
    }
    if (tid < kTile) sP[tid] = pr;
  }
};

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ bf16x8 zero_bf16x8() {
  return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
}

// rows of KV head g handled by lane: row = base + rb*32 + col
struct RowInfo {
  int row;     // row inside the KV head (0 .. rows-1), or >= rows if padding
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

template <int D, int RB>
__device__ __forceinline__ void load_q(const AttnGeom& a, int g, const RowInfo (&ri)[RB],
                                       int half, bf16x8 (&qf)[RB][D / 16]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int h = g * a.group + (ri[rb].ok ? ri[rb].row / a.W : 0);
    const int p = ri[rb].ok ? ri[rb].row % a.W : 0;
    const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)p * a.q_row_stride;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
      qf[rb][ks] = ri[rb].ok ? load_bf16x8(qrow + 16 * ks + 8 * half) : zero_bf16x8();
  }
}

// ---------------------------------------------------------------------------
// A. split window attention
// ---------------------------------------------------------------------------
template <int D, int RB, int NW>
__global__ __launch_bounds__(NW * 64, 1) void window_attention_kernel(AttnGeom a, AttnSplit sp) {
  constexpr int NT = NW * 64, KS = D / 16, DB = D / 32;
  using St = Stager<D, NT>;
  __shared__ __align__(16) uint16_t sK[2][kTile * St::KP];
  __shared__ __align__(16) _Float16 sV[2][D * St::VP];
  __shared__ __align__(16) int sP[2][kTile];

  const int g = blockIdx.z, split = blockIdx.x, rblk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int t_begin = split * sp.chunk;
  const int t_end = min(a.S, t_begin + sp.chunk);
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;

  RowInfo ri[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
    ri[rb] = row_info(a, g, (rblk * NW + wave) * (32 * RB) + rb * 32 + col);
  bf16x8 qf[RB][KS];
  load_q<D, RB>(a, g, ri, half, qf);

  f32x16 oacc[RB][DB];
  float m[RB], l[RB];
  int cnt[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
    cnt[rb] = 0;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[rb][db] = zero16();
  }

  const int n_tiles = t_end > t_begin ? (t_end - t_begin + kTile - 1) / kTile : 0;
  St st;
  if (n_tiles > 0) {
    st.issue(kh, vh, a.kv_tok_stride, a.pos, t_begin, min(kTile, t_end - t_begin), tid);
    st.commit(sK[0], sV[0], sP[0], tid);
  }
  __syncthreads();

  for (int it = 0; it < n_tiles; ++it) {
    const int b = it & 1;
    const int tn = t_begin + (it + 1) * kTile;
    if (it + 1 < n_tiles) st.issue(kh, vh, a.kv_tok_stride, a.pos, tn, min(kTile, t_end - tn), tid);

    // S^T = K Q^T for 64 tokens (two 32-token blocks)
    f32x16 sacc[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sacc[rb][0] = sacc[rb][1] = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const bf16x8 af = load_bf16x8(&sK[b][(32 * tb + col) * St::KP + 16 * ks + 8 * half]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) sacc[rb][tb] = mfma_bf16(af, qf[rb][ks], sacc[rb][tb]);
      }
    }
    // causal mask by absolute position, online softmax (log2 units)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float mx = -INFINITY;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int4 pq = *reinterpret_cast<const int4*>(&sP[b][32 * tb + 8 * i + 4 * half]);
          const int pv[4] = {pq.x, pq.y, pq.z, pq.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool vis = ri[rb].ok && pv[j] <= ri[rb].qp;
            const float x = vis ? sacc[rb][tb][4 * i + j] * a.sl2 : -INFINITY;
            cnt[rb] += vis ? 1 : 0;
            sacc[rb][tb][4 * i + j] = x;
            mx = fmaxf(mx, x);
          }
        }
      }
      mx = fmaxf(mx, xor32(mx));
      const float mn = fmaxf(m[rb], mx);
      const float base = (mn == -INFINITY) ? 0.f : mn;
      const float alpha = __builtin_amdgcn_exp2f(m[rb] - base);
      float ls = 0.f;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(sacc[rb][tb][r] - base);
          sacc[rb][tb][r] = p;
          ls += p;
        }
      }
      l[rb] = l[rb] * alpha + ls;
      m[rb] = mn;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[rb][db] *= alpha;
    }
    // O^T += V^T P^T (fp16 weights and values, fp32 accumulation)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f16x8 bfr[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int e = 0; e < 8; ++e) bfr[rb][e] = (_Float16)sacc[rb][tb][8 * u + e];
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const f16x8 af = *reinterpret_cast<const f16x8*>(
              &sV[b][(32 * db + col) * St::VP + 32 * tb + 16 * u + 8 * half]);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) oacc[rb][db] = mfma_f16(af, bfr[rb], oacc[rb][db]);
        }
      }
    }
    if (it + 1 < n_tiles) st.commit(sK[b ^ 1], sV[b ^ 1], sP[b ^ 1], tid);
    __syncthreads();
  }

  // partial results of this split
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float lt = l[rb] + xor32(l[rb]);
    const int ct = cnt[rb] + xor32i(cnt[rb]);
    if (!ri[rb].ok) continue;
    const size_t idx = ((size_t)(g * sp.n_splits + split) * sp.rows_pad + ri[rb].row);
    if (half == 0) {
      sp.part_m[idx] = m[rb];
      sp.part_l[idx] = lt;
      sp.part_c[idx] = ct;
    }
    float* po = sp.part_o + idx * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v4;
#pragma unroll
        for (int j = 0; j < 4; ++j) v4[j] = oacc[rb][db][4 * i + j];
        *reinterpret_cast<f32x4*>(po + 32 * db + 8 * i + 4 * half) = v4;
      }
  }
}

// one wave per window row: merge the splits, write o, lse, ||o||, n_vis
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(AttnGeom a, AttnSplit sp, RowStats rs,
                                                      float* lse_out, ZeroList zl) {
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  // zero the outputs that later kernels reduce into with atomic max
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < zl.n0; i += (size_t)gridDim.x * blockDim.x)
    zl.p0[i] = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < zl.n1; i += (size_t)gridDim.x * blockDim.x)
    zl.p1[i] = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < zl.n2; i += (size_t)gridDim.x * blockDim.x)
    zl.p2[i] = 0.f;
  if (wid >= a.Hkv * a.rows) return;
  const int g = wid / a.rows, row = wid % a.rows;
  const int rg = g * a.rows + row;
  float M = -INFINITY;
  int nv = 0;
  for (int s = 0; s < sp.n_splits; ++s) {
    const size_t idx = (size_t)(g * sp.n_splits + s) * sp.rows_pad + row;
    M = fmaxf(M, sp.part_m[idx]);
    nv += sp.part_c[idx];
  }
  float wsum = 0.f;
  float acc[D / 64];
#pragma unroll
  for (int j = 0; j < D / 64; ++j) acc[j] = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < sp.n_splits; ++s) {
      const size_t idx = (size_t)(g * sp.n_splits + s) * sp.rows_pad + row;
      const float ms = sp.part_m[idx];
      if (ms == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(ms - M);
      wsum += sp.part_l[idx] * w;
#pragma unroll
      for (int j = 0; j < D / 64; ++j) acc[j] += sp.part_o[idx * D + lane + 64 * j] * w;
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  float n2 = 0.f;
#pragma unroll
  for (int j = 0; j < D / 64; ++j) {
    const float ov = acc[j] * inv;
    rs.o[(size_t)rg * D + lane + 64 * j] = ov;
    n2 += ov * ov;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) n2 += __shfl_xor(n2, off, 64);
  if (lane == 0) {
    const float l2 = wsum > 0.f ? M + __log2f(wsum) : -INFINITY;
    rs.lse2[rg] = l2;
    rs.onorm[rg] = sqrtf(n2);
    rs.nvis[rg] = nv;
    if (lse_out) lse_out[rg] = l2 * kLn2;
  }
}

// ---------------------------------------------------------------------------
// B. per-page deletion effect (MODE 0) or per-candidate residual (MODE 1)
// ---------------------------------------------------------------------------
template <int D, int RB, int NW, int MODE>
__global__ __launch_bounds__(NW * 64, 1) void page_kernel(AttnGeom a, PageWork pw, RowStats rs) {
  constexpr int NT = NW * 64, KS = D / 16, DB = D / 32, RWG = 32 * RB * NW;
  using St = Stager<D, NT>;
  __shared__ __align__(16) uint16_t sK[2][kTile * St::KP];
  __shared__ __align__(16) _Float16 sV[2][D * St::VP];
  __shared__ __align__(16) int sP[2][kTile];
  __shared__ unsigned int sMax[2][RWG + 2];

  const int g = blockIdx.z, rblk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  int n_items = pw.n_items;
  if (MODE == 1) n_items = min(*pw.n_cand, pw.n_items);
  const int i_begin = blockIdx.x * pw.items_per_block;
  const int i_end = min(n_items, i_begin + pw.items_per_block);
  if (i_begin >= i_end) return;
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const uint16_t* vh = a.v + (int64_t)g * a.kv_head_stride;

  RowInfo ri[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
    ri[rb] = row_info(a, g, (rblk * NW + wave) * (32 * RB) + rb * 32 + col);
  bf16x8 qf[RB][KS];
  load_q<D, RB>(a, g, ri, half, qf);
  // o_p in accumulator layout: register r of block db holds width 32db + 8(r/4) + 4h + r%4
  f32x16 of[RB][DB];
  float lse2[RB], onorm[RB];
  int nvis[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float* orow = rs.o + (size_t)ri[rb].rg * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 v4 = ri[rb].ok ? *reinterpret_cast<const f32x4*>(orow + 32 * db + 8 * i + 4 * half)
                                   : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) of[rb][db][4 * i + j] = v4[j];
      }
    lse2[rb] = ri[rb].ok ? rs.lse2[ri[rb].rg] : -INFINITY;
    onorm[rb] = ri[rb].ok ? rs.onorm[ri[rb].rg] : 0.f;
    nvis[rb] = ri[rb].ok ? rs.nvis[ri[rb].rg] : 0;
  }
  const int row0 = rblk * RWG;                 // first row of this block
  const int head0 = row0 / a.W;                // first local head touched
  const int n_heads_blk = min(a.group, (min(a.rows, row0 + RWG) - 1) / a.W + 1) - head0;
  if (MODE == 0) {
    for (int i = tid; i < 2 * (RWG + 2); i += NT) (&sMax[0][0])[i] = 0u;
  }

  // page of an item; a candidate index outside the page list is an empty page
  auto page_of = [&](int item) { return MODE == 0 ? item : pw.cand[item]; };
  auto page_ok = [&](int pg) { return pg >= 0 && pg < pw.n_pages; };
  auto pstart = [&](int item) { const int pg = page_of(item); return page_ok(pg) ? pw.start[pg] : 0; };
  auto plen = [&](int item) { const int pg = page_of(item); return page_ok(pg) ? pw.len[pg] : 0; };
  St st;
  st.issue(kh, vh, a.kv_tok_stride, a.pos, pstart(i_begin), plen(i_begin), tid);
  st.commit(sK[0], sV[0], sP[0], tid);
  __syncthreads();

  for (int it = i_begin; it < i_end; ++it) {
    const int b = (it - i_begin) & 1;
    if (it + 1 < i_end) st.issue(kh, vh, a.kv_tok_stride, a.pos, pstart(it + 1), plen(it + 1), tid);
    // flush the previous item's per-head maxima (its LDS slots are final)
    if (MODE == 0 && it > i_begin && tid < n_heads_blk) {
      const int pb = b ^ 1;
      const float v = __uint_as_float(sMax[pb][tid]);
      const int page = it - 1;
      const int h = g * a.group + head0 + tid;
      if (pw.R_head) atomic_max_nonneg(&pw.R_head[(size_t)page * pw.Hq + h], v);
      atomic_max_nonneg(&pw.R[page], v);
      sMax[pb][tid] = 0u;
    }

    const int len = plen(it);
    const int nblk = len > 32 ? 2 : 1;
    f32x16 sacc[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sacc[rb][0] = sacc[rb][1] = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        if (tb < nblk) {
          const bf16x8 af = load_bf16x8(&sK[b][(32 * tb + col) * St::KP + 16 * ks + 8 * half]);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) sacc[rb][tb] = mfma_bf16(af, qf[rb][ks], sacc[rb][tb]);
        }
      }
    }
    float lhat[RB], mE[RB];
    int cE[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float mx = -INFINITY;
      int c = 0;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t0 = 32 * tb + 8 * i + 4 * half;
          const int4 pq = *reinterpret_cast<const int4*>(&sP[b][t0]);
          const int pv[4] = {pq.x, pq.y, pq.z, pq.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool vis = ri[rb].ok && (t0 + j) < len && pv[j] <= ri[rb].qp;
            const float x = vis ? sacc[rb][tb][4 * i + j] * a.sl2 : -INFINITY;
            c += vis ? 1 : 0;
            sacc[rb][tb][4 * i + j] = x;
            mx = fmaxf(mx, x);
          }
        }
      }
      mx = fmaxf(mx, xor32(mx));
      c += xor32i(c);
      const float base = (mx == -INFINITY) ? 0.f : mx;
      float ls = 0.f;
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(sacc[rb][tb][r] - base);
          sacc[rb][tb][r] = p;
          ls += p;
        }
      lhat[rb] = ls + xor32(ls);
      mE[rb] = mx;
      cE[rb] = c;
    }
    // U^T = V_E^T P^T
    f32x16 uacc[RB][DB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int db = 0; db < DB; ++db) uacc[rb][db] = zero16();
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      if (tb < nblk) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          f16x8 bfr[RB];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int e = 0; e < 8; ++e) bfr[rb][e] = (_Float16)sacc[rb][tb][8 * u + e];
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const f16x8 af = *reinterpret_cast<const f16x8*>(
                &sV[b][(32 * db + col) * St::VP + 32 * tb + 16 * u + 8 * half]);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) uacc[rb][db] = mfma_f16(af, bfr[rb], uacc[rb][db]);
          }
        }
      }
    }
    // residual r^ = U^ - l^ o, its norm, and the ratio of Eq. (6)-(7)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float n2 = 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float rv = uacc[rb][db][r] - lhat[rb] * of[rb][db][r];
          uacc[rb][db][r] = rv;
          n2 += rv * rv;
        }
      n2 += xor32(n2);
      const bool touched = cE[rb] > 0;
      const float f = touched ? __builtin_amdgcn_exp2f(mE[rb] - lse2[rb]) : 0.f;
      const float A = f * lhat[rb];
      if (MODE == 0) {
        float ratio = 0.f;
        if (touched) {
          const float keep = 1.f - A;
          if (cE[rb] >= nvis[rb] || !(keep > 0.f)) ratio = INFINITY;
          else if (onorm[rb] > 0.f) ratio = f * sqrtf(n2) / (keep * onorm[rb]);
          else ratio = n2 > 0.f ? INFINITY : 0.f;
        }
        if (ri[rb].ok && half == 0)
          atomicMax(&sMax[b][ri[rb].row / a.W - head0], __float_as_uint(ratio));
      } else {
        if (ri[rb].ok) {
          const size_t base = (size_t)it * pw.total_rows + ri[rb].rg;
          float* rrow = pw.resid + base * D;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              f32x4 v4;
#pragma unroll
              for (int j = 0; j < 4; ++j) v4[j] = f * uacc[rb][db][4 * i + j];
              *reinterpret_cast<f32x4*>(rrow + 32 * db + 8 * i + 4 * half) = v4;
            }
          if (half == 0) {
            pw.resA[base] = A;
            pw.resC[base] = cE[rb];
          }
        }
      }
    }
    if (it + 1 < i_end) st.commit(sK[b ^ 1], sV[b ^ 1], sP[b ^ 1], tid);
    __syncthreads();
  }
  if (MODE == 0 && tid < n_heads_blk) {
    const int pb = (i_end - 1 - i_begin) & 1;
    const float v = __uint_as_float(sMax[pb][tid]);
    const int page = i_end - 1;
    const int h = g * a.group + head0 + tid;
    if (pw.R_head) atomic_max_nonneg(&pw.R_head[(size_t)page * pw.Hq + h], v);
    atomic_max_nonneg(&pw.R[page], v);
  }
}

// ---------------------------------------------------------------------------
// C. window-attention mass of every token: max_h sum_p a_hpi
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void token_mass_kernel(AttnGeom a, RowStats rs, float* mass,
                                                             int chunk) {
  constexpr int NT = NW * 64, KS = D / 16;
  constexpr int KP = D + 8, CPR = D / 8, KCH = kTile * CPR;
  __shared__ __align__(16) uint16_t sK[kTile * KP];
  __shared__ int sP[kTile];
  __shared__ unsigned int sM[kTile];
  const int g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int t_begin = blockIdx.x * chunk;
  const int t_end = min(a.S, t_begin + chunk);
  const uint16_t* kh = a.k + (int64_t)g * a.kv_head_stride;
  const int nrb = (a.W + 31) / 32;
  for (int t0 = t_begin; t0 < t_end; t0 += kTile) {
    const int nv = min(kTile, t_end - t0);
    for (int c = tid; c < KCH; c += NT) {
      const int tr = c / CPR, cc = c % CPR;
      *reinterpret_cast<uint4*>(&sK[tr * KP + cc * 8]) =
          tr < nv ? *reinterpret_cast<const uint4*>(kh + (int64_t)(t0 + tr) * a.kv_tok_stride + cc * 8)
                  : make_uint4(0, 0, 0, 0);
    }
    if (tid < kTile) {
      sP[tid] = tid < nv ? a.pos[t0 + tid] : INT_MAX;
      sM[tid] = 0u;
    }
    __syncthreads();
    for (int hl = wave; hl < a.group; hl += NW) {
      const int h = g * a.group + hl;
      float msum[2] = {0.f, 0.f};
      for (int rb = 0; rb < nrb; ++rb) {
        const int prow = 32 * rb + col;          // A operand row of this lane
        const bool aok = prow < a.W;
        const uint16_t* qrow = a.q + (int64_t)h * a.q_head_stride + (int64_t)(aok ? prow : 0) * a.q_row_stride;
        bf16x8 qa[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qa[ks] = aok ? load_bf16x8(qrow + 16 * ks + 8 * half) : zero_bf16x8();
        // rows of the C layout held by this lane
        int qpr[16];
        float l2r[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int p = 32 * rb + 8 * (r >> 2) + 4 * half + (r & 3);
          qpr[r] = p < a.W ? a.qpos[p] : INT_MIN;
          l2r[r] = p < a.W ? rs.lse2[h * a.W + p] : 0.f;
        }
#pragma unroll
        for (int tb = 0; tb < 2; ++tb) {
          f32x16 acc = zero16();
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 kb = load_bf16x8(&sK[(32 * tb + col) * KP + 16 * ks + 8 * half]);
            acc = mfma_bf16(qa[ks], kb, acc);
          }
          const int pt = sP[32 * tb + col];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool vis = qpr[r] != INT_MIN && pt <= qpr[r];
            msum[tb] += vis ? __builtin_amdgcn_exp2f(acc[r] * a.sl2 - l2r[r]) : 0.f;
          }
        }
      }
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const float s = msum[tb] + xor32(msum[tb]);
        if (half == 0) atomicMax(&sM[32 * tb + col], __float_as_uint(s));
      }
    }
    __syncthreads();
    if (tid < nv) atomic_max_nonneg(&mass[t0 + tid], __uint_as_float(sM[tid]));
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
namespace {
constexpr int kNW = 4;
constexpr int kRBA = 2;     // row blocks per wave in pass A
constexpr int kRBB = 2;     // row blocks per wave in pass B
}  // namespace

int rows_per_block_attention() { return 32 * kRBA * kNW; }
int rows_per_block_page() { return 32 * kRBB * kNW; }

hipError_t launch_window_attention(const AttnGeom& a, const AttnSplit& sp, hipStream_t s) {
  const int nrb = (a.rows + rows_per_block_attention() - 1) / rows_per_block_attention();
  dim3 grid(sp.n_splits, nrb, a.Hkv), block(kNW * 64);
  if (a.D == 128)
    hipLaunchKernelGGL((window_attention_kernel<128, kRBA, kNW>), grid, block, 0, s, a, sp);
  else
    hipLaunchKernelGGL((window_attention_kernel<64, kRBA, kNW>), grid, block, 0, s, a, sp);
  return hipGetLastError();
}

hipError_t launch_combine(const AttnGeom& a, const AttnSplit& sp, const RowStats& rs, float* lse_out,
                          const ZeroList& zl, hipStream_t s) {
  const int waves = a.Hkv * a.rows;
  dim3 grid((waves + 3) / 4), block(256);
  if (a.D == 128)
    hipLaunchKernelGGL((combine_kernel<128>), grid, block, 0, s, a, sp, rs, lse_out, zl);
  else
    hipLaunchKernelGGL((combine_kernel<64>), grid, block, 0, s, a, sp, rs, lse_out, zl);
  return hipGetLastError();
}

hipError_t launch_page_kernel(const AttnGeom& a, const PageWork& pw, const RowStats& rs, int mode,
                              hipStream_t s) {
  const int nrb = (a.rows + rows_per_block_page() - 1) / rows_per_block_page();
  const int nblk = (pw.n_items + pw.items_per_block - 1) / pw.items_per_block;
  if (nblk == 0) return hipSuccess;
  dim3 grid(nblk, nrb, a.Hkv), block(kNW * 64);
  if (a.D == 128) {
    if (mode == 0) hipLaunchKernelGGL((page_kernel<128, kRBB, kNW, 0>), grid, block, 0, s, a, pw, rs);
    else hipLaunchKernelGGL((page_kernel<128, kRBB, kNW, 1>), grid, block, 0, s, a, pw, rs);
  } else {
    if (mode == 0) hipLaunchKernelGGL((page_kernel<64, kRBB, kNW, 0>), grid, block, 0, s, a, pw, rs);
    else hipLaunchKernelGGL((page_kernel<64, kRBB, kNW, 1>), grid, block, 0, s, a, pw, rs);
  }
  return hipGetLastError();
}

hipError_t launch_token_mass(const AttnGeom& a, const RowStats& rs, float* mass, int chunk,
                             hipStream_t s) {
  dim3 grid((a.S + chunk - 1) / chunk, a.Hkv), block(kNW * 64);
  if (a.D == 128)
    hipLaunchKernelGGL((token_mass_kernel<128, kNW>), grid, block, 0, s, a, rs, mass, chunk);
  else
    hipLaunchKernelGGL((token_mass_kernel<64, kNW>), grid, block, 0, s, a, rs, mass, chunk);
  return hipGetLastError();
}

}  // namespace ckv
