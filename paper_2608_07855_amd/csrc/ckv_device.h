// Device-side building blocks shared by the CommitKV kernels (gfx950 only).
//
// MFMA fragment layouts used throughout (v_mfma_f32_32x32x16_{bf16,f16},
// one wave of 64 lanes, lane l, half h = l / 32, column c = l % 32):
//   A operand (32 x 16): lane holds A[c][8h .. 8h+7]
//   B operand (16 x 32): lane holds B[8h .. 8h+7][c]
//   C/D (32 x 32), 16 floats: register r holds C[8(r/4) + 4h + r%4][c]
//
// The attention kernels compute the TRANSPOSED scores S^T = K Q^T so that a
// window row sits on a lane column: per-row max/sum/norm reductions are then
// lane-local plus one exchange with the partner lane (l ^ 32), and the
// per-row rescaling of the output accumulator is a per-lane scalar.  The
// value-weighted sum O^T = V^T P^T takes P^T straight from the score
// accumulator: registers 8u .. 8u+7 of a 32-token score block are the B
// operand of the u-th 16-token step, provided V^T is staged in LDS with the
// token order inside each 16-token group permuted by swapping bits 2 and 3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ckv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kTile = 64;            // tokens per staged tile / max page length
constexpr int kMaxPage = 64;

__device__ __forceinline__ f32x16 mfma_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma_f16(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) {
  return __uint_as_float(b << 16);
}

// 8 bf16 (one 16-byte chunk) -> 8 fp16, exact inside the fp16 normal range.
__device__ __forceinline__ f16x4 bf16x4_to_f16(uint32_t lo, uint32_t hi) {
  f16x4 r;
  r[0] = (_Float16)bf16_bits_to_float(lo & 0xFFFFu);
  r[1] = (_Float16)bf16_bits_to_float(lo >> 16);
  r[2] = (_Float16)bf16_bits_to_float(hi & 0xFFFFu);
  r[3] = (_Float16)bf16_bits_to_float(hi >> 16);
  return r;
}

// bf16 element j (0..7) of a 16-byte chunk
template <class V4>
__device__ __forceinline__ uint32_t chunk_elem(const V4& c, int j) {
  const uint32_t w = c[j >> 1];
  return (j & 1) ? (w >> 16) : (w & 0xFFFFu);
}

// slot of token t (0..63) in the V^T tile: swap bits 2 and 3
__device__ __forceinline__ int vt_slot(int t) {
  return (t & ~0xC) | ((t & 4) << 1) | ((t & 8) >> 1);
}

// Stored column of slot s in row r of the V^T tile: the 8-slot (16-byte)
// group index is XOR-ed with bits 4..6 of the row.  With the padded row
// stride (36 dwords) and gfx950's 64 LDS banks, a 16-byte read of sixteen
// consecutive rows at one group stays conflict-free, and the transposing
// 4-byte writes of sixteen rows 8 apart (one 16-byte chunk of V per lane)
// spread over distinct bank groups instead of a few.
__device__ __forceinline__ int vt_col(int r, int s) {
  return (((s >> 3) ^ (r >> 4)) & 7) << 3 | (s & 7);
}

// Element offset of the 16-byte V^T fragment that lane (col, half) reads as
// the A operand for width block db (< 4), 32-token slot tb and 16-token step
// u: row r = 32 db + col, slots 32 tb + 16 u + 8 half .. + 7, i.e.
// r * VP + vt_col(r, 32 tb + 16 u + 8 half).  The XOR of vt_col splits bit by
// bit into a per-lane part (bit 0: half ^ (col >> 4)) and a part fixed by
// (db, tb, u), so every fragment of a lane is one base register plus an
// immediate offset.
template <int VP>
__device__ __forceinline__ int vt_frag_lane(int col, int half) {
  return col * VP + 8 * (half ^ (col >> 4));
}
__device__ __forceinline__ constexpr int vt_frag_const(int VP, int db, int tb, int u) {
  return 32 * db * VP + 8 * (((tb ^ (db >> 1)) << 2) | ((u ^ (db & 1)) << 1));
}

// Device bounds checks (builds with -DCKV_DEBUG): an index outside [0, n)
// stores the check's site number in the context's debug word (pinned host
// memory, reported by the next call or ckv_sync as CKV_ERR_DEVICE_CHECK) and
// is clamped into the range, so the access itself stays inside the buffer.
// Other builds use the index as it is.
#ifdef CKV_DEBUG
__device__ __forceinline__ int64_t checked_index(int64_t i, int64_t n, uint32_t* word, uint32_t site) {
  if (i >= 0 && i < n) return i;
  if (word) __hip_atomic_store(word, site, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  return (i < 0 || n <= 0) ? 0 : n - 1;
}
#define CKV_IDX(i, n, word, site) ::ckv::checked_index((int64_t)(i), (int64_t)(n), (word), (site))
#else
#define CKV_IDX(i, n, word, site) (i)
#endif

// loads through the global address space (pointers inside by-value argument
// structs otherwise compile to flat accesses)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 ldg_u4(const void* p) {
  typedef const __attribute__((address_space(1))) u32x4* gptr;
  return *(gptr)(p);
}
__device__ __forceinline__ int ldg_i32(const void* p) {
  typedef const __attribute__((address_space(1))) int* gptr;
  return *(gptr)(p);
}

__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, 64); }
__device__ __forceinline__ int xor32i(int v) { return __shfl_xor(v, 32, 64); }

// Both halves of a wave combined lane by lane (lane l with lane l ^ 32) in
// one VALU op: v_permlane32_swap hands lanes 0-31 the upper half and lanes
// 32-63 the lower half, so {lo, hi} below is {v[l % 32], v[l % 32 + 32]} in
// every lane and the result is bit-identical in both halves.
__device__ __forceinline__ void halves(float v, float& lo, float& hi) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum32(float v) {
  float lo, hi;
  halves(v, lo, hi);
  return lo + hi;
}
__device__ __forceinline__ float max32(float v) {
  float lo, hi;
  halves(v, lo, hi);
  return fmaxf(lo, hi);
}
__device__ __forceinline__ int sum32i(int v) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)(r[0] + r[1]);
}

// bit pattern of a non-negative float (including +inf) keeps its order as uint
__device__ __forceinline__ void atomic_max_nonneg(float* addr, float v) {
  atomicMax(reinterpret_cast<unsigned int*>(addr), __float_as_uint(v));
}

}  // namespace ckv
