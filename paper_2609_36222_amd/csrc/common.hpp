// Device-side building blocks shared by the BASE kernels (gfx950, wave64).
//
// Every translation unit is compiled with -ffp-contract=off: a multiply and
// an add are fused only where the code says fmaf().  The scoring path relies
// on that to follow one fixed fp32 operation order (see dot partials and
// base_exp below).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace basek {

constexpr int WAVE = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }
// the same, known to the compiler to be uniform over the wavefront (values
// derived from it stay in scalar registers)
__device__ __forceinline__ int wave_id_u() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
}

// LDS writes of this wavefront complete, then the workgroup meets.  Unlike
// __syncthreads() this does not wait for the wavefront's global loads, so
// loads requested ahead stay in flight across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt, expcnt: no wait
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// ---------------------------------------------------------------- bf16 ---
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}
// round to nearest, ties to even (finite inputs)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Four consecutive activations as fp32 (exact widening for bf16).
__device__ __forceinline__ void load4(const float *p, float v[4]) {
  float4 q = *reinterpret_cast<const float4 *>(p);
  v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
}
__device__ __forceinline__ void load4(const uint16_t *p, float v[4]) {
  u32x2 q = *reinterpret_cast<const u32x2 *>(p);
  v[0] = __uint_as_float(q.x << 16);
  v[1] = __uint_as_float(q.x & 0xFFFF0000u);
  v[2] = __uint_as_float(q.y << 16);
  v[3] = __uint_as_float(q.y & 0xFFFF0000u);
}

// ---------------------------------------------------------- wave sums ---
// The value of lane j ^ H in lane j: quad permutations (DPP) for H = 1, 2,
// an LDS-free swizzle inside 32-lane halves for H = 4, 8, 16, a permute
// across the halves for H = 32.
template <int H>
__device__ __forceinline__ float xor_lane(float v) {
  static_assert(H == 1 || H == 2 || H == 4 || H == 8 || H == 16 || H == 32, "lane distance");
  const int i = __float_as_int(v);
  int r;
  if constexpr (H == 1)
    r = __builtin_amdgcn_update_dpp(0, i, 0xB1, 0xF, 0xF, false);   // quad_perm [1, 0, 3, 2]
  else if constexpr (H == 2)
    r = __builtin_amdgcn_update_dpp(0, i, 0x4E, 0xF, 0xF, false);   // quad_perm [2, 3, 0, 1]
  else if constexpr (H < 32)
    r = __builtin_amdgcn_ds_swizzle(i, (H << 10) | 0x1F);          // bit mode: lane ^ H
  else
    r = __shfl_xor(i, 32, WAVE);
  return __int_as_float(r);
}

// Butterfly over the 64 lanes.  At step h lane j adds the value of lane
// j^h; since fp32 addition is commutative this is, value for value, the
// halving tree "s[j] = s[j] + s[j+h] for j < h" (h = 32 .. 1), and every
// lane ends with the tree's s[0].
__device__ __forceinline__ float wave_tree_sum(float v) {
  v = v + xor_lane<32>(v);
  v = v + xor_lane<16>(v);
  v = v + xor_lane<8>(v);
  v = v + xor_lane<4>(v);
  v = v + xor_lane<2>(v);
  v = v + xor_lane<1>(v);
  return v;
}

// (value desc, index asc): does (a, ia) rank before (b, ib)?
__device__ __forceinline__ bool ranks_before(float a, int ia, float b, int ib) {
  return (a > b) || (a == b && ia < ib);
}

// A 64-bit key whose unsigned order is the order (value desc, index asc) of
// ranks_before, for finite values: the high word maps the float's order onto
// the unsigned integers (with -0 taken as +0, equal as floats), the low word
// is larger for smaller indices.
__device__ __forceinline__ uint64_t rank_key(float v, int e) {
  uint32_t u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)o << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)e);
}

// Wave-wide maximum of a 64-bit key (rank_key order); every lane gets it.
// Within each row of 16 lanes by DPP moves (quad permutations, then the
// half-row and row mirrors: after each step every lane holds the maximum of
// its group), then over the four rows' values read out as uniform values.
template <int CTRL>
__device__ __forceinline__ uint64_t max_dpp(uint64_t k) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)k, CTRL, 0xF, 0xF, false);
  const uint32_t hi =
      (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(k >> 32), CTRL, 0xF, 0xF, false);
  const uint64_t o = ((uint64_t)hi << 32) | lo;
  return o > k ? o : k;
}

__device__ __forceinline__ uint64_t lane_key(uint64_t k, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(k >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  k = max_dpp<0xB1>(k);    // quad_perm [1, 0, 3, 2]: pairs
  k = max_dpp<0x4E>(k);    // quad_perm [2, 3, 0, 1]: quads
  k = max_dpp<0x141>(k);   // row_half_mirror: 8 lanes
  k = max_dpp<0x140>(k);   // row_mirror: 16 lanes
  const uint64_t a = lane_key(k, 0), b = lane_key(k, 16), c = lane_key(k, 32),
                 d = lane_key(k, 48);
  const uint64_t ab = a > b ? a : b, cd = c > d ? c : d;
  return ab > cd ? ab : cd;
}

// ------------------------------------------------------------ base_exp ---
// exp(x) by Cody-Waite reduction and a degree-7 Taylor polynomial:
//   x <- clamp(x, -86, 88); n = rint(x * log2 e);
//   r = fma(-n, C1, x); r = fma(-n, C2, r)   (C1 + C2 = ln 2, C1 short);
//   p = 1/7!; p = fma(p, r, 1/k!) for k = 6 .. 0;  result p * 2^n.
// Constants are the binary32 values nearest the stated reals; C1 is ln 2
// with its 9 low significand bits cleared so that n * C1 is exact.
__device__ __forceinline__ float base_exp(float x) {
  const float C1 = __uint_as_float(0x3F317200u);
  const float C2 = __uint_as_float(0x35BFBE8Eu);
  x = fminf(fmaxf(x, -86.0f), 88.0f);
  float t = x * 1.44269504088896341f;
  float n = __builtin_rintf(t);
  float r = __builtin_fmaf(-n, C1, x);
  r = __builtin_fmaf(-n, C2, r);
  float p = 1.0f / 5040.0f;
  p = __builtin_fmaf(p, r, 1.0f / 720.0f);
  p = __builtin_fmaf(p, r, 1.0f / 120.0f);
  p = __builtin_fmaf(p, r, 1.0f / 24.0f);
  p = __builtin_fmaf(p, r, 1.0f / 6.0f);
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  return __builtin_ldexpf(p, (int)n);
}

// SwiGLU activation of the expert FFN (not part of the bit-exact path).
// silu(a) = a / (1 + exp(-a)) for fp32 results
__device__ __forceinline__ float silu(float a) {
  return a / (1.0f + __expf(-a));
}

// The same for a result that is rounded to bf16 next: the quotient as a
// product with the hardware reciprocal (within an ulp or two of fp32, far
// below bf16's rounding; the limits agree with the quotient's: -0 for a ->
// -inf, a for large a, NaN for NaN)
__device__ __forceinline__ float silu_bf16(float a) {
  return a * __builtin_amdgcn_rcpf(1.0f + __expf(-a));
}

}  // namespace basek
