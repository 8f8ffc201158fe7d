// Device-side building blocks shared by the FMMformer attention kernels:
// storage types, matrix-core (MFMA) fragment helpers, feature maps and
// wavefront reductions, all for gfx950 (CDNA4, 64-wide wavefronts).
//
// Fragment convention used by every contraction in this library
// ---------------------------------------------------------------
// A 16x16 MFMA tile is held by one wavefront: lane L has column r = L % 16 and
// lane group g = L / 16 (0..3).  The output (C/D) of
// v_mfma_f32_16x16x{4f32,32_bf16} holds rows 4g..4g+3 of column r.
// For the operands, the contraction index runs over 16-wide blocks, and in
// every block lane group g supplies the four consecutive indices 4g..4g+3
// (a "quad").  One MFMA step consumes:
//   fp32 16x16x4   : one element of one quad      (4 steps per block)
//   bf16 16x16x32  : two quads of two blocks      (1 step per 2 blocks; a
//                    single quad is padded with a zero quad)
// A and B use the same index for the same (lane group, element) slot, so any
// such assignment contracts correctly; the quad assignment is chosen because
// the MFMA output already has it (rows 4g..4g+3), so a score tile can be fed
// back as the next product's operand without moving data between lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fmm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// bf16 values are stored as their raw 16-bit patterns.
typedef uint16_t bf16_t;

// ---------------------------------------------------------------- quads
// Four consecutive contraction-index values of one lane.
template <typename T> struct QuadOf;
template <> struct QuadOf<float> { typedef float4 type; };
template <> struct QuadOf<bf16_t> { typedef uint2 type; };   // 4 x bf16 bits

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
  __bf16 h = (__bf16)x;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Two floats to two bf16 (round to nearest even) in one 32-bit word, low
// half first; a single v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// quad <-> 4 floats
__device__ __forceinline__ void quad_to_f32(const float4& q, float* f) {
  f[0] = q.x; f[1] = q.y; f[2] = q.z; f[3] = q.w;
}
__device__ __forceinline__ void quad_to_f32(const uint2& q, float* f) {
  f[0] = bf16_to_f32(q.x & 0xffffu); f[1] = bf16_to_f32(q.x >> 16);
  f[2] = bf16_to_f32(q.y & 0xffffu); f[3] = bf16_to_f32(q.y >> 16);
}
template <typename T> __device__ __forceinline__ typename QuadOf<T>::type f32_to_quad(const float* f);
template <> __device__ __forceinline__ float4 f32_to_quad<float>(const float* f) {
  return make_float4(f[0], f[1], f[2], f[3]);
}
template <> __device__ __forceinline__ uint2 f32_to_quad<bf16_t>(const float* f) {
  return make_uint2(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]));
}
// Value actually used by the matrix core for a float rounded to T.
template <typename T> __device__ __forceinline__ float round_as(float x);
template <> __device__ __forceinline__ float round_as<float>(float x) { return x; }
template <> __device__ __forceinline__ float round_as<bf16_t>(float x) {
  return bf16_to_f32(f32_to_bf16_bits(x));
}

// ---------------------------------------------------------------- MFMA
__device__ __forceinline__ f32x4 mma_step(const float4& a, const float4& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
  return c;
}
// One bf16 quad: issued as v_mfma_f32_16x16x32_bf16 with the second quad of
// both operands zero.  (The 16x16x16 bf16 instruction gave wrong sums in some
// instruction schedules of the causal kernel at d = 16 with this toolchain;
// the zero-padded 32-wide form is exact and only d = 16 contractions use it.)
__device__ __forceinline__ f32x4 mma_step(const uint2& a, const uint2& b, f32x4 c) {
  const uint4 ua = make_uint4(a.x, a.y, 0u, 0u), ub = make_uint4(b.x, b.y, 0u, 0u);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ua),
                                                 __builtin_bit_cast(bf16x8, ub), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_step2(const uint2& a0, const uint2& a1,
                                           const uint2& b0, const uint2& b1, f32x4 c) {
  uint4 ua = make_uint4(a0.x, a0.y, a1.x, a1.y);
  uint4 ub = make_uint4(b0.x, b0.y, b1.x, b1.y);
  bf16x8 av = __builtin_bit_cast(bf16x8, ua);
  bf16x8 bv = __builtin_bit_cast(bf16x8, ub);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_step2(const float4& a0, const float4& a1,
                                           const float4& b0, const float4& b1, f32x4 c) {
  return mma_step(a1, b1, mma_step(a0, b0, c));
}

// Contract NQ quads (NQ 16-wide blocks of the contraction index).
template <int NQ, typename Q>
__device__ __forceinline__ f32x4 contract(const Q* a, const Q* b, f32x4 c) {
  if constexpr (NQ % 2 == 0) {
#pragma unroll
    for (int t = 0; t < NQ; t += 2) c = mma_step2(a[t], a[t + 1], b[t], b[t + 1], c);
  } else {
#pragma unroll
    for (int t = 0; t < NQ; ++t) c = mma_step(a[t], b[t], c);
  }
  return c;
}

// ---------------------------------------------------------------- maps
// phi_1(x) = elu(x) + 1 and phi_2(x) = elu(-x) + 1 share e = exp(-|x|).
// Since exp(y) >= 1 + y for every y, phi_1(x) = max(1 + x, e) (for x > 0, e <
// 1 < 1 + x; for x <= 0, e = exp(x) >= 1 + x) and likewise phi_2(x) =
// max(1 - x, e): one exponential, two adds, two max.
__device__ __forceinline__ void phi12(float x, float& p1, float& p2) {
  const float e = __expf(-fabsf(x));
  p1 = fmaxf(1.f + x, e);
  p2 = fmaxf(1.f - x, e);
}
__device__ __forceinline__ float phi_l(float x, int l) {
  float p1, p2;
  phi12(x, p1, p2);
  return l == 0 ? p1 : p2;
}
// The first R feature maps of x: phi_1, phi_2 as above and phi_3(x) = tanh(x)
// (the third map of Sec. 3.2.1).
template <int R>
__device__ __forceinline__ void phi_maps(float x, float* p) {
  float p1, p2;
  phi12(x, p1, p2);
  p[0] = p1;
  if constexpr (R >= 2) p[1] = p2;
  if constexpr (R >= 3) p[2] = tanhf(x);
}
// Feature map l (0-based) of x, for a map index known only at run time.
__device__ __forceinline__ float phi_any(float x, int l) {
  if (l == 2) return tanhf(x);
  return phi_l(x, l);
}

__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

__device__ __forceinline__ float sigmoidf_exact(float w) {
  // 1/(1+exp(-w)); w = +inf -> 1, w = -inf -> 0
  return 1.0f / (1.0f + expf(-w));
}

// Sum / max over the four lanes that share a column (lanes r, r+16, r+32,
// r+48), with the gfx950 lane-swap instructions: permlane32_swap exchanges
// the upper half of one register with the lower half of another, so (a, b)
// = swap(x, x) holds x's two halves in opposite order; permlane16_swap does
// the same for odd and even 16-lane rows.  Plain VALU, no LDS round trip.
__device__ __forceinline__ float col_max(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float y = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false,
                                                  false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
__device__ __forceinline__ float col_sum(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float y = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false,
                                                  false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// Workgroup index remap so that consecutive logical tiles land on the same
// XCD (the hardware deals workgroups round-robin over the 8 XCDs, each with
// its own L2); neighbouring tiles share key/value halo rows.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int xcd = bid & 7, idx = bid >> 3;
  const int q = nblocks >> 3, rem = nblocks & 7;
  return xcd * q + min(xcd, rem) + idx;
}

}  // namespace fmm
