// Building blocks of the bf16 strip kernels (fmm_pair.hip, fmm_causal.hip):
// oct operands, raw buffer accesses and the swizzled LDS rows of K, V and
// phi(K).
//
// Operands contracted over the head width (scores, far terms) are "octs": the
// contraction index runs over 32-wide blocks and lane group g holds the eight
// consecutive indices 8g..8g+7 of a block, so a row's slice is one 16-byte LDS
// read.  Products contracted over keys (P V, the state sums) take their key
// operands from transposed 8-byte reads, four keys per lane group and block.
#pragma once

#include "fmm_device.h"

namespace fmm {

typedef uint4 Oct;  // 8 bf16

__device__ __forceinline__ f32x4 mma8(const Oct& a, const Oct& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ Oct oct_of(const uint2& lo, const uint2& hi) {
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}
__device__ __forceinline__ Oct oct_pack(const float* f) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                    pack_bf16x2(f[6], f[7]));
}
__device__ __forceinline__ void oct_unpack(const Oct& o, float* f) {
  const uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ uint2 quad_pack(const f32x4& x) {
  return make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
}
// bf16 1.0 in all eight slots
__device__ __forceinline__ Oct oct_ones() {
  return make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
}
// Larger of two bf16 pairs, lane by lane, for pairs whose second operand is
// >= +0: for such values the order of the bit patterns read as signed 16-bit
// integers is the order of the numbers (a negative first operand has its sign
// bit set and compares below), and rounding to bf16 is monotone, so
// max(bf16(a), bf16(b)) = bf16(max(a, b)).  One v_pk_max_i16 per pair.
__device__ __forceinline__ uint32_t pk_max_bf16_nonneg(uint32_t a, uint32_t b) {
  typedef short s16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, a),
                                                                __builtin_bit_cast(s16x2, b)));
}
// phi_1 and phi_2 of eight values.  Of the two numbers 1 + |x| and
// e = exp(-|x|), phi_1(x) = elu(x) + 1 takes 1 + |x| for x >= 0 and e for
// x < 0, phi_2(x) = elu(-x) + 1 the other one (both are 1 at x = 0).  Both are
// packed to bf16 (the same bits as rounding phi_1, phi_2 themselves), and each
// 16-bit half is picked by the sign bit of its input: a byte permute whose
// selectors 8 and 9 replicate bits 15 and 31 turns the two signs into
// half-word masks, a bit-select per map does the rest.
__device__ __forceinline__ void phi_oct(const Oct& x, Oct& p1, Oct& p2) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(w[i] << 16), hi = __uint_as_float(w[i] & 0xffff0000u);
    const uint32_t e = pack_bf16x2(__expf(-fabsf(lo)), __expf(-fabsf(hi)));
    const uint32_t o = pack_bf16x2(1.f + fabsf(lo), 1.f + fabsf(hi));
    // 0xffff in each half whose input has its sign bit set
    const uint32_t m = __builtin_amdgcn_perm(0u, w[i], 0x09090808u);
    a[i] = (e & m) | (o & ~m);
    b[i] = (o & m) | (e & ~m);
  }
  p1 = make_uint4(a[0], a[1], a[2], a[3]);
  p2 = make_uint4(b[0], b[1], b[2], b[3]);
}

// Buffer resource over one head's [N, D] bf16 rows.  Raw buffer loads past
// its end (or at a negative offset, i.e. a huge unsigned one) return zeros
// without touching memory and stores there are dropped, so every global access
// of a walk is branch-free: rows outside [0, N) and skipped prefetches just
// use out-of-range offsets.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr uint32_t OOB = 0x80000000u;
__device__ __forceinline__ Rsrc head_rsrc(const bf16_t* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(p), 0, bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(Rsrc rs, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

// Byte offset of 16-byte chunk c of LDS row r.  The LDS serves 64 banks of 4
// bytes per cycle: an 8-byte read in two passes of 32 consecutive lanes, a
// 16-byte read in four passes of 16 lanes, the lanes of each half-wave split by
// bit2 ^ bit3 ^ bit4 of the lane index; a pass is conflict-free when its lanes
// touch distinct banks.  Rows are unpadded and chunk c of row r sits at chunk
// c ^ swz(r), with swz linear in the bits of r % 16, chosen so that the row
// reads of the oct operands (row r, chunk 4p + g), the transposed reads of
// the key operands (rows 4g + t/4, 8-byte halves of chunks t % 4 or
// 2nb + (t % 4)/2) and the row stores all run without conflicts.
template <int D> struct RingRows;
template <> struct RingRows<64> {
  static constexpr int RB = 128;
  __device__ __forceinline__ static int swz(int r) { return ((r & 2) ? 3 : 0) ^ ((r & 4) ? 4 : 0); }
  __device__ __forceinline__ static int off(int r, int c) { return r * RB + ((c ^ swz(r)) << 4); }
};
template <> struct RingRows<32> {
  static constexpr int RB = 64;
  __device__ __forceinline__ static int swz(int r) { return (r & 4) ? 3 : 0; }
  __device__ __forceinline__ static int off(int r, int c) { return r * RB + ((c ^ swz(r)) << 4); }
};

// Per-lane byte offsets of the reads within a 16-row block (blocks start at
// multiples of 16 rows, so the swizzle of a row depends only on its index
// within the block).  koff[p]: the lane's oct of row r, chunk 4p + g.
// voff[nb]: the lane's transposed read for columns 16nb .. 16nb+15: lane t of
// group g reads row 4g + t/4, columns 16nb + 4(t%4) .. +3, and the hardware
// hands lane (j, g) the values X[4g + e][16nb + j], e = 0..3.
template <int D>
struct RingOffsets {
  int koff[D / 32];
  int voff[D / 16];
  __device__ __forceinline__ RingOffsets() {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4, t = lane & 15;
#pragma unroll
    for (int p = 0; p < D / 32; ++p) koff[p] = RingRows<D>::off(r, 4 * p + g);
#pragma unroll
    for (int nb = 0; nb < D / 16; ++nb)
      voff[nb] = RingRows<D>::off(4 * g + (t >> 2), 2 * nb + ((t & 3) >> 1)) + 8 * (t & 1);
  }
};

__device__ __forceinline__ uint2 ld_tr16(const unsigned char* p) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  return __builtin_bit_cast(uint2, v);
}

// ROWS consecutive K or V rows [k0, k0 + ROWS) of a head in registers (zero
// outside [0, N), or everywhere when !on); thread t of NTHR holds chunk
// t % CPR of row t / CPR + (NTHR / CPR) * it.
template <int D, int ROWS, int NTHR>
struct RowsCopy {
  static constexpr int CPR = D / 8;
  static constexpr int IT = ROWS * CPR / NTHR;
  static_assert(ROWS * CPR % NTHR == 0, "whole rows per pass");
  uint4 r[IT];
  __device__ __forceinline__ void load(Rsrc rs, int k0, bool on) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * NTHR;
      const int e = (k0 + x / CPR) * D + (x % CPR) * 8;
      r[it] = buf_load16(rs, on ? (uint32_t)(2 * e) : OOB);
    }
  }
  // 32-row unit j of the copied rows goes to ring slot slot_of(j) (skipped if < 0).
  template <typename F>
  __device__ __forceinline__ void store(unsigned char* ring, F slot_of) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * NTHR;
      const int i = x / CPR;
      const int slot = slot_of(i >> 5);
      if (slot >= 0)
        *reinterpret_cast<uint4*>(ring + RingRows<D>::off(slot * 32 + (i & 31), x % CPR)) = r[it];
    }
  }
};

// Store a 16-row strip of output rows row0 .. row0+15 held in the MFMA output
// layout (lane (r, g) has row r, columns 16nb + 4g .. +3 in fo[nb]) as bf16
// with 16-byte stores: a lane-group swap exchanges the quads of column blocks
// 2c and 2c+1 between groups g and g^1, after which lane (r, g) holds the
// eight consecutive columns 32c + 16(g&1) + 8(g>>1) .. +7 and the four lanes
// of a row write 64 contiguous bytes per instruction.  Rows at or beyond the
// buffer's end are dropped.
template <int D>
__device__ __forceinline__ void store_strip(Rsrc oh, int row0, const f32x4* fo) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int c = 0; c < D / 32; ++c) {
    const uint2 a = quad_pack(fo[2 * c]), b = quad_pack(fo[2 * c + 1]);
    // odd lane groups of the first operand trade places with the even groups
    // of the second
    const auto x = __builtin_amdgcn_permlane16_swap(a.x, b.x, false, false);
    const auto y = __builtin_amdgcn_permlane16_swap(a.y, b.y, false, false);
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    const i32x4 o = {(int)x[0], (int)y[0], (int)x[1], (int)y[1]};
    const int col = 32 * c + 16 * (g & 1) + 8 * (g >> 1);
    __builtin_amdgcn_raw_buffer_store_b128(o, oh, 2 * ((row0 + r) * D + col), 0, 0);
  }
}

// Query octs of the lane's row of NS consecutive 16-row strips:
// qo[s][p] = q[i0 + 16s + r][32p + 8g .. +7] (zero for rows at or beyond N,
// or everywhere when !on).
template <int D, int NS>
__device__ __forceinline__ void load_qo(Rsrc rs, int i0, bool on, Oct (*qo)[D / 32]) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int p = 0; p < D / 32; ++p) {
      const int e = (i0 + 16 * s + r) * D + 32 * p + 8 * g;
      qo[s][p] = buf_load16(rs, on ? (uint32_t)(2 * e) : OOB);
    }
}

}  // namespace fmm
