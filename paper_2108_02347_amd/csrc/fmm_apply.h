// Building blocks of the apply kernels (near field, far field, blend), shared
// by the tuned kernels of fmm_kernels.hip and the general kernel of
// fmm_wide.hip: workgroup shape, raw-buffer global access, LDS operand reads,
// row staging, the online-softmax near field over staged key units, the far
// products with state fragments, and the blend and store of a row strip.
#pragma once

#include "fmm_device.h"

namespace fmm {

constexpr int NW = 4;            // wavefronts per apply workgroup
constexpr int NT = NW * 64;      // threads per apply workgroup
constexpr int TM = 16 * NW;      // query rows per tile (= 2 key units)

template <typename T> struct Lay {
  static constexpr int ES = (int)sizeof(T);
  static constexpr int EPC = 16 / ES;          // elements per 16-byte chunk
  static constexpr int PAD = ES == 2 ? 8 : 4;  // row pad (rows stay 16-B aligned)
};

// LDS budgets of the apply kernels.  Ring kernels: ring + state fragments (+
// the causal tile's feature rows) within 78 KiB, so two workgroups fit on a
// CU whatever the band (narrower bands use less and fit more); U_NC / U_C is
// the widest ring, in 32-key units, of the non-causal / causal walk.  Rounds
// kernels (bands wider than the ring): up to UR units per round within 150 KiB.
template <typename T, int D, int R> struct Ring {
  static constexpr int ST = D + Lay<T>::PAD;
  static constexpr int UNIT_BYTES = 2 * 32 * ST * (int)sizeof(T);  // K + V
  static constexpr int FRAG_BYTES = R * (D / 16) * (D / 16) * 64 * 4 * (int)sizeof(T) + R * D * 4;
  static constexpr int PHI_BYTES = R * TM * ST * (int)sizeof(T);   // causal only
  static constexpr int BUDGET = 78 * 1024, RBUDGET = 150 * 1024;
  static constexpr int U_NC = (BUDGET - FRAG_BYTES) / UNIT_BYTES;
  static constexpr int U_C = (BUDGET - FRAG_BYTES - PHI_BYTES) / UNIT_BYTES;
  static constexpr int UR_FIT = (RBUDGET - FRAG_BYTES - PHI_BYTES) / UNIT_BYTES;
  static constexpr int UR = UR_FIT > 6 ? 6 : UR_FIT;
  static_assert(UR >= 2, "a round must hold one tile of keys");
  static size_t bytes(int u, bool causal) {
    return (size_t)u * UNIT_BYTES + FRAG_BYTES + (causal ? PHI_BYTES : 0);
  }
};

// ------------------------------------------------------------------ global access
// Rows [r0, r0 + nrows) of a [N, D] head, clipped to [0, N), as a raw buffer
// whose offsets count from row max(r0, 0).  Buffer loads outside it (rows
// before 0 give negative, i.e. huge unsigned, offsets; rows at or beyond the
// clip give offsets past its size) return zeros without touching memory and
// stores there are dropped, so row-range checks need no branches and the
// compiler's memory-counter waits stay exact across the prefetch pipeline.
typedef __amdgpu_buffer_rsrc_t Rsrc;
template <typename T, int D>
__device__ __forceinline__ Rsrc rows_rsrc(const T* head, int r0, int nrows, int N) {
  const int b = max(r0, 0);
  const int n = max(0, min(r0 + nrows, N) - b);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(head + (size_t)b * D), 0,
                                           n * D * (int)sizeof(T), 0x00020000);
}
__device__ __forceinline__ uint4 buf_ld(Rsrc rs, int off, uint4*) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}
__device__ __forceinline__ float4 buf_ld(Rsrc rs, int off, float4*) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}
__device__ __forceinline__ uint2 buf_ld(Rsrc rs, int off, uint2*) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
}
__device__ __forceinline__ void buf_st(Rsrc rs, int off, const float4& v) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), rs, off, 0, 0);
}
__device__ __forceinline__ void buf_st(Rsrc rs, int off, const uint2& v) {
  typedef int i32x2 __attribute__((ext_vector_type(2)));
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(i32x2, v), rs, off, 0, 0);
}
// First row of the lane's 16-row strip (wave-uniform): row - r.
__device__ __forceinline__ int strip_row0(int row) {
  return __builtin_amdgcn_readfirstlane(row - (threadIdx.x & 15));
}

// ------------------------------------------------------------------ LDS operand reads
// Row-major quad: X[row][col .. col+3].
template <typename T>
__device__ __forceinline__ typename QuadOf<T>::type ld_quad(const T* x, int row, int col, int ld) {
  return *reinterpret_cast<const typename QuadOf<T>::type*>(x + row * ld + col);
}

// Transposed quad: lane (r, g) receives X[row0 + 4g + e][col0 + r], e = 0..3.
// bf16 uses the gfx950 LDS transpose read: within each 16-lane group, lane t
// reads the 4 values X[row0 + 4g + t/4][col0 + 4(t%4) .. +3] and the hardware
// hands lane j the j%4-th value of lane 4e + j/4 as element e.
__device__ __forceinline__ uint2 ld_tquad(const bf16_t* x, int row0, int col0, int ld) {
  const int lane = threadIdx.x & 63, g = lane >> 4, t = lane & 15;
  const bf16_t* p = x + (row0 + 4 * g + (t >> 2)) * ld + col0 + 4 * (t & 3);
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  return __builtin_bit_cast(uint2, v);
}
__device__ __forceinline__ float4 ld_tquad(const float* x, int row0, int col0, int ld) {
  const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
  const float* p = x + (row0 + 4 * g) * ld + col0 + r;
  return make_float4(p[0], p[ld], p[2 * ld], p[3 * ld]);
}

template <typename T> __device__ __forceinline__ typename QuadOf<T>::type quad_fill(float x) {
  const float f[4] = {x, x, x, x};
  return f32_to_quad<T>(f);
}

// ------------------------------------------------------------------ row staging
// Copy rows [k0, k0 + nrows) of a [N, D] head into LDS (row-major, stride ST);
// rows outside [0, N) are zero.  `dst_row(i)` gives the LDS row of the i-th
// copied row.
template <typename T, int D, int NTHR, int MAXROWS>
struct RowCopy {
  static constexpr int CPR = D / Lay<T>::EPC;
  static constexpr int IT = (MAXROWS * CPR + NTHR - 1) / NTHR;
  uint4 r[IT];
  __device__ __forceinline__ void load(const T* __restrict__ src, int k0, int nrows, int N) {
    const Rsrc rs = rows_rsrc<T, D>(src, k0, nrows, N);
    const int b = max(k0, 0);
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NTHR;
      const int key = k0 + t / CPR;
      r[it] = buf_ld(rs, ((key - b) * D + (t % CPR) * Lay<T>::EPC) * (int)sizeof(T), (uint4*)0);
    }
  }
  // A full copy (nrows == MAXROWS filling every thread's passes) stores
  // without a row test: a test the compiler cannot fold would sink the
  // copy's loads behind it, after a wait for every load in flight.
  template <typename F>
  __device__ __forceinline__ void store(T* dst, int ST, int nrows, F dst_row) const {
    const bool full = MAXROWS * CPR == IT * NTHR && nrows == MAXROWS;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NTHR;
      if (full || t < nrows * CPR)
        *reinterpret_cast<uint4*>(dst + dst_row(t / CPR) * ST + (t % CPR) * Lay<T>::EPC) = r[it];
    }
  }
};

// LDS row of the first key of absolute 32-key unit ua.
struct RingMap {
  int ua0, U;
  __device__ __forceinline__ int operator()(int ua) const { return ((ua - ua0) % U) * 32; }
};
struct RoundMap {
  int ks;
  __device__ __forceinline__ int operator()(int ua) const { return ua * 32 - ks; }
};

// ------------------------------------------------------------------ near field
// Softmax state of one wavefront's 16-row strip.  Lane (r, g) holds row r;
// o[nb] (nb < NB) holds output columns 16nb + 4g + {0..3}; o[NB] holds the
// row's sum of weights in all four entries; m is the running maximum of the
// raw scores q.k of the row.
template <int D> struct NearState {
  f32x4 o[D / 16 + 1];
  float m;
  int fresh;  // wave-uniform: nothing accumulated yet
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int nb = 0; nb <= D / 16; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    fresh = 1;
  }
};

// Band units [ua_lo, ua_hi] (32 keys each, in LDS through `map`) for the strip
// of rows [i0, i0 + 16).  Up to GU units are scored at once, then one row
// maximum, one exponentiation pass and the P V products; the accumulator is
// rescaled only between groups.  Exponentials use exp2 with tau*log2(e)
// folded into the subtraction of the maximum.
template <typename T, int D, bool CAUSAL, int GU, class Map>
__device__ __forceinline__ void near_units(NearState<D>& st, const typename QuadOf<T>::type* qq,
                                           const T* kr, const T* vr, int ST, Map map, int ua_lo,
                                           int ua_hi, int i0, int N, int band_k, float scale2) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int row = i0 + r;
  const Q ones = quad_fill<T>(1.f);
  for (int u0 = ua_lo; u0 <= ua_hi; u0 += GU) {
    f32x4 sc[GU][2];
    float mloc = -INFINITY;
#pragma unroll
    for (int gi = 0; gi < GU; ++gi) {
      const int ua = u0 + gi;
      if (ua > ua_hi) break;
      const T* kx = kr + map(ua) * ST;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        Q ka[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) ka[cb] = ld_quad(kx, 16 * b + r, 16 * cb + 4 * g, ST);
        sc[gi][b] = contract<NB>(ka, qq, f32x4{0.f, 0.f, 0.f, 0.f});
      }
      const int j0 = ua * 32;
      const bool interior = j0 >= 0 && j0 + 31 < N && j0 >= i0 + 15 - band_k &&
                            (CAUSAL ? j0 + 31 <= i0 : j0 + 31 <= i0 + band_k);
      if (!interior) {
        // valid keys of this lane's row form one interval; in unit-local
        // offsets c = 16b + i (lane group g adds 4g) it is [lo, lo + span]
        int lo = max(row - band_k, 0) - j0 - 4 * g;
        int span = min(CAUSAL ? row : row + band_k, N - 1) - j0 - 4 * g - lo;
        if (span < 0) { lo = 64; span = 0; }
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if ((unsigned)(16 * b + i - lo) > (unsigned)span) sc[gi][b][i] = -INFINITY;
      }
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) mloc = fmaxf(mloc, sc[gi][b][i]);
    }
    const float mnew = fmaxf(st.m, col_max(mloc));
    const float ms = (mnew == -INFINITY ? 0.f : mnew) * scale2;
    if (!__builtin_amdgcn_readfirstlane(st.fresh)) {
      const float alpha = __builtin_amdgcn_exp2f(st.m * scale2 - ms);
#pragma unroll
      for (int nb = 0; nb <= NB; ++nb) st.o[nb] *= alpha;
    }
    st.m = mnew;
    st.fresh = 0;
#pragma unroll
    for (int gi = 0; gi < GU; ++gi) {
      const int ua = u0 + gi;
      if (ua > ua_hi) break;
      float p[2][4];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) p[b][i] = __builtin_amdgcn_exp2f(fmaf(sc[gi][b][i], scale2, -ms));
      const Q pq0 = f32_to_quad<T>(p[0]), pq1 = f32_to_quad<T>(p[1]);
      const T* vx = vr + map(ua) * ST;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        st.o[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), pq0,
                             pq1, st.o[nb]);
      st.o[NB] = mma_step2(ones, ones, pq0, pq1, st.o[NB]);
    }
  }
}

// Straight-line form of near_units for a strip whose band is exactly the NU
// units [ua_lo, ua_lo + NU) with units 1 .. NU-2 inside the band for every
// row of the strip (and inside [0, N)): no per-unit branches, so the
// compiler can overlap one unit's score products with another's softmax
// arithmetic; only the two end units are masked.  Fresh state only.
template <typename T, int D, bool CAUSAL, int NU, class Map>
__device__ __forceinline__ void near_fixed(NearState<D>& st, const typename QuadOf<T>::type* qq,
                                           const T* kr, const T* vr, int ST, Map map, int ua_lo,
                                           int i0, int N, int band_k, float scale2) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int row = i0 + r;
  const Q ones = quad_fill<T>(1.f);
  f32x4 sc[NU][2];
  int urow[NU];
#pragma unroll
  for (int gi = 0; gi < NU; ++gi) urow[gi] = map(ua_lo + gi);
#pragma unroll
  for (int gi = 0; gi < NU; ++gi) {
    const T* kx = kr + urow[gi] * ST;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      Q ka[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) ka[cb] = ld_quad(kx, 16 * b + r, 16 * cb + 4 * g, ST);
      sc[gi][b] = contract<NB>(ka, qq, f32x4{0.f, 0.f, 0.f, 0.f});
    }
  }
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int gi = e == 0 ? 0 : NU - 1;
    const int j0 = (ua_lo + gi) * 32;
    int lo = max(row - band_k, 0) - j0 - 4 * g;
    int span = min(CAUSAL ? row : row + band_k, N - 1) - j0 - 4 * g - lo;
    if (span < 0) { lo = 64; span = 0; }
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((unsigned)(16 * b + i - lo) > (unsigned)span) sc[gi][b][i] = -INFINITY;
  }
  float mloc = -INFINITY;
#pragma unroll
  for (int gi = 0; gi < NU; ++gi)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) mloc = fmaxf(mloc, sc[gi][b][i]);
  const float mnew = col_max(mloc);
  const float ms = mnew * scale2;
  st.m = mnew;
  st.fresh = 0;
#pragma unroll
  for (int gi = 0; gi < NU; ++gi) {
    float p[2][4];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) p[b][i] = __builtin_amdgcn_exp2f(fmaf(sc[gi][b][i], scale2, -ms));
    const Q pq0 = f32_to_quad<T>(p[0]), pq1 = f32_to_quad<T>(p[1]);
    const T* vx = vr + urow[gi] * ST;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      st.o[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), pq0, pq1,
                           st.o[nb]);
    st.o[NB] = mma_step2(ones, ones, pq0, pq1, st.o[NB]);
  }
}

// True when the strip [i0, i0 + 16) takes the near_fixed<NU> path: its band
// spans exactly NU units, the middle ones inside the band for all its rows
// and the whole span inside [0, N).
template <bool CAUSAL, int NU>
__device__ __forceinline__ bool fixed_strip(int i0, int N, int band_k) {
  const int lo = i0 - band_k, hi = CAUSAL ? i0 + 15 : i0 + 15 + band_k;
  if (lo < 0 || hi >= N) return false;
  const int ul = lo >> 5;
  if ((hi >> 5) - ul != NU - 1) return false;
  if (NU < 3) return true;
  const int first_mid = (ul + 1) * 32, last_mid_end = (ul + NU - 2) * 32 + 31;
  return first_mid >= i0 + 15 - band_k && last_mid_end <= (CAUSAL ? i0 : i0 + band_k);
}

// ------------------------------------------------------------------ far field
// phi_1(q), phi_2(q) of the lane's row as operand quads.
template <typename T, int D, int R>
__device__ __forceinline__ void phi_q(const typename QuadOf<T>::type* qq,
                                      typename QuadOf<T>::type (*pq)[D / 16]) {
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb) {
    float x[4], p1[4], p2[4];
    quad_to_f32(qq[cb], x);
#pragma unroll
    for (int i = 0; i < 4; ++i) phi12(x[i], p1[i], p2[i]);
    pq[0][cb] = f32_to_quad<T>(p1);
    if constexpr (R == 2) pq[1][cb] = f32_to_quad<T>(p2);
  }
}

// num[l][nb] (+)= S_l^T phi_l(Q)^T for nb < NB and num[l][NB] (+)= phi_l(q) . z_l
// (z_l broadcast over the 16 rows of an extra A block).  State fragments:
// sf[(l*NB + nb)*NB + cb][lane] = S_l[16cb + 4g + {0..3}][16nb + r];
// szq[(l*NB + cb)*4 + g] = z_l[16cb + 4g + {0..3}].  ACC = false starts the
// sums from zero.
template <typename T, int D, int R, bool ACC>
__device__ __forceinline__ void far_terms(const typename QuadOf<T>::type* sf,
                                          const typename QuadOf<T>::type* szq,
                                          const typename QuadOf<T>::type (*pq)[D / 16],
                                          f32x4 (*num)[D / 16 + 1]) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int l = 0; l < R; ++l) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      Q a[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) a[cb] = sf[((l * NB + nb) * NB + cb) * 64 + lane];
      num[l][nb] = contract<NB>(a, pq[l], ACC ? num[l][nb] : zero);
    }
    Q zq[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) zq[cb] = szq[(l * NB + cb) * 4 + g];
    num[l][NB] = contract<NB>(zq, pq[l], ACC ? num[l][NB] : zero);
  }
}

// The same terms for one map l, accumulated into num (NB + 1 tiles).
template <typename T, int D>
__device__ __forceinline__ void far_terms_map(const typename QuadOf<T>::type* sf,
                                              const typename QuadOf<T>::type* szq, int l,
                                              const typename QuadOf<T>::type* pql, f32x4* num) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    Q a[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) a[cb] = sf[((l * NB + nb) * NB + cb) * 64 + lane];
    num[nb] = contract<NB>(a, pql, num[nb]);
  }
  Q zq[NB];
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) zq[cb] = szq[(l * NB + cb) * 4 + g];
  num[NB] = contract<NB>(zq, pql, num[NB]);
}

// Near part of the output, sigmoid(w_near) * near, in the lane's output layout.
template <int D>
__device__ __forceinline__ void near_out(const NearState<D>& st, float sn, f32x4* fo) {
  constexpr int NB = D / 16;
  const float a = sn > 0.f ? sn * fast_rcp(st.o[NB][0]) : 0.f;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) fo[nb] = st.o[nb] * a;
}

// fo += sigmoid(w_far) * num / den for one map (den in num[NB]).
template <int D>
__device__ __forceinline__ void add_far_map(const f32x4* num, float sfw, f32x4* fo) {
  constexpr int NB = D / 16;
  const float f = sfw > 0.f ? sfw * fast_rcp(num[NB][0]) : 0.f;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) fo[nb] += num[nb] * f;
}

template <typename T, int D>
__device__ __forceinline__ void store_row(T* __restrict__ oh, int row, int N, const f32x4* fo) {
  const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
  const Rsrc rs = rows_rsrc<T, D>(oh, strip_row0(row), 16, N);
#pragma unroll
  for (int nb = 0; nb < D / 16; ++nb) {
    const float o[4] = {fo[nb][0], fo[nb][1], fo[nb][2], fo[nb][3]};
    buf_st(rs, (r * D + 16 * nb + 4 * g) * (int)sizeof(T), f32_to_quad<T>(o));
  }
}

// out = sigmoid(w_near) near + sigmoid(w_far) sum_l num_l / den_l  (Eq. (11)).
template <typename T, int D, int R>
__device__ __forceinline__ void blend_store(T* __restrict__ oh, int row, int N, float sn,
                                            float sfw, const NearState<D>& st,
                                            const f32x4 (*num)[D / 16 + 1]) {
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
  const Rsrc rs = rows_rsrc<T, D>(oh, strip_row0(row), 16, N);
  const float a = sn > 0.f ? sn * fast_rcp(st.o[NB][0]) : 0.f;
  float f[R];
#pragma unroll
  for (int l = 0; l < R; ++l) f[l] = sfw > 0.f ? sfw * fast_rcp(num[l][NB][0]) : 0.f;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float x = st.o[nb][i] * a;
#pragma unroll
      for (int l = 0; l < R; ++l) x = fmaf(num[l][nb][i], f[l], x);
      o[i] = x;
    }
    buf_st(rs, (r * D + 16 * nb + 4 * g) * (int)sizeof(T), f32_to_quad<T>(o));
  }
}

// Fill state fragments from a tile-order record (non-causal final state).
template <typename T, int D, int R, int NTHR>
__device__ __forceinline__ void load_state_frags(const float* __restrict__ rec,
                                                 typename QuadOf<T>::type* sf,
                                                 typename QuadOf<T>::type* szq) {
  constexpr int NB = D / 16;
  constexpr int E = R * NB * NB * 64;
  for (int t = threadIdx.x; t < E; t += NTHR) {
    const int lane = t & 63, blk = t >> 6;
    const int cb = blk % NB, nb = (blk / NB) % NB, l = blk / (NB * NB);
    const float4 v = *reinterpret_cast<const float4*>(
        rec + (size_t)l * D * (D + 1) + ((cb * NB + nb) * 64 + lane) * 4);
    const float f[4] = {v.x, v.y, v.z, v.w};
    sf[t] = f32_to_quad<T>(f);
  }
  for (int t = threadIdx.x; t < R * NB * 4; t += NTHR) {
    const int l = t / (NB * 4), c0 = 4 * (t % (NB * 4));
    const float* z = rec + (size_t)l * D * (D + 1) + D * D + c0;
    const float f[4] = {z[0], z[1], z[2], z[3]};
    szq[t] = f32_to_quad<T>(f);
  }
}

// Query quads of one row: lane (r, g) gets q[row][16cb + 4g + {0..3}].
template <typename T, int D>
__device__ __forceinline__ void load_q(const T* __restrict__ qh, int row, int N,
                                       typename QuadOf<T>::type* qq) {
  using Q = typename QuadOf<T>::type;
  const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
  const Rsrc rs = rows_rsrc<T, D>(qh, strip_row0(row), 16, N);
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb)
    qq[cb] = buf_ld(rs, (r * D + 16 * cb + 4 * g) * (int)sizeof(T), (Q*)0);
}

}  // namespace fmm
