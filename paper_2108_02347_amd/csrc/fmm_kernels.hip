// HIP kernels of the FMMformer attention forward operator for gfx950.
//
//   k_seg_state      per-segment far-field totals  T_l = phi_l(K)^T [V | 1]
//                    (Eq. (5), Eq. (7): the regrouped products phi_l(K)^T V and
//                    the normaliser phi_l(K)^T 1), MFMA over the keys
//   k_state_combine  fixed-order sum over segments (non-causal S_l, z_l) or
//                    exclusive scan over segments (causal prefix, Sec. 3.2.1)
//   k_band_ring      non-causal, band fits the LDS ring: each workgroup walks the
//                    64-row tiles of a segment; the key/value window slides
//                    through an LDS ring and the next tile is prefetched into
//                    registers during compute.  Per tile: banded online softmax
//                    (Eq. (3)), far apply phi_l(Q) S_l / phi_l(Q) z_l
//                    (Eq. (8)-(9)), sigmoid blend (Eq. (11)), store
//   k_causal_ring    causal, band fits the ring: same walk, with the running
//                    state carried in registers; per tile the causal band
//                    [i-k, i], the intra-tile lower-triangular far part, the
//                    prefix far part, the blend and the state update
//   k_band_rounds,   the same two operators for bands wider than the ring: every
//   k_causal_rounds  tile stages its key window in rounds
//
// Every workgroup of the apply kernels has NW = 4 wavefronts; wave w owns query
// rows [16w, 16w+16) of a TM = 64-row tile.  All sums are accumulated in fp32
// in a fixed order, so results are bit-reproducible run to run.
//
// State records (one per segment, and one final record per (batch, head) in
// the non-causal form) are kept in MFMA tile order: for map l, the d x d block
// S_l is stored as tiles (cb, eb) of 16 x 16, each as 64 lanes x 4 floats with
// lane 16g + r holding S_l[16cb + 4g + i][16eb + r], i = 0..3; z_l (d floats)
// follows.  A wave's accumulator tile is then one coalesced float4 per lane.
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {

constexpr int NW = 4;            // wavefronts per apply workgroup
constexpr int NT = NW * 64;      // threads per apply workgroup
constexpr int TM = 16 * NW;      // query rows per tile (= 2 key units)
constexpr int WK = 192;          // keys staged per round in the rounds kernels

template <typename T> struct Lay {
  static constexpr int ES = (int)sizeof(T);
  static constexpr int EPC = 16 / ES;          // elements per 16-byte chunk
  static constexpr int PAD = ES == 2 ? 8 : 4;  // row pad (rows stay 16-B aligned)
};

// Ring capacity limit (in 32-key units) for the apply kernels: the LDS of one
// workgroup (ring + state fragments) stays within 78 KiB, so two workgroups
// fit on a CU whatever the band; narrower bands use less and fit more.
template <typename T, int D, int R> struct Ring {
  static constexpr int ST = D + Lay<T>::PAD;
  static constexpr int UNIT_BYTES = 2 * 32 * ST * (int)sizeof(T);  // K + V
  static constexpr int FRAG_BYTES = R * (D / 16) * (D / 16) * 64 * 4 * (int)sizeof(T) + R * D * 4;
  static constexpr int BUDGET = 78 * 1024;
  static constexpr int U = (BUDGET - FRAG_BYTES) / UNIT_BYTES;
  static size_t bytes(int u) { return (size_t)u * UNIT_BYTES + FRAG_BYTES; }
};

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

// ------------------------------------------------------------------ row staging
// Copy rows [k0, k0 + nrows) of a [N, D] head into LDS rows `dst` (row-major,
// stride ST); rows outside [0, N) are zero.  `dst_row(i)` gives the LDS row of
// the i-th copied row.
template <typename T, int D, int NTHR, int MAXROWS>
struct RowCopy {
  static constexpr int CPR = D / Lay<T>::EPC;
  static constexpr int IT = (MAXROWS * CPR + NTHR - 1) / NTHR;
  uint4 r[IT];
  __device__ __forceinline__ void load(const T* __restrict__ src, int k0, int nrows, int N) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NTHR;
      const int key = k0 + t / CPR;
      r[it] = make_uint4(0, 0, 0, 0);
      if (t < nrows * CPR && key >= 0 && key < N)
        r[it] = *reinterpret_cast<const uint4*>(src + (size_t)key * D + (t % CPR) * Lay<T>::EPC);
    }
  }
  template <typename F>
  __device__ __forceinline__ void store(T* dst, int ST, int nrows, F dst_row) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NTHR;
      if (t < nrows * CPR)
        *reinterpret_cast<uint4*>(dst + dst_row(t / CPR) * ST + (t % CPR) * Lay<T>::EPC) = r[it];
    }
  }
};

// ------------------------------------------------------------------ near field
// Online-softmax state of one wavefront's 16-row strip.  Lane (r, g) holds
// row r; o[nb] holds output columns 16nb + 4g + {0..3}; lsum is this lane's
// share of the row normaliser (summed over the four lane groups at the end).
template <int D> struct NearState {
  f32x4 o[D / 16];
  float m, lsum;
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int nb = 0; nb < D / 16; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    lsum = 0.f;
  }
};

// One 32-key unit of the band for the strip whose lane row is `row`.  kx, vx
// point at the unit's first K / V row in LDS (row-major, stride ST); j0 is the
// absolute index of its first key.  Scores use exp2 with tau*log2(e) folded in.
template <typename T, int D, bool CAUSAL>
__device__ __forceinline__ void near_unit(NearState<D>& st, const typename QuadOf<T>::type* qq,
                                          const T* kx, const T* vx, int ST, int j0, int row,
                                          int N, int band_k, float scale2) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  f32x4 sc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    Q ka[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) ka[cb] = ld_quad(kx, 16 * b + r, 16 * cb + 4 * g, ST);
    sc[b] = contract<NB>(ka, qq, f32x4{0.f, 0.f, 0.f, 0.f});
  }
  float x[2][4];
  float mloc = -INFINITY;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = j0 + 16 * b + 4 * g + i;
      const bool ok = j >= 0 && j < N && j >= row - band_k &&
                      (CAUSAL ? j <= row : j <= row + band_k);
      x[b][i] = ok ? sc[b][i] * scale2 : -INFINITY;
      mloc = fmaxf(mloc, x[b][i]);
    }
  const float mnew = fmaxf(st.m, col_max(mloc));
  const float muse = mnew == -INFINITY ? 0.f : mnew;
  const float alpha = __builtin_amdgcn_exp2f(st.m - muse);
  st.m = mnew;
  float p[2][4];
  float ps = 0.f;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[b][i] = round_as<T>(__builtin_amdgcn_exp2f(x[b][i] - muse));
      ps += p[b][i];
    }
  st.lsum = st.lsum * alpha + ps;
  const Q pq0 = f32_to_quad<T>(p[0]), pq1 = f32_to_quad<T>(p[1]);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const Q va0 = ld_tquad(vx, 0, 16 * nb, ST);
    const Q va1 = ld_tquad(vx, 16, 16 * nb, ST);
    st.o[nb] = mma_step2(va0, va1, pq0, pq1, st.o[nb] * alpha);
  }
}

// ------------------------------------------------------------------ far field
// State fragments in LDS: sf[(l*NB + nb)*NB + cb][lane] is the quad
// S_l[16cb + 4g + {0..3}][16nb + r], the A operand of F^T = S_l^T phi_l(Q)^T;
// sz[l*D + c] = z_l[c].
template <typename T, int D>
__device__ __forceinline__ void far_prefix(const typename QuadOf<T>::type* sf, const float* sz,
                                           const float* qf, int l, f32x4* num, float& den) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  float pf[D / 4];
  float dpart = 0.f;
#pragma unroll
  for (int t = 0; t < D / 4; ++t) {
    pf[t] = phi_l(qf[t], l);
    dpart += round_as<T>(pf[t]) * sz[l * D + 16 * (t >> 2) + 4 * g + (t & 3)];
  }
  den += col_sum(dpart);
  Q pq[NB];
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) pq[cb] = f32_to_quad<T>(pf + 4 * cb);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    Q a[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) a[cb] = sf[((l * NB + nb) * NB + cb) * 64 + lane];
    num[nb] = contract<NB>(a, pq, num[nb]);
  }
}

// Fill state fragments from a tile-order record (non-causal final state).
template <typename T, int D, int R, int NTHR>
__device__ __forceinline__ void load_state_frags(const float* __restrict__ rec,
                                                 typename QuadOf<T>::type* sf, float* sz) {
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
  for (int t = threadIdx.x; t < R * D; t += NTHR)
    sz[t] = rec[(size_t)(t / D) * D * (D + 1) + D * D + t % D];
}

// Query quads of one row: lane (r, g) gets q[row][16cb + 4g + {0..3}].
template <typename T, int D>
__device__ __forceinline__ void load_q(const T* __restrict__ qh, int row, int N,
                                       typename QuadOf<T>::type* qq) {
  using Q = typename QuadOf<T>::type;
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb)
    qq[cb] = row < N ? *reinterpret_cast<const Q*>(qh + (size_t)row * D + 16 * cb + 4 * g) : Q{};
}

template <typename T, int D>
__device__ __forceinline__ void q_floats(const typename QuadOf<T>::type* qq, float* qf) {
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb) quad_to_f32(qq[cb], qf + 4 * cb);
}

// Blend (Eq. (11)) and store one lane's 4 x (D/16) outputs.
template <typename T, int D>
__device__ __forceinline__ void blend_store(T* __restrict__ oh, int row, int N, float sn,
                                            float sfw, const NearState<D>& st, const f32x4* far) {
  using Q = typename QuadOf<T>::type;
  const int g = (threadIdx.x & 63) >> 4;
  const float inv_l = 1.f / col_sum(st.lsum);
#pragma unroll
  for (int nb = 0; nb < D / 16; ++nb) {
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a = sn > 0.f ? sn * (st.o[nb][i] * inv_l) : 0.f;
      const float b = sfw > 0.f ? sfw * far[nb][i] : 0.f;
      o[i] = a + b;
    }
    if (row < N)
      *reinterpret_cast<Q*>(oh + (size_t)row * D + 16 * nb + 4 * g) = f32_to_quad<T>(o);
  }
}

// Non-causal far apply for one strip: sum_l phi_l(q) S_l / phi_l(q) z_l.
template <typename T, int D, int R>
__device__ __forceinline__ void far_apply(const typename QuadOf<T>::type* sf, const float* sz,
                                          const float* qf, f32x4* far) {
  constexpr int NB = D / 16;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) far[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int l = 0; l < R; ++l) {
    f32x4 num[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) num[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    far_prefix<T, D>(sf, sz, qf, l, num, den);
    const float inv = 1.f / den;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) far[nb] += num[nb] * inv;
  }
}

// ------------------------------------------------------------------ state tiles
// A wave's share of the state T_l = phi_l(K)^T [V | 1]: the (map, feature
// block) groups ag = w + NW2*a (l = ag / NB, cb = ag % NB), every value block
// eb < NB plus the ones column eb = NB that yields z_l.
template <typename T, int D, int R, int NW2>
struct StateTiles {
  using Q = typename QuadOf<T>::type;
  static constexpr int NB = D / 16;
  static constexpr int AG = R * NB;
  static constexpr int AGPW = AG >= NW2 ? AG / NW2 : 1;
  f32x4 acc[AGPW][NB + 1];

  __device__ __forceinline__ static bool active(int w) { return w < AG; }
  __device__ __forceinline__ static int group(int w, int a) { return w + NW2 * a; }

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int a = 0; a < AGPW; ++a)
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb) acc[a][eb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // acc += phi_l(K)^T [V | 1] over one 32-key unit at LDS rows kx / vx.
  // Keys with index >= kvalid (relative to the unit) contribute nothing.
  __device__ __forceinline__ void add_unit(int w, const T* kx, const T* vx, int ST, int kvalid) {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
    Q vb0[NB + 1], vb1[NB + 1];
#pragma unroll
    for (int eb = 0; eb < NB; ++eb) {
      vb0[eb] = ld_tquad(vx, 0, 16 * eb, ST);
      vb1[eb] = ld_tquad(vx, 16, 16 * eb, ST);
    }
    {
      float f[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) f[i] = r == 0 ? 1.f : 0.f;
      vb0[NB] = f32_to_quad<T>(f);
      vb1[NB] = vb0[NB];
    }
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
      Q aq[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float kf[4], p1[4], p2[4];
        quad_to_f32(ld_tquad(kx, 16 * b, 16 * cb, ST), kf);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          phi12(kf[i], p1[i], p2[i]);
          if (16 * b + 4 * g + i >= kvalid) { p1[i] = 0.f; p2[i] = 0.f; }
        }
        aq[b] = f32_to_quad<T>(l == 0 ? p1 : p2);
      }
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb)
        acc[a][eb] = mma_step2(aq[0], aq[1], vb0[eb], vb1[eb], acc[a][eb]);
    }
  }
  // Tile-order record I/O (see the file header).
  __device__ __forceinline__ void store(int w, float* rec) const {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
      float* sl = rec + (size_t)l * D * (D + 1);
#pragma unroll
      for (int eb = 0; eb < NB; ++eb)
        *reinterpret_cast<f32x4*>(sl + ((cb * NB + eb) * 64 + lane) * 4) = acc[a][eb];
      if (r == 0) *reinterpret_cast<f32x4*>(sl + D * D + 16 * cb + 4 * g) = acc[a][NB];
    }
  }
  __device__ __forceinline__ void load(int w, const float* rec) {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
      const float* sl = rec + (size_t)l * D * (D + 1);
#pragma unroll
      for (int eb = 0; eb < NB; ++eb)
        acc[a][eb] = *reinterpret_cast<const f32x4*>(sl + ((cb * NB + eb) * 64 + lane) * 4);
      acc[a][NB] = r == 0 ? *reinterpret_cast<const f32x4*>(sl + D * D + 16 * cb + 4 * g)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  // Write this wave's tiles as apply fragments (sf, sz) for the prefix far part.
  __device__ __forceinline__ void to_frags(int w, Q* sf, float* sz) const {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) {
        const float f[4] = {acc[a][eb][0], acc[a][eb][1], acc[a][eb][2], acc[a][eb][3]};
        sf[((l * NB + eb) * NB + cb) * 64 + lane] = f32_to_quad<T>(f);
      }
      if (r == 0)
#pragma unroll
        for (int i = 0; i < 4; ++i) sz[l * D + 16 * cb + 4 * g + i] = acc[a][NB][i];
    }
  }
};

// ------------------------------------------------------------------ k_seg_state
// grid.x = nseg * BH (segment fastest), 8 waves.  Segment s of head bh covers
// rows [s*L, min(N, s*L + L)), walked in chunks of 64 keys double-buffered in
// LDS, the next chunk's loads in flight during compute.  Waves sharing a
// feature block split the 32-key units and are summed in a fixed tree at the
// end.  Output: the segment's tile-order state record.
constexpr int SW = 8;          // waves in k_seg_state
constexpr int SNT = SW * 64;
template <typename T, int D, int R>
__global__ __launch_bounds__(SNT) void k_seg_state(const T* __restrict__ k,
                                                   const T* __restrict__ v,
                                                   float* __restrict__ part, int N, int L,
                                                   int nseg) {
  constexpr int NB = D / 16;
  constexpr int ST = D + Lay<T>::PAD;
  constexpr int TK = 64;
  // waves are laid out as (rs, cb): cb = w % NB, rs = w / NB splits the units
  constexpr int RS = SW / NB;
  __shared__ __attribute__((aligned(16))) T s_kv[2][2][TK * ST];  // [buffer][K, V]

  const int seg = blockIdx.x % nseg, bh = blockIdx.x / nseg;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int cbw = w % NB, rs = w / NB;
  const int r0 = seg * L, r1 = min(N, r0 + L);
  const T* kh = k + (size_t)bh * N * D;
  const T* vh = v + (size_t)bh * N * D;
  const int nchunk = (r1 - r0 + TK - 1) / TK;

  // this wave accumulates both maps of feature block cbw: groups ag = l*NB + cbw
  f32x4 acc[R][NB + 1];
#pragma unroll
  for (int l = 0; l < R; ++l)
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) acc[l][eb] = f32x4{0.f, 0.f, 0.f, 0.f};

  RowCopy<T, D, SNT, TK> ck, cv;
  auto ident = [](int i) { return i; };
  ck.load(kh, r0, min(TK, r1 - r0), r1);
  cv.load(vh, r0, min(TK, r1 - r0), r1);
  ck.store(s_kv[0][0], ST, TK, ident);
  cv.store(s_kv[0][1], ST, TK, ident);
  if (nchunk > 1) {
    ck.load(kh, r0 + TK, min(TK, r1 - r0 - TK), r1);
    cv.load(vh, r0 + TK, min(TK, r1 - r0 - TK), r1);
  }
  const int r = lane & 15, g = lane >> 4;
  using Q = typename QuadOf<T>::type;
  for (int c = 0; c < nchunk; ++c) {
    __syncthreads();
    if (c + 1 < nchunk) {
      ck.store(s_kv[(c + 1) & 1][0], ST, TK, ident);
      cv.store(s_kv[(c + 1) & 1][1], ST, TK, ident);
    }
    if (c + 2 < nchunk) {
      const int ks = r0 + (c + 2) * TK;
      ck.load(kh, ks, min(TK, r1 - ks), r1);
      cv.load(vh, ks, min(TK, r1 - ks), r1);
    }
    const T* kx = s_kv[c & 1][0];
    const T* vx = s_kv[c & 1][1];
    const int kvalid_chunk = r1 - (r0 + c * TK);
#pragma unroll
    for (int u = 0; u < TK / 32; ++u) {
      if (((c * (TK / 32) + u) % RS) != rs) continue;
      const int kvalid = kvalid_chunk - 32 * u;
      if (kvalid <= 0) continue;
      Q vb0[NB + 1], vb1[NB + 1];
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) {
        vb0[eb] = ld_tquad(vx, 32 * u, 16 * eb, ST);
        vb1[eb] = ld_tquad(vx, 32 * u + 16, 16 * eb, ST);
      }
      {
        float f[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) f[i] = r == 0 ? 1.f : 0.f;
        vb0[NB] = f32_to_quad<T>(f);
        vb1[NB] = vb0[NB];
      }
      float p[2][2][4];  // [b][map][i]
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float kf[4];
        quad_to_f32(ld_tquad(kx, 32 * u + 16 * b, 16 * cbw, ST), kf);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          phi12(kf[i], p[b][0][i], p[b][1][i]);
          if (16 * b + 4 * g + i >= kvalid) { p[b][0][i] = 0.f; p[b][1][i] = 0.f; }
        }
      }
#pragma unroll
      for (int l = 0; l < R; ++l) {
        const Q a0 = f32_to_quad<T>(p[0][l]), a1 = f32_to_quad<T>(p[1][l]);
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb) acc[l][eb] = mma_step2(a0, a1, vb0[eb], vb1[eb], acc[l][eb]);
      }
    }
  }

  // fixed-order tree over the RS waves sharing a feature block, one map at a
  // time, through the (now free) staging buffers
  f32x4* red = reinterpret_cast<f32x4*>(&s_kv[0][0][0]);
  static_assert(SW / 2 * (NB + 1) * 64 * 16 <= (int)sizeof(s_kv), "reduction buffer");
#pragma unroll
  for (int l = 0; l < R; ++l) {
#pragma unroll
    for (int s = RS / 2; s >= 1; s >>= 1) {
      __syncthreads();
      if (rs >= s && rs < 2 * s)
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb)
          red[(((rs - s) * NB + cbw) * (NB + 1) + eb) * 64 + lane] = acc[l][eb];
      __syncthreads();
      if (rs < s)
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb)
          acc[l][eb] += red[((rs * NB + cbw) * (NB + 1) + eb) * 64 + lane];
    }
  }
  if (rs != 0) return;
  float* out = part + ((size_t)bh * nseg + seg) * (R * D * (D + 1));
#pragma unroll
  for (int l = 0; l < R; ++l) {
    float* sl = out + (size_t)l * D * (D + 1);
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
      *reinterpret_cast<f32x4*>(sl + ((cbw * NB + eb) * 64 + lane) * 4) = acc[l][eb];
    if (r == 0) *reinterpret_cast<f32x4*>(sl + D * D + 16 * cbw + 4 * g) = acc[l][NB];
  }
}

// ------------------------------------------------------------------ k_state_combine
// Each workgroup: 64 record elements x 4 segment ranges.  Non-causal: every
// thread sums its range in order, then the four range sums are added in
// order.  Causal: range totals first, then each range is scanned in order
// from the sum of the totals before it, writing the exclusive prefix in place.
template <bool CAUSAL>
__global__ __launch_bounds__(256) void k_state_combine(float* __restrict__ part,
                                                       float* __restrict__ fin, int nseg,
                                                       int rec) {
  __shared__ float tot[4][64];
  const int el = threadIdx.x & 63, qr = threadIdx.x >> 6;
  const int e = blockIdx.x * 64 + el, bh = blockIdx.y;
  const int per = (nseg + 3) / 4;
  const int s0 = min(nseg, qr * per), s1 = min(nseg, s0 + per);
  float* p = part + (size_t)bh * nseg * rec + e;
  float s = 0.f;
  if (e < rec) {
    int j = s0;
    for (; j + 4 <= s1; j += 4) {
      const float a0 = p[(size_t)j * rec], a1 = p[(size_t)(j + 1) * rec];
      const float a2 = p[(size_t)(j + 2) * rec], a3 = p[(size_t)(j + 3) * rec];
      s += a0; s += a1; s += a2; s += a3;
    }
    for (; j < s1; ++j) s += p[(size_t)j * rec];
  }
  tot[qr][el] = s;
  __syncthreads();
  if (e >= rec) return;
  if constexpr (!CAUSAL) {
    if (qr == 0) fin[(size_t)bh * rec + e] = ((tot[0][el] + tot[1][el]) + tot[2][el]) + tot[3][el];
  } else {
    float run = 0.f;
    for (int q2 = 0; q2 < qr; ++q2) run += tot[q2][el];
    for (int j = s0; j < s1; ++j) {
      const float t = p[(size_t)j * rec];
      p[(size_t)j * rec] = run;
      run += t;
    }
  }
}

// ------------------------------------------------------------------ ring helpers
// LDS ring of U 32-key units; window of tile t of a segment = absolute units
// [ua0 + 2t, ua0 + 2t + U), unit ua lives at ring rows ((ua - ua0) % U) * 32.
template <typename T, int D, int R>
struct RingSmem {
  using Q = typename QuadOf<T>::type;
  static constexpr int ST = Ring<T, D, R>::ST, NB = D / 16;
  T* k;
  T* v;
  Q* sf;
  float* sz;
  __device__ __forceinline__ RingSmem(unsigned char* base, int U) {
    k = reinterpret_cast<T*>(base);
    v = k + U * 32 * ST;
    sf = reinterpret_cast<Q*>(v + U * 32 * ST);
    sz = reinterpret_cast<float*>(sf + R * NB * NB * 64);
  }
};

// Copy absolute units [ua, ua + n) of K and V into the ring (synchronously).
template <typename T, int D, int R>
__device__ __forceinline__ void ring_fill(const RingSmem<T, D, R>& sm, const T* kh, const T* vh,
                                          int ua, int n, int ua0, int U, int N) {
  constexpr int ST = RingSmem<T, D, R>::ST;
  for (int x = 0; x < n; x += 2) {
    const int m = min(2, n - x);
    RowCopy<T, D, NT, 64> ck, cv;
    ck.load(kh, (ua + x) * 32, 32 * m, N);
    cv.load(vh, (ua + x) * 32, 32 * m, N);
    auto row = [&](int i) { return ((ua + x + (i >> 5) - ua0) % U) * 32 + (i & 31); };
    ck.store(sm.k, ST, 32 * m, row);
    cv.store(sm.v, ST, 32 * m, row);
  }
}

// ------------------------------------------------------------------ k_band_ring
// Non-causal.  grid.x = BH * nseg (XCD-aware remap); the workgroup walks the
// 64-row tiles of rows [s*L, min(N, s*L + L)).  Window of a tile starting at
// t0: keys [t0 - 32*ceil(k/32), t0 + 64 + 32*ceil(k/32)) = U = 2 + 2*ceil(k/32) units.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_band_ring(const T* __restrict__ q,
                                                  const T* __restrict__ k,
                                                  const T* __restrict__ v, T* __restrict__ out,
                                                  const float* __restrict__ fin,
                                                  const float* __restrict__ w_near,
                                                  const float* __restrict__ w_far, int H, int N,
                                                  int band_k, int L, int nseg, float scale2) {
  using Q = typename QuadOf<T>::type;
  using SM = RingSmem<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  const int kc = (band_k + 31) >> 5;        // band half-width in units (rounded up)
  const int U = 2 + 2 * kc;
  const SM sm(dyn_smem, U);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const T* qh = q + base;
  const T* kh = k + base;
  const T* vh = v + base;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + TM - 1) / TM;
  const int ua0 = (s0 >> 5) - kc;

  load_state_frags<T, D, R, NT>(fin + (size_t)bh * R * D * (D + 1), sm.sf, sm.sz);
  ring_fill<T, D, R>(sm, kh, vh, ua0, U, ua0, U, N);
  Q qq[NB], qn[NB];
  load_q<T, D>(qh, s0 + 16 * w + r, N, qq);
  RowCopy<T, D, NT, 64> pk, pv;
  if (ntile > 1) {
    pk.load(kh, (ua0 + U) * 32, 64, N);
    pv.load(vh, (ua0 + U) * 32, 64, N);
    load_q<T, D>(qh, s0 + TM + 16 * w + r, N, qn);
  }
  for (int t = 0; t < ntile; ++t) {
    __syncthreads();  // ring holds the window of tile t
    const int t0 = s0 + t * TM, i0 = t0 + 16 * w, row = i0 + r;
    NearState<D> st;
    st.init();
    const int lo = max(0, i0 - band_k), hi = min(N - 1, i0 + 15 + band_k);
    for (int ua = lo >> 5; ua <= hi >> 5; ++ua) {
      const int rr = ((ua - ua0) % U) * 32;
      near_unit<T, D, false>(st, qq, sm.k + rr * ST, sm.v + rr * ST, ST, ua * 32, row, N,
                             band_k, scale2);
    }
    float qf[D / 4];
    q_floats<T, D>(qq, qf);
    f32x4 far[NB];
    far_apply<T, D, R>(sm.sf, sm.sz, qf, far);
    blend_store<T, D>(out + base, row, N, sn, sfw, st, far);
    if (t + 1 < ntile) {
      __syncthreads();  // every wave is done with the window of tile t
      const int ua_new = ua0 + 2 * t + U;  // the two units tile t+1 adds
      auto rowmap = [&](int i) { return ((ua_new + (i >> 5) - ua0) % U) * 32 + (i & 31); };
      pk.store(sm.k, ST, 64, rowmap);
      pv.store(sm.v, ST, 64, rowmap);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) qq[cb] = qn[cb];
      if (t + 2 < ntile) {
        pk.load(kh, (ua_new + 2) * 32, 64, N);
        pv.load(vh, (ua_new + 2) * 32, 64, N);
        load_q<T, D>(qh, t0 + 2 * TM + 16 * w + r, N, qn);
      }
    }
  }
}

// ------------------------------------------------------------------ causal tile body
// Intra-tile far part of one strip: keys [t0, row] of the tile, per map,
// accumulated into fnum / fden.  kt, vt: LDS rows of the tile's first key.
template <typename T, int D, int R>
__device__ __forceinline__ void causal_intra(const T* kt, const T* vt, int ST, int t0, int row,
                                             int w, const typename QuadOf<T>::type (*pq)[D / 16],
                                             f32x4 (*fnum)[D / 16], float* fden) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  for (int u = 0; u <= (w >> 1); ++u) {
    float kf[2][D / 4];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
        quad_to_f32(ld_quad(kt, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST), kf[b] + 4 * cb);
    float pk[2][2][D / 4];  // [b][map][t]
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < D / 4; ++t) phi12(kf[b][t], pk[b][0][t], pk[b][1][t]);
#pragma unroll
    for (int l = 0; l < R; ++l) {
      f32x4 at[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        Q ka[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) ka[cb] = f32_to_quad<T>(pk[b][l] + 4 * cb);
        at[b] = contract<NB>(ka, pq[l], f32x4{0.f, 0.f, 0.f, 0.f});
      }
      float pa[2][4];
      float dp = 0.f;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = t0 + 32 * u + 16 * b + 4 * g + i;
          pa[b][i] = j <= row ? round_as<T>(at[b][i]) : 0.f;
          dp += pa[b][i];
        }
      fden[l] += col_sum(dp);
      const Q p0 = f32_to_quad<T>(pa[0]), p1 = f32_to_quad<T>(pa[1]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const Q va0 = ld_tquad(vt, 32 * u, 16 * nb, ST);
        const Q va1 = ld_tquad(vt, 32 * u + 16, 16 * nb, ST);
        fnum[l][nb] = mma_step2(va0, va1, p0, p1, fnum[l][nb]);
      }
    }
  }
}

template <typename T, int D, int R>
__device__ __forceinline__ void causal_finish(T* __restrict__ oh, int row, int N, float sn,
                                              float sfw, const NearState<D>& st,
                                              const typename QuadOf<T>::type* sf,
                                              const float* sz, const float* qf,
                                              f32x4 (*fnum)[D / 16], float* fden) {
  constexpr int NB = D / 16;
  f32x4 far[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) far[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int l = 0; l < R; ++l) {
    far_prefix<T, D>(sf, sz, qf, l, fnum[l], fden[l]);
    const float inv = 1.f / fden[l];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) far[nb] += fnum[l][nb] * inv;
  }
  blend_store<T, D>(oh, row, N, sn, sfw, st, far);
}

template <typename T, int D, int R>
__device__ __forceinline__ void phi_q_quads(const float* qf,
                                            typename QuadOf<T>::type (*pq)[D / 16]) {
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb) {
    float p1[4], p2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) phi12(qf[4 * cb + i], p1[i], p2[i]);
    pq[0][cb] = f32_to_quad<T>(p1);
    if constexpr (R == 2) pq[1][cb] = f32_to_quad<T>(p2);
  }
}

// ------------------------------------------------------------------ k_causal_ring
// Causal.  grid.x = BH * nseg (XCD-aware remap); the workgroup walks the tiles
// of segment s in order, state (exclusive prefix at the current tile) in
// registers.  Window of a tile at t0: [t0 - 32*ceil(k/32), t0 + 64) = U = 2 +
// ceil(k/32) units; its last two units are the tile's own keys.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_causal_ring(const T* __restrict__ q,
                                                    const T* __restrict__ k,
                                                    const T* __restrict__ v, T* __restrict__ out,
                                                    const float* __restrict__ prefix,
                                                    const float* __restrict__ w_near,
                                                    const float* __restrict__ w_far, int H,
                                                    int N, int band_k, int L, int nseg,
                                                    float scale2) {
  using Q = typename QuadOf<T>::type;
  using SM = RingSmem<T, D, R>;
  using Tiles = StateTiles<T, D, R, NW>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  const int kc = (band_k + 31) >> 5;
  const int U = 2 + kc;
  const SM sm(dyn_smem, U);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const T* qh = q + base;
  const T* kh = k + base;
  const T* vh = v + base;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + TM - 1) / TM;
  const int ua0 = (s0 >> 5) - kc;
  const bool has_ag = Tiles::active(w);

  Tiles tiles;
  if (has_ag) tiles.load(w, prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1));
  ring_fill<T, D, R>(sm, kh, vh, ua0, U, ua0, U, N);
  Q qq[NB], qn[NB];
  load_q<T, D>(qh, s0 + 16 * w + r, N, qq);
  RowCopy<T, D, NT, 64> pk, pv;
  if (ntile > 1) {
    pk.load(kh, (ua0 + U) * 32, 64, N);
    pv.load(vh, (ua0 + U) * 32, 64, N);
    load_q<T, D>(qh, s0 + TM + 16 * w + r, N, qn);
  }
  for (int t = 0; t < ntile; ++t) {
    const int t0 = s0 + t * TM, i0 = t0 + 16 * w, row = i0 + r;
    if (has_ag) tiles.to_frags(w, sm.sf, sm.sz);
    __syncthreads();  // ring window and prefix fragments of tile t are in LDS
    NearState<D> st;
    st.init();
    const int lo = max(0, i0 - band_k), hi = min(N - 1, i0 + 15);
    for (int ua = lo >> 5; ua <= hi >> 5; ++ua) {
      const int rr = ((ua - ua0) % U) * 32;
      near_unit<T, D, true>(st, qq, sm.k + rr * ST, sm.v + rr * ST, ST, ua * 32, row, N,
                            band_k, scale2);
    }
    float qf[D / 4];
    q_floats<T, D>(qq, qf);
    Q pq[R][NB];
    phi_q_quads<T, D, R>(qf, pq);
    f32x4 fnum[R][NB];
    float fden[R];
#pragma unroll
    for (int l = 0; l < R; ++l) {
      fden[l] = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fnum[l][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int rt = (((t0 >> 5) - ua0) % U) * 32;  // ring row of the tile's first key
    // the tile's two units are consecutive ring units unless the ring wraps
    const int rt2 = (((t0 >> 5) + 1 - ua0) % U) * 32;
    if (rt2 == rt + 32) {
      causal_intra<T, D, R>(sm.k + rt * ST, sm.v + rt * ST, ST, t0, row, w, pq, fnum, fden);
    } else {
      // wrapped: handle the two units separately (unit 1 only matters for w >= 2)
      causal_intra<T, D, R>(sm.k + rt * ST, sm.v + rt * ST, ST, t0, row, 0, pq, fnum, fden);
      if (w >= 2)
        causal_intra<T, D, R>(sm.k + rt2 * ST, sm.v + rt2 * ST, ST, t0 + 32, row, 0, pq, fnum,
                              fden);
    }
    causal_finish<T, D, R>(out + base, row, N, sn, sfw, st, sm.sf, sm.sz, qf, fnum, fden);
    if (has_ag && t + 1 < ntile) {
      tiles.add_unit(w, sm.k + rt * ST, sm.v + rt * ST, ST, N - t0);
      tiles.add_unit(w, sm.k + rt2 * ST, sm.v + rt2 * ST, ST, N - t0 - 32);
    }
    if (t + 1 < ntile) {
      __syncthreads();  // every wave is done with the window and fragments of tile t
      const int ua_new = ua0 + 2 * t + U;
      auto rowmap = [&](int i) { return ((ua_new + (i >> 5) - ua0) % U) * 32 + (i & 31); };
      pk.store(sm.k, ST, 64, rowmap);
      pv.store(sm.v, ST, 64, rowmap);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) qq[cb] = qn[cb];
      if (t + 2 < ntile) {
        pk.load(kh, (ua_new + 2) * 32, 64, N);
        pv.load(vh, (ua_new + 2) * 32, 64, N);
        load_q<T, D>(qh, t0 + 2 * TM + 16 * w + r, N, qn);
      }
    }
  }
}

// ------------------------------------------------------------------ rounds variants
// Bands too wide for the ring: every tile stages its window in rounds of up to
// WK keys (row-major K and V, like the ring).
template <typename T, int D, int R> struct RoundSmem {
  using Q = typename QuadOf<T>::type;
  static constexpr int ST = D + Lay<T>::PAD, NB = D / 16;
  T k[WK * ST];
  T v[WK * ST];
  Q sf[R * NB * NB * 64];
  float sz[R * D];
};

template <typename T, int D, int R>
__device__ __forceinline__ void round_stage(RoundSmem<T, D, R>& sm, const T* kh, const T* vh,
                                            int ks, int nk, int kend) {
  constexpr int ST = RoundSmem<T, D, R>::ST;
  auto ident = [](int i) { return i; };
  for (int x = 0; x < nk; x += 64) {
    const int m = min(64, nk - x);
    RowCopy<T, D, NT, 64> ck, cv;
    ck.load(kh, ks + x, m, kend);
    cv.load(vh, ks + x, m, kend);
    ck.store(sm.k + x * ST, ST, m, ident);
    cv.store(sm.v + x * ST, ST, m, ident);
  }
}

// Non-causal, one 64-row tile per workgroup.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_band_rounds(const T* __restrict__ q,
                                                    const T* __restrict__ k,
                                                    const T* __restrict__ v, T* __restrict__ out,
                                                    const float* __restrict__ fin,
                                                    const float* __restrict__ w_near,
                                                    const float* __restrict__ w_far, int H,
                                                    int N, int band_k, int ntile, float scale2) {
  using Q = typename QuadOf<T>::type;
  using SM = RoundSmem<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  __shared__ __attribute__((aligned(16))) SM sm;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / ntile, tile = lin % ntile, h = bh % H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r = lane & 15;
  const int t0 = tile * TM, i0 = t0 + 16 * w, row = i0 + r;
  const size_t base = (size_t)bh * N * D;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  load_state_frags<T, D, R, NT>(fin + (size_t)bh * R * D * (D + 1), sm.sf, sm.sz);
  Q qq[NB];
  load_q<T, D>(q + base, row, N, qq);
  NearState<D> st;
  st.init();
  const int ka = (max(0, t0 - band_k) >> 5) << 5;
  const int kend = min(N, t0 + TM + band_k);
  for (int ks = ka; ks < kend; ks += WK) {
    const int nk = min(WK, ((kend - ks) + 31) & ~31);
    __syncthreads();
    round_stage<T, D, R>(sm, k + base, v + base, ks, nk, kend);
    __syncthreads();
    const int lo = max(max(0, i0 - band_k), ks), hi = min(min(N - 1, i0 + 15 + band_k), ks + nk - 1);
    for (int j = lo & ~31; j <= hi; j += 32)
      near_unit<T, D, false>(st, qq, sm.k + (j - ks) * ST, sm.v + (j - ks) * ST, ST, j, row, N,
                             band_k, scale2);
  }
  float qf[D / 4];
  q_floats<T, D>(qq, qf);
  f32x4 far[NB];
  far_apply<T, D, R>(sm.sf, sm.sz, qf, far);
  blend_store<T, D>(out + base, row, N, sn, sfw, st, far);
}

// Causal, walks the tiles of a segment; per tile the window [t0 - k, t0 + 64)
// is staged in rounds, last keys first, so that round 0 holds the tile itself.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_causal_rounds(const T* __restrict__ q,
                                                      const T* __restrict__ k,
                                                      const T* __restrict__ v,
                                                      T* __restrict__ out,
                                                      const float* __restrict__ prefix,
                                                      const float* __restrict__ w_near,
                                                      const float* __restrict__ w_far, int H,
                                                      int N, int band_k, int L, int nseg,
                                                      float scale2) {
  using Q = typename QuadOf<T>::type;
  using SM = RoundSmem<T, D, R>;
  using Tiles = StateTiles<T, D, R, NW>;
  constexpr int NB = D / 16, ST = SM::ST;
  static_assert(WK >= TM, "round 0 must hold the whole tile");
  __shared__ __attribute__((aligned(16))) SM sm;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const bool has_ag = Tiles::active(w);
  Tiles tiles;
  if (has_ag) tiles.load(w, prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1));
  const int s0 = seg * L, s1 = min(N, s0 + L);
  for (int t0 = s0; t0 < s1; t0 += TM) {
    const int i0 = t0 + 16 * w, row = i0 + r;
    __syncthreads();  // every wave is done with the previous tile's LDS
    if (has_ag) tiles.to_frags(w, sm.sf, sm.sz);
    Q qq[NB];
    load_q<T, D>(q + base, row, N, qq);
    float qf[D / 4];
    q_floats<T, D>(qq, qf);
    Q pq[R][NB];
    phi_q_quads<T, D, R>(qf, pq);
    NearState<D> st;
    st.init();
    f32x4 fnum[R][NB];
    float fden[R];
#pragma unroll
    for (int l = 0; l < R; ++l) {
      fden[l] = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fnum[l][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int ka = (max(0, t0 - band_k) >> 5) << 5;
    const int hi = t0 + TM;
    for (int ke = hi; ke > ka; ke -= WK) {
      const int ks = max(ka, ke - WK), nk = ke - ks;
      __syncthreads();
      round_stage<T, D, R>(sm, k + base, v + base, ks, nk, min(N, ke));
      __syncthreads();
      const int lo = max(max(0, i0 - band_k), ks), hj = min(min(N - 1, i0 + 15), ks + nk - 1);
      for (int j = lo & ~31; j <= hj; j += 32)
        near_unit<T, D, true>(st, qq, sm.k + (j - ks) * ST, sm.v + (j - ks) * ST, ST, j, row, N,
                              band_k, scale2);
      if (ke != hi) continue;
      const int tk = t0 - ks;
      causal_intra<T, D, R>(sm.k + tk * ST, sm.v + tk * ST, ST, t0, row, w, pq, fnum, fden);
      if (has_ag && t0 + TM < s1) {
        tiles.add_unit(w, sm.k + tk * ST, sm.v + tk * ST, ST, N - t0);
        tiles.add_unit(w, sm.k + (tk + 32) * ST, sm.v + (tk + 32) * ST, ST, N - t0 - 32);
      }
    }
    causal_finish<T, D, R>(out + base, row, N, sn, sfw, st, sm.sf, sm.sz, qf, fnum, fden);
  }
}

// ------------------------------------------------------------------ launchers
template <typename T, int D, int R>
static hipError_t launch_all(const LaunchArgs& a, LaunchTimer* timer) {
  const int BH = a.B * a.H;
  const float scale2 = 1.4426950408889634f / sqrtf((float)D);
  const int REC = R * D * (D + 1);
  hipStream_t s = (hipStream_t)a.stream;
  const T* q = (const T*)a.q;
  const T* k = (const T*)a.k;
  const T* v = (const T*)a.v;
  T* o = (T*)a.out;
  float* part = a.ws;
  float* fin = a.ws + (size_t)BH * a.nseg * REC;
  const int kc = (a.band_k + 31) / 32;
  const int U = a.causal ? 2 + kc : 2 + 2 * kc;
  const bool ring = U <= Ring<T, D, R>::U;
  const size_t ring_lds = Ring<T, D, R>::bytes(U);
  static const bool lds_attr = [] {
    const int mx = (int)Ring<T, D, R>::bytes(Ring<T, D, R>::U);
    hipFuncSetAttribute((const void*)k_band_ring<T, D, R>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, mx);
    hipFuncSetAttribute((const void*)k_causal_ring<T, D, R>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, mx);
    return true;
  }();
  (void)lds_attr;

  timer->begin(FMM_KERNEL_SEG_STATE, s);
  hipLaunchKernelGGL((k_seg_state<T, D, R>), dim3(a.nseg * BH), dim3(SNT), 0, s, k, v, part,
                     a.N, a.L, a.nseg);
  timer->end(FMM_KERNEL_SEG_STATE, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;

  timer->begin(FMM_KERNEL_STATE_COMBINE, s);
  const dim3 cgrid((REC + 63) / 64, BH);
  if (a.causal)
    hipLaunchKernelGGL((k_state_combine<true>), cgrid, dim3(256), 0, s, part, fin, a.nseg, REC);
  else
    hipLaunchKernelGGL((k_state_combine<false>), cgrid, dim3(256), 0, s, part, fin, a.nseg, REC);
  timer->end(FMM_KERNEL_STATE_COMBINE, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;

  if (a.causal) {
    timer->begin(FMM_KERNEL_CAUSAL_APPLY, s);
    if (ring)
      hipLaunchKernelGGL((k_causal_ring<T, D, R>), dim3(BH * a.nseg), dim3(NT), ring_lds, s, q, k, v,
                         o, part, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg, scale2);
    else
      hipLaunchKernelGGL((k_causal_rounds<T, D, R>), dim3(BH * a.nseg), dim3(NT), 0, s, q, k,
                         v, o, part, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg,
                         scale2);
    timer->end(FMM_KERNEL_CAUSAL_APPLY, s);
  } else {
    timer->begin(FMM_KERNEL_BAND_APPLY, s);
    if (ring) {
      hipLaunchKernelGGL((k_band_ring<T, D, R>), dim3(BH * a.nseg_apply), dim3(NT), ring_lds, s, q, k,
                         v, o, fin, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L_apply,
                         a.nseg_apply, scale2);
    } else {
      const int ntile = (a.N + TM - 1) / TM;
      hipLaunchKernelGGL((k_band_rounds<T, D, R>), dim3(BH * ntile), dim3(NT), 0, s, q, k, v,
                         o, fin, a.w_near, a.w_far, a.H, a.N, a.band_k, ntile, scale2);
    }
    timer->end(FMM_KERNEL_BAND_APPLY, s);
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t dispatch_d(const LaunchArgs& a, LaunchTimer* t) {
  switch (a.d * 4 + a.rank) {
    case 16 * 4 + 1: return launch_all<T, 16, 1>(a, t);
    case 16 * 4 + 2: return launch_all<T, 16, 2>(a, t);
    case 32 * 4 + 1: return launch_all<T, 32, 1>(a, t);
    case 32 * 4 + 2: return launch_all<T, 32, 2>(a, t);
    case 64 * 4 + 1: return launch_all<T, 64, 1>(a, t);
    case 64 * 4 + 2: return launch_all<T, 64, 2>(a, t);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_forward(const LaunchArgs& a, LaunchTimer* t) {
  return a.dtype == FMM_DTYPE_BF16 ? dispatch_d<bf16_t>(a, t) : dispatch_d<float>(a, t);
}

int tile_rows() { return TM; }

}  // namespace fmm
