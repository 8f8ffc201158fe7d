// HIP kernels of the FMMformer attention forward operator for gfx950.
//
//   k_seg_state      per-segment far-field totals  T_l = phi_l(K)^T [V | 1]
//                    (Eq. (5), Eq. (7): the regrouped products phi_l(K)^T V and
//                    the normaliser phi_l(K)^T 1), MFMA over the keys
//   k_state_combine  sum over segments (non-causal state S_l, z_l) or
//                    exclusive scan over segments (causal prefix, Sec. 3.2.1)
//   k_band_apply     non-causal: banded online softmax (Eq. (3)) over a key
//                    window staged in LDS, far apply phi_l(Q) S_l / phi_l(Q) z_l
//                    (Eq. (8)-(9)), sigmoid blend (Eq. (11)), store
//   k_causal_apply   causal: walks the tiles of one segment in order, carrying
//                    the running state in registers; per tile the causal band
//                    [i-k, i], the intra-tile lower-triangular far part, the
//                    prefix far part, the blend and the state update
//
// Every workgroup has NW wavefronts; wave w owns query rows [16w, 16w+16) of a
// TM = 16*NW row tile.  All sums are accumulated in fp32 in a fixed order, so
// results are bit-reproducible run to run.
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {

constexpr int NW = 4;            // wavefronts per workgroup
constexpr int NT = NW * 64;      // threads per workgroup
constexpr int TM = 16 * NW;      // query rows per tile
constexpr int WK = 192;          // keys staged in LDS per round (multiple of 32)

template <typename T> struct Lay {
  static constexpr int ES = (int)sizeof(T);
  static constexpr int EPC = 16 / ES;          // elements per 16-byte chunk
  static constexpr int KPAD = ES == 2 ? 8 : 4; // row pad (keeps rows 16-B aligned)
  static constexpr int VPAD = 4;               // transposed rows stay 8/16-B aligned
};

// ------------------------------------------------------------------ staging
// Stage keys [ks, ks + nk) of one head: K row-major into sk[nk][D + KPAD] and
// V transposed into svt[D][WK + VPAD].  Keys at or beyond `kend` are zero.
template <typename T, int D>
__device__ __forceinline__ void stage_kv(const T* __restrict__ kh, const T* __restrict__ vh,
                                         int ks, int nk, int kend, T* sk, T* svt) {
  using L = Lay<T>;
  constexpr int CPR = D / L::EPC;               // 16-B chunks per row
  constexpr int KST = D + L::KPAD, VST = WK + L::VPAD;
  constexpr int KIT = (WK * CPR + NT - 1) / NT;         // K chunks per thread
  constexpr int VIT = (WK / 4 * CPR + NT - 1) / NT;     // V (4-key x chunk) tasks per thread
  const int tid = threadIdx.x;
  uint4 kreg[KIT];
  uint4 vreg[VIT][4];
  const int kt = nk * CPR, vt = nk / 4 * CPR;
#pragma unroll
  for (int it = 0; it < KIT; ++it) {
    const int t = tid + it * NT;
    kreg[it] = make_uint4(0, 0, 0, 0);
    if (t < kt) {
      const int key = ks + t / CPR, c = t % CPR;
      if (key < kend)
        kreg[it] = *reinterpret_cast<const uint4*>(kh + (size_t)key * D + c * L::EPC);
    }
  }
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int t = tid + it * NT;
#pragma unroll
    for (int e = 0; e < 4; ++e) vreg[it][e] = make_uint4(0, 0, 0, 0);
    if (t < vt) {
      const int quad = t / CPR, c = t % CPR;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = ks + 4 * quad + e;
        if (key < kend)
          vreg[it][e] = *reinterpret_cast<const uint4*>(vh + (size_t)key * D + c * L::EPC);
      }
    }
  }
#pragma unroll
  for (int it = 0; it < KIT; ++it) {
    const int t = tid + it * NT;
    if (t < kt) {
      const int key = t / CPR, c = t % CPR;
      *reinterpret_cast<uint4*>(sk + key * KST + c * L::EPC) = kreg[it];
    }
  }
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int t = tid + it * NT;
    if (t < vt) {
      const int quad = t / CPR, c = t % CPR;
      if constexpr (sizeof(T) == 2) {
        const uint16_t* e0 = reinterpret_cast<const uint16_t*>(&vreg[it][0]);
        const uint16_t* e1 = reinterpret_cast<const uint16_t*>(&vreg[it][1]);
        const uint16_t* e2 = reinterpret_cast<const uint16_t*>(&vreg[it][2]);
        const uint16_t* e3 = reinterpret_cast<const uint16_t*>(&vreg[it][3]);
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          uint2 w = make_uint2((uint32_t)e0[x] | ((uint32_t)e1[x] << 16),
                               (uint32_t)e2[x] | ((uint32_t)e3[x] << 16));
          *reinterpret_cast<uint2*>(svt + (c * 8 + x) * VST + 4 * quad) = w;
        }
      } else {
        const float* e0 = reinterpret_cast<const float*>(&vreg[it][0]);
        const float* e1 = reinterpret_cast<const float*>(&vreg[it][1]);
        const float* e2 = reinterpret_cast<const float*>(&vreg[it][2]);
        const float* e3 = reinterpret_cast<const float*>(&vreg[it][3]);
#pragma unroll
        for (int x = 0; x < 4; ++x)
          *reinterpret_cast<float4*>(svt + (c * 4 + x) * VST + 4 * quad) =
              make_float4(e0[x], e1[x], e2[x], e3[x]);
      }
    }
  }
}

// ------------------------------------------------------------------ near field
// Online-softmax state of one wavefront's 16-row strip.  Lane (r, g) holds row
// r; o[nb] holds output columns 16nb + 4g + {0..3}; lsum is this lane's share
// of the row's normaliser (summed over the four lane groups at the end).
template <int D> struct NearState {
  f32x4 o[D / 16];
  float m, lsum;
};

// Process the staged keys [ks, ks + nk) for the strip starting at row i0.
// Scores use exp2 with the scale tau*log2(e) folded in.
template <typename T, int D, bool CAUSAL>
__device__ __forceinline__ void near_round(NearState<D>& st,
                                           const typename QuadOf<T>::type* qq,
                                           const T* sk, const T* svt, int ks, int nk,
                                           int i0, int N, int band_k, float scale2) {
  using Q = typename QuadOf<T>::type;
  using L = Lay<T>;
  constexpr int NB = D / 16;
  constexpr int KST = D + L::KPAD, VST = WK + L::VPAD;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int slo = max(0, i0 - band_k);
  const int shi = CAUSAL ? min(N - 1, i0 + 15) : min(N - 1, i0 + 15 + band_k);
  const int lo = max(slo, ks), hi = min(shi, ks + nk - 1);
  if (lo > hi) return;
  const int row = i0 + r;
  for (int u = (lo - ks) >> 5; u <= (hi - ks) >> 5; ++u) {
    f32x4 sc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const T* krow = sk + (32 * u + 16 * b + r) * KST + 4 * g;
      Q ka[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) ka[cb] = *reinterpret_cast<const Q*>(krow + 16 * cb);
      sc[b] = contract<NB>(ka, qq, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    float x[2][4];
    float mloc = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = ks + 32 * u + 16 * b + 4 * g + i;
        const bool ok = j < N && j >= row - band_k && (CAUSAL ? j <= row : j <= row + band_k);
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
      const T* vrow = svt + (16 * nb + r) * VST + 32 * u + 4 * g;
      const Q va0 = *reinterpret_cast<const Q*>(vrow);
      const Q va1 = *reinterpret_cast<const Q*>(vrow + 16);
      f32x4 o = st.o[nb] * alpha;
      st.o[nb] = mma_step2(va0, va1, pq0, pq1, o);
    }
  }
}

// ------------------------------------------------------------------ far apply
// State fragments in LDS: sf[l][nb][cb][lane] is the quad
// S_l[16cb + 4g + {0..3}][16nb + r] (lane = 16g + r), i.e. the A operand of
// F^T = S_l^T phi_l(Q)^T; sz[l][c] = z_l[c].
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

// Fill the state fragments from a plain state record (S_l row-major d x d,
// then z_l), for every map.
template <typename T, int D, int R>
__device__ __forceinline__ void load_state_frags(const float* __restrict__ rec,
                                                 typename QuadOf<T>::type* sf, float* sz) {
  constexpr int NB = D / 16;
  constexpr int E = R * NB * NB * 64;
  for (int t = threadIdx.x; t < E; t += NT) {
    const int lane = t & 63, blk = t >> 6;
    const int cb = blk % NB, nb = (blk / NB) % NB, l = blk / (NB * NB);
    const int r = lane & 15, g = lane >> 4;
    const float* s = rec + (size_t)l * D * (D + 1) + (16 * cb + 4 * g) * D + 16 * nb + r;
    float f[4] = {s[0], s[D], s[2 * D], s[3 * D]};
    sf[t] = f32_to_quad<T>(f);
  }
  for (int t = threadIdx.x; t < R * D; t += NT) {
    const int l = t / D, c = t % D;
    sz[t] = rec[(size_t)l * D * (D + 1) + D * D + c];
  }
}

// Load the strip's queries: lane (r, g) gets q[row][16cb + 4g + {0..3}].
template <typename T, int D>
__device__ __forceinline__ void load_q(const T* __restrict__ qh, int row, int N,
                                       typename QuadOf<T>::type* qq, float* qf) {
  using Q = typename QuadOf<T>::type;
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int cb = 0; cb < D / 16; ++cb) {
    Q v;
    if (row < N) v = *reinterpret_cast<const Q*>(qh + (size_t)row * D + 16 * cb + 4 * g);
    else v = Q{};
    qq[cb] = v;
    quad_to_f32(v, qf + 4 * cb);
  }
}

template <typename T, int D>
__device__ __forceinline__ void store_out(T* __restrict__ oh, int row, int N, const float* vals,
                                          int nb) {
  using Q = typename QuadOf<T>::type;
  const int g = (threadIdx.x & 63) >> 4;
  if (row < N)
    *reinterpret_cast<Q*>(oh + (size_t)row * D + 16 * nb + 4 * g) = f32_to_quad<T>(vals);
}

// ------------------------------------------------------------------ k_seg_state
// grid.x = nseg * BH (segment fastest).  Segment s of head bh covers rows
// [s*L, min(N, s*L + L)).  Output: part[(bh*nseg + s)*REC ...] with, for each
// map l, S_l (d x d, row-major, row = feature c, column = value e) followed by
// z_l (d).
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_seg_state(const T* __restrict__ k,
                                                  const T* __restrict__ v,
                                                  float* __restrict__ part, int N, int L,
                                                  int nseg) {
  using Q = typename QuadOf<T>::type;
  using Ly = Lay<T>;
  constexpr int NB = D / 16;
  constexpr int AG = R * NB;                     // (map, feature block) groups
  constexpr int AGPW = AG >= NW ? AG / NW : 1;   // groups per wave
  constexpr int RS = AG >= NW ? 1 : NW / AG;     // waves sharing one group split the keys
  static_assert(AG < NW ? NW % AG == 0 : AG % NW == 0, "group split");
  constexpr int TK = sizeof(T) == 2 ? 128 : 64;  // keys per staging round
  constexpr int PST = TK + Ly::VPAD;
  constexpr int CPR = D / Ly::EPC;
  constexpr int REC = R * D * (D + 1);
  __shared__ __attribute__((aligned(16))) T s_pk[R][D][PST];  // phi_l(K)^T
  __shared__ __attribute__((aligned(16))) T s_vt[D][PST];     // V^T
  __shared__ f32x4 s_red[RS > 1 ? NW * (NB + 1) * 64 : 1];

  const int seg = blockIdx.x % nseg, bh = blockIdx.x / nseg;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r = lane & 15, g = lane >> 4;
  const int r0 = seg * L, r1 = min(N, r0 + L);
  const T* kh = k + (size_t)bh * N * D;
  const T* vh = v + (size_t)bh * N * D;

  f32x4 acc[AGPW][NB + 1];
#pragma unroll
  for (int a = 0; a < AGPW; ++a)
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) acc[a][eb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ones column for z: B(key, e) = (e == 0)
  Q ones;
  {
    float f[4];
    for (int i = 0; i < 4; ++i) f[i] = r == 0 ? 1.f : 0.f;
    ones = f32_to_quad<T>(f);
  }
  const int rgrp = RS > 1 ? w / AG : 0;

  constexpr int TASKS = TK / 4 * CPR;
  constexpr int IT = (TASKS + NT - 1) / NT;
  int unit_base = 0;
  for (int ks = r0; ks < r1; ks += TK, unit_base += TK / 32) {
    // stage phi_l(K)^T and V^T for keys [ks, ks + TK)
    uint4 kr[IT][4], vr[IT][4];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NT;
#pragma unroll
      for (int e = 0; e < 4; ++e) { kr[it][e] = make_uint4(0, 0, 0, 0); vr[it][e] = kr[it][e]; }
      if (t < TASKS) {
        const int quad = t / CPR, c = t % CPR;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = ks + 4 * quad + e;
          if (key < r1) {
            kr[it][e] = *reinterpret_cast<const uint4*>(kh + (size_t)key * D + c * Ly::EPC);
            vr[it][e] = *reinterpret_cast<const uint4*>(vh + (size_t)key * D + c * Ly::EPC);
          }
        }
      }
    }
    __syncthreads();  // previous round's LDS reads are done
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int t = threadIdx.x + it * NT;
      if (t < TASKS) {
        const int quad = t / CPR, c = t % CPR;
#pragma unroll
        for (int x = 0; x < Ly::EPC; ++x) {
          float kv[4], vv[4], p1[4], p2[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (sizeof(T) == 2) {
              kv[e] = bf16_to_f32(reinterpret_cast<const uint16_t*>(&kr[it][e])[x]);
              vv[e] = bf16_to_f32(reinterpret_cast<const uint16_t*>(&vr[it][e])[x]);
            } else {
              kv[e] = reinterpret_cast<const float*>(&kr[it][e])[x];
              vv[e] = reinterpret_cast<const float*>(&vr[it][e])[x];
            }
            const bool ok = ks + 4 * quad + e < r1;
            phi12(kv[e], p1[e], p2[e]);
            if (!ok) { p1[e] = 0.f; p2[e] = 0.f; }
          }
          const int col = c * Ly::EPC + x;
          *reinterpret_cast<Q*>(&s_vt[col][4 * quad]) = f32_to_quad<T>(vv);
          *reinterpret_cast<Q*>(&s_pk[0][col][4 * quad]) = f32_to_quad<T>(p1);
          if constexpr (R == 2) *reinterpret_cast<Q*>(&s_pk[R - 1][col][4 * quad]) = f32_to_quad<T>(p2);
        }
      }
    }
    __syncthreads();
    const int nunits = (min(TK, r1 - ks) + 31) >> 5;
    for (int u = 0; u < nunits; ++u) {
      if (RS > 1 && ((unit_base + u) % RS) != rgrp) continue;
      Q vb0[NB + 1], vb1[NB + 1];
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) {
        vb0[eb] = *reinterpret_cast<const Q*>(&s_vt[16 * eb + r][32 * u + 4 * g]);
        vb1[eb] = *reinterpret_cast<const Q*>(&s_vt[16 * eb + r][32 * u + 16 + 4 * g]);
      }
      vb0[NB] = ones;
      vb1[NB] = ones;
#pragma unroll
      for (int a = 0; a < AGPW; ++a) {
        const int ag = AG >= NW ? w + NW * a : w % AG;
        const int l = ag / NB, cb = ag % NB;
        const Q a0 = *reinterpret_cast<const Q*>(&s_pk[l][16 * cb + r][32 * u + 4 * g]);
        const Q a1 = *reinterpret_cast<const Q*>(&s_pk[l][16 * cb + r][32 * u + 16 + 4 * g]);
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb) acc[a][eb] = mma_step2(a0, a1, vb0[eb], vb1[eb], acc[a][eb]);
      }
    }
  }

  if constexpr (RS > 1) {
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) s_red[(w * (NB + 1) + eb) * 64 + lane] = acc[0][eb];
    __syncthreads();
    if (rgrp != 0) return;
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) {
      f32x4 s = s_red[(w * (NB + 1) + eb) * 64 + lane];
      for (int j = 1; j < RS; ++j) s += s_red[((w + j * AG) * (NB + 1) + eb) * 64 + lane];
      acc[0][eb] = s;
    }
  }
  float* out = part + ((size_t)bh * nseg + seg) * REC;
#pragma unroll
  for (int a = 0; a < AGPW; ++a) {
    const int ag = AG >= NW ? w + NW * a : w % AG;
    const int l = ag / NB, cb = ag % NB;
    float* sl = out + (size_t)l * D * (D + 1);
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
#pragma unroll
      for (int i = 0; i < 4; ++i) sl[(16 * cb + 4 * g + i) * D + 16 * eb + r] = acc[a][eb][i];
    if (r == 0)
#pragma unroll
      for (int i = 0; i < 4; ++i) sl[D * D + 16 * cb + 4 * g + i] = acc[a][NB][i];
  }
}

// ------------------------------------------------------------------ k_state_combine
// grid (ceil(REC/256), BH).  Non-causal: fin[bh] = sum_s part[bh][s] in order
// s = 0, 1, ...  Causal: part[bh][s] <- sum_{s' < s} part[bh][s'] (in place).
template <bool CAUSAL>
__global__ __launch_bounds__(256) void k_state_combine(float* __restrict__ part,
                                                       float* __restrict__ fin, int nseg,
                                                       int rec) {
  const int e = blockIdx.x * 256 + threadIdx.x, bh = blockIdx.y;
  if (e >= rec) return;
  float* p = part + (size_t)bh * nseg * rec + e;
  float s = 0.f;
  if constexpr (!CAUSAL) {
    for (int j = 0; j < nseg; ++j) s += p[(size_t)j * rec];
    fin[(size_t)bh * rec + e] = s;
  } else {
    for (int j = 0; j < nseg; ++j) {
      const float t = p[(size_t)j * rec];
      p[(size_t)j * rec] = s;
      s += t;
    }
  }
}

// ------------------------------------------------------------------ shared LDS
template <typename T, int D, int R> struct ApplySmem {
  using Q = typename QuadOf<T>::type;
  static constexpr int KST = D + Lay<T>::KPAD, VST = WK + Lay<T>::VPAD, NB = D / 16;
  T sk[WK * KST];
  T svt[D * VST];
  Q sf[R * NB * NB * 64];
  float sz[R * D];
};

// ------------------------------------------------------------------ k_band_apply
// Non-causal.  grid.x = BH * ntile (XCD-aware remap), one TM-row tile each.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_band_apply(const T* __restrict__ q,
                                                   const T* __restrict__ k,
                                                   const T* __restrict__ v, T* __restrict__ out,
                                                   const float* __restrict__ fin,
                                                   const float* __restrict__ w_near,
                                                   const float* __restrict__ w_far, int H,
                                                   int N, int band_k, int ntile,
                                                   float scale2) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  __shared__ __attribute__((aligned(16))) ApplySmem<T, D, R> sm;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / ntile, tile = lin % ntile, h = bh % H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r = lane & 15;
  const int t0 = tile * TM, i0 = t0 + 16 * w, row = i0 + r;
  const size_t base = (size_t)bh * N * D;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);

  load_state_frags<T, D, R>(fin + (size_t)bh * R * D * (D + 1), sm.sf, sm.sz);
  Q qq[NB];
  float qf[D / 4];
  load_q<T, D>(q + base, row, N, qq, qf);

  NearState<D> st;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) st.o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.lsum = 0.f;
  const int ka = (max(0, t0 - band_k) >> 5) << 5;
  const int kend = min(N, t0 + TM + band_k);
  for (int ks = ka; ks < kend; ks += WK) {
    const int nk = min(WK, ((kend - ks) + 31) & ~31);
    __syncthreads();
    stage_kv<T, D>(k + base, v + base, ks, nk, kend, sm.sk, sm.svt);
    __syncthreads();
    near_round<T, D, false>(st, qq, sm.sk, sm.svt, ks, nk, i0, N, band_k, scale2);
  }
  const float lrow = col_sum(st.lsum);
  f32x4 far[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) far[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int l = 0; l < R; ++l) {
    f32x4 num[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) num[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    far_prefix<T, D>(sm.sf, sm.sz, qf, l, num, den);
    const float inv = 1.f / den;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) far[nb] += num[nb] * inv;
  }
  const float inv_l = 1.f / lrow;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a = sn > 0.f ? sn * (st.o[nb][i] * inv_l) : 0.f;
      const float b = sfw > 0.f ? sfw * far[nb][i] : 0.f;
      o[i] = a + b;
    }
    store_out<T, D>(out + base, row, N, o, nb);
  }
}

// ------------------------------------------------------------------ k_causal_apply
// Causal.  grid.x = BH * nseg (XCD-aware remap); the workgroup walks the
// TM-row tiles of segment s in order.  Waves own state tiles exactly as in
// k_seg_state (group ag = (map, feature block), all value blocks + z), kept
// in registers; at the start of each tile they are written to LDS as the
// exclusive prefix state for that tile.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_causal_apply(const T* __restrict__ q,
                                                     const T* __restrict__ k,
                                                     const T* __restrict__ v,
                                                     T* __restrict__ out,
                                                     const float* __restrict__ prefix,
                                                     const float* __restrict__ w_near,
                                                     const float* __restrict__ w_far, int H,
                                                     int N, int band_k, int L, int nseg,
                                                     float scale2) {
  using Q = typename QuadOf<T>::type;
  using Ly = Lay<T>;
  constexpr int NB = D / 16;
  constexpr int AG = R * NB;
  constexpr int AGPW = AG >= NW ? AG / NW : 1;
  constexpr int KST = D + Ly::KPAD, VST = WK + Ly::VPAD;
  static_assert(WK >= TM, "round 0 must hold the whole tile");
  __shared__ __attribute__((aligned(16))) ApplySmem<T, D, R> sm;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r = lane & 15, g = lane >> 4;
  const size_t base = (size_t)bh * N * D;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const bool has_ag = w < AG;   // waves beyond the group count do no state work

  // running state (exclusive prefix at the current tile), wave-owned tiles
  f32x4 acc[AGPW][NB + 1];
  {
    const float* rec = prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1);
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = w + NW * a;
      const int l = ag / NB, cb = ag % NB;
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float val = 0.f;
          if (has_ag) {
            const float* sl = rec + (size_t)l * D * (D + 1);
            if (eb < NB) val = sl[(16 * cb + 4 * g + i) * D + 16 * eb + r];
            else if (r == 0) val = sl[D * D + 16 * cb + 4 * g + i];
          }
          acc[a][eb][i] = val;
        }
    }
  }
  Q ones;
  {
    float f[4];
    for (int i = 0; i < 4; ++i) f[i] = r == 0 ? 1.f : 0.f;
    ones = f32_to_quad<T>(f);
  }

  const int s0 = seg * L, s1 = min(N, s0 + L);
  for (int t0 = s0; t0 < s1; t0 += TM) {
    const int i0 = t0 + 16 * w, row = i0 + r;
    __syncthreads();  // every wave is done with the previous tile's LDS
    if (has_ag) {
#pragma unroll
      for (int a = 0; a < AGPW; ++a) {
        const int ag = w + NW * a;
        const int l = ag / NB, cb = ag % NB;
#pragma unroll
        for (int eb = 0; eb < NB; ++eb) {
          float f[4] = {acc[a][eb][0], acc[a][eb][1], acc[a][eb][2], acc[a][eb][3]};
          sm.sf[((l * NB + eb) * NB + cb) * 64 + lane] = f32_to_quad<T>(f);
        }
        if (r == 0)
#pragma unroll
          for (int i = 0; i < 4; ++i) sm.sz[l * D + 16 * cb + 4 * g + i] = acc[a][NB][i];
      }
    }
    Q qq[NB];
    float qf[D / 4];
    load_q<T, D>(q + base, row, N, qq, qf);

    NearState<D> st;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) st.o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    st.m = -INFINITY;
    st.lsum = 0.f;
    f32x4 fnum[R][NB];
    float fden[R];
#pragma unroll
    for (int l = 0; l < R; ++l) {
      fden[l] = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fnum[l][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // key rounds, last keys first: round 0 = [max(ka, hi - WK), hi) holds the tile
    const int ka = (max(0, t0 - band_k) >> 5) << 5;
    const int hi = t0 + TM;
    for (int ke = hi; ke > ka; ke -= WK) {
      const int ks = max(ka, ke - WK), nk = ke - ks;
      __syncthreads();
      stage_kv<T, D>(k + base, v + base, ks, nk, min(N, ke), sm.sk, sm.svt);
      __syncthreads();
      near_round<T, D, true>(st, qq, sm.sk, sm.svt, ks, nk, i0, N, band_k, scale2);
      if (ke != hi) continue;
      // ---- intra-tile far part: keys [t0, row], per map
      const int tk = t0 - ks;  // tile's first key inside the staged round
      Q pq[R][NB];             // phi_l(q) quads of this lane's row
#pragma unroll
      for (int l = 0; l < R; ++l)
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          float fq[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) fq[i] = phi_l(qf[4 * cb + i], l);
          pq[l][cb] = f32_to_quad<T>(fq);
        }
      for (int u = 0; u <= (w >> 1); ++u) {
        // phi_l(K) rows for key blocks 2u, 2u+1 of the tile (A operand, keys as rows)
        float kf[2][D / 4];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const T* krow = sm.sk + (tk + 32 * u + 16 * b + r) * KST + 4 * g;
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            const Q x = *reinterpret_cast<const Q*>(krow + 16 * cb);
            quad_to_f32(x, kf[b] + 4 * cb);
          }
        }
#pragma unroll
        for (int l = 0; l < R; ++l) {
          f32x4 at[2];
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            Q ka_[NB];
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) {
              float fk[4];
#pragma unroll
              for (int i = 0; i < 4; ++i) fk[i] = phi_l(kf[b][4 * cb + i], l);
              ka_[cb] = f32_to_quad<T>(fk);
            }
            at[b] = contract<NB>(ka_, pq[l], f32x4{0.f, 0.f, 0.f, 0.f});
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
            const T* vrow = sm.svt + (16 * nb + r) * VST + tk + 32 * u + 4 * g;
            const Q va0 = *reinterpret_cast<const Q*>(vrow);
            const Q va1 = *reinterpret_cast<const Q*>(vrow + 16);
            fnum[l][nb] = mma_step2(va0, va1, p0, p1, fnum[l][nb]);
          }
        }
      }
      // ---- state update with the tile's keys (not needed after the last tile)
      if (has_ag && t0 + TM < s1) {
#pragma unroll
        for (int u = 0; u < TM / 32; ++u) {
          Q vb0[NB + 1], vb1[NB + 1];
#pragma unroll
          for (int eb = 0; eb < NB; ++eb) {
            const T* vrow = sm.svt + (16 * eb + r) * VST + tk + 32 * u + 4 * g;
            vb0[eb] = *reinterpret_cast<const Q*>(vrow);
            vb1[eb] = *reinterpret_cast<const Q*>(vrow + 16);
          }
          vb0[NB] = ones;
          vb1[NB] = ones;
#pragma unroll
          for (int a = 0; a < AGPW; ++a) {
            const int ag = w + NW * a;
            const int l = ag / NB, cb = ag % NB;
            // A operand phi_l(K)^T: lane (feature 16cb + r, g) holds keys 4g..4g+3
            float fa[2][4];
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int key = tk + 32 * u + 16 * b + 4 * g + i;
                const T raw = sm.sk[key * KST + 16 * cb + r];
                float x;
                if constexpr (sizeof(T) == 2) x = bf16_to_f32(raw);
                else x = raw;
                fa[b][i] = (t0 + 32 * u + 16 * b + 4 * g + i) < N ? phi_l(x, l) : 0.f;
              }
            const Q a0 = f32_to_quad<T>(fa[0]), a1 = f32_to_quad<T>(fa[1]);
#pragma unroll
            for (int eb = 0; eb <= NB; ++eb)
              acc[a][eb] = mma_step2(a0, a1, vb0[eb], vb1[eb], acc[a][eb]);
          }
        }
      }
    }
    // ---- prefix far part, blend, store
    const float lrow = col_sum(st.lsum);
    f32x4 far[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) far[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int l = 0; l < R; ++l) {
      far_prefix<T, D>(sm.sf, sm.sz, qf, l, fnum[l], fden[l]);
      const float inv = 1.f / fden[l];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) far[nb] += fnum[l][nb] * inv;
    }
    const float inv_l = 1.f / lrow;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a = sn > 0.f ? sn * (st.o[nb][i] * inv_l) : 0.f;
        const float b = sfw > 0.f ? sfw * far[nb][i] : 0.f;
        o[i] = a + b;
      }
      store_out<T, D>(out + base, row, N, o, nb);
    }
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

  timer->begin(FMM_KERNEL_SEG_STATE, s);
  hipLaunchKernelGGL((k_seg_state<T, D, R>), dim3(a.nseg * BH), dim3(NT), 0, s, k, v, part,
                     a.N, a.L, a.nseg);
  timer->end(FMM_KERNEL_SEG_STATE, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;

  timer->begin(FMM_KERNEL_STATE_COMBINE, s);
  if (a.causal)
    hipLaunchKernelGGL((k_state_combine<true>), dim3((REC + 255) / 256, BH), dim3(256), 0, s,
                       part, fin, a.nseg, REC);
  else
    hipLaunchKernelGGL((k_state_combine<false>), dim3((REC + 255) / 256, BH), dim3(256), 0, s,
                       part, fin, a.nseg, REC);
  timer->end(FMM_KERNEL_STATE_COMBINE, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;

  if (a.causal) {
    timer->begin(FMM_KERNEL_CAUSAL_APPLY, s);
    hipLaunchKernelGGL((k_causal_apply<T, D, R>), dim3(BH * a.nseg), dim3(NT), 0, s, q, k, v,
                       o, part, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg, scale2);
    timer->end(FMM_KERNEL_CAUSAL_APPLY, s);
  } else {
    const int ntile = (a.N + TM - 1) / TM;
    timer->begin(FMM_KERNEL_BAND_APPLY, s);
    hipLaunchKernelGGL((k_band_apply<T, D, R>), dim3(BH * ntile), dim3(NT), 0, s, q, k, v, o,
                       fin, a.w_near, a.w_far, a.H, a.N, a.band_k, ntile, scale2);
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
