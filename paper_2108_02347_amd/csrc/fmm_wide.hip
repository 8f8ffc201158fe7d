// General apply kernel of the FMMformer attention forward: every head width
// (16, 32, 64, 128), one to three feature maps (phi_3 = tanh, Sec. 3.2.1) and
// both far-field normalisations (each map on its own as Eq. (9) writes it, or
// the maps' numerators summed over their summed denominators), both forms.
// The tuned kernels of fmm_kernels.hip, fmm_pair.hip and fmm_causal.hip serve
// widths up to 64 with one or two maps normalised per map; this kernel serves
// the rest.
//
// Differences from the tuned kernels, chosen so that any width fits:
//   * the far state is read as the record itself (fp32, tile order) rather
//     than as operand fragments: for widths up to 64 the records of up to
//     three maps are copied into LDS once per workgroup; at d = 128 they stay
//     in the workspace (global memory, read through the caches), since the
//     fp32 records alone would fill the CU's LDS;
//   * the causal running state is that record, advanced after each tile (one
//     map and one 16-feature block at a time, 36 accumulator registers),
//     instead of in registers;
//   * the maps are processed one after another, so only one map's numerator
//     tiles are live at a time.
// Per 64-row tile (4 waves, one 16-row strip each): the key window is staged
// in rounds (ascending; the last round holds the tile's own keys), the banded
// softmax runs over each round (Eq. (3)); then per map l: phi_l(q), the
// intra-tile lower-triangular part (causal), the product with the record
// S_l, z_l (Eq. (8)-(9)), the map's share of the blend (Eq. (11)), and
// (causal) the record update with the tile's keys (the prefix of Sec. 3.2.1).
#include "fmm_apply.h"
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {
namespace {

// TWO: an LDS budget of half a CU's LDS, so that two workgroups (two waves
// per SIMD) share a CU, where a round still holds a tile of keys (FITS);
// else the budget of one workgroup per CU.
template <typename T, int D, bool TWO = false>
struct WideCfg {
  static constexpr int ST = D + Lay<T>::PAD;
  static constexpr int ROW = ST * (int)sizeof(T);
  static constexpr int PK_BYTES = TM * ROW;     // phi_l of the tile's keys (causal)
  static constexpr int UNIT2 = 2 * 32 * ROW;    // K and V rows of one 32-key unit
  // the state records of up to three maps, kept in LDS for widths up to 64
  // (read every tile; the causal ones are also advanced there)
  static constexpr int REC_BYTES = D <= 64 ? 3 * D * (D + 1) * 4 : 0;
  static constexpr bool FITS = (80 * 1024 - PK_BYTES - REC_BYTES) / UNIT2 >= 2;
  static constexpr int BUDGET = TWO && FITS ? 80 * 1024 : 150 * 1024;
  static constexpr int UR_FIT = (BUDGET - PK_BYTES - REC_BYTES) / UNIT2;
  static constexpr int UR = UR_FIT > 8 ? 8 : UR_FIT;
  static_assert(UR >= 2, "a round must hold one tile of keys");
  static constexpr int WK = 32 * UR;            // keys per round
  static constexpr int REC_OFF = 2 * WK * ROW + PK_BYTES;
  static constexpr int LDS = REC_OFF + REC_BYTES;
};

// Wait states after a loop whose last matrix-core results are read by vector
// instructions after the loop exits: the required distance is provided here
// explicitly instead of relying on the hazard tracking across the loop's
// branches.
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"); }

// Rows [ks, ks + nk) of K and V (rows at or beyond kend read as zero) into
// row-major LDS buffers of stride ST.
template <typename T, int D>
__device__ __forceinline__ void stage_kv(T* sk, T* sv, const T* kh, const T* vh, int ks, int nk,
                                         int kend) {
  constexpr int ST = D + Lay<T>::PAD;
  auto ident = [](int i) { return i; };
  for (int x = 0; x < nk; x += 64) {
    const int m = min(64, nk - x);
    RowCopy<T, D, NT, 64> ck, cv;
    ck.load(kh, ks + x, m, kend);
    cv.load(vh, ks + x, m, kend);
    ck.store(sk + x * ST, ST, m, ident);
    cv.store(sv + x * ST, ST, m, ident);
  }
}

// phi_l of the tile's 64 keys (LDS rows kr .. kr+63 of the key buffer) into
// pk (row-major, stride ST); keys at or beyond N give 0.
template <typename T, int D>
__device__ __forceinline__ void stage_phi_map(const T* kbuf, int kr, int t0, int N, int l,
                                              T* pk) {
  using LY = Lay<T>;
  constexpr int ST = D + LY::PAD, CPR = D / LY::EPC;
  for (int t = threadIdx.x; t < TM * CPR; t += NT) {
    const int key = t / CPR, c = t % CPR;
    const uint4 raw = *reinterpret_cast<const uint4*>(kbuf + (kr + key) * ST + c * LY::EPC);
    float x[LY::EPC];
    if constexpr (sizeof(T) == 2) {
      const uint16_t* e = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int i = 0; i < LY::EPC; ++i) x[i] = bf16_to_f32(e[i]);
    } else {
      const float* e = reinterpret_cast<const float*>(&raw);
#pragma unroll
      for (int i = 0; i < LY::EPC; ++i) x[i] = e[i];
    }
    const bool ok = t0 + key < N;
    float p[LY::EPC];
#pragma unroll
    for (int i = 0; i < LY::EPC; ++i) p[i] = ok ? phi_any(x[i], l) : 0.f;
    uint4 outw;
    if constexpr (sizeof(T) == 2) {
      outw = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                        pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
    } else {
      outw = make_uint4(__float_as_uint(p[0]), __float_as_uint(p[1]), __float_as_uint(p[2]),
                        __float_as_uint(p[3]));
    }
    *reinterpret_cast<uint4*>(pk + key * ST + c * LY::EPC) = outw;
  }
}

// A record value block (4 consecutive floats) as a matrix-core operand quad.
template <typename T>
__device__ __forceinline__ typename QuadOf<T>::type rec_quad(const float* p) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  const float f[4] = {v.x, v.y, v.z, v.w};
  return f32_to_quad<T>(f);
}

// Intra-tile far part of one map for the strip of wave w (causal): keys
// [t0, row] of the tile, A = tril(phi_l(K_t) phi_l(q)^T) from pk, num[nb] +=
// V^T A and the row sums of A into num[NB].  vt: LDS row of the tile's first
// value row.
template <typename T, int D>
__device__ __forceinline__ void intra_map(const T* pk, const T* vt, int ST, int t0, int w,
                                          const typename QuadOf<T>::type* pq, f32x4* num) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int row = t0 + 16 * w + r;
  const Q ones = quad_fill<T>(1.f);
  for (int u = 0; u <= (w >> 1); ++u) {
    const bool diag = u == (w >> 1);
    float a[2][4];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      Q ka[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) ka[cb] = ld_quad(pk, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
      const f32x4 at = contract<NB>(ka, pq, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = t0 + 32 * u + 16 * b + 4 * g + i;
        a[b][i] = (!diag || j <= row) ? at[i] : 0.f;
      }
    }
    const Q p0 = f32_to_quad<T>(a[0]), p1 = f32_to_quad<T>(a[1]);
    const T* vx = vt + 32 * u * ST;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      num[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), p0, p1,
                          num[nb]);
    num[NB] = mma_step2(ones, ones, p0, p1, num[NB]);
  }
  mfma_drain();
}

template <typename T, int D, bool CAUSAL, bool JOINT, bool TWO>
__global__ __launch_bounds__(NT, TWO && D > 64 && (CAUSAL || JOINT) ? 2 : 1) void k_wide(const T* __restrict__ q, const T* __restrict__ k,
                                             const T* __restrict__ v, T* __restrict__ out,
                                             float* __restrict__ recs,
                                             const float* __restrict__ w_near,
                                             const float* __restrict__ w_far, int H, int N,
                                             int band_k, int L, int nseg, int rank,
                                             float scale2) {
  using Q = typename QuadOf<T>::type;
  using C = WideCfg<T, D, TWO>;
  constexpr int NB = D / 16, ST = C::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  T* sk = reinterpret_cast<T*>(dyn_smem);
  T* sv = sk + C::WK * ST;
  T* pk = sv + C::WK * ST;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const size_t base = (size_t)bh * N * D;
  const size_t REC = (size_t)rank * D * (D + 1);
  // non-causal: the slice's final record; causal: the segment's exclusive
  // prefix record, advanced tile by tile
  float* grec = CAUSAL ? recs + ((size_t)bh * nseg + seg) * REC : recs + (size_t)bh * REC;
  float* srec = reinterpret_cast<float*>(dyn_smem + C::REC_OFF);
  if constexpr (C::REC_BYTES > 0) {
    // (the first tile's staging barriers order the copy before any read)
    for (int t = threadIdx.x; 4 * t < (int)REC; t += NT)
      *reinterpret_cast<float4*>(srec + 4 * t) = *reinterpret_cast<const float4*>(grec + 4 * t);
  }
  float* rec = C::REC_BYTES > 0 ? srec : grec;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const int s0 = seg * L, s1 = min(N, s0 + L);
  for (int t0 = s0; t0 < s1; t0 += TM) {
    const int i0 = t0 + 16 * w, row = i0 + r;
    Q qq[NB];
    load_q<T, D>(q + base, row, N, qq);
    NearState<D> st;
    st.init();
    // key window [ka, hi): causal keys up to the tile's end (rows past N
    // stage as zeros), non-causal up to the band's end
    const int ka = (max(0, t0 - band_k) >> 5) << 5;
    const int hi = CAUSAL ? t0 + TM : ((min(N, t0 + TM + band_k) + 31) & ~31);
    const int nr = (hi - ka + C::WK - 1) / C::WK;
    int ks = ka;
    for (int rr = nr - 1; rr >= 0; --rr) {
      const int ke = hi - rr * C::WK;
      ks = max(ka, ke - C::WK);
      __syncthreads();  // every wave is done with the previous round / tile
      stage_kv<T, D>(sk, sv, k + base, v + base, ks, ke - ks, N);
      __syncthreads();
      const int lo = max(max(0, i0 - band_k), ks);
      const int hj = min(min(N - 1, CAUSAL ? i0 + 15 : i0 + 15 + band_k), ke - 1);
      if (lo <= hj)
        near_units<T, D, CAUSAL, 2>(st, qq, sk, sv, ST, RoundMap{ks}, lo >> 5, hj >> 5, i0, N,
                                    band_k, scale2);
    }
    mfma_drain();
    f32x4 fo[NB];
    near_out<D>(st, sn, fo);
    // far part, one map at a time; ks is the last round's first key, so the
    // tile's keys sit at LDS rows t0 - ks .. t0 - ks + 63
    f32x4 nsum[NB];
    float dsum = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) nsum[nb] = zero;
    for (int l = 0; l < rank; ++l) {
      Q pq[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        float x[4], p[4];
        quad_to_f32(qq[cb], x);
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = phi_any(x[i], l);
        pq[cb] = f32_to_quad<T>(p);
      }
      float* rl = rec + (size_t)l * D * (D + 1);
      f32x4 num[NB + 1];
#pragma unroll
      for (int nb = 0; nb <= NB; ++nb) num[nb] = zero;
      if constexpr (CAUSAL) {
        __syncthreads();  // the previous map's phi rows are no longer read
        stage_phi_map<T, D>(sk, t0 - ks, t0, N, l, pk);
        __syncthreads();
        intra_map<T, D>(pk, sv + (t0 - ks) * ST, ST, t0, w, pq, num);
      }
      // the product with the record: S_l tiles (cb, nb), then z_l
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        Q a[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) a[cb] = rec_quad<T>(rl + ((cb * NB + nb) * 64 + lane) * 4);
        num[nb] = contract<NB>(a, pq, num[nb]);
      }
      {
        Q zq[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) zq[cb] = rec_quad<T>(rl + D * D + 16 * cb + 4 * g);
        num[NB] = contract<NB>(zq, pq, num[NB]);
      }
      if constexpr (JOINT) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) nsum[nb] += num[nb];
        dsum += num[NB][0];
      } else {
        add_far_map<D>(num, sfw, fo);
      }
      if constexpr (CAUSAL) {
        if (t0 + TM < s1) {
          // advance the record by the tile's keys: S_l += phi_l(K_t)^T V_t,
          // z_l += phi_l(K_t)^T 1; wave w owns feature blocks w, w + 4, ...
          __syncthreads();  // every wave has read record l for this tile
          const T* vt = sv + (t0 - ks) * ST;
          const Q one0 = quad_fill<T>(r == 0 ? 1.f : 0.f);
          for (int cb = w; cb < NB; cb += NW) {
            f32x4 acc[NB + 1];
#pragma unroll
            for (int eb = 0; eb < NB; ++eb)
              acc[eb] = *reinterpret_cast<const f32x4*>(rl + ((cb * NB + eb) * 64 + lane) * 4);
            acc[NB] = r == 0 ? *reinterpret_cast<const f32x4*>(rl + D * D + 16 * cb + 4 * g)
                             : zero;
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const Q a0 = ld_tquad(pk, 32 * u, 16 * cb, ST);
              const Q a1 = ld_tquad(pk, 32 * u + 16, 16 * cb, ST);
              const T* vx = vt + 32 * u * ST;
#pragma unroll
              for (int eb = 0; eb < NB; ++eb)
                acc[eb] = mma_step2(a0, a1, ld_tquad(vx, 0, 16 * eb, ST),
                                    ld_tquad(vx, 16, 16 * eb, ST), acc[eb]);
              acc[NB] = mma_step2(a0, a1, one0, one0, acc[NB]);
            }
#pragma unroll
            for (int eb = 0; eb < NB; ++eb)
              *reinterpret_cast<f32x4*>(rl + ((cb * NB + eb) * 64 + lane) * 4) = acc[eb];
            if (r == 0) *reinterpret_cast<f32x4*>(rl + D * D + 16 * cb + 4 * g) = acc[NB];
          }
        }
      }
    }
    if constexpr (JOINT) {
      const float f = sfw > 0.f ? sfw * fast_rcp(dsum) : 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fo[nb] += nsum[nb] * f;
    }
    store_row<T, D>(out + base, row, N, fo);
  }
}

template <typename T, int D, bool CAUSAL, bool JOINT>
hipError_t launch_wide_k(const LaunchArgs& a, Launcher& L, float* recs) {
  // two workgroups per CU where the LDS allows it (bf16 at any width, fp32
  // up to 32); the kernels then stay within 256 registers (held there at
  // d = 128 causal or joint, a few of them spilled, which still pays)
  constexpr bool TWO = (D <= 64 || sizeof(T) == 2) && WideCfg<T, D, true>::FITS;
  using C = WideCfg<T, D, TWO>;
  static std::atomic<unsigned long long> lds_set{0};
  if (L.note(lds_limit_once((const void*)k_wide<T, D, CAUSAL, JOINT, TWO>, C::LDS, lds_set)) !=
      hipSuccess)
    return L.err;
  const float scale2 = 1.4426950408889634f / sqrtf((float)D);
  L(a.causal ? FMM_KERNEL_CAUSAL_APPLY : FMM_KERNEL_BAND_APPLY, k_wide<T, D, CAUSAL, JOINT, TWO>,
    dim3(a.B * a.H * a.nseg), dim3(NT), (size_t)C::LDS, (hipStream_t)a.stream, (const T*)a.q,
    (const T*)a.k, (const T*)a.v, (T*)a.out, recs, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L,
    a.nseg, a.rank, scale2);
  return L.err;
}

template <typename T, int D>
hipError_t launch_wide_d(const LaunchArgs& a, Launcher& L, float* recs) {
  const bool joint = a.far_norm == FMM_FAR_NORM_JOINT;
  if (a.causal)
    return joint ? launch_wide_k<T, D, true, true>(a, L, recs)
                 : launch_wide_k<T, D, true, false>(a, L, recs);
  return joint ? launch_wide_k<T, D, false, true>(a, L, recs)
               : launch_wide_k<T, D, false, false>(a, L, recs);
}

template <typename T>
hipError_t launch_wide_t(const LaunchArgs& a, Launcher& L, float* recs) {
  switch (a.d) {
    case 16: return launch_wide_d<T, 16>(a, L, recs);
    case 32: return launch_wide_d<T, 32>(a, L, recs);
    case 64: return launch_wide_d<T, 64>(a, L, recs);
    case 128: return launch_wide_d<T, 128>(a, L, recs);
    default: return L.note(hipErrorInvalidValue);
  }
}

}  // namespace

hipError_t launch_wide(const LaunchArgs& a, Launcher& L, float* recs) {
  return a.dtype == FMM_DTYPE_BF16 ? launch_wide_t<bf16_t>(a, L, recs)
                                   : launch_wide_t<float>(a, L, recs);
}

}  // namespace fmm
