// Backward pass of the FMMformer attention operator: the gradients of a loss
// L through g = dL/dout with respect to q, k, v and the two blend logits.
// For one (batch, head) slice, with a = sigmoid(w_near), c = sigmoid(w_far):
//
//   near field (Eq. (3)), p_ij the banded softmax of tau q_i.k_j:
//     D_i = a g_i . near_i
//     ds_ij = p_ij (a g_i . v_j - D_i)
//     dq_i += tau sum_j ds_ij k_j,  dk_j += tau sum_i ds_ij q_i,
//     dv_j += a sum_i p_ij g_i
//   far field (Eq. (7)-(9)), per map l with num_i = phi(q_i)^T S(i),
//   den_i = phi(q_i)^T z(i):
//     dnum_i = c g_i / den_i,  dden_i = -c g_i . num_i / den_i^2
//     dphi(q_i) = S(i) dnum_i + z(i) dden_i
//     dS(j) = sum_{i in G(j)} phi(q_i) dnum_i^T,  dz(j) = sum_{i in G(j)} phi(q_i) dden_i
//             (G(j): every row; causal: the rows i >= j, a suffix sum)
//     dphi(k_j) = dS(j) v_j + dz(j),  dv_j += dS(j)^T phi(k_j)
//     dq += phi'(q) * dphi(q),  dk += phi'(k) * dphi(k)
//   blend (Eq. (11)): dw_near = a (1 - a) sum g . near, dw_far = c (1 - c) sum g . far
//   joint normalisation (far = sum_l num_l / Den, Den = sum_l den_l): the
//   same with dnum_i = c g_i / Den_i and dden_i = -c g_i . far_i / Den_i for
//   every map, which the row pass forms in a first sweep over the maps
//
// Launch sequence (after the forward state k_seg_state + k_state_combine):
//   k_bwd_rows   per state segment, walking 64-row tiles: recomputes the near
//                softmax statistics (row maximum, sum) and D_i, then dq of the
//                near field in a second sweep over the staged keys; per map
//                the far numerator and denominator (state record, plus the
//                intra-tile part and the running prefix in the causal form),
//                dq of the far field, and the segment's partial
//                dS = sum phi(q_i) [dnum_i | dden_i]^T; writes dq, the per-row
//                softmax statistics and (1/den, dden) per map, and the
//                segment's sums of g . near and g . far
//   k_state_combine / k_suffix_scan
//                the dS partials summed per slice (non-causal) or turned into
//                exclusive suffix sums over segments (causal)
//   k_bwd_keys   per state segment, walking 64-key tiles (last tile first in
//                the causal form): near-field dk and dv over the rows whose
//                band holds the key, the far-field dk and dv from dS (causal:
//                the segment's suffix record advanced tile by tile plus the
//                intra-tile rows i >= j); writes dk, dv
//   k_dw_reduce  the blend-logit gradients, summed in a fixed order
//
// Fragment conventions are those of fmm_device.h: a 16-row strip per wave,
// row-quad accumulators (lane 16g + r holds row r, columns 16cb + 4g + {0..3}),
// products over 32 buffer rows through the transposed LDS reads.
#include "fmm_apply.h"
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {

// The fp32 d = 128 passes, defined in the second compilation of this file
// (with FMM_BWD_F32_D128, see the end of the file).
hipError_t launch_backward_f32_d128(const BwdArgs& a, Launcher& L);

namespace {

// NM: maps the record area holds (2 or 3).  TWO: an LDS budget of half a
// CU's LDS, so that two workgroups (two waves per SIMD) share a CU, where the
// rounds still hold a tile (FITS); else the budget of one workgroup per CU.
template <typename T, int D, int NM = 3, bool TWO = false>
struct BwdCfg {
  static constexpr int ST = D + Lay<T>::PAD;
  static constexpr int ROW = ST * (int)sizeof(T);
  static constexpr int TILE = TM * ROW;         // 64 staged rows
  static constexpr int UNIT2 = 2 * 32 * ROW;    // two buffers of one 32-row unit
  static constexpr int STAT_UNIT = 32 * 3 * 4;  // key pass: m, 1/l, D per row
  // the far-field records of up to NM maps, kept in LDS for widths up to
  // 64 (read every tile; the causal ones are also advanced there): fp32
  // records (causal), or their bf16 fragments (non-causal bf16:
  // RecFrags::PER_MAP per map)
  static constexpr int FRAG_MAP = 2 * (D / 16) * (D / 16) * 64 * 8 + (D / 16) * 32 + D * 4;
  static constexpr int REC_F32 = NM * D * (D + 1) * 4;
  static constexpr int REC_FRAG = NM * FRAG_MAP;
  static constexpr int REC_BYTES = D > 64 ? 0 : (REC_F32 > REC_FRAG ? REC_F32 : REC_FRAG);
  // tile buffers: phi and dnum rows of the tile
  static constexpr int NTB = 2;
  static constexpr int FIXED = NTB * TILE + 256 + 2 * NT * 4 + REC_BYTES;
  static constexpr bool FITS = (80 * 1024 - FIXED) / (UNIT2 + STAT_UNIT) >= 2;
  static constexpr int BUDGET = TWO && FITS ? 80 * 1024 : 150 * 1024;
  static constexpr int UR_FIT = (BUDGET - FIXED) / (UNIT2 + STAT_UNIT);
  static constexpr int UR = UR_FIT > 8 ? 8 : UR_FIT;
  static_assert(UR >= 2, "a round must hold one tile");
  static constexpr int WK = 32 * UR;  // rows per staging round
  // per staged row of the key pass: scaled maximum, 1/l, D; the row pass
  // reuses the area for its block reduction (2 x NT floats)
  static constexpr int STAT_BYTES = WK * 12 > 2 * NT * 4 ? WK * 12 : 2 * NT * 4;
  // [buffer A: WK rows][buffer B: WK rows][tile buffers 1, 2][64 floats][stats]
  // [records]
  static constexpr int REC_OFF = 2 * WK * ROW + 2 * TILE + 256 + STAT_BYTES;
  static constexpr int LDS = REC_OFF + REC_BYTES;
};

__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"); }

constexpr int SWB = 8;          // waves of k_seg_grad
constexpr int SNTB = SWB * 64;

// Rows [r0, r0 + n) of two [N, D] tensors (rows at or beyond kend read as
// zero) into row-major LDS buffers of stride ST.
template <typename T, int D>
__device__ __forceinline__ void stage_pair(T* sa, T* sb, const T* ha, const T* hb, int r0, int n,
                                           int kend) {
  constexpr int ST = D + Lay<T>::PAD;
  auto ident = [](int i) { return i; };
  for (int x = 0; x < n; x += 64) {
    const int m = min(64, n - x);
    RowCopy<T, D, NT, 64> ca, cb;
    ca.load(ha, r0 + x, m, kend);
    cb.load(hb, r0 + x, m, kend);
    ca.store(sa + x * ST, ST, m, ident);
    cb.store(sb + x * ST, ST, m, ident);
  }
}

// phi_l of 64 rows staged at src (stride ST) into dst; rows at or beyond
// N - r0 give 0.
template <typename T, int D>
__device__ __forceinline__ void stage_phi_rows(const T* src, int r0, int N, int l, T* dst) {
  using LY = Lay<T>;
  constexpr int ST = D + LY::PAD, CPR = D / LY::EPC;
  for (int t = threadIdx.x; t < TM * CPR; t += NT) {
    const int row = t / CPR, c = t % CPR;
    const uint4 raw = *reinterpret_cast<const uint4*>(src + row * ST + c * LY::EPC);
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
    const bool ok = r0 + row < N;
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
    *reinterpret_cast<uint4*>(dst + row * ST + c * LY::EPC) = outw;
  }
}

// The slice's or segment's records (n floats) into LDS, 16 bytes per thread
// and pass; the caller synchronises before reading them.
__device__ __forceinline__ void stage_records(float* dst, const float* src, int n) {
  for (int t = threadIdx.x; 4 * t < n; t += NT)
    *reinterpret_cast<float4*>(dst + 4 * t) = *reinterpret_cast<const float4*>(src + 4 * t);
}

template <typename T>
__device__ __forceinline__ typename QuadOf<T>::type rec_quad(const float* p) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  const float f[4] = {v.x, v.y, v.z, v.w};
  return f32_to_quad<T>(f);
}

// Transposed operand from a tile-order record: lane (r, g) gets
// X[16cb + r][16eb + 4g + {0..3}] where the record tile (cb, eb) stores
// X[16cb + 4g' + i][16eb + r'] at lane 16g' + r'.
template <typename T>
__device__ __forceinline__ typename QuadOf<T>::type rec_quad_t(const float* rl, int NB, int cb,
                                                               int eb) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const float* p = rl + ((cb * NB + eb) * 64 + 16 * (r >> 2) + 4 * g) * 4 + (r & 3);
  const float f[4] = {p[0], p[4], p[8], p[12]};
  return f32_to_quad<T>(f);
}

template <typename T>
__device__ __forceinline__ typename QuadOf<T>::type to_quad(const f32x4& x) {
  const float f[4] = {x[0], x[1], x[2], x[3]};
  return f32_to_quad<T>(f);
}

// bf16 operands of a constant record (the non-causal forward state and dS
// total), built once per workgroup in LDS so that every later use is one
// 8-byte read with no conversion.  Per map l, at l * PER_MAP bytes:
//   A[(cb * NB + nb) * 64 + lane] = rec_quad of tile (cb, nb) (lane's row of
//                                   the tile's quad layout)
//   B[(cb * NB + eb) * 64 + lane] = rec_quad_t of tile (cb, eb)
//   Z[cb * 4 + g]                 = rec_quad of z[16cb + 4g .. +3]
//   zf[D]                         = z in fp32
template <int D>
struct RecFrags {
  static constexpr int NB = D / 16;
  static constexpr int A_OFF = 0, B_OFF = NB * NB * 64 * 8, Z_OFF = 2 * NB * NB * 64 * 8,
                       ZF_OFF = Z_OFF + NB * 4 * 8;
  static constexpr int PER_MAP = ZF_OFF + D * 4;
  // from the fp32 record (tile order, rank maps) in global memory; the
  // caller synchronises before the first read
  __device__ __forceinline__ static void build(unsigned char* base, const float* rec, int rank) {
    const int nq = rank * NB * NB * 64;
    for (int t = threadIdx.x; t < nq; t += NT) {
      const int l = t / (NB * NB * 64), x = t % (NB * NB * 64), ln = x & 63, tile = x >> 6;
      const int cb = tile / NB, eb = tile % NB, r = ln & 15, g = ln >> 4;
      const float* rl = rec + (size_t)l * D * (D + 1);
      unsigned char* ml = base + l * PER_MAP;
      const float4 a = *reinterpret_cast<const float4*>(rl + (tile * 64 + ln) * 4);
      const float fa[4] = {a.x, a.y, a.z, a.w};
      const float* pb = rl + ((cb * NB + eb) * 64 + 16 * (r >> 2) + 4 * g) * 4 + (r & 3);
      const float fb[4] = {pb[0], pb[4], pb[8], pb[12]};
      reinterpret_cast<uint2*>(ml + A_OFF)[x] = f32_to_quad<bf16_t>(fa);
      reinterpret_cast<uint2*>(ml + B_OFF)[x] = f32_to_quad<bf16_t>(fb);
    }
    for (int t = threadIdx.x; t < rank * D; t += NT) {
      const int l = t / D, c = t % D;
      const float zv = rec[(size_t)l * D * (D + 1) + D * D + c];
      reinterpret_cast<float*>(base + l * PER_MAP + ZF_OFF)[c] = zv;
      if ((c & 3) == 0) {
        const float* zp = rec + (size_t)l * D * (D + 1) + D * D + c;
        const float fz[4] = {zp[0], zp[1], zp[2], zp[3]};
        reinterpret_cast<uint2*>(base + l * PER_MAP + Z_OFF)[c >> 2] = f32_to_quad<bf16_t>(fz);
      }
    }
  }
  __device__ __forceinline__ static uint2 a(const unsigned char* base, int l, int cb, int nb) {
    return reinterpret_cast<const uint2*>(base + l * PER_MAP + A_OFF)[(cb * NB + nb) * 64 +
                                                                       (threadIdx.x & 63)];
  }
  __device__ __forceinline__ static uint2 b(const unsigned char* base, int l, int cb, int eb) {
    return reinterpret_cast<const uint2*>(base + l * PER_MAP + B_OFF)[(cb * NB + eb) * 64 +
                                                                       (threadIdx.x & 63)];
  }
  __device__ __forceinline__ static uint2 z(const unsigned char* base, int l, int cb) {
    return reinterpret_cast<const uint2*>(base + l * PER_MAP + Z_OFF)[cb * 4 +
                                                                       ((threadIdx.x & 63) >> 4)];
  }
  __device__ __forceinline__ static const float* zf(const unsigned char* base, int l) {
    return reinterpret_cast<const float*>(base + l * PER_MAP + ZF_OFF);
  }
};

// rec_l += phi(X)^T [Y | y] over the 64 staged rows: px holds phi of the rows
// (stride ST), py the second factor's rows, ycol (64 floats) the extra column
// that lands in z; wave w updates feature blocks w, w + 4, ...
//
// With frl (bf16 only), the wave also rebuilds the RecFrags operands of its
// blocks from the updated tiles (A and Z from its registers, B read back
// transposed from the tiles it has just stored).
template <typename T, int D>
__device__ __forceinline__ void record_add(float* rl, const T* px, const T* py,
                                           const float* ycol, int ST, int w,
                                           unsigned char* frl = nullptr) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  for (int cb = w; cb < NB; cb += NW) {
    f32x4 acc[NB + 1];
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
      acc[eb] = *reinterpret_cast<const f32x4*>(rl + ((cb * NB + eb) * 64 + lane) * 4);
    acc[NB] = r == 0 ? *reinterpret_cast<const f32x4*>(rl + D * D + 16 * cb + 4 * g) : zero;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const Q a0 = ld_tquad(px, 32 * u, 16 * cb, ST);
      const Q a1 = ld_tquad(px, 32 * u + 16, 16 * cb, ST);
#pragma unroll
      for (int eb = 0; eb < NB; ++eb)
        acc[eb] = mma_step2(a0, a1, ld_tquad(py, 32 * u, 16 * eb, ST),
                            ld_tquad(py, 32 * u + 16, 16 * eb, ST), acc[eb]);
      float c0[4], c1[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        c0[i] = r == 0 ? ycol[32 * u + 4 * g + i] : 0.f;
        c1[i] = r == 0 ? ycol[32 * u + 16 + 4 * g + i] : 0.f;
      }
      acc[NB] = mma_step2(a0, a1, f32_to_quad<T>(c0), f32_to_quad<T>(c1), acc[NB]);
    }
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
      *reinterpret_cast<f32x4*>(rl + ((cb * NB + eb) * 64 + lane) * 4) = acc[eb];
    if (r == 0) *reinterpret_cast<f32x4*>(rl + D * D + 16 * cb + 4 * g) = acc[NB];
    if constexpr (sizeof(T) == 2) {
      if (frl) {
        using RF = RecFrags<D>;
#pragma unroll
        for (int eb = 0; eb < NB; ++eb) {
          reinterpret_cast<uint2*>(frl + RF::A_OFF)[(cb * NB + eb) * 64 + lane] =
              to_quad<bf16_t>(acc[eb]);
          reinterpret_cast<uint2*>(frl + RF::B_OFF)[(cb * NB + eb) * 64 + lane] =
              rec_quad_t<bf16_t>(rl, NB, cb, eb);
        }
        if (r == 0) reinterpret_cast<uint2*>(frl + RF::Z_OFF)[cb * 4 + g] = to_quad<bf16_t>(acc[NB]);
      }
    }
  }
}

// Band validity of key j (unit-local offset 16b + 4g + i from j0) for query
// row `row`: the interval logic of near_units.
template <bool CAUSAL>
__device__ __forceinline__ void band_interval(int row, int j0, int g, int N, int band_k, int& lo,
                                              int& span) {
  lo = max(row - band_k, 0) - j0 - 4 * g;
  span = min(CAUSAL ? row : row + band_k, N - 1) - j0 - 4 * g - lo;
  if (span < 0) {
    lo = 64;
    span = 0;
  }
}

// ------------------------------------------------------------------ row pass
// Near-field dq of the strip over key units [ua_lo, ua_hi] staged through map:
// dq += tau sum_j p_ij (a g_i . v_j - D_i) k_j with p from the final row
// statistics (maximum m of the raw scores, 1/l).
template <typename T, int D, bool CAUSAL, class Map>
__device__ __forceinline__ void near_dq_units(f32x4* dq, const typename QuadOf<T>::type* qq,
                                              const typename QuadOf<T>::type* gq, const T* kr,
                                              const T* vr, int ST, Map map, int ua_lo, int ua_hi,
                                              int i0, int N, int band_k, float scale2, float ms,
                                              float inv_l, float Di, float a_tau, float a) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int row = i0 + r;
  for (int ua = ua_lo; ua <= ua_hi; ++ua) {
    const T* kx = kr + map(ua) * ST;
    const T* vx = vr + map(ua) * ST;
    int lo, span;
    band_interval<CAUSAL>(row, ua * 32, g, N, band_k, lo, span);
    float ds[2][4];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      Q ka[NB], va[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        ka[cb] = ld_quad(kx, 16 * b + r, 16 * cb + 4 * g, ST);
        va[cb] = ld_quad(vx, 16 * b + r, 16 * cb + 4 * g, ST);
      }
      const f32x4 s = contract<NB>(ka, qq, f32x4{0.f, 0.f, 0.f, 0.f});
      const f32x4 dp = contract<NB>(va, gq, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = (unsigned)(16 * b + i - lo) <= (unsigned)span;
        const float p = ok ? __builtin_amdgcn_exp2f(fmaf(s[i], scale2, -ms)) * inv_l : 0.f;
        ds[b][i] = p * fmaf(a, dp[i], -Di) * a_tau;
      }
    }
    const Q d0 = f32_to_quad<T>(ds[0]), d1 = f32_to_quad<T>(ds[1]);
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
      dq[cb] = mma_step2(ld_tquad(kx, 0, 16 * cb, ST), ld_tquad(kx, 16, 16 * cb, ST), d0, d1,
                         dq[cb]);
  }
  mfma_drain();
}

template <typename T, int D, bool CAUSAL, int NM, bool TWO, bool JOINT>
__global__ __launch_bounds__(NT, TWO && CAUSAL ? 2 : 1) void k_bwd_rows(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, T* __restrict__ dq, float* __restrict__ recs,
    float* __restrict__ rowstat, float* __restrict__ rowfar,
    float* __restrict__ dwpart, const float* __restrict__ w_near, const float* __restrict__ w_far,
    int H, int N, int band_k, int L, int nseg, int rank, float scale2) {
  using Q = typename QuadOf<T>::type;
  using C = BwdCfg<T, D, NM, TWO>;
  constexpr int NB = D / 16, ST = C::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  T* sk = reinterpret_cast<T*>(dyn_smem);
  T* sv = sk + C::WK * ST;
  T* tb1 = sv + C::WK * ST;  // phi_l of the tile's keys, then of its queries
  T* tb2 = tb1 + TM * ST;    // dnum rows of the tile
  float* dden_s = reinterpret_cast<float*>(tb2 + TM * ST);
  float* red = dden_s + 64;  // block reduction of the blend-logit sums
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const size_t base = (size_t)bh * N * D;
  const size_t REC = (size_t)rank * D * (D + 1);
  float* grec = CAUSAL ? recs + ((size_t)bh * nseg + seg) * REC : recs + (size_t)bh * REC;
  // bf16 operands of the record: the non-causal record is constant and they
  // are built once
  constexpr bool FR = !CAUSAL && sizeof(T) == 2 && C::REC_BYTES > 0;
  unsigned char* frb = dyn_smem + C::REC_OFF;
  float* srec = reinterpret_cast<float*>(dyn_smem + C::REC_OFF);
  if constexpr (FR) RecFrags<D>::build(frb, grec, rank);
  if constexpr (C::REC_BYTES > 0 && (!FR || CAUSAL)) stage_records(srec, grec, (int)REC);
  float* rec = C::REC_BYTES > 0 ? srec : grec;  // (the first tile's barriers order the copy)
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const float tau = scale2 * 0.69314718055994531f;  // 1/sqrt(d)
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  float acc_near = 0.f, acc_far = 0.f;  // this lane's share of g . near and g . far
  // the ones column of the forward record's update (z), for every tile
  float* ones_col = dden_s;
  if (threadIdx.x < 64) ones_col[threadIdx.x] = 1.f;
  const int s0 = seg * L, s1 = min(N, s0 + L);
  for (int t0 = s0; t0 < s1; t0 += TM) {
    const int i0 = t0 + 16 * w, row = i0 + r;
    const bool row_ok = row < N;
    Q qq[NB], gq[NB];
    load_q<T, D>(q + base, row, N, qq);
    load_q<T, D>(dout + base, row, N, gq);
    float gf[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) quad_to_f32(gq[cb], gf[cb]);
    // ---- near field: statistics, then dq in a second sweep
    NearState<D> st;
    st.init();
    const int ka = (max(0, t0 - band_k) >> 5) << 5;
    const int hi = CAUSAL ? t0 + TM : ((min(N, t0 + TM + band_k) + 31) & ~31);
    const int nr = (hi - ka + C::WK - 1) / C::WK;
    int ks = ka;
    for (int rr = nr - 1; rr >= 0; --rr) {
      const int ke = hi - rr * C::WK;
      ks = max(ka, ke - C::WK);
      __syncthreads();
      stage_pair<T, D>(sk, sv, k + base, v + base, ks, ke - ks, N);
      __syncthreads();
      const int lo = max(max(0, i0 - band_k), ks);
      const int hj = min(min(N - 1, CAUSAL ? i0 + 15 : i0 + 15 + band_k), ke - 1);
      if (lo <= hj)
        near_units<T, D, CAUSAL, 2>(st, qq, sk, sv, ST, RoundMap{ks}, lo >> 5, hj >> 5, i0, N,
                                    band_k, scale2);
    }
    mfma_drain();
    const float inv_l = row_ok ? 1.f / st.o[NB][0] : 0.f;
    float gn = 0.f;  // g . (unnormalised near) over this lane's columns
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) gn = fmaf(gf[nb][i], st.o[nb][i], gn);
    const float gnear = col_sum(gn) * inv_l;  // g_i . near_i
    acc_near += gn * inv_l;
    const float Di = sn * gnear;
    const float ms = (st.m == -INFINITY ? 0.f : st.m) * scale2;
    if (row_ok && g == 0) {
      float* sp = rowstat + ((size_t)bh * N + row) * 3;
      sp[0] = ms;
      sp[1] = inv_l;
      sp[2] = Di;
    }
    f32x4 dqa[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) dqa[cb] = zero;
    for (int rr = nr - 1; rr >= 0; --rr) {
      const int ke = hi - rr * C::WK;
      const int ks2 = max(ka, ke - C::WK);
      if (nr > 1) {
        __syncthreads();
        stage_pair<T, D>(sk, sv, k + base, v + base, ks2, ke - ks2, N);
        __syncthreads();
      }
      const int lo = max(max(0, i0 - band_k), ks2);
      const int hj = min(min(N - 1, CAUSAL ? i0 + 15 : i0 + 15 + band_k), ke - 1);
      if (lo <= hj)
        near_dq_units<T, D, CAUSAL>(dqa, qq, gq, sk, sv, ST, RoundMap{ks2}, lo >> 5, hj >> 5, i0,
                                    N, band_k, scale2, ms, inv_l, Di, tau, sn);
    }
    // ks: first key of the last staged round, which holds the tile's keys
    // (causal form)
    // ---- far field, one map at a time (joint normalisation: below)
    if constexpr (!JOINT) {
      const T* vt = sv + (t0 - ks) * ST;
      for (int l = 0; l < rank; ++l) {
        const T* tbl = tb1;
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
          // the tile's keys: phi_l(K_t) into tb1; intra-tile part of num, den
          __syncthreads();
          stage_phi_rows<T, D>(sk + (t0 - ks) * ST, t0, N, l, tb1);
          __syncthreads();
          const Q ones = quad_fill<T>(1.f);
          for (int u = 0; u <= (w >> 1); ++u) {
            const bool diag = u == (w >> 1);
            float a2[2][4];
  #pragma unroll
            for (int b = 0; b < 2; ++b) {
              Q ka2[NB];
  #pragma unroll
              for (int cb = 0; cb < NB; ++cb)
                ka2[cb] = ld_quad(tbl, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
              const f32x4 at = contract<NB>(ka2, pq, zero);
  #pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int j = t0 + 32 * u + 16 * b + 4 * g + i;
                a2[b][i] = (!diag || j <= row) ? at[i] : 0.f;
              }
            }
            const Q p0 = f32_to_quad<T>(a2[0]), p1 = f32_to_quad<T>(a2[1]);
            const T* vx = vt + 32 * u * ST;
  #pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              num[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), p0,
                                  p1, num[nb]);
            num[NB] = mma_step2(ones, ones, p0, p1, num[NB]);
          }
          mfma_drain();
        }
        // the product with the record (non-causal: the slice's total; causal:
        // the prefix before the tile)
  #pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          Q a[NB];
  #pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            if constexpr (FR) a[cb] = RecFrags<D>::a(frb, l, cb, nb);
            else a[cb] = rec_quad<T>(rl + ((cb * NB + nb) * 64 + lane) * 4);
          }
          num[nb] = contract<NB>(a, pq, num[nb]);
        }
        {
          Q zq[NB];
  #pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            if constexpr (FR) zq[cb] = RecFrags<D>::z(frb, l, cb);
            else zq[cb] = rec_quad<T>(rl + D * D + 16 * cb + 4 * g);
          }
          num[NB] = contract<NB>(zq, pq, num[NB]);
        }
        // quotient rule
        const float inv_den = row_ok ? fast_rcp(num[NB][0]) : 0.f;
        float gnum = 0.f;
  #pragma unroll
        for (int nb = 0; nb < NB; ++nb)
  #pragma unroll
          for (int i = 0; i < 4; ++i) gnum = fmaf(gf[nb][i], num[nb][i], gnum);
        acc_far += gnum * inv_den;
        const float dden = -sfw * col_sum(gnum) * inv_den * inv_den;
        const float cid = sfw * inv_den;
        Q dnq[NB];
  #pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          float f[4];
  #pragma unroll
          for (int i = 0; i < 4; ++i) f[i] = gf[nb][i] * cid;
          dnq[nb] = f32_to_quad<T>(f);
        }
        if (row_ok && g == 0) {
          float* fp = rowfar + (((size_t)bh * N + row) * rank + l) * 2;
          fp[0] = inv_den;
          fp[1] = dden;
        }
        // dphi(q) = S dnum + z dden (+ intra-tile keys in the causal form)
        f32x4 dph[NB];
  #pragma unroll
        for (int cb = 0; cb < NB; ++cb) dph[cb] = zero;
        if constexpr (CAUSAL) {
          for (int u = 0; u <= (w >> 1); ++u) {
            const bool diag = u == (w >> 1);
            float a2[2][4];
  #pragma unroll
            for (int b = 0; b < 2; ++b) {
              Q va[NB];
  #pragma unroll
              for (int eb = 0; eb < NB; ++eb)
                va[eb] = ld_quad(vt, 32 * u + 16 * b + r, 16 * eb + 4 * g, ST);
              const f32x4 at = contract<NB>(va, dnq, zero);
  #pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int j = t0 + 32 * u + 16 * b + 4 * g + i;
                a2[b][i] = (!diag || j <= row) ? at[i] + dden : 0.f;
              }
            }
            const Q p0 = f32_to_quad<T>(a2[0]), p1 = f32_to_quad<T>(a2[1]);
  #pragma unroll
            for (int cb = 0; cb < NB; ++cb)
              dph[cb] = mma_step2(ld_tquad(tbl, 32 * u, 16 * cb, ST),
                                  ld_tquad(tbl, 32 * u + 16, 16 * cb, ST), p0, p1, dph[cb]);
          }
          mfma_drain();
        }
  #pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          Q a[NB];
  #pragma unroll
          for (int eb = 0; eb < NB; ++eb) {
            if constexpr (FR) a[eb] = RecFrags<D>::b(frb, l, cb, eb);
            else a[eb] = rec_quad_t<T>(rl, NB, cb, eb);
          }
          dph[cb] = contract<NB>(a, dnq, dph[cb]);
        }
        const float* zl = FR && !CAUSAL ? RecFrags<D>::zf(frb, l) : rl + D * D;
  #pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 z = *reinterpret_cast<const float4*>(zl + 16 * cb + 4 * g);
          const float zf[4] = {z.x, z.y, z.z, z.w};
          float x[4];
          quad_to_f32(qq[cb], x);
  #pragma unroll
          for (int i = 0; i < 4; ++i) {
            float dg = 0.f;
            if (l == 0) dg = x[i] > 0.f ? 1.f : __expf(x[i]);
            else if (l == 1) dg = x[i] < 0.f ? -1.f : -__expf(-x[i]);
            else {
              const float t = tanhf(x[i]);
              dg = 1.f - t * t;
            }
            dqa[cb][i] = fmaf(dg, dph[cb][i] + zf[i] * dden, dqa[cb][i]);
          }
        }
        if constexpr (CAUSAL) {
          // advance the forward prefix record by the tile's keys (tb1 still
          // holds phi_l(K_t)), unless this is the segment's last tile
          if (t0 + TM < s1) {
            __syncthreads();  // every wave has read record l for this tile
            record_add<T, D>(rl, tb1, vt, ones_col, ST, w, nullptr);
          }
        }
      }
    } else {
      const T* vt = sv + (t0 - ks) * ST;
      const T* tbl = tb1;
      auto phi_q = [&](int l, Q* pq) {
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          float x[4], p[4];
          quad_to_f32(qq[cb], x);
#pragma unroll
          for (int i = 0; i < 4; ++i) p[i] = phi_any(x[i], l);
          pq[cb] = f32_to_quad<T>(p);
        }
      };
      // the causal form's phi_l(K_t) rows into tb1 (for the intra-tile parts
      // and the record's advance)
      auto stage_keys = [&](int l) {
        __syncthreads();
        stage_phi_rows<T, D>(sk + (t0 - ks) * ST, t0, N, l, tb1);
        __syncthreads();
      };
      // num and den (column NB) of map l for the strip's rows
      auto far_num = [&](int l, const Q* pq, f32x4* num) {
        const float* rl = rec + (size_t)l * D * (D + 1);
#pragma unroll
        for (int nb = 0; nb <= NB; ++nb) num[nb] = zero;
        if constexpr (CAUSAL) {
          // the tile's keys: intra-tile part of num, den
          stage_keys(l);
          const Q ones = quad_fill<T>(1.f);
          for (int u = 0; u <= (w >> 1); ++u) {
            const bool diag = u == (w >> 1);
            float a2[2][4];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
              Q ka2[NB];
#pragma unroll
              for (int cb = 0; cb < NB; ++cb)
                ka2[cb] = ld_quad(tbl, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
              const f32x4 at = contract<NB>(ka2, pq, zero);
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int j = t0 + 32 * u + 16 * b + 4 * g + i;
                a2[b][i] = (!diag || j <= row) ? at[i] : 0.f;
              }
            }
            const Q p0 = f32_to_quad<T>(a2[0]), p1 = f32_to_quad<T>(a2[1]);
            const T* vx = vt + 32 * u * ST;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              num[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), p0,
                                  p1, num[nb]);
            num[NB] = mma_step2(ones, ones, p0, p1, num[NB]);
          }
          mfma_drain();
        }
        // the product with the record (non-causal: the slice's total; causal:
        // the prefix before the tile)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          Q a[NB];
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            if constexpr (FR) a[cb] = RecFrags<D>::a(frb, l, cb, nb);
            else a[cb] = rec_quad<T>(rl + ((cb * NB + nb) * 64 + lane) * 4);
          }
          num[nb] = contract<NB>(a, pq, num[nb]);
        }
        {
          Q zq[NB];
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            if constexpr (FR) zq[cb] = RecFrags<D>::z(frb, l, cb);
            else zq[cb] = rec_quad<T>(rl + D * D + 16 * cb + 4 * g);
          }
          num[NB] = contract<NB>(zq, pq, num[NB]);
        }
      };
      // one quotient for all maps: far = sum_l num_l / Den, Den = sum_l
      // den_l, so dnum_l = c g / Den and dden_l = -c g . (sum_l num_l) / Den^2
      // for every l; a first sweep over the maps forms Den and g . sum_l num_l
      float den = 0.f, gsum = 0.f;
      for (int l = 0; l < rank; ++l) {
        Q pq[NB];
        phi_q(l, pq);
        f32x4 num[NB + 1];
        far_num(l, pq, num);
        den += num[NB][0];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) gsum = fmaf(gf[nb][i], num[nb][i], gsum);
      }
      const float inv_den = row_ok ? fast_rcp(den) : 0.f;
      acc_far += gsum * inv_den;
      const float dden = -sfw * col_sum(gsum) * inv_den * inv_den;
      const float cid = sfw * inv_den;
      // then, per map, dq through phi_l'(q) and (causal) the record's advance
      for (int l = 0; l < rank; ++l) {
        float* rl = rec + (size_t)l * D * (D + 1);
        Q pq[NB];
        phi_q(l, pq);
        if constexpr (CAUSAL) stage_keys(l);
        Q dnq[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          float f[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) f[i] = gf[nb][i] * cid;
          dnq[nb] = f32_to_quad<T>(f);
        }
        if (row_ok && g == 0) {
          float* fp = rowfar + (((size_t)bh * N + row) * rank + l) * 2;
          fp[0] = inv_den;
          fp[1] = dden;
        }
        // dphi(q) = S dnum + z dden (+ intra-tile keys in the causal form)
        f32x4 dph[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) dph[cb] = zero;
        if constexpr (CAUSAL) {
          for (int u = 0; u <= (w >> 1); ++u) {
            const bool diag = u == (w >> 1);
            float a2[2][4];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
              Q va[NB];
#pragma unroll
              for (int eb = 0; eb < NB; ++eb)
                va[eb] = ld_quad(vt, 32 * u + 16 * b + r, 16 * eb + 4 * g, ST);
              const f32x4 at = contract<NB>(va, dnq, zero);
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int j = t0 + 32 * u + 16 * b + 4 * g + i;
                a2[b][i] = (!diag || j <= row) ? at[i] + dden : 0.f;
              }
            }
            const Q p0 = f32_to_quad<T>(a2[0]), p1 = f32_to_quad<T>(a2[1]);
#pragma unroll
            for (int cb = 0; cb < NB; ++cb)
              dph[cb] = mma_step2(ld_tquad(tbl, 32 * u, 16 * cb, ST),
                                  ld_tquad(tbl, 32 * u + 16, 16 * cb, ST), p0, p1, dph[cb]);
          }
          mfma_drain();
        }
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          Q a[NB];
#pragma unroll
          for (int eb = 0; eb < NB; ++eb) {
            if constexpr (FR) a[eb] = RecFrags<D>::b(frb, l, cb, eb);
            else a[eb] = rec_quad_t<T>(rl, NB, cb, eb);
          }
          dph[cb] = contract<NB>(a, dnq, dph[cb]);
        }
        const float* zl = FR && !CAUSAL ? RecFrags<D>::zf(frb, l) : rl + D * D;
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 z = *reinterpret_cast<const float4*>(zl + 16 * cb + 4 * g);
          const float zf[4] = {z.x, z.y, z.z, z.w};
          float x[4];
          quad_to_f32(qq[cb], x);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float dg = 0.f;
            if (l == 0) dg = x[i] > 0.f ? 1.f : __expf(x[i]);
            else if (l == 1) dg = x[i] < 0.f ? -1.f : -__expf(-x[i]);
            else {
              const float t = tanhf(x[i]);
              dg = 1.f - t * t;
            }
            dqa[cb][i] = fmaf(dg, dph[cb][i] + zf[i] * dden, dqa[cb][i]);
          }
        }
        if constexpr (CAUSAL) {
          // advance the forward prefix record by the tile's keys (tb1 still
          // holds phi_l(K_t)), unless this is the segment's last tile
          if (t0 + TM < s1) {
            __syncthreads();  // every wave has read record l for this tile
            record_add<T, D>(rl, tb1, vt, ones_col, ST, w, nullptr);
          }
        }
      }
    }
    store_row<T, D>(dq + base, row, N, dqa);
  }
  // the segment's sums of g . near and g . far, in a fixed order
  __syncthreads();
  red[threadIdx.x] = acc_near;
  red[NT + threadIdx.x] = acc_far;
  __syncthreads();
  if (threadIdx.x < 2) {
    float s = 0.f;
    for (int t = 0; t < NT; ++t) s += red[threadIdx.x * NT + t];
    dwpart[((size_t)bh * nseg + seg) * 2 + threadIdx.x] = s;
  }
}

// ------------------------------------------------------------------ suffix scan
// Causal dS: each segment's record becomes the sum of the records of the
// segments after it (exclusive suffix), in place, in a fixed order.
__global__ __launch_bounds__(256) void k_suffix_scan(float* __restrict__ part, int nseg, int rec,
                                                     int nchunk) {
  const int bh = blockIdx.x / nchunk;
  const int e = (blockIdx.x - bh * nchunk) * 256 + threadIdx.x;
  if (e >= rec) return;
  float* p = part + (size_t)bh * nseg * rec + e;
  float run = 0.f;
  for (int s = nseg - 1; s >= 0; --s) {
    const float t = p[(size_t)s * rec];
    p[(size_t)s * rec] = run;
    run += t;
  }
}

// ------------------------------------------------------------------ dS partials
// Per state segment, the far-field gradient state of map l:
//   dS_l = sum_i phi_l(q_i) dnum_i^T,  dz_l = sum_i phi_l(q_i) dden_i,
//   dnum_i = c g_i / den_l,i  (c = sigmoid(w_far[h]))
// from q, dout and the row pass's (1/den, dden), in the record's tile order.
// Same structure as k_seg_state: 8 waves, (rs, cb) = wave split of the
// 32-row units and feature block, 64-row chunks staged in LDS, a fixed-order
// tree over the waves sharing a feature block.
template <typename T, int D, int R>
__global__ __launch_bounds__(SNTB) void k_seg_grad(const T* __restrict__ q,
                                                   const T* __restrict__ dout,
                                                   const float* __restrict__ rowfar,
                                                   const float* __restrict__ w_far,
                                                   float* __restrict__ dpart, int H, int N, int L,
                                                   int nseg) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  constexpr int ST = D + Lay<T>::PAD;
  constexpr int RS = SWB / NB > 0 ? SWB / NB : 1;
  constexpr int TK = 64;
  // two 64-row chunks of q and dout double-buffered (the next chunk's loads
  // in flight during the current one's products), reused for the reduction
  // tree at the end
  constexpr int STAGE = 2 * 2 * TK * ST * (int)sizeof(T);
  constexpr int REDB = SWB / 2 * (NB + 1) * 64 * 16;
  __shared__ __attribute__((aligned(16))) unsigned char s_buf[STAGE > REDB ? STAGE : REDB];
  __shared__ float s_sc[2][R][TK], s_dd[2][R][TK];
  const int seg = blockIdx.x % nseg, bh = blockIdx.x / nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int cbw = w % NB, rs = w / NB;
  const bool owner = w < NB * RS;
  const int r0 = seg * L, r1 = min(N, r0 + L);
  const size_t base = (size_t)bh * N * D;
  const float sfw = sigmoidf_exact(w_far[h]);
  const int nchunk = (r1 - r0 + TK - 1) / TK;
  f32x4 acc[R][NB + 1];
#pragma unroll
  for (int l = 0; l < R; ++l)
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) acc[l][eb] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto ident = [](int i) { return i; };
  // a chunk's per-row (c / den, dden) pairs: thread t < R TK holds map t / TK,
  // row t % TK (zeros past the segment)
  // (a buffer over the segment's rows: pairs past it read as zeros, so the
  // loads need no branch)
  static_assert(R * TK <= SNTB, "one pair per thread");
  const __amdgpu_buffer_rsrc_t far_rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(rowfar + ((size_t)bh * N + r0) * R * 2), 0, (r1 - r0) * R * 8,
      0x00020000);
  auto load_far = [&](int c0) {
    const int t = threadIdx.x, l = t / TK, i = t % TK;
    const bool on = t < R * TK && c0 + i < r1;
    const uint32_t off = on ? (uint32_t)(((c0 - r0 + i) * R + l) * 8) : 0x80000000u;
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(far_rs, off, 0, 0));
  };
  auto store_far = [&](int buf, float2 f) {
    const int t = threadIdx.x;
    if (t < R * TK) {
      s_sc[buf][t / TK][t % TK] = sfw * f.x;
      s_dd[buf][t / TK][t % TK] = f.y;
    }
  };
  auto sq_of = [&](int buf) { return reinterpret_cast<T*>(s_buf) + buf * 2 * TK * ST; };
  // the first two chunks' loads together, the first stored
  RowCopy<T, D, SNTB, TK> cq, cg, cq0, cg0;
  cq0.load(q + base, r0, min(TK, r1 - r0), r1);
  cg0.load(dout + base, r0, min(TK, r1 - r0), r1);
  float2 f0 = load_far(r0);
  cq.load(q + base, r0 + TK, min(TK, r1 - r0 - TK), r1);
  cg.load(dout + base, r0 + TK, min(TK, r1 - r0 - TK), r1);
  float2 f1 = load_far(r0 + TK);
  cq0.store(sq_of(0), ST, TK, ident);
  cg0.store(sq_of(0) + TK * ST, ST, TK, ident);
  store_far(0, f0);
  for (int c = 0; c < nchunk; ++c) {
    const int c0 = r0 + c * TK;
    __syncthreads();  // chunk c is in its buffer; chunk c - 1's buffer is free
    if (c + 1 < nchunk) {
      cq.store(sq_of((c + 1) & 1), ST, TK, ident);
      cg.store(sq_of((c + 1) & 1) + TK * ST, ST, TK, ident);
      store_far((c + 1) & 1, f1);
    }
    if (c + 2 < nchunk) {
      const int cn = c0 + 2 * TK;
      cq.load(q + base, cn, min(TK, r1 - cn), r1);
      cg.load(dout + base, cn, min(TK, r1 - cn), r1);
      f1 = load_far(cn);
    }
    const T* s_q = sq_of(c & 1);
    const T* s_g = s_q + TK * ST;
    const float(*sc)[TK] = s_sc[c & 1];
    const float(*dd)[TK] = s_dd[c & 1];
    if (owner) {
#pragma unroll
      for (int u = 0; u < TK / 32; ++u) {
        if ((u % RS) != rs) continue;
        float qf[2][4];
#pragma unroll
        for (int b = 0; b < 2; ++b) quad_to_f32(ld_tquad(s_q, 32 * u + 16 * b, 16 * cbw, ST), qf[b]);
#pragma unroll
        for (int l = 0; l < R; ++l) {
          float pa[2][4];
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = 32 * u + 16 * b + 4 * g + i;
              pa[b][i] = c0 + row < r1 ? phi_any(qf[b][i], l) : 0.f;
            }
          const Q a0 = f32_to_quad<T>(pa[0]), a1 = f32_to_quad<T>(pa[1]);
#pragma unroll
          for (int eb = 0; eb < NB; ++eb) {
            float gb[2][4];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
              quad_to_f32(ld_tquad(s_g, 32 * u + 16 * b, 16 * eb, ST), gb[b]);
#pragma unroll
              for (int i = 0; i < 4; ++i) gb[b][i] *= sc[l][32 * u + 16 * b + 4 * g + i];
            }
            acc[l][eb] = mma_step2(a0, a1, f32_to_quad<T>(gb[0]), f32_to_quad<T>(gb[1]),
                                   acc[l][eb]);
          }
          float zb[2][4];
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              zb[b][i] = r == 0 ? dd[l][32 * u + 16 * b + 4 * g + i] : 0.f;
          acc[l][NB] = mma_step2(a0, a1, f32_to_quad<T>(zb[0]), f32_to_quad<T>(zb[1]),
                                 acc[l][NB]);
        }
      }
    }
  }
  mfma_drain();
  // fixed-order tree over the RS waves of a feature block, through s_q
  f32x4* red = reinterpret_cast<f32x4*>(s_buf);
#pragma unroll
  for (int l = 0; l < R; ++l) {
#pragma unroll
    for (int st = RS / 2; st >= 1; st >>= 1) {
      __syncthreads();
      if (owner && rs >= st && rs < 2 * st)
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb)
          red[(((rs - st) * NB + cbw) * (NB + 1) + eb) * 64 + lane] = acc[l][eb];
      __syncthreads();
      if (owner && rs < st)
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb)
          acc[l][eb] += red[((rs * NB + cbw) * (NB + 1) + eb) * 64 + lane];
    }
  }
  if (!owner || rs != 0) return;
  float* outp = dpart + ((size_t)bh * nseg + seg) * (R * D * (D + 1));
#pragma unroll
  for (int l = 0; l < R; ++l) {
    float* sl = outp + (size_t)l * D * (D + 1);
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
      *reinterpret_cast<f32x4*>(sl + ((cbw * NB + eb) * 64 + lane) * 4) = acc[l][eb];
    if (r == 0) *reinterpret_cast<f32x4*>(sl + D * D + 16 * cbw + 4 * g) = acc[l][NB];
  }
}

template <typename T, int D>
void launch_seg_grad(const BwdArgs& a, Launcher& L) {
  const dim3 grid(a.B * a.H * a.nseg);
  hipStream_t s = (hipStream_t)a.stream;
  switch (a.rank) {
    case 1:
      L(FMM_KERNEL_BWD_SEG_GRAD, k_seg_grad<T, D, 1>, grid, dim3(SNTB), 0, s, (const T*)a.q,
        (const T*)a.dout, (const float*)a.rowfar, a.w_far, a.dpart, a.H, a.N, a.L, a.nseg);
      break;
    case 2:
      L(FMM_KERNEL_BWD_SEG_GRAD, k_seg_grad<T, D, 2>, grid, dim3(SNTB), 0, s, (const T*)a.q,
        (const T*)a.dout, (const float*)a.rowfar, a.w_far, a.dpart, a.H, a.N, a.L, a.nseg);
      break;
    default:
      L(FMM_KERNEL_BWD_SEG_GRAD, k_seg_grad<T, D, 3>, grid, dim3(SNTB), 0, s, (const T*)a.q,
        (const T*)a.dout, (const float*)a.rowfar, a.w_far, a.dpart, a.H, a.N, a.L, a.nseg);
      break;
  }
}

// ------------------------------------------------------------------ key pass
template <typename T, int D, bool CAUSAL, int NM, bool TWO>
__global__ __launch_bounds__(NT, TWO && CAUSAL ? 2 : 1) void k_bwd_keys(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ drecs,
    const float* __restrict__ rowstat, const float* __restrict__ rowfar,
    const float* __restrict__ w_near, const float* __restrict__ w_far, int H, int N, int band_k,
    int L, int nseg, int rank, float scale2) {
  using Q = typename QuadOf<T>::type;
  using C = BwdCfg<T, D, NM, TWO>;
  constexpr int NB = D / 16, ST = C::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  T* sq = reinterpret_cast<T*>(dyn_smem);
  T* sg = sq + C::WK * ST;
  T* tb1 = sg + C::WK * ST;  // phi_l of the tile's query rows
  T* tb2 = tb1 + TM * ST;    // dnum rows of the tile
  float* dden_s = reinterpret_cast<float*>(tb2 + TM * ST);
  float* stat = dden_s + 64;  // per staged row: scaled maximum, 1/l, D
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const size_t base = (size_t)bh * N * D;
  const size_t REC = (size_t)rank * D * (D + 1);
  float* gdrec = CAUSAL ? drecs + ((size_t)bh * nseg + seg) * REC : drecs + (size_t)bh * REC;
  // bf16 operands of the dS record, as in the row pass
  constexpr bool FR = !CAUSAL && sizeof(T) == 2 && C::REC_BYTES > 0;
  unsigned char* frb = dyn_smem + C::REC_OFF;
  float* sdrec = reinterpret_cast<float*>(dyn_smem + C::REC_OFF);
  if constexpr (FR) RecFrags<D>::build(frb, gdrec, rank);
  if constexpr (C::REC_BYTES > 0 && (!FR || CAUSAL)) stage_records(sdrec, gdrec, (int)REC);
  float* drec = C::REC_BYTES > 0 ? sdrec : gdrec;  // (the first tile's barriers order the copy)
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const float tau = scale2 * 0.69314718055994531f;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + TM - 1) / TM;
  for (int tt = 0; tt < ntile; ++tt) {
    // causal: last tile first, so that the suffix record covers the rows
    // after the tile
    const int t0 = CAUSAL ? s0 + (ntile - 1 - tt) * TM : s0 + tt * TM;
    const int j0 = t0 + 16 * w, key = j0 + r;
    Q kq[NB], vq[NB];
    load_q<T, D>(k + base, key, N, kq);
    load_q<T, D>(v + base, key, N, vq);
    f32x4 dka[NB], dva[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      dka[cb] = zero;
      dva[cb] = zero;
    }
    // ---- near field over the rows whose band holds the strip's keys
    const int ra = CAUSAL ? t0 : (max(0, t0 - band_k) >> 5) << 5;
    const int rb = (min(N, t0 + TM + band_k) + 31) & ~31;
    // causal, one staging round of at least the tile's 64 rows: the staged
    // rows start with the tile's own rows t0 .. t0+63 (zero at or beyond N),
    // which the far part reads again
    const bool staged_tile = CAUSAL && rb - ra <= C::WK && rb - ra >= TM;
    for (int rs = ra; rs < rb; rs += C::WK) {
      const int nrow = min(C::WK, rb - rs);
      __syncthreads();
      stage_pair<T, D>(sq, sg, q + base, dout + base, rs, nrow, N);
      // per staged row (three arrays, read four rows at a time): the scaled
      // maximum, 1/l and D
      float* sm = stat;
      float* sli = stat + C::WK;
      float* sD = stat + 2 * C::WK;
      for (int t = threadIdx.x; t < nrow; t += NT) {
        const int i = rs + t;
        const bool ok = i < N;
        const float* sp = rowstat + ((size_t)bh * N + (ok ? i : 0)) * 3;
        sm[t] = ok ? sp[0] : 0.f;
        sli[t] = ok ? sp[1] : 0.f;
        sD[t] = ok ? sp[2] : 0.f;
      }
      __syncthreads();
      // rows of this round that can hold the strip's keys in their band
      const int lo = max(max(0, j0 - (CAUSAL ? 0 : band_k)), rs);
      const int hj = min(min(N - 1, j0 + 15 + band_k), rs + nrow - 1);
      // rows whose band holds this lane's key: [rlo, rhi] (empty past N)
      const int rlo = max(key - (CAUSAL ? 0 : band_k), 0);
      const int rhi = key < N ? min(key + band_k, N - 1) : -1;
      for (int ua = lo >> 5; ua <= (hj >> 5) && lo <= hj; ++ua) {
        const int ur = ua * 32 - rs;  // LDS row of the unit (a multiple of 32)
        const T* qx = sq + ur * ST;
        const T* gx = sg + ur * ST;
        // unit-local row offsets c = 16b + i of this lane group (rows
        // ua*32 + 4g + c) inside the interval
        int ilo = rlo - ua * 32 - 4 * g, ispan = rhi - rlo;
        if (ispan < 0) { ilo = 64; ispan = 0; }
        float pp[2][4], ds[2][4];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          Q qa[NB], ga[NB];
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            qa[cb] = ld_quad(qx, 16 * b + r, 16 * cb + 4 * g, ST);
            ga[cb] = ld_quad(gx, 16 * b + r, 16 * cb + 4 * g, ST);
          }
          const f32x4 s = contract<NB>(qa, kq, zero);
          const f32x4 dp = contract<NB>(ga, vq, zero);
          const int lr0 = ur + 16 * b + 4 * g;  // staged rows lr0 .. lr0+3
          const float4 m4 = *reinterpret_cast<const float4*>(sm + lr0);
          const float4 l4 = *reinterpret_cast<const float4*>(sli + lr0);
          const float4 d4 = *reinterpret_cast<const float4*>(sD + lr0);
          const float mv[4] = {m4.x, m4.y, m4.z, m4.w}, lv[4] = {l4.x, l4.y, l4.z, l4.w},
                      dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool ok = (unsigned)(16 * b + i - ilo) <= (unsigned)ispan;
            const float p = ok ? __builtin_amdgcn_exp2f(fmaf(s[i], scale2, -mv[i])) * lv[i] : 0.f;
            pp[b][i] = p * sn;
            ds[b][i] = p * fmaf(sn, dp[i], -dv4[i]) * tau;
          }
        }
        const Q p0 = f32_to_quad<T>(pp[0]), p1 = f32_to_quad<T>(pp[1]);
        const Q d0 = f32_to_quad<T>(ds[0]), d1 = f32_to_quad<T>(ds[1]);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          dva[cb] = mma_step2(ld_tquad(gx, 0, 16 * cb, ST), ld_tquad(gx, 16, 16 * cb, ST), p0, p1,
                              dva[cb]);
          dka[cb] = mma_step2(ld_tquad(qx, 0, 16 * cb, ST), ld_tquad(qx, 16, 16 * cb, ST), d0, d1,
                              dka[cb]);
        }
      }
      mfma_drain();
    }
    // ---- far field, one map at a time.  Causal: per map the tile's rows as
    // phi_l(q) rows, dnum = c g / den rows, and dden
    auto reload_tile = [&]() {
      if (!staged_tile) {
        RowCopy<T, D, NT, 64> cq, cg;
        cq.load(q + base, t0, TM, N);
        cg.load(dout + base, t0, TM, N);
        auto ident = [](int i) { return i; };
        cq.store(sq, ST, TM, ident);
        cg.store(sg, ST, TM, ident);
      }
    };
    auto far_row_terms = [&](int l) {  // dden and c / den of the tile's rows
      if (threadIdx.x < 64) {
        const int i = t0 + threadIdx.x;
        const bool ok = i < N;
        const float* fp = rowfar + (((size_t)bh * N + (ok ? i : 0)) * rank + l) * 2;
        dden_s[threadIdx.x] = ok ? fp[1] : 0.f;
        stat[threadIdx.x] = ok ? sfw * fp[0] : 0.f;
      }
    };
    auto dnum_rows = [&](T* dst, const float* cd) {
      using LY = Lay<T>;
      constexpr int CPR = D / LY::EPC;
      for (int t = threadIdx.x; t < TM * CPR; t += NT) {
        const int rr = t / CPR, c = t % CPR;
        const uint4 raw = *reinterpret_cast<const uint4*>(sg + rr * ST + c * LY::EPC);
        const float f = cd[rr];
        uint4 outw;
        if constexpr (sizeof(T) == 2) {
          const uint16_t* e = reinterpret_cast<const uint16_t*>(&raw);
          float x[8];
#pragma unroll
          for (int ii = 0; ii < 8; ++ii) x[ii] = bf16_to_f32(e[ii]) * f;
          outw = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]),
                            pack_bf16x2(x[4], x[5]), pack_bf16x2(x[6], x[7]));
        } else {
          const float* e = reinterpret_cast<const float*>(&raw);
          outw = make_uint4(__float_as_uint(e[0] * f), __float_as_uint(e[1] * f),
                            __float_as_uint(e[2] * f), __float_as_uint(e[3] * f));
        }
        *reinterpret_cast<uint4*>(dst + rr * ST + c * LY::EPC) = outw;
      }
    };
    for (int l = 0; l < rank; ++l) {
      const T* phq = tb1;
      const T* dnr = tb2;
      const float* ddl = dden_s;
      Q pk[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        float x[4], p[4];
        quad_to_f32(kq[cb], x);
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = phi_any(x[i], l);
        pk[cb] = f32_to_quad<T>(p);
      }
      float* drl = drec + (size_t)l * D * (D + 1);
      f32x4 dph[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) dph[cb] = zero;
      if constexpr (CAUSAL) {
        __syncthreads();
        reload_tile();
        far_row_terms(l);
        __syncthreads();
        stage_phi_rows<T, D>(sq, t0, N, l, tb1);
        dnum_rows(tb2, stat);
        __syncthreads();
        // rows i >= j of the tile: units (w >> 1) .. 1, the first one masked
        for (int u = (w >> 1); u < 2; ++u) {
          const bool diag = u == (w >> 1);
          float cc[2][4], ee[2][4];
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            Q na[NB], fa[NB];
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) {
              na[cb] = ld_quad(dnr, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
              fa[cb] = ld_quad(phq, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
            }
            const f32x4 c1 = contract<NB>(na, vq, zero);
            const f32x4 e1 = contract<NB>(fa, pk, zero);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int lr = 32 * u + 16 * b + 4 * g + i;
              const bool ok = !diag || t0 + lr >= key;
              cc[b][i] = ok ? c1[i] + ddl[lr] : 0.f;
              ee[b][i] = ok ? e1[i] : 0.f;
            }
          }
          const Q c0q = f32_to_quad<T>(cc[0]), c1q = f32_to_quad<T>(cc[1]);
          const Q e0q = f32_to_quad<T>(ee[0]), e1q = f32_to_quad<T>(ee[1]);
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            dph[cb] = mma_step2(ld_tquad(phq, 32 * u, 16 * cb, ST),
                                ld_tquad(phq, 32 * u + 16, 16 * cb, ST), c0q, c1q, dph[cb]);
            dva[cb] = mma_step2(ld_tquad(dnr, 32 * u, 16 * cb, ST),
                                ld_tquad(dnr, 32 * u + 16, 16 * cb, ST), e0q, e1q, dva[cb]);
          }
        }
        mfma_drain();
      }
      // dS (j) from the record: dphi(k) += dS v + dz, dv += dS^T phi(k)
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        Q a[NB];
#pragma unroll
        for (int eb = 0; eb < NB; ++eb) {
          if constexpr (FR) a[eb] = RecFrags<D>::b(frb, l, cb, eb);
          else a[eb] = rec_quad_t<T>(drl, NB, cb, eb);
        }
        dph[cb] = contract<NB>(a, vq, dph[cb]);
      }
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) {
        Q a[NB];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          if constexpr (FR) a[cb] = RecFrags<D>::a(frb, l, cb, eb);
          else a[cb] = rec_quad<T>(drl + ((cb * NB + eb) * 64 + lane) * 4);
        }
        dva[eb] = contract<NB>(a, pk, dva[eb]);
      }
      const float* zl = FR && !CAUSAL ? RecFrags<D>::zf(frb, l) : drl + D * D;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 z = *reinterpret_cast<const float4*>(zl + 16 * cb + 4 * g);
        const float zf[4] = {z.x, z.y, z.z, z.w};
        float x[4];
        quad_to_f32(kq[cb], x);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float dg = 0.f;
          if (l == 0) dg = x[i] > 0.f ? 1.f : __expf(x[i]);
          else if (l == 1) dg = x[i] < 0.f ? -1.f : -__expf(-x[i]);
          else {
            const float t = tanhf(x[i]);
            dg = 1.f - t * t;
          }
          dka[cb][i] = fmaf(dg, dph[cb][i] + zf[i], dka[cb][i]);
        }
      }
      if constexpr (CAUSAL) {
        // advance the suffix record by the tile's rows, unless this is the
        // segment's first tile (the last one walked)
        if (tt + 1 < ntile) {
          __syncthreads();  // every wave has read record l for this tile
          record_add<T, D>(drl, tb1, tb2, dden_s, ST, w, nullptr);
        }
      }
    }
    store_row<T, D>(dk + base, key, N, dka);
    store_row<T, D>(dv + base, key, N, dva);
  }
}

// ------------------------------------------------------------------ dw
__global__ void k_dw_reduce(const float* __restrict__ dwpart, const float* __restrict__ w_near,
                            const float* __restrict__ w_far, float* __restrict__ dw_near,
                            float* __restrict__ dw_far, int B, int H, int nseg) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= H) return;
  float sn = 0.f, sf = 0.f;
  for (int b = 0; b < B; ++b)
    for (int s = 0; s < nseg; ++s) {
      const float* p = dwpart + (((size_t)b * H + h) * nseg + s) * 2;
      sn += p[0];
      sf += p[1];
    }
  const float a = sigmoidf_exact(w_near[h]), c = sigmoidf_exact(w_far[h]);
  dw_near[h] = a * (1.f - a) * sn;
  dw_far[h] = c * (1.f - c) * sf;
}

template <typename T, int D, bool CAUSAL, int NM = 3, bool TWO = false>
hipError_t launch_bwd_dcf(const BwdArgs& a, Launcher& L) {
  using C = BwdCfg<T, D, NM, TWO>;
  const bool joint = a.far_norm == FMM_FAR_NORM_JOINT;
  static std::atomic<unsigned long long> set_rows{0}, set_rows_j{0}, set_keys{0};
  if (L.note(joint ? lds_limit_once((const void*)k_bwd_rows<T, D, CAUSAL, NM, TWO, true>,
                                    C::LDS, set_rows_j)
                   : lds_limit_once((const void*)k_bwd_rows<T, D, CAUSAL, NM, TWO, false>,
                                    C::LDS, set_rows)) != hipSuccess ||
      L.note(lds_limit_once((const void*)k_bwd_keys<T, D, CAUSAL, NM, TWO>, C::LDS,
                            set_keys)) != hipSuccess)
    return L.err;
  const float scale2 = 1.4426950408889634f / sqrtf((float)D);
  const int BH = a.B * a.H;
  const size_t REC = (size_t)a.rank * D * (D + 1);
  hipStream_t s = (hipStream_t)a.stream;
  const dim3 grid(BH * a.nseg);
  auto rows = [&](auto kern) {
    L(FMM_KERNEL_BWD_ROWS, kern, grid, dim3(NT), (size_t)C::LDS, s, (const T*)a.q,
      (const T*)a.k, (const T*)a.v, (const T*)a.dout, (T*)a.dq, CAUSAL ? a.part : a.fin,
      a.rowstat, a.rowfar, a.dwpart, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg,
      a.rank, scale2);
  };
  if (joint) rows(k_bwd_rows<T, D, CAUSAL, NM, TWO, true>);
  else rows(k_bwd_rows<T, D, CAUSAL, NM, TWO, false>);
  launch_seg_grad<T, D>(a, L);
  const int nchunk = (int)((REC + 255) / 256);
  const dim3 sgrid((unsigned)std::min<long long>((long long)nchunk * BH, 0xFFFFFFFFll));
  if constexpr (CAUSAL) {
    L(FMM_KERNEL_STATE_COMBINE, k_suffix_scan, sgrid, dim3(256), 0, s, a.dpart, a.nseg, (int)REC,
      nchunk);
  } else {
    (void)launch_state_sum(L, a.dpart, a.dfin, a.nseg, (int)REC, BH, s);
  }
  L(FMM_KERNEL_BWD_KEYS, k_bwd_keys<T, D, CAUSAL, NM, TWO>, grid, dim3(NT), (size_t)C::LDS, s,
    (const T*)a.q, (const T*)a.k, (const T*)a.v, (const T*)a.dout, (T*)a.dk, (T*)a.dv,
    CAUSAL ? a.dpart : a.dfin, (const float*)a.rowstat, (const float*)a.rowfar, a.w_near, a.w_far,
    a.H, a.N, a.band_k, a.L, a.nseg, a.rank, scale2);
  L(FMM_KERNEL_BWD_DW, k_dw_reduce, dim3((a.H + 63) / 64), dim3(64), 0, s,
    (const float*)a.dwpart, a.w_near, a.w_far, a.dw_near, a.dw_far, a.B, a.H, a.nseg);
  return L.err;
}

template <typename T, int D>
hipError_t launch_bwd_d(const BwdArgs& a, Launcher& L) {
  // at d <= 64 with one or two maps the records of two maps leave room for
  // two workgroups per CU (two waves per SIMD; the causal passes are held
  // to 256 registers for it)
  if constexpr (D <= 64) {
    if (a.rank <= 2) {
      constexpr bool two = BwdCfg<T, D, 2, true>::FITS;
      return a.causal ? launch_bwd_dcf<T, D, true, 2, two>(a, L)
                      : launch_bwd_dcf<T, D, false, 2, two>(a, L);
    }
  }
  return a.causal ? launch_bwd_dcf<T, D, true>(a, L) : launch_bwd_dcf<T, D, false>(a, L);
}

#ifndef FMM_BWD_F32_D128
template <typename T>
hipError_t launch_bwd_t(const BwdArgs& a, Launcher& L) {
  switch (a.d) {
    case 16: return launch_bwd_d<T, 16>(a, L);
    case 32: return launch_bwd_d<T, 32>(a, L);
    case 64: return launch_bwd_d<T, 64>(a, L);
    case 128:
      // fp32 at d = 128 is built in a translation unit of its own (below)
      if constexpr (sizeof(T) == 2) return launch_bwd_d<T, 128>(a, L);
      return launch_backward_f32_d128(a, L);
    default: return L.note(hipErrorInvalidValue);
  }
}
#endif

}  // namespace

#ifdef FMM_BWD_F32_D128
// fp32 storage at d = 128 holds twice the operand registers of bf16: its
// passes run at one workgroup per CU and need the accumulation registers
// beside the 256 vector registers, so this file is compiled a second time,
// with this macro and without forcing MFMA results into vector registers
// (with that option the compiler fails on the causal key pass).
hipError_t launch_backward_f32_d128(const BwdArgs& a, Launcher& L) {
  return launch_bwd_d<float, 128>(a, L);
}
#else
hipError_t launch_backward_tail(const BwdArgs& a, Launcher& L) {
  return a.dtype == FMM_DTYPE_BF16 ? launch_bwd_t<bf16_t>(a, L) : launch_bwd_t<float>(a, L);
}
#endif

}  // namespace fmm
