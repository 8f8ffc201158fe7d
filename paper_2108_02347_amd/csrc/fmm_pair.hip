// Non-causal FMMformer apply for bf16 heads of width 32 or 64 and band
// half-widths up to 64, with two 16-row strips per wavefront.
//
// k_band_pair walks the 128-row tiles of a row segment like k_band_ring, but
// each of its four wavefronts owns 32 consecutive query rows (strip A = rows
// i0 .. i0+15, strip B = i0+16 .. i0+31).  The two strips share every operand
// read from LDS: a key block's K rows feed both strips' score products
// (Eq. (3)), a key unit's V^T quads both strips' P V products, and the state
// fragments both strips' far products (Eq. (8)-(9)); the blend (Eq. (11)) and
// store follow per strip.
//
// Operands of the products contracted over the head width (scores, far
// terms) are "octs": the contraction index runs over 32-wide blocks and lane
// group g holds the eight consecutive indices 8g..8g+7 of a block, so a K
// row's slice is one 16-byte LDS read.  The P V product keeps the quad
// convention of the score output (keys 4g..4g+3 of each 16-key block).
//
// K and V rows sit unpadded in an LDS ring; for d = 64 the 16-byte chunk c of
// ring row r is stored at chunk c ^ swz(r), which keeps the 16-byte K reads,
// the transposed 8-byte V reads and the 16-byte row stores free of bank
// conflicts.  d = 32 rows are padded to 80 bytes instead.
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {
namespace {

constexpr int PW = 4;           // wavefronts per workgroup
constexpr int PNT = PW * 64;    // threads per workgroup
constexpr int PTM = 32 * PW;    // query rows per tile

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

// Byte offset of 16-byte chunk c of ring row r.
template <int D> struct PairRows;
template <> struct PairRows<64> {
  static constexpr int RB = 128;
  // a permutation of 0..7 on every aligned 8-row group; rows r and r + 8 and
  // the even (odd) rows of a 16-row group get distinct chunk positions, and
  // four aligned consecutive rows distinct chunk pairs
  __device__ __forceinline__ static int swz(int r) {
    const int a = (r >> 2) & 1;
    return ((((r & 3) ^ a) << 1) | a) ^ ((r >> 3) & 1);
  }
  __device__ __forceinline__ static int off(int r, int c) { return r * RB + ((c ^ swz(r)) << 4); }
};
template <> struct PairRows<32> {
  static constexpr int RB = 80;
  __device__ __forceinline__ static int off(int r, int c) { return r * RB + (c << 4); }
};

template <int D, int R, int KC>
struct PairCfg {
  static constexpr int NB = D / 16, NQ = D / 32;
  static constexpr int U = 4 + 2 * KC;   // ring units of 32 keys: a tile's window
  static constexpr int NU = 2 * KC + 1;  // key units spanned by one wavefront's rows
  static constexpr int RING = U * 32 * PairRows<D>::RB;
  static constexpr int FRAG = R * NB * NQ * 64 * 16;
  static constexpr int LDS = 2 * RING + FRAG;
};

// K or V rows [k0, k0 + 128) of a head in registers (zero outside [0, N));
// thread t holds chunk t % CPR of row t / CPR + (PNT / CPR) * it.
template <int D>
struct PairCopy {
  static constexpr int CPR = D / 8;
  static constexpr int IT = PTM * CPR / PNT;
  uint4 r[IT];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ src, int k0, int N) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * PNT;
      const int key = k0 + x / CPR;
      r[it] = make_uint4(0, 0, 0, 0);
      if (key >= 0 && key < N)
        r[it] = *reinterpret_cast<const uint4*>(src + (size_t)key * D + (x % CPR) * 8);
    }
  }
  // Unit j (0..3) of the copied rows goes to ring slot slot_of(j) (skipped if < 0).
  template <typename F>
  __device__ __forceinline__ void store(unsigned char* ring, F slot_of) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * PNT;
      const int i = x / CPR;
      const int slot = slot_of(i >> 5);
      if (slot >= 0)
        *reinterpret_cast<uint4*>(ring + PairRows<D>::off(slot * 32 + (i & 31), x % CPR)) = r[it];
    }
  }
};

// V^T quad of the 16-key block starting at ring row r0, columns 16nb .. 16nb+15:
// lane (j, g) receives V[r0 + 4g + e][16nb + j], e = 0..3 (see ld_tquad).
template <int D>
__device__ __forceinline__ uint2 vt_quad(const unsigned char* vr, int r0, int nb) {
  const int lane = threadIdx.x & 63, g = lane >> 4, t = lane & 15;
  const int row = r0 + 4 * g + (t >> 2);
  const unsigned char* p = vr + PairRows<D>::off(row, 2 * nb + ((t & 3) >> 1)) + 8 * (t & 1);
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  return __builtin_bit_cast(uint2, v);
}

// Query octs of the lane's row of each strip: qo[s][p] = q[i0 + 16s + r][32p + 8g .. +7].
template <int D>
__device__ __forceinline__ void load_qo(const bf16_t* __restrict__ qh, int i0, int N,
                                        Oct (*qo)[D / 32]) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int row = i0 + 16 * s + r;
#pragma unroll
    for (int p = 0; p < D / 32; ++p)
      qo[s][p] = row < N ? *reinterpret_cast<const Oct*>(qh + (size_t)row * D + 32 * p + 8 * g)
                         : make_uint4(0, 0, 0, 0);
  }
}

// State fragments from the non-causal tile-order record (see k_seg_state):
// sf[((l*NB + nb)*NQ + p)*64 + lane] holds S_l[32p + 8g + i][16nb + r],
// i = 0..7, as an oct; zo[l][p] holds z_l[32p + 8g + i].
template <int D, int R>
__device__ __forceinline__ void pair_frags(const float* __restrict__ rec, Oct* sf,
                                           Oct (*zo)[D / 32]) {
  constexpr int NB = D / 16, NQ = D / 32;
  for (int x = threadIdx.x; x < R * NB * NQ * 64; x += PNT) {
    const int ln = x & 63, blk = x >> 6;
    const int p = blk % NQ, nb = (blk / NQ) % NB, l = blk / (NQ * NB);
    const int gg = ln >> 4, rr = ln & 15;
    const int cb = 2 * p + (gg >> 1);
    const float* t0 = rec + (size_t)l * D * (D + 1) + ((cb * NB + nb) * 64 + 32 * (gg & 1) + rr) * 4;
    const float4 a = *reinterpret_cast<const float4*>(t0);
    const float4 b = *reinterpret_cast<const float4*>(t0 + 64);
    const float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    sf[x] = oct_pack(f);
  }
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int l = 0; l < R; ++l)
#pragma unroll
    for (int p = 0; p < NQ; ++p) {
      const float* z = rec + (size_t)l * D * (D + 1) + D * D + 32 * p + 8 * g;
      const float4 a = *reinterpret_cast<const float4*>(z);
      const float4 b = *reinterpret_cast<const float4*>(z + 4);
      const float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      zo[l][p] = oct_pack(f);
    }
}

// Banded softmax of both strips of the wavefront whose rows start at i0 (a
// multiple of 32).  Key units u = 0 .. NU-1 (absolute unit i0/32 - KC + u)
// sit in ring slots (slot0 + u) % U.  Strip A never needs the last 16-key
// block of the span and strip B never the first.  EXACT: k = 32*KC and the
// span lies inside [0, N), so only the first and last block of each strip
// cut the band (triangles); otherwise every block is masked against the
// row's band clipped to [0, N).  On return o[s][nb] holds the unnormalised
// P V of strip s and o[s][NB] its row sums.
template <int D, int R, int KC, bool EXACT>
__device__ __forceinline__ void pair_near(f32x4 (*o)[D / 16 + 1], Oct (*qo)[D / 32],
                                          const unsigned char* kr, const unsigned char* vr,
                                          int slot0, int i0, int N, int band_k, float scale2) {
  using C = PairCfg<D, R, KC>;
  constexpr int NB = C::NB, NQ = C::NQ, NU = C::NU, NBK = 2 * NU;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  int urow[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) urow[u] = ((slot0 + u) % C::U) * 32;

  // scores S^T = K Q^T of every (strip, block) the strip needs
  f32x4 sc[2][NBK];
#pragma unroll
  for (int b = 0; b < NBK; ++b) {
    Oct ko[NQ];
#pragma unroll
    for (int p = 0; p < NQ; ++p)
      ko[p] = *reinterpret_cast<const Oct*>(
          kr + PairRows<D>::off(urow[b >> 1] + 16 * (b & 1) + r, 4 * p + g));
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if ((s == 0 && b == NBK - 1) || (s == 1 && b == 0)) continue;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < NQ; ++p) acc = mma8(ko[p], qo[s][p], acc);
      sc[s][b] = acc;
    }
  }

  // band masks
  if constexpr (EXACT) {
    // lower edge (first block of the strip): key offset 4g + i >= r;
    // upper edge (last block): 4g + i <= r
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool lo_ok = 4 * g + i >= r, hi_ok = 4 * g + i <= r;
      if (!lo_ok) { sc[0][0][i] = -INFINITY; sc[1][1][i] = -INFINITY; }
      if (!hi_ok) { sc[0][NBK - 2][i] = -INFINITY; sc[1][NBK - 1][i] = -INFINITY; }
    }
  } else {
    const int kbase = (i0 / 32 - KC) * 32 + 4 * g;  // key of (block 0, element 0) of this lane
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int row = i0 + 16 * s + r;
      int lo = max(row - band_k, 0) - kbase;
      int span = min(row + band_k, N - 1) - kbase - lo;
      if (span < 0) { lo = 0x40000000; span = 0; }
#pragma unroll
      for (int b = 0; b < NBK; ++b) {
        if ((s == 0 && b == NBK - 1) || (s == 1 && b == 0)) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if ((unsigned)(16 * b + i - lo) > (unsigned)span) sc[s][b][i] = -INFINITY;
      }
    }
  }

  // per-strip row maximum, exponentials, P quads paired per key unit
  Oct pq[2][NU];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    float mloc = -INFINITY;
#pragma unroll
    for (int b = 0; b < NBK; ++b) {
      if ((s == 0 && b == NBK - 1) || (s == 1 && b == 0)) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) mloc = fmaxf(mloc, sc[s][b][i]);
    }
    const float m = col_max(mloc);
    const float ms = (m == -INFINITY ? 0.f : m) * scale2;
    uint2 qd[NBK];
#pragma unroll
    for (int b = 0; b < NBK; ++b) {
      if ((s == 0 && b == NBK - 1) || (s == 1 && b == 0)) {
        qd[b] = make_uint2(0, 0);
        continue;
      }
      float pv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[s][b][i], scale2, -ms));
      qd[b] = make_uint2(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]));
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) pq[s][u] = oct_of(qd[2 * u], qd[2 * u + 1]);
  }

  // O^T = V^T P^T and the row sums (ones block), V^T shared by both strips
  const Oct ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int nb = 0; nb <= NB; ++nb) o[s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < NU; ++u) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const Oct vt = oct_of(vt_quad<D>(vr, urow[u], nb), vt_quad<D>(vr, urow[u] + 16, nb));
      o[0][nb] = mma8(vt, pq[0][u], o[0][nb]);
      o[1][nb] = mma8(vt, pq[1][u], o[1][nb]);
    }
    o[0][NB] = mma8(ones, pq[0][u], o[0][NB]);
    o[1][NB] = mma8(ones, pq[1][u], o[1][NB]);
  }
}

// Far part and blend of both strips, then the store (Eq. (8)-(9), Eq. (11)).
template <int D, int R>
__device__ __forceinline__ void pair_far_store(bf16_t* __restrict__ oh, int i0, int N, float sn,
                                               float sfw, f32x4 (*o)[D / 16 + 1],
                                               Oct (*qo)[D / 32], const Oct* sf,
                                               Oct (*zo)[D / 32]) {
  constexpr int NB = D / 16, NQ = D / 32;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  // phi_1, phi_2 of the query octs (one exp(-|x|) serves both maps)
  Oct ph[R][2][NQ];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int p = 0; p < NQ; ++p) {
      float x[8], p1[8], p2[8];
      oct_unpack(qo[s][p], x);
#pragma unroll
      for (int i = 0; i < 8; ++i) phi12(x[i], p1[i], p2[i]);
      ph[0][s][p] = oct_pack(p1);
      if constexpr (R == 2) ph[1][s][p] = oct_pack(p2);
    }
  f32x4 fo[2][NB];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const float a = sn > 0.f ? sn * fast_rcp(o[s][NB][0]) : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) fo[s][nb] = o[s][nb] * a;
  }
#pragma unroll
  for (int l = 0; l < R; ++l) {
    f32x4 num[2][NB + 1];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < NQ; ++p) {
        const Oct f = sf[((l * NB + nb) * NQ + p) * 64 + lane];
        a0 = mma8(f, ph[l][0][p], a0);
        a1 = mma8(f, ph[l][1][p], a1);
      }
      num[0][nb] = a0;
      num[1][nb] = a1;
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f32x4 den = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < NQ; ++p) den = mma8(zo[l][p], ph[l][s][p], den);
      const float f = sfw > 0.f ? sfw * fast_rcp(den[0]) : 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fo[s][nb] += num[s][nb] * f;
    }
  }
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int row = i0 + 16 * s + r;
    if (row >= N) continue;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      *reinterpret_cast<uint2*>(oh + (size_t)row * D + 16 * nb + 4 * g) =
          make_uint2(pack_bf16x2(fo[s][nb][0], fo[s][nb][1]),
                     pack_bf16x2(fo[s][nb][2], fo[s][nb][3]));
  }
}

// grid.x = BH * nseg (XCD-aware remap); the workgroup walks the 128-row tiles
// of rows [s*L, min(N, s*L + L)), L a multiple of 128.  The window of the
// tile at t0 is the U units [t0/32 - KC, t0/32 + 4 + KC); unit ua0 + m lives
// in ring slot m % U, and the ring slides by four units per tile, the next
// four units and the next query rows prefetched into registers.
template <int D, int R, int KC>
__global__ __launch_bounds__(PNT) void k_band_pair(const bf16_t* __restrict__ q,
                                                   const bf16_t* __restrict__ k,
                                                   const bf16_t* __restrict__ v,
                                                   bf16_t* __restrict__ out,
                                                   const float* __restrict__ fin,
                                                   const float* __restrict__ w_near,
                                                   const float* __restrict__ w_far, int H, int N,
                                                   int band_k, int L, int nseg, float scale2) {
  using C = PairCfg<D, R, KC>;
  constexpr int NB = C::NB, NQ = C::NQ, U = C::U;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  unsigned char* kr = dyn_smem;
  unsigned char* vr = dyn_smem + C::RING;
  Oct* sf = reinterpret_cast<Oct*>(dyn_smem + 2 * C::RING);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const size_t base = (size_t)bh * N * D;
  const bf16_t* qh = q + base;
  const bf16_t* kh = k + base;
  const bf16_t* vh = v + base;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + PTM - 1) / PTM;
  const int ua0 = (s0 >> 5) - KC;

  Oct zo[R][NQ];
  pair_frags<D, R>(fin + (size_t)bh * R * D * (D + 1), sf, zo);
#pragma unroll
  for (int x = 0; x < U; x += 4) {
    PairCopy<D> ck, cv;
    ck.load(kh, (ua0 + x) * 32, N);
    cv.load(vh, (ua0 + x) * 32, N);
    auto slot = [=](int j) { return x + j < U ? x + j : -1; };
    ck.store(kr, slot);
    cv.store(vr, slot);
  }
  Oct qo[2][NQ], qn[2][NQ];
  load_qo<D>(qh, s0 + 32 * w, N, qo);
  PairCopy<D> pk, pv;
  if (ntile > 1) {
    pk.load(kh, (ua0 + U) * 32, N);
    pv.load(vh, (ua0 + U) * 32, N);
    load_qo<D>(qh, s0 + PTM + 32 * w, N, qn);
  }
  for (int t = 0; t < ntile; ++t) {
    __syncthreads();  // the ring holds the window of tile t
    const int i0 = s0 + t * PTM + 32 * w;
    const int slot0 = (4 * t + w) % U;
    f32x4 o[2][NB + 1];
    if (band_k == 32 * KC && i0 - band_k >= 0 && i0 + 31 + band_k < N)
      pair_near<D, R, KC, true>(o, qo, kr, vr, slot0, i0, N, band_k, scale2);
    else
      pair_near<D, R, KC, false>(o, qo, kr, vr, slot0, i0, N, band_k, scale2);
    pair_far_store<D, R>(out + base, i0, N, sn, sfw, o, qo, sf, zo);
    if (t + 1 < ntile) {
      __syncthreads();  // every wave is done with the window of tile t
      auto slot = [=](int j) { return (4 * t + j) % U; };
      pk.store(kr, slot);
      pv.store(vr, slot);
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int p = 0; p < NQ; ++p) qo[s][p] = qn[s][p];
      if (t + 2 < ntile) {
        pk.load(kh, (ua0 + U + 4 * (t + 1)) * 32, N);
        pv.load(vh, (ua0 + U + 4 * (t + 1)) * 32, N);
        load_qo<D>(qh, s0 + (t + 2) * PTM + 32 * w, N, qn);
      }
    }
  }
}

template <int D, int R, int KC>
hipError_t launch_pair_kc(const LaunchArgs& a, LaunchTimer* timer, const float* fin,
                          float scale2) {
  using C = PairCfg<D, R, KC>;
  static const hipError_t attr = [] {
    const hipError_t e = hipFuncSetAttribute((const void*)k_band_pair<D, R, KC>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    (void)hipGetLastError();
    return e;
  }();
  if (attr != hipSuccess) return attr;
  launch_timed(timer, FMM_KERNEL_BAND_APPLY, k_band_pair<D, R, KC>,
               dim3(a.B * a.H * a.nseg_apply), dim3(PNT), (size_t)C::LDS,
               (hipStream_t)a.stream, (const bf16_t*)a.q, (const bf16_t*)a.k,
               (const bf16_t*)a.v, (bf16_t*)a.out, fin, a.w_near, a.w_far, a.H, a.N, a.band_k,
               a.L_apply, a.nseg_apply, scale2);
  return hipGetLastError();
}

template <int D, int R>
hipError_t launch_pair_d(const LaunchArgs& a, LaunchTimer* t, const float* fin, float scale2) {
  return a.band_k <= 32 ? launch_pair_kc<D, R, 1>(a, t, fin, scale2)
                        : launch_pair_kc<D, R, 2>(a, t, fin, scale2);
}

}  // namespace

bool band_pair_applies(int dtype, int d, int band_k, int causal) {
  return dtype == FMM_DTYPE_BF16 && (d == 32 || d == 64) && band_k <= 64 && !causal;
}

int pair_tile_rows() { return PTM; }

hipError_t launch_band_pair(const LaunchArgs& a, LaunchTimer* t, const float* fin) {
  const float scale2 = 1.4426950408889634f / sqrtf((float)a.d);
  switch (a.d * 4 + a.rank) {
    case 32 * 4 + 1: return launch_pair_d<32, 1>(a, t, fin, scale2);
    case 32 * 4 + 2: return launch_pair_d<32, 2>(a, t, fin, scale2);
    case 64 * 4 + 1: return launch_pair_d<64, 1>(a, t, fin, scale2);
    case 64 * 4 + 2: return launch_pair_d<64, 2>(a, t, fin, scale2);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fmm
