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
// K and V rows sit unpadded in an LDS ring, their 16-byte chunks permuted per
// row so that the 16-byte K reads, the transposed 8-byte V reads and the row
// stores are free of bank conflicts.
#include <type_traits>

#include "fmm_device.h"
#include "fmm_launch.h"
#include "fmm_oct.h"
#include "fmm_xchg.h"

namespace fmm {
namespace {

constexpr int PW = 4;           // wavefronts per workgroup
constexpr int PNT = PW * 64;    // threads per workgroup
constexpr int PTM = 32 * PW;    // query rows per tile

template <int D, int R, int KC>
struct PairCfg {
  static constexpr int NB = D / 16, NQ = D / 32;
  static constexpr int U = 4 + 2 * KC;   // ring units of 32 keys: a tile's window
  static constexpr int NU = 2 * KC + 1;  // key units spanned by one wavefront's rows
  static constexpr int RING = U * 32 * RingRows<D>::RB;
  static constexpr int FRAG = R * NB * NQ * 64 * 16;
  static constexpr int LDS = 2 * RING + FRAG;
};

// State fragments from the non-causal tile-order record (see k_seg_state):
// sf[((l*NB + nb)*NQ + p)*64 + lane] holds S_l[32p + 8g + i][16nb + r],
// i = 0..7, as an oct; zo[l][p] holds z_l[32p + 8g + i].  load() issues every
// read of the record, store() packs and writes the fragments, so the
// workgroup's other prologue loads can be in flight in between.
template <int D, int R>
struct PairFrags {
  static constexpr int NB = D / 16, NQ = D / 32;
  static constexpr int TOT = R * NB * NQ * 64, IT = (TOT + PNT - 1) / PNT;
  float4 s[IT][2];
  float4 z[R][NQ][2];
  __device__ __forceinline__ void load(const float* __restrict__ rec) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * PNT;
      if (TOT % PNT != 0 && x >= TOT) break;
      const int ln = x & 63, blk = x >> 6;
      const int p = blk % NQ, nb = (blk / NQ) % NB, l = blk / (NQ * NB);
      const int gg = ln >> 4, rr = ln & 15;
      const int cb = 2 * p + (gg >> 1);
      const float* t0 = rec + (size_t)l * D * (D + 1) + ((cb * NB + nb) * 64 + 32 * (gg & 1) + rr) * 4;
      s[it][0] = *reinterpret_cast<const float4*>(t0);
      s[it][1] = *reinterpret_cast<const float4*>(t0 + 64);
    }
    const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
    for (int l = 0; l < R; ++l)
#pragma unroll
      for (int p = 0; p < NQ; ++p) {
        const float* zp = rec + (size_t)l * D * (D + 1) + D * D + 32 * p + 8 * g;
        z[l][p][0] = *reinterpret_cast<const float4*>(zp);
        z[l][p][1] = *reinterpret_cast<const float4*>(zp + 4);
      }
  }
  __device__ __forceinline__ void store(Oct* sf, Oct (*zo)[D / 32]) const {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int x = threadIdx.x + it * PNT;
      if (TOT % PNT != 0 && x >= TOT) break;
      const float f[8] = {s[it][0].x, s[it][0].y, s[it][0].z, s[it][0].w,
                          s[it][1].x, s[it][1].y, s[it][1].z, s[it][1].w};
      sf[x] = oct_pack(f);
    }
#pragma unroll
    for (int l = 0; l < R; ++l)
#pragma unroll
      for (int p = 0; p < NQ; ++p) {
        const float f[8] = {z[l][p][0].x, z[l][p][0].y, z[l][p][0].z, z[l][p][0].w,
                            z[l][p][1].x, z[l][p][1].y, z[l][p][1].z, z[l][p][1].w};
        zo[l][p] = oct_pack(f);
      }
  }
};

// One 128-row tile of a wavefront: both strips' banded softmax (Eq. (3)),
// far part (Eq. (8)-(9)), blend (Eq. (11)) and store.  The rows start at i0
// (a multiple of 32); key units u = 0 .. NU-1 (absolute unit i0/32 - KC + u)
// sit in ring slots (slot0 + u) % U.  Strip A (s = 0) never needs the last
// 16-key block of the span and strip B (s = 1) never the first, so strip s
// scores blocks s .. s + NBK - 2.  Exact tiles (!GENERAL: k = 32*KC and every
// wavefront's span inside [0, N)) have only the first and last block of each
// strip cut by the band (triangles); GENERAL tiles mask every block against
// the row's band clipped to [0, N).
//
// Every LDS operand is read once per wavefront and feeds both strips.  The
// work runs as phases separated by scheduling fences:
//   scores of A and B + phi(q) | softmax of A and B |
//   far products and P V of A and B (at a raised wave priority) |
//   near normalisation, blend, store
// mid() runs after the first phase, once phi(q) is formed.  With FAR_LAST
// the far products move behind the near field's P V product and
// normalisation, and pre_far() runs just before them: the state fragments
// (sf, zo) need to be in place only from then on.
struct NoStep {
  __device__ __forceinline__ void operator()() const {}
};

// Far part of both strips (Eq. (8)-(9), each map normalised on its own),
// each state fragment read once per map, added to fo with weight sfw.
template <int D, int R>
__device__ __forceinline__ void pair_far(const Oct* sf, Oct (*zo)[D / 32],
                                         Oct (*ph)[2][D / 32], float sfw,
                                         f32x4 (*fo)[D / 16]) {
  constexpr int NB = D / 16, NQ = D / 32;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int l = 0; l < R; ++l) {
    f32x4 nA[NB + 1], nB[NB + 1];
#pragma unroll
    for (int nb = 0; nb <= NB; ++nb) nA[nb] = nB[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < NQ; ++p) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const Oct f = sf[((l * NB + nb) * NQ + p) * 64 + lane];
        nA[nb] = mma8(f, ph[l][0][p], nA[nb]);
        nB[nb] = mma8(f, ph[l][1][p], nB[nb]);
      }
      nA[NB] = mma8(zo[l][p], ph[l][0][p], nA[NB]);
      nB[NB] = mma8(zo[l][p], ph[l][1][p], nB[NB]);
    }
    const float fa = sfw > 0.f ? sfw * fast_rcp(nA[NB][0]) : 0.f;
    const float fb = sfw > 0.f ? sfw * fast_rcp(nB[NB][0]) : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      fo[0][nb] += nA[nb] * fa;
      fo[1][nb] += nB[nb] * fb;
    }
  }
}

template <int D, int R, int KC, bool GENERAL, bool FAR_LAST = false, class Mid,
          class PreFar = NoStep>
__device__ __forceinline__ void pair_tile(Rsrc oh, int i0, int N, int band_k,
                                          float scale2, float sn, float sfw, Oct (*qo)[D / 32],
                                          const unsigned char* kr, const unsigned char* vr,
                                          int slot0, const RingOffsets<D>& ro, const Oct* sf,
                                          Oct (*zo)[D / 32], Mid mid, PreFar pre_far = {}) {
  using C = PairCfg<D, R, KC>;
  constexpr int NB = C::NB, NQ = C::NQ, NU = C::NU, NBK = 2 * NU, NS = NBK - 1;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  // byte offset of each key unit's first ring row (wave-uniform)
  int ubase[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u)
    ubase[u] = __builtin_amdgcn_readfirstlane(((slot0 + u) % C::U) * 32 * RingRows<D>::RB);
  const Oct ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);

  // Exact tiles: the band cuts the first block of each strip below the
  // diagonal offset (key offset 4g + i < r) and the last block above it; the
  // score products start from these -inf / 0 biases, so no mask is applied.
  f32x4 bias_lo, bias_hi;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bias_lo[i] = (!GENERAL && 4 * g + i < r) ? -INFINITY : 0.f;
    bias_hi[i] = (!GENERAL && 4 * g + i > r) ? -INFINITY : 0.f;
  }
  // band mask of the general tiles
  auto mask = [&](int s, f32x4* sc) {
    if constexpr (GENERAL) {
      const int kbase = (i0 / 32 - KC) * 32 + 4 * g;
      const int row = i0 + 16 * s + r;
      int lo = max(row - band_k, 0) - kbase;
      int span = min(row + band_k, N - 1) - kbase - lo;
      if (span < 0) { lo = 0x40000000; span = 0; }
#pragma unroll
      for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if ((unsigned)(16 * (j + s) + i - lo) > (unsigned)span) sc[j][i] = -INFINITY;
    }
  };
  // row maximum, exponentials; P quads paired per key unit
  auto softmax = [&](int s, f32x4* sc, Oct* pq) {
    float mloc = -INFINITY;
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) mloc = fmaxf(mloc, sc[j][i]);
    const float m = col_max(mloc);
    const float ms = (m == -INFINITY ? 0.f : m) * scale2;
    uint2 qd[NBK];
    qd[s == 0 ? NBK - 1 : 0] = make_uint2(0, 0);
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      float pv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[j][i], scale2, -ms));
      qd[j + s] = make_uint2(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]));
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) pq[u] = oct_of(qd[2 * u], qd[2 * u + 1]);
  };
  f32x4 scA[NS], scB[NS];
  Oct pqA[NU], pqB[NU];
  Oct ph[R][2][NQ];

  // ---- phase 1: scores of both strips, each key block read once (block b
  // is strip A's block b and strip B's block b - 1) | phi(q)
#pragma unroll
  for (int b = 0; b < NBK; ++b) {
    Oct ko[NQ];
#pragma unroll
    for (int p = 0; p < NQ; ++p)
      ko[p] = *reinterpret_cast<const Oct*>(kr + ubase[b >> 1] + ro.koff[p] +
                                            16 * RingRows<D>::RB * (b & 1));
    if (b < NS) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!GENERAL) acc = b == 0 ? bias_lo : b == NS - 1 ? bias_hi : acc;
#pragma unroll
      for (int p = 0; p < NQ; ++p) acc = mma8(ko[p], qo[0][p], acc);
      scA[b] = acc;
    }
    if (b >= 1) {
      const int j = b - 1;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!GENERAL) acc = j == 0 ? bias_lo : j == NS - 1 ? bias_hi : acc;
#pragma unroll
      for (int p = 0; p < NQ; ++p) acc = mma8(ko[p], qo[1][p], acc);
      scB[j] = acc;
    }
  }
  // phi_1, phi_2 of the query octs (one exp(-|x|) serves both maps)
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int p = 0; p < NQ; ++p) {
      Oct p2;
      phi_oct(qo[s][p], ph[0][s][p], p2);
      if constexpr (R == 2) ph[1][s][p] = p2;
    }
  __builtin_amdgcn_sched_barrier(0);
  // the query octs are dead: the caller's step between the phases (it
  // reloads them with the next tile's rows)
  mid();

  // ---- phase 2: band masks and softmax of both strips | far products of
  // both strips, each state fragment read once per map (each map normalised
  // on its own)
  mask(0, scA);
  mask(1, scB);
  softmax(0, scA, pqA);
  softmax(1, scB, pqB);
  __builtin_amdgcn_sched_barrier(0);
  // the far and P V products run at a raised wave priority, so the other
  // wavefront on the SIMD fills their shadow with its vector phases
  // (measured: 59.2 -> 57.2 us on the 2^16-token workload)
  __builtin_amdgcn_s_setprio(1);
  f32x4 fo[2][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) fo[0][nb] = fo[1][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (!FAR_LAST) pair_far<D, R>(sf, zo, ph, sfw, fo);
  __builtin_amdgcn_sched_barrier(0);

  // ---- phase 3: O^T = V^T P^T and the row sums of both strips, each value
  // unit read once; near normalisation and blend
  f32x4 oA[NB + 1], oB[NB + 1];
#pragma unroll
  for (int nb = 0; nb <= NB; ++nb) oA[nb] = oB[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < NU; ++u) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const unsigned char* vp = vr + ubase[u] + ro.voff[nb];
      const Oct vt = oct_of(ld_tr16(vp), ld_tr16(vp + 16 * RingRows<D>::RB));
      oA[nb] = mma8(vt, pqA[u], oA[nb]);
      oB[nb] = mma8(vt, pqB[u], oB[nb]);
    }
    oA[NB] = mma8(ones, pqA[u], oA[NB]);
    oB[NB] = mma8(ones, pqB[u], oB[NB]);
  }
  __builtin_amdgcn_s_setprio(0);
  {
    const float a0 = sn > 0.f ? sn * fast_rcp(oA[NB][0]) : 0.f;
    const float a1 = sn > 0.f ? sn * fast_rcp(oB[NB][0]) : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      fo[0][nb] += oA[nb] * a0;
      fo[1][nb] += oB[nb] * a1;
    }
  }
  if constexpr (FAR_LAST) {
    pre_far();
    pair_far<D, R>(sf, zo, ph, sfw, fo);
  }
  // rows at or beyond N fall outside the output buffer and are dropped
  for (int s = 0; s < 2; ++s) store_strip<D>(oh, i0 + 16 * s, fo[s]);
}

// grid.x = BH * nseg (XCD-aware remap); the workgroup walks the 128-row tiles
// of rows [s*L, min(N, s*L + L)), L a multiple of 128.  The window of the
// tile at t0 is the U units [t0/32 - KC, t0/32 + 4 + KC); unit ua0 + m lives
// in ring slot m % U, and the ring slides by four units per tile, the next
// four units and the next tile's query rows prefetched into registers a tile
// ahead.
template <int D, int R, int KC>
__global__ __launch_bounds__(PNT, 2) void k_band_pair(const bf16_t* __restrict__ q,
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
  const int hbytes = N * D * 2;
  const Rsrc qh = head_rsrc(q + base, hbytes), kh = head_rsrc(k + base, hbytes),
             vh = head_rsrc(v + base, hbytes), oh = head_rsrc(out + base, hbytes);
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + PTM - 1) / PTM;
  const int ua0 = (s0 >> 5) - KC;

  // prologue: every load (the ring's first window in rounds of four units,
  // the first query rows, the state record) is issued before the first LDS
  // store, so the workgroup waits for one round trip instead of several
  constexpr int NR = U / 4, UREM = U % 4;  // rounds of four units, then the rest
  static_assert(UREM == 0 || UREM == 2, "ring of 4 + 2 KC units");
  RowsCopy<D, PTM, PNT> rk[NR], rv[NR];
  RowsCopy<D, 32 * (UREM ? UREM : 2), PNT> tk, tv;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    rk[i].load(kh, (ua0 + 4 * i) * 32, true);
    rv[i].load(vh, (ua0 + 4 * i) * 32, true);
  }
  if constexpr (UREM != 0) {
    tk.load(kh, (ua0 + 4 * NR) * 32, true);
    tv.load(vh, (ua0 + 4 * NR) * 32, true);
  }
  Oct qo[2][NQ];
  load_qo<D, 2>(qh, s0 + 32 * w, true, qo);
  Oct zo[R][NQ];
  {
    PairFrags<D, R> fr;
    fr.load(fin + (size_t)bh * R * D * (D + 1));
    fr.store(sf, zo);
  }
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    auto slot = [=](int j) { return 4 * i + j; };
    rk[i].store(kr, slot);
    rv[i].store(vr, slot);
  }
  if constexpr (UREM != 0) {
    auto slot = [=](int j) { return 4 * NR + j; };
    tk.store(kr, slot);
    tv.store(vr, slot);
  }
  const RingOffsets<D> ro;
  RowsCopy<D, PTM, PNT> pk, pv;
  pk.load(kh, (ua0 + U) * 32, ntile > 1);
  pv.load(vh, (ua0 + U) * 32, ntile > 1);
  // one tile, then the ring slides by the four prefetched units (past the
  // last tile the loads and stores are harmless no-ops on zeros); the next
  // tile's query rows are loaded into the query registers as soon as phi(q)
  // has consumed them (separate prefetch registers cost more in register
  // pressure than the shorter lead costs in latency)
  auto step = [&](int t, auto general) {
    __syncthreads();  // the ring holds the window of tile t
    const int i0 = s0 + t * PTM + 32 * w;
    const int slot0 = (4 * t + w) % U;
    auto mid = [&]() { load_qo<D, 2>(qh, i0 + PTM, t + 1 < ntile, qo); };
    pair_tile<D, R, KC, decltype(general)::value>(oh, i0, N, band_k, scale2, sn, sfw, qo, kr, vr,
                                                  slot0, ro, sf, zo, mid);
    __syncthreads();  // every wave is done with the window of tile t
    auto slot = [=](int j) { return (4 * t + j) % U; };
    pk.store(kr, slot);
    pv.store(vr, slot);
    pk.load(kh, (ua0 + U + 4 * (t + 1)) * 32, t + 2 < ntile);
    pv.load(vh, (ua0 + U + 4 * (t + 1)) * 32, t + 2 < ntile);
  };
  // exact tiles: k = 32*KC and every row's band inside [0, N); they form one
  // contiguous run of the walk, between the leading and trailing general tiles
  const bool fit = band_k == 32 * KC;
  auto interior = [&](int t) {
    const int t0 = s0 + t * PTM;
    return fit && t0 - band_k >= 0 && t0 + PTM - 1 + band_k < N;
  };
  int t = 0;
  for (; t < ntile && !interior(t); ++t) step(t, std::true_type{});
  for (; t < ntile && interior(t); ++t) step(t, std::false_type{});
  for (; t < ntile; ++t) step(t, std::true_type{});
}

// ------------------------------------------------------------------ one launch for short slices
// For short sequences the three dependent launches of the state, its sum and
// the apply cost more than their bytes.  k_band_fused does all three in one
// launch: workgroup j of a (batch, head) slice owns rows [128 j, 128 j + 128)
// and, besides its tile of the operator, the partial far-field state of those
// rows.  The slice's G workgroups exchange their partial states through
// memory: each writes its record and then a stamp; once every stamp of the
// slice is there, workgroup j sums elements [j C, (j + 1) C) of the G records
// (C = ceil(rec / G)) in slice order and stamps again; once all of those are
// there, each reads the slice's total.  The tile's near field covers the
// waits: the first stamp goes out after the score phase (by when the
// record's stores have long reached L2), the first wait comes after the P V
// product.
//
// The exchange relies on the slice's workgroups sharing one L2: the grid is
// ordered so that each slice's workgroups are consecutive after xcd_remap,
// which places them on one XCD when B*H is a multiple of 8.  A record is
// written with ordinary stores and s_waitcnt vmcnt(0) (the stores have
// reached L2) precedes its stamp; stamps are written and polled with
// device-scope atomics (which bypass the vector L1; plain loads of a stamp
// can keep hitting a stale L1 line), and a workgroup reads the records only
// after it has seen their stamps, so no line of them is in its L1 before.  A
// stamp holds the launch's epoch and the XCC id of its writer.  The epoch
// differs from launch to launch, also between replays of a captured graph
// (it includes the dispatch id), so stamps left by an earlier launch in the
// same workspace never count as this launch's.  Any stamp from another XCC (or one
// marking a workgroup that gave up), or a wait beyond spin_limit polls, makes
// the workgroup compute its slice's total itself from K and V in memory: the
// same partial states (same products, same order) summed in the same order,
// so every path gives the same bits.  Waits are bounded, so the kernel always
// drains, and no workgroup's result depends on where its peers ran.


// Partial far-field state of the 128 keys r0 .. r0+127 held in ring slots
// slot0 .. slot0+3 (keys at or beyond N excluded): T_l = phi_l(K)^T [V | 1]
// for the feature block cb, in record order: acc[l][eb], lane (r, g) holds
// T_l[16cb + 4g + i][16eb + r]; acc[l][NB] (lanes r = 0) holds z_l[16cb + 4g
// + i].  The key operands are the transposed ring reads of the P V product,
// so phi_l(K)^T and [V | 1] share one key order.
template <int D, int R>
__device__ __forceinline__ void tile_state(const unsigned char* kr, const unsigned char* vr,
                                           int slot0, int r0, int N, const RingOffsets<D>& ro,
                                           int cb, f32x4 (*acc)[D / 16 + 1]) {
  constexpr int NB = D / 16, RB = RingRows<D>::RB;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const Oct onecol = r == 0 ? oct_ones() : make_uint4(0u, 0u, 0u, 0u);
  // the transposed read of columns 16cb .. 16cb+15 (RingOffsets::voff[cb],
  // formed here since cb is not a compile-time index)
  const int kcol = RingRows<D>::off(4 * g + (r >> 2), 2 * cb + ((r & 3) >> 1)) + 8 * (r & 1);
#pragma unroll
  for (int l = 0; l < R; ++l)
#pragma unroll
    for (int eb = 0; eb <= NB; ++eb) acc[l][eb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ub = (slot0 + u) * 32 * RB;
    const unsigned char* kp = kr + ub + kcol;
    Oct pk[2];
    phi_oct(oct_of(ld_tr16(kp), ld_tr16(kp + 16 * RB)), pk[0], pk[1]);
    // slot 2i (low half of word i) and 2i + 1 hold keys 4g + 2i, 4g + 2i + 1
    // (i < 2) or 16 + 4g + 2(i - 2), ... of the unit
    const int kvalid = N - (r0 + 32 * u);
    if (kvalid < 32) {
#pragma unroll
      for (int l = 0; l < R; ++l) {
        uint32_t wv[4] = {pk[l].x, pk[l].y, pk[l].z, pk[l].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k0 = i < 2 ? 4 * g + 2 * i : 16 + 4 * g + 2 * (i - 2);
          wv[i] &= (k0 < kvalid ? 0x0000ffffu : 0u) | (k0 + 1 < kvalid ? 0xffff0000u : 0u);
        }
        pk[l] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
      }
    }
#pragma unroll
    for (int eb = 0; eb < NB; ++eb) {
      const unsigned char* vp = vr + ub + ro.voff[eb];
      const Oct vt = oct_of(ld_tr16(vp), ld_tr16(vp + 16 * RB));
#pragma unroll
      for (int l = 0; l < R; ++l) acc[l][eb] = mma8(pk[l], vt, acc[l][eb]);
    }
#pragma unroll
    for (int l = 0; l < R; ++l) acc[l][NB] = mma8(pk[l], onecol, acc[l][NB]);
  }
}

// The tiles of feature block cb in a state record (the layout k_seg_state writes).
template <int D, int R>
__device__ __forceinline__ void store_record_block(float* rec, int cb,
                                                   const f32x4 (*acc)[D / 16 + 1]) {
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int l = 0; l < R; ++l) {
    float* sl = rec + (size_t)l * D * (D + 1);
#pragma unroll
    for (int eb = 0; eb < NB; ++eb)
      *reinterpret_cast<f32x4*>(sl + ((cb * NB + eb) * 64 + lane) * 4) = acc[l][eb];
    if (r == 0) *reinterpret_cast<f32x4*>(sl + D * D + 16 * cb + 4 * g) = acc[l][NB];
  }
}


// grid.x = BH * G, G = ceil(N / 128) <= 64.  part: G records per slice; tot:
// one record per slice; stamp: 2 G per slice.  exchange = 0 skips the exchange
// (every workgroup computes its slice's total itself).
template <int D, int R, int KC>
__global__ __launch_bounds__(PNT, 2) void k_band_fused(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    bf16_t* __restrict__ out, float* __restrict__ part, float* __restrict__ tot,
    unsigned long long* __restrict__ stamp, const float* __restrict__ w_near,
    const float* __restrict__ w_far, int H, int N, int band_k, int G, float scale2,
    unsigned long long host_epoch, int spin_limit, int exchange) {
  using C = PairCfg<D, R, KC>;
  constexpr int NB = C::NB, NQ = C::NQ, U = C::U;
  constexpr int REC = R * D * (D + 1);
  static_assert(REC * 4 <= 2 * C::RING, "the ring holds a record in the fallback");
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  unsigned char* kr = dyn_smem;
  unsigned char* vr = dyn_smem + C::RING;
  Oct* sf = reinterpret_cast<Oct*>(dyn_smem + 2 * C::RING);
  // the waits' flag lives in the ring once the near field is done with it
  // (a static LDS word would take d = 64 past two workgroups per CU)
  int* s_flag = reinterpret_cast<int*>(dyn_smem);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / G, j = lin % G, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const size_t base = (size_t)bh * N * D;
  const int hbytes = N * D * 2;
  const Rsrc qh = head_rsrc(q + base, hbytes), kh = head_rsrc(k + base, hbytes),
             vh = head_rsrc(v + base, hbytes), oh = head_rsrc(out + base, hbytes);
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int t0 = j * PTM;
  const int ua0 = (t0 >> 5) - KC;

  // the tile's window: units ua0 + m in ring slot m; the wavefront's query
  // rows (every load issued before the first LDS store)
  constexpr int NR = U / 4, UREM = U % 4;
  static_assert(UREM == 0 || UREM == 2, "ring of 4 + 2 KC units");
  Oct qo[2][NQ];
  {
    RowsCopy<D, PTM, PNT> rk[NR], rv[NR];
    RowsCopy<D, 32 * (UREM ? UREM : 2), PNT> tk, tv;
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      rk[i].load(kh, (ua0 + 4 * i) * 32, true);
      rv[i].load(vh, (ua0 + 4 * i) * 32, true);
    }
    if constexpr (UREM != 0) {
      tk.load(kh, (ua0 + 4 * NR) * 32, true);
      tv.load(vh, (ua0 + 4 * NR) * 32, true);
    }
    load_qo<D, 2>(qh, t0 + 32 * w, true, qo);
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      auto slot = [=](int jj) { return 4 * i + jj; };
      rk[i].store(kr, slot);
      rv[i].store(vr, slot);
    }
    if constexpr (UREM != 0) {
      auto slot = [=](int jj) { return 4 * NR + jj; };
      tk.store(kr, slot);
      tv.store(vr, slot);
    }
  }
  __syncthreads();
  const RingOffsets<D> ro;
  const unsigned long long epoch = launch_epoch(host_epoch);
  const unsigned long long mine = (epoch << 8) | xcc_id();
  unsigned long long* st = stamp + (size_t)bh * G * 2;
  float* prec = part + (size_t)bh * G * REC;
  float* trec = tot + (size_t)bh * REC;

  // the partial state of the tile's own 128 keys (ring slots KC .. KC+3);
  // its stamp follows the near field's first phase, by when the stores have
  // long reached L2, so no wave stalls on them
  if (exchange && w < NB) {
    f32x4 acc[R][NB + 1];
    tile_state<D, R>(kr, vr, KC, t0, N, ro, w, acc);
    store_record_block<D, R>(prec + (size_t)j * REC, w, acc);
  }
  auto publish = [&]() {
    if (exchange) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the record is in L2
      __syncthreads();
      if (threadIdx.x == 0) put_stamp(st + 2 * j, mine);
    }
  };

  Oct zo[R][NQ];
  auto pre_far = [&]() {
    __syncthreads();  // every wave is done with the ring
    bool ok = exchange != 0 && wait_stamps(st, 2, 0, G, epoch, mine, spin_limit, s_flag);
    if (ok) {
      // elements [e0, e0 + cnt) of the G records: every value loaded at
      // once (flat index f = i CH + el, record i, element e0 + el), staged
      // in LDS, then each element summed over the records in slice order
      const int CH = (REC + G - 1) / G;
      const int e0 = j * CH, cnt = min(CH, REC - e0), nflat = G * CH;
      // i = f / CH as umulhi(f, M), exact for f, CH < 2^16
      const unsigned M = 0xffffffffu / (unsigned)CH + 1u;
      const Rsrc ph = __builtin_amdgcn_make_buffer_rsrc(prec, 0, G * REC * 4, 0x00020000);
      constexpr int IT = (REC + 63 + PNT - 1) / PNT;  // G CH < REC + G <= REC + 64
      float* stage = reinterpret_cast<float*>(dyn_smem + 256);  // past the flag
      static_assert(256 + 4 * (REC + 64) <= 2 * C::RING, "staging fits the ring");
      float x[IT];
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const unsigned f = threadIdx.x + PNT * it;
        const unsigned i = __umulhi(f, M), el = f - i * CH;
        const bool on = (int)f < nflat && (int)el < cnt;
        x[it] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(ph, on ? 4 * (i * REC + e0 + el) : OOB,
                                                        0, 0));
      }
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int f = threadIdx.x + PNT * it;
        if (f < nflat) stage[f] = x[it];
      }
      __syncthreads();
      for (int el = threadIdx.x; el < cnt; el += PNT) {
        float sum = 0.f;
#pragma unroll 8
        for (int i = 0; i < G; ++i) sum += stage[i * CH + el];
        trec[e0 + el] = sum;
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (threadIdx.x == 0) put_stamp(st + 2 * j + 1, mine);
      ok = wait_stamps(st, 2, 1, G, epoch, mine, spin_limit, s_flag);
    } else if (exchange && threadIdx.x == 0) {
      // peers waiting for this workgroup's sum stop waiting
      put_stamp(st + 2 * j + 1, (epoch << 8) | kGaveUp);
    }
    if (ok) {
      PairFrags<D, R> fr;
      fr.load(trec);
      fr.store(sf, zo);
    } else {
      // the slice's total from K and V in memory: each tile's partial state
      // as its own workgroup forms it, added in slice order
      f32x4 tacc[R][NB + 1];
#pragma unroll
      for (int l = 0; l < R; ++l)
#pragma unroll
        for (int eb = 0; eb <= NB; ++eb) tacc[l][eb] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int i = 0; i < G; ++i) {
        RowsCopy<D, PTM, PNT> fk, fv;
        fk.load(kh, i * PTM, true);
        fv.load(vh, i * PTM, true);
        __syncthreads();  // the ring is free (the previous tile's products are done)
        auto slot = [](int jj) { return jj; };
        fk.store(kr, slot);
        fv.store(vr, slot);
        __syncthreads();
        if (w < NB) {
          f32x4 pacc[R][NB + 1];
          tile_state<D, R>(kr, vr, 0, i * PTM, N, ro, w, pacc);
#pragma unroll
          for (int l = 0; l < R; ++l)
#pragma unroll
            for (int eb = 0; eb <= NB; ++eb) tacc[l][eb] += pacc[l][eb];
        }
      }
      __syncthreads();
      float* lrec = reinterpret_cast<float*>(dyn_smem);
      if (w < NB) store_record_block<D, R>(lrec, w, tacc);
      __syncthreads();
      PairFrags<D, R> fr;
      fr.load(lrec);
      fr.store(sf, zo);
    }
    __syncthreads();  // the fragments are in place
  };
  const int i0 = t0 + 32 * w;
  const bool exact = band_k == 32 * KC && t0 - band_k >= 0 && t0 + PTM - 1 + band_k < N;
  if (exact)
    pair_tile<D, R, KC, false, true>(oh, i0, N, band_k, scale2, sn, sfw, qo, kr, vr, w, ro, sf,
                                     zo, publish, pre_far);
  else
    pair_tile<D, R, KC, true, true>(oh, i0, N, band_k, scale2, sn, sfw, qo, kr, vr, w, ro, sf,
                                    zo, publish, pre_far);
}

template <int D, int R, int KC>
hipError_t launch_fused_kc(const LaunchArgs& a, Launcher& L, float scale2) {
  using C = PairCfg<D, R, KC>;
  static std::atomic<unsigned long long> lds_set{0};
  if (L.note(lds_limit_once((const void*)k_band_fused<D, R, KC>, C::LDS, lds_set)) !=
      hipSuccess)
    return L.err;
  const int BH = a.B * a.H, G = a.fused_g;
  const FusedLayout f = fused_layout(BH, G, R * D * (D + 1));
  // (integer arithmetic: the dry pass runs with no workspace yet)
  const uintptr_t ws = reinterpret_cast<uintptr_t>(a.ws);
  L(FMM_KERNEL_BAND_APPLY, k_band_fused<D, R, KC>, dim3(BH * G), dim3(PNT), (size_t)C::LDS,
    (hipStream_t)a.stream, (const bf16_t*)a.q, (const bf16_t*)a.k, (const bf16_t*)a.v,
    (bf16_t*)a.out, reinterpret_cast<float*>(ws + f.off_part),
    reinterpret_cast<float*>(ws + f.off_tot),
    reinterpret_cast<unsigned long long*>(ws + f.off_stamp), a.w_near, a.w_far, a.H, a.N,
    a.band_k, G, scale2, a.epoch, kFusedSpinLimit, a.exchange);
  return L.err;
}

template <int D, int R, int KC>
hipError_t launch_pair_kc(const LaunchArgs& a, Launcher& L, const float* fin,
                          float scale2) {
  using C = PairCfg<D, R, KC>;
  static std::atomic<unsigned long long> lds_set{0};
  if (L.note(lds_limit_once((const void*)k_band_pair<D, R, KC>, C::LDS, lds_set)) != hipSuccess)
    return L.err;
  L(FMM_KERNEL_BAND_APPLY, k_band_pair<D, R, KC>,
               dim3(a.B * a.H * a.nseg_apply), dim3(PNT), (size_t)C::LDS,
               (hipStream_t)a.stream, (const bf16_t*)a.q, (const bf16_t*)a.k,
               (const bf16_t*)a.v, (bf16_t*)a.out, fin, a.w_near, a.w_far, a.H, a.N, a.band_k,
               a.L_apply, a.nseg_apply, scale2);
  return L.err;
}

template <int D, int R>
hipError_t launch_pair_d(const LaunchArgs& a, Launcher& t, const float* fin, float scale2) {
  return a.band_k <= 32 ? launch_pair_kc<D, R, 1>(a, t, fin, scale2)
                        : launch_pair_kc<D, R, 2>(a, t, fin, scale2);
}

}  // namespace

bool band_pair_applies(int dtype, int d, int band_k, int causal, long long n) {
  // 32-bit buffer offsets: one head's rows must stay below 2 GiB
  return dtype == FMM_DTYPE_BF16 && (d == 32 || d == 64) && band_k <= 64 && !causal &&
         n * d * 2 < (1LL << 31);
}

int fused_groups(int dtype, int d, int band_k, int rank, int causal, long long bh, long long n,
                 int max_workgroups) {
  // one or two maps (the pair kernel's tile); B*H a multiple of 8, so that
  // each slice's workgroups share an XCD; at most 64 tiles per slice (one
  // wave polls the stamps); every workgroup resident at once (two per CU)
  if (!band_pair_applies(dtype, d, band_k, causal, n) || rank > 2 || bh % 8 != 0 || n < 1)
    return 0;
  const long long G = (n + PTM - 1) / PTM;
  if (G > 64 || bh * G > max_workgroups) return 0;
  return (int)G;
}

int pair_tile_rows() { return PTM; }

hipError_t launch_band_fused(const LaunchArgs& a, Launcher& t) {
  const float scale2 = 1.4426950408889634f / sqrtf((float)a.d);
  const bool kc1 = a.band_k <= 32;
  switch (a.d * 4 + a.rank) {
    case 32 * 4 + 1:
      return kc1 ? launch_fused_kc<32, 1, 1>(a, t, scale2) : launch_fused_kc<32, 1, 2>(a, t, scale2);
    case 32 * 4 + 2:
      return kc1 ? launch_fused_kc<32, 2, 1>(a, t, scale2) : launch_fused_kc<32, 2, 2>(a, t, scale2);
    case 64 * 4 + 1:
      return kc1 ? launch_fused_kc<64, 1, 1>(a, t, scale2) : launch_fused_kc<64, 1, 2>(a, t, scale2);
    case 64 * 4 + 2:
      return kc1 ? launch_fused_kc<64, 2, 1>(a, t, scale2) : launch_fused_kc<64, 2, 2>(a, t, scale2);
    default: return t.note(hipErrorInvalidValue);
  }
}

hipError_t launch_band_pair(const LaunchArgs& a, Launcher& t, const float* fin) {
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
