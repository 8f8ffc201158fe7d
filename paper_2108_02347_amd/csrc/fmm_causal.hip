// Causal FMMformer apply for bf16 heads of width 32 or 64 and band
// half-widths up to 64, one 16-row strip per wavefront.
//
// k_causal_strip walks the 64-row tiles of a state segment in order, with the
// running far-field sums of the keys before the current tile (the prefix form
// of Eq. (9): S_l = sum_j phi_l(k_j) v_j^T and z_l = sum_j phi_l(k_j)) in
// registers.  Per tile, each of the four wavefronts takes a strip of 16 query
// rows i and computes
//   near: softmax over the causal band [i - k, i] (Eq. (3)),
//   far:  phi_l(q_i) . S_l(i) / phi_l(q_i) . z_l(i) with the sums over keys
//         [0, i]: the sums at the tile start (fragments in LDS) plus the
//         tile's own keys up to the row (an explicit lower-triangular
//         product phi_l(q) phi_l(K)^T [V | 1]),
//   the blend of Eq. (11) and the store;
// then the sums advance by the tile's 64 keys.
//
// K and V rows sit in a swizzled LDS ring like the paired-strip kernel's, the
// tile's phi_l(K) rows in the same row layout: the intra-tile scores read them
// as octs (like K rows), the state update reads them transposed (like V rows).
// The state is held as tiles whose feature order makes every pair of tiles one
// oct per lane, so a tile's packed sums are stored straight into the
// fragments the far product reads.
#include <type_traits>

#include "fmm_device.h"
#include "fmm_launch.h"
#include "fmm_oct.h"

namespace fmm {
namespace {

constexpr int CW = 4;          // wavefronts per workgroup
constexpr int CNT = CW * 64;   // threads per workgroup
constexpr int CTM = 16 * CW;   // query rows (and keys) per tile

template <int D, int R, int KC>
struct CausalCfg {
  static constexpr int NB = D / 16, NQ = D / 32;
  static constexpr int U = 2 + KC;        // ring units of 32 keys: a tile's window
  static constexpr int NS = 2 * KC + 1;   // 16-key blocks of one strip's band
  static constexpr int RB = RingRows<D>::RB;
  static constexpr int RING = U * 32 * RB;
  static constexpr int PHI = CTM * RB;    // one map's phi rows of the tile's keys
  static constexpr int FRAG = R * NB * NQ * 64 * 16;
  static constexpr int ZO = R * NQ * 4 * 16;
  static constexpr int LDS = 2 * RING + R * PHI + FRAG + ZO;
};

// The running sums of the walk, T_l = phi_l(K)^T [V | 1], as 16x16 fp32 tiles
// spread over the wavefronts.  Feature tile (l, p, h) covers the features
// f(4q + i) = 32p + 8q + 4((q & 1) ^ h) + i, q, i = 0..3, so lane (e, g) of its
// column block eb holds S_l[32p + 8g + 4((g & 1) ^ h) + {0..3}][16eb + e]: the
// h = 0 and h = 1 tiles of (l, p) are the two halves of lane (e, g)'s oct of
// the far product's fragment (in swapped order for odd g), and their
// transposed phi-row reads alternate between the chunk halves, which keeps
// those reads free of bank conflicts.  Column block NB is the ones column:
// every lane holds z_l at the same features.
template <int D, int R>
struct CausalState {
  static constexpr int NB = D / 16, NQ = D / 32;
  static constexpr int FT = R * NQ * 2;                 // feature tiles
  static constexpr int AG = FT >= CW ? FT / CW : 1;     // tiles per wavefront
  static_assert(AG <= 2, "a wavefront holds at most the two halves of one oct");
  f32x4 acc[AG][NB + 1];
  int aoff[AG];  // transposed phi-row read of each tile (lane offset, map base)

  // Wavefronts beyond the FT tiles (d = 32, rank 1) repeat the first ones:
  // they load, update and pack their copies like the owners, so no branch
  // separates the update's matrix-core products from the vector code that
  // follows, and only their fragment stores are skipped.
  __device__ __forceinline__ static bool active(int w) { return w * AG < FT; }
  __device__ __forceinline__ static void tile_of(int w, int a, int& l, int& p, int& h) {
    const int ft = (w * AG + a) % FT;
    h = ft & 1;
    p = (ft >> 1) % NQ;
    l = (ft >> 1) / NQ;
  }

  // Sums from a tile-order record (see k_seg_state: tile (cb, eb) lane
  // (g, e) holds S_l[16cb + 4g + {0..3}][16eb + e]; z_l at offset D*D).
  __device__ __forceinline__ void load(int w, const float* __restrict__ rec) {
    const int lane = threadIdx.x & 63, e = lane & 15, g = lane >> 4, t = lane & 15;
#pragma unroll
    for (int a = 0; a < AG; ++a) {
      int l, p, h;
      tile_of(w, a, l, p, h);
      const float* sl = rec + (size_t)l * D * (D + 1);
      const int hq = (g & 1) ^ h;
      const int cb = 2 * p + (g >> 1), gp = (2 * g + hq) & 3;
#pragma unroll
      for (int eb = 0; eb < NB; ++eb)
        acc[a][eb] = *reinterpret_cast<const f32x4*>(sl + ((cb * NB + eb) * 64 + gp * 16 + e) * 4);
      acc[a][NB] = *reinterpret_cast<const f32x4*>(sl + D * D + 32 * p + 8 * g + 4 * hq);
      // lane t of group g reads key 4g + t/4, features 32p + 8(t%4) + 4((t%2) ^ h) .. +3
      aoff[a] = l * CTM * RingRows<D>::RB + RingRows<D>::off(4 * g + (t >> 2), 4 * p + (t & 3)) +
                8 * ((t & 1) ^ h);
    }
  }

  // acc += phi_l(K_u)^T [V_u | 1] over key unit u (32 keys) of the tile: phi
  // rows at phr, vt[eb] the unit's V^T octs (columns 16eb .. 16eb+15).
  __device__ __forceinline__ void add_unit(const unsigned char* phr, int u, const Oct* vt) {
    constexpr int RB = RingRows<D>::RB;
    const Oct ones = oct_ones();
#pragma unroll
    for (int a = 0; a < AG; ++a) {
      const unsigned char* pp = phr + 32 * u * RB + aoff[a];
      const Oct ao = oct_of(ld_tr16(pp), ld_tr16(pp + 16 * RB));
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) acc[a][eb] = mma8(ao, vt[eb], acc[a][eb]);
      acc[a][NB] = mma8(ao, ones, acc[a][NB]);
    }
  }

  struct Frags {
    uint2 q[AG][NB + 1];
  };
  __device__ __forceinline__ Frags pack() const {
    Frags f;
#pragma unroll
    for (int a = 0; a < AG; ++a)
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb) f.q[a][eb] = quad_pack(acc[a][eb]);
    return f;
  }
  // Fragments of the far product: sf[((l*NB + nb)*NQ + p)*64 + lane] is lane
  // (e, g)'s oct S_l[32p + 8g + {0..7}][16nb + e]; szo[(l*NQ + p)*4 + g] is
  // z_l[32p + 8g + {0..7}].
  __device__ __forceinline__ static void store(int w, const Frags& f, Oct* sf, Oct* szo) {
    const int lane = threadIdx.x & 63, e = lane & 15, g = lane >> 4;
    // tile h holds the first half of lane (e, g)'s oct when (g & 1) == h: each
    // half goes to its place with an 8-byte store (no lane-dependent select)
#pragma unroll
    for (int a = 0; a < AG; ++a) {
      int l, p, h;
      tile_of(w, a, l, p, h);
      const int hb = 8 * ((g & 1) ^ h);
#pragma unroll
      for (int eb = 0; eb < NB; ++eb)
        *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(
                                      sf + ((l * NB + eb) * NQ + p) * 64 + lane) + hb) = f.q[a][eb];
      if (e == 0)
        *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(szo + (l * NQ + p) * 4 + g) +
                                  hb) = f.q[a][NB];
    }
  }
};

// phi_l of the tile's 64 key rows from the registers of a RowsCopy (thread x
// holds chunk x % CPR of row x / CPR + it * (CNT / CPR)), stored in the ring
// row layout, map l at byte offset l * CTM * RB.
template <int D, int R>
struct PhiRows {
  using RC = RowsCopy<D, CTM, CNT>;
  Oct v[R][RC::IT];
  __device__ __forceinline__ void compute(const RC& ck) {
#pragma unroll
    for (int it = 0; it < RC::IT; ++it) {
      Oct p2;
      phi_oct(ck.r[it], v[0][it], p2);
      if constexpr (R == 2) v[1][it] = p2;
    }
  }
  __device__ __forceinline__ void store(unsigned char* phr) const {
#pragma unroll
    for (int it = 0; it < RC::IT; ++it) {
      const int x = threadIdx.x + it * CNT;
      const int o = RingRows<D>::off(x / RC::CPR, x % RC::CPR);
#pragma unroll
      for (int l = 0; l < R; ++l)
        *reinterpret_cast<Oct*>(phr + l * CTM * RingRows<D>::RB + o) = v[l][it];
    }
  }
};

// One tile of a wavefront: the strip rows i0 .. i0+15 (i0 = t0 + 16w).  The
// ring holds the window units [t0/32 - KC, t0/32 + 2), window unit m in ring
// slot (m0 + m) % U; window block j (16 keys) is unit j/2, half j%2.  The
// strip's band is window blocks w .. w + 2KC.  Exact tiles (!GENERAL: k =
// 32*KC and the whole window inside [0, N)) cut only the first block (keys
// below i - k) and the last (keys above i) and start those score products from
// -inf biases; GENERAL tiles mask every block against the band clipped to
// [0, N).  The intra-tile product runs over the tile's four blocks in two
// pairs for every strip, tmask[j] masking tile block j: kept below the
// strip's own block w, lower-triangular on it, empty above it (the strips of
// the tile's first half thus spend products on an empty pair, which keeps
// every wavefront on one straight-line path; they would otherwise wait for
// the others at the next barrier).
//
// The near and far parts are independent until the blend, so the work runs
// as phases that pair matrix-core products of one part with vector
// arithmetic of the other (scheduling fences keep the phases apart):
//   1: near scores + phi(q)
//   2: softmax + far products of both maps with the sums before the tile
//   3: P V + intra-tile scores of both maps (masked, packed)
//   4: per tile key unit, its V^T octs read once for the intra-tile far
//      products of both maps and the running sums' update (unit()), beside
//      phi of the next tile's keys (late())
//   then near normalisation, blend, store.
// mid() runs once phi(q) is formed (the query octs are dead then).
template <int D, int R, int KC, bool GENERAL, class Mid, class Unit, class Late>
__device__ __forceinline__ void tile_work(Rsrc oh, int t0, int w, int m0, int N, int band_k,
                                          float scale2, float sn, float sfw, const Oct* qo,
                                          const unsigned char* kr, const unsigned char* vr,
                                          const unsigned char* phr, const RingOffsets<D>& ro,
                                          const Oct* sf, const Oct* szo, const uint2* tmask,
                                          Mid mid, Unit unit, Late late) {
  using C = CausalCfg<D, R, KC>;
  constexpr int NB = C::NB, NQ = C::NQ, NS = C::NS, RB = C::RB, U = C::U;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int i0 = t0 + 16 * w;
  const Oct ones = oct_ones();
  auto wblock = [&](int j) {  // ring byte offset of window block j (wave-uniform)
    return __builtin_amdgcn_readfirstlane(((m0 + (j >> 1)) % U) * 32 * RB + (j & 1) * 16 * RB);
  };
  int kb[NS];
#pragma unroll
  for (int b = 0; b < NS; ++b) kb[b] = wblock(w + b);
  int tb[4];  // tile blocks 0..3 are window blocks 2KC..2KC+3
#pragma unroll
  for (int j = 0; j < 4; ++j) tb[j] = wblock(2 * KC + j);

  // ---- phase 1: near scores S^T = K Q^T over the strip's NS blocks | phi(q)
  f32x4 sc[NS];
  {
    f32x4 bias_lo, bias_hi;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bias_lo[i] = (!GENERAL && 4 * g + i < r) ? -INFINITY : 0.f;
      bias_hi[i] = (!GENERAL && 4 * g + i > r) ? -INFINITY : 0.f;
    }
#pragma unroll
    for (int b = 0; b < NS; ++b) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!GENERAL) acc = b == 0 ? bias_lo : b == NS - 1 ? bias_hi : acc;
#pragma unroll
      for (int p = 0; p < NQ; ++p)
        acc = mma8(*reinterpret_cast<const Oct*>(kr + kb[b] + ro.koff[p]), qo[p], acc);
      sc[b] = acc;
    }
  }
  Oct ph[R][NQ];
#pragma unroll
  for (int p = 0; p < NQ; ++p) {
    Oct p2;
    phi_oct(qo[p], ph[0][p], p2);
    if constexpr (R == 2) ph[1][p] = p2;
  }
  __builtin_amdgcn_sched_barrier(0);

  // Phases 2-4 carry most of the tile's matrix-core products and run at a
  // raised wave priority: the other wavefront on the SIMD is then usually in
  // phase 1, the store or phi of the next keys (vector work), so the arbiter
  // keeps the matrix pipe fed and fills its shadow with that vector work
  // (measured: 81.5 -> 77.7 us on the 2^16-token causal workload).
  __builtin_amdgcn_s_setprio(1);
  // ---- phase 2: softmax numerators | far products with the sums before the
  // tile (Eq. (9) numerator and denominator)
  mid();
  if constexpr (GENERAL) {
    const int kbase = i0 - 32 * KC + 4 * g;
    const int row = i0 + r;
    int lo = max(row - band_k, 0) - kbase;
    int span = min(row, N - 1) - kbase - lo;
    if (span < 0) { lo = 0x40000000; span = 0; }
#pragma unroll
    for (int b = 0; b < NS; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((unsigned)(16 * b + i - lo) > (unsigned)span) sc[b][i] = -INFINITY;
  }
  uint2 pq[NS + 1];
  {
    float mloc = -INFINITY;
#pragma unroll
    for (int b = 0; b < NS; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) mloc = fmaxf(mloc, sc[b][i]);
    const float m = col_max(mloc);
    const float ms = (m == -INFINITY ? 0.f : m) * scale2;
#pragma unroll
    for (int b = 0; b < NS; ++b) {
      f32x4 pv;
#pragma unroll
      for (int i = 0; i < 4; ++i) pv[i] = __builtin_amdgcn_exp2f(fmaf(sc[b][i], scale2, -ms));
      pq[b] = quad_pack(pv);
    }
    pq[NS] = make_uint2(0u, 0u);
  }
  // far products of both maps with the sums before the tile (Eq. (9)
  // numerator and denominator)
  f32x4 num[R][NB + 1];
#pragma unroll
  for (int l = 0; l < R; ++l) {
#pragma unroll
    for (int nb = 0; nb <= NB; ++nb) num[l][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < NQ; ++p) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        num[l][nb] = mma8(sf[((l * NB + nb) * NQ + p) * 64 + lane], ph[l][p], num[l][nb]);
      num[l][NB] = mma8(szo[(l * NQ + p) * 4 + g], ph[l][p], num[l][NB]);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- phase 3: O^T = V^T P^T and the row sums | intra-tile scores
  // phi_l(K) phi_l(q)^T of both maps over the tile's blocks in two pairs,
  // masked to keys t0 .. i (tile blocks 0 .. w, block w lower-triangular)
  f32x4 o[NB + 1];
#pragma unroll
  for (int nb = 0; nb <= NB; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < (NS + 1) / 2; ++c) {
    const Oct pc = oct_of(pq[2 * c], pq[2 * c + 1]);
    const bool two = 2 * c + 1 < NS;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const uint2 v0 = ld_tr16(vr + kb[2 * c] + ro.voff[nb]);
      const uint2 v1 = two ? ld_tr16(vr + kb[2 * c + 1] + ro.voff[nb]) : make_uint2(0u, 0u);
      o[nb] = mma8(oct_of(v0, v1), pc, o[nb]);
    }
    o[NB] = mma8(ones, pc, o[NB]);
  }
  Oct ac[R][2];
#pragma unroll
  for (int l = 0; l < R; ++l) {
    const unsigned char* pl = phr + l * CTM * RB;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < NQ; ++p) {
        a0 = mma8(*reinterpret_cast<const Oct*>(pl + 32 * c * RB + ro.koff[p]), ph[l][p], a0);
        a1 = mma8(*reinterpret_cast<const Oct*>(pl + (32 * c + 16) * RB + ro.koff[p]), ph[l][p],
                  a1);
      }
      uint2 q0 = quad_pack(a0), q1 = quad_pack(a1);
      q0.x &= tmask[2 * c].x; q0.y &= tmask[2 * c].y;
      q1.x &= tmask[2 * c + 1].x; q1.y &= tmask[2 * c + 1].y;
      ac[l][c] = oct_of(q0, q1);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- phase 4: per key unit c of the tile, its V^T octs are read once and
  // feed the intra-tile far products of both maps and the running sums'
  // update (the caller's) | phi of the next tile's keys (the caller's),
  // near normalisation, blend
  late();
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    Oct vt[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      vt[nb] = oct_of(ld_tr16(vr + tb[2 * c] + ro.voff[nb]),
                      ld_tr16(vr + tb[2 * c + 1] + ro.voff[nb]));
#pragma unroll
    for (int l = 0; l < R; ++l) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) num[l][nb] = mma8(vt[nb], ac[l][c], num[l][nb]);
      num[l][NB] = mma8(ones, ac[l][c], num[l][NB]);
    }
    unit(c, vt);
  }
  __builtin_amdgcn_s_setprio(0);
  f32x4 fo[NB];
  {
    const float a = sn > 0.f ? sn * fast_rcp(o[NB][0]) : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) fo[nb] = o[nb] * a;
  }
#pragma unroll
  for (int l = 0; l < R; ++l) {
    const float f = sfw > 0.f ? sfw * fast_rcp(num[l][NB][0]) : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) fo[nb] += num[l][nb] * f;
  }
  __builtin_amdgcn_sched_barrier(0);

  // rows at or beyond N fall outside the output buffer and are dropped
  store_strip<D>(oh, i0, fo);
}

// grid.x = BH * nseg (XCD-aware remap); the workgroup walks the 64-row tiles
// of segment s, rows [s*L, min(N, s*L + L)) with L a multiple of 64, starting
// from the segment's exclusive prefix sums (tile-order record).  Window of the
// tile at t0: the U units [t0/32 - KC, t0/32 + 2); unit ua0 + m lives in ring
// slot m % U and the ring slides by two units (the next tile's keys) per
// tile, those units prefetched into registers a tile ahead.
template <int D, int R, int KC>
__global__ __launch_bounds__(CNT, 2) void k_causal_strip(const bf16_t* __restrict__ q,
                                                      const bf16_t* __restrict__ k,
                                                      const bf16_t* __restrict__ v,
                                                      bf16_t* __restrict__ out,
                                                      const float* __restrict__ prefix,
                                                      const float* __restrict__ w_near,
                                                      const float* __restrict__ w_far, int H,
                                                      int N, int band_k, int L, int nseg,
                                                      float scale2) {
  using C = CausalCfg<D, R, KC>;
  using St = CausalState<D, R>;
  constexpr int NQ = C::NQ, U = C::U, RB = C::RB;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  unsigned char* kr = dyn_smem;
  unsigned char* vr = kr + C::RING;
  unsigned char* phr = vr + C::RING;
  Oct* sf = reinterpret_cast<Oct*>(phr + R * C::PHI);
  Oct* szo = sf + C::FRAG / 16;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const size_t base = (size_t)bh * N * D;
  const int hbytes = N * D * 2;
  const Rsrc qh = head_rsrc(q + base, hbytes), kh = head_rsrc(k + base, hbytes),
             vh = head_rsrc(v + base, hbytes), oh = head_rsrc(out + base, hbytes);
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + CTM - 1) / CTM;
  const int ua0 = (s0 >> 5) - KC;
  constexpr bool all_st = St::FT >= CW;  // every wave owns state tiles
  const bool has_st = St::active(w);

  // prologue: every load (the segment's prefix sums, the ring's first window
  // in rounds of two units, the first tile's keys for their phi rows, the
  // first query rows) is issued before the first LDS store, so the workgroup
  // waits for one round trip instead of several
  using RC = RowsCopy<D, CTM, CNT>;
  constexpr int NR = (U + 1) / 2;
  St st;
  st.load(w, prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1));
  RC rk[NR], rv[NR], ck;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    rk[i].load(kh, (ua0 + 2 * i) * 32, true);
    rv[i].load(vh, (ua0 + 2 * i) * 32, true);
  }
  ck.load(kh, s0, true);
  Oct qo[1][NQ];
  load_qo<D, 1>(qh, s0 + 16 * w, true, qo);
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    // full rounds need no range test (one the compiler cannot fold would
    // sink their loads behind a branch and a wait)
    auto slot = [=](int j) { return (U % 2 == 0 || i + 1 < NR) ? 2 * i + j : (j == 0 ? 2 * i : -1); };
    rk[i].store(kr, slot);
    rv[i].store(vr, slot);
  }
  {
    PhiRows<D, R> ph;
    ph.compute(ck);
    ph.store(phr);
  }
  if (all_st || has_st) St::store(w, st.pack(), sf, szo);
  const RingOffsets<D> ro;
  RC pk, pv;
  pk.load(kh, (ua0 + U) * 32, ntile > 1);
  pv.load(vh, (ua0 + U) * 32, ntile > 1);

  // masks of the four tile blocks in this strip's intra-tile product: keys
  // below the strip's block kept, its own block lower-triangular (key 4g + i
  // <= row r), the blocks above empty
  uint2 tmask[4];
  {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
    uint2 dm;
    dm.x = (4 * g <= r ? 0xffffu : 0u) | (4 * g + 1 <= r ? 0xffff0000u : 0u);
    dm.y = (4 * g + 2 <= r ? 0xffffu : 0u) | (4 * g + 3 <= r ? 0xffff0000u : 0u);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      tmask[j] = j < w ? make_uint2(~0u, ~0u) : j == w ? dm : make_uint2(0u, 0u);
  }
  // one tile, then the ring slides by the prefetched units and their phi rows
  // replace the tile's (past the last tile the loads and stores are harmless
  // no-ops on zeros, and the sums are not read again)
  auto step = [&](int t, auto general) {
    constexpr bool G = decltype(general)::value;
    __syncthreads();  // ring, phi rows and fragments hold tile t's
    const int t0 = s0 + t * CTM;
    const int m0 = 2 * t;
    auto mid = [&]() { load_qo<D, 1>(qh, t0 + CTM + 16 * w, t + 1 < ntile, qo); };
    PhiRows<D, R> phn;
    // the sums advance by the tile's 64 keys inside the tile's last phase,
    // which hands over each key unit's V^T octs; phi of the next tile's keys
    // is formed there too, beside the matrix-core products
    auto unit = [&](int c, const Oct* vt) { st.add_unit(phr, c, vt); };
    auto late = [&]() { phn.compute(pk); };
    tile_work<D, R, KC, G>(oh, t0, w, m0, N, band_k, scale2, sn, sfw, qo[0], kr, vr, phr, ro,
                           sf, szo, tmask, mid, unit, late);
    const typename St::Frags fr = st.pack();
    __syncthreads();  // every wave is done with tile t's LDS
    auto slot = [=](int j) { return (m0 + j) % U; };
    pk.store(kr, slot);
    pv.store(vr, slot);
    phn.store(phr);
    if (all_st || has_st) St::store(w, fr, sf, szo);
    pk.load(kh, (ua0 + U + m0 + 2) * 32, t + 2 < ntile);
    pv.load(vh, (ua0 + U + m0 + 2) * 32, t + 2 < ntile);
  };
  // exact tiles: k = 32*KC and the tile's window inside [0, N); they form one
  // contiguous run of the walk, between the leading and trailing general tiles
  const bool fit = band_k == 32 * KC;
  auto interior = [&](int t) {
    const int t0 = s0 + t * CTM;
    return fit && t0 - 32 * KC >= 0 && t0 + CTM - 1 < N;
  };
  int t = 0;
  for (; t < ntile && !interior(t); ++t) step(t, std::true_type{});
  for (; t < ntile && interior(t); ++t) step(t, std::false_type{});
  for (; t < ntile; ++t) step(t, std::true_type{});
}

template <int D, int R, int KC>
hipError_t launch_strip_kc(const LaunchArgs& a, Launcher& L, const float* prefix,
                           float scale2) {
  using C = CausalCfg<D, R, KC>;
  static std::atomic<unsigned long long> lds_set{0};
  if (L.note(lds_limit_once((const void*)k_causal_strip<D, R, KC>, C::LDS, lds_set)) !=
      hipSuccess)
    return L.err;
  L(FMM_KERNEL_CAUSAL_APPLY, k_causal_strip<D, R, KC>, dim3(a.B * a.H * a.nseg),
               dim3(CNT), (size_t)C::LDS, (hipStream_t)a.stream, (const bf16_t*)a.q,
               (const bf16_t*)a.k, (const bf16_t*)a.v, (bf16_t*)a.out, prefix, a.w_near,
               a.w_far, a.H, a.N, a.band_k, a.L, a.nseg, scale2);
  return L.err;
}

template <int D, int R>
hipError_t launch_strip_d(const LaunchArgs& a, Launcher& t, const float* prefix,
                          float scale2) {
  return a.band_k <= 32 ? launch_strip_kc<D, R, 1>(a, t, prefix, scale2)
                        : launch_strip_kc<D, R, 2>(a, t, prefix, scale2);
}

}  // namespace

bool causal_strip_applies(int dtype, int d, int band_k, int causal, long long n) {
  // 32-bit buffer offsets: one head's rows must stay below 2 GiB
  return dtype == FMM_DTYPE_BF16 && (d == 32 || d == 64) && band_k <= 64 && causal &&
         n * d * 2 < (1LL << 31);
}

hipError_t launch_causal_strip(const LaunchArgs& a, Launcher& t, const float* prefix) {
  const float scale2 = 1.4426950408889634f / sqrtf((float)a.d);
  switch (a.d * 4 + a.rank) {
    case 32 * 4 + 1: return launch_strip_d<32, 1>(a, t, prefix, scale2);
    case 32 * 4 + 2: return launch_strip_d<32, 2>(a, t, prefix, scale2);
    case 64 * 4 + 1: return launch_strip_d<64, 1>(a, t, prefix, scale2);
    case 64 * 4 + 2: return launch_strip_d<64, 2>(a, t, prefix, scale2);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fmm
