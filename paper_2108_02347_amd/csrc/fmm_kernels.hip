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
//                    registers during compute.  Per tile: banded softmax
//                    (Eq. (3)), far apply phi_l(Q) S_l / phi_l(Q) z_l
//                    (Eq. (8)-(9)), sigmoid blend (Eq. (11)), store
//   k_causal_ring    causal, band fits the ring: same walk, with the running
//                    state carried in registers; per tile the causal band
//                    [i-k, i], the intra-tile lower-triangular far part, the
//                    prefix far part, the blend and the state update
//   k_band_rounds,   the same two operators for bands wider than the ring: every
//   k_causal_rounds  tile stages its key window in rounds
//
// bf16 heads of width 32 or 64 with band half-widths up to 64 take the strip
// kernels of fmm_pair.hip (non-causal, two 16-row strips per wavefront) and
// fmm_causal.hip (causal); the ring and rounds kernels here serve every other
// case (fp32 storage, d = 16, wider bands).
//
// Every workgroup of the apply kernels has NW = 4 wavefronts; wave w owns query
// rows [16w, 16w+16) of a TM = 64-row tile.  All sums are accumulated in fp32
// in a fixed order, so results are bit-reproducible run to run.
//
// Row sums of the softmax weights and the far-field denominators
// phi_l(q) . z_l are taken on the matrix cores too: an extra 16-row A block of
// ones (resp. of z_l broadcast over rows) yields the sum in every lane of the
// row, so no cross-lane reduction is needed for them.
//
// State records (one per segment, and one final record per (batch, head) in
// the non-causal form) are kept in MFMA tile order: for map l, the d x d block
// S_l is stored as tiles (cb, eb) of 16 x 16, each as 64 lanes x 4 floats with
// lane 16g + r holding S_l[16cb + 4g + i][16eb + r], i = 0..3; z_l (d floats)
// follows.  A wave's accumulator tile is then one coalesced float4 per lane.
#include "fmm_apply.h"
#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {

// ------------------------------------------------------------------ causal pieces
// phi_l of the tile's 64 keys (LDS rows kt0 .. kt0+31 and kt1 .. kt1+31 of the
// key buffer) into pk[l] (row-major, TM rows); keys at or beyond N give 0.
template <typename T, int D, int R>
__device__ __forceinline__ void stage_phi_tile(const T* kbuf, int kt0, int kt1, int ST, int t0,
                                               int N, T* pk) {
  using L = Lay<T>;
  constexpr int CPR = D / L::EPC;
  for (int t = threadIdx.x; t < TM * CPR; t += NT) {
    const int key = t / CPR, c = t % CPR;
    const int src = key < 32 ? kt0 + key : kt1 + key - 32;
    const uint4 raw = *reinterpret_cast<const uint4*>(kbuf + src * ST + c * L::EPC);
    float x[L::EPC], p1[L::EPC], p2[L::EPC];
    if constexpr (sizeof(T) == 2) {
      const uint16_t* e = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int i = 0; i < L::EPC; ++i) x[i] = bf16_to_f32(e[i]);
    } else {
      const float* e = reinterpret_cast<const float*>(&raw);
#pragma unroll
      for (int i = 0; i < L::EPC; ++i) x[i] = e[i];
    }
    const bool ok = t0 + key < N;
#pragma unroll
    for (int i = 0; i < L::EPC; ++i) {
      phi12(x[i], p1[i], p2[i]);
      if (!ok) { p1[i] = 0.f; p2[i] = 0.f; }
    }
#pragma unroll
    for (int l = 0; l < R; ++l) {
      const float* p = l == 0 ? p1 : p2;
      uint4 outw;
      if constexpr (sizeof(T) == 2) {
        outw = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                          pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
      } else {
        outw = make_uint4(__float_as_uint(p[0]), __float_as_uint(p[1]), __float_as_uint(p[2]),
                          __float_as_uint(p[3]));
      }
      *reinterpret_cast<uint4*>(pk + l * TM * ST + key * ST + c * L::EPC) = outw;
    }
  }
}

// phi_l of the 64 key rows a RowCopy holds in registers (rows k0 .. k0+63 of
// the head), computed into registers (same chunk-to-thread assignment as
// RowCopy) and later stored as pk[l]; rows at or beyond N give 0.
template <typename T, int D, int R>
struct PhiRows {
  using L = Lay<T>;
  using RC = RowCopy<T, D, NT, 64>;
  uint4 v[R][RC::IT];
  __device__ __forceinline__ void compute(const RC& ck, int k0, int N) {
#pragma unroll
    for (int it = 0; it < RC::IT; ++it) {
      const int t = threadIdx.x + it * NT;
      const int key = t / RC::CPR;
      const uint4 raw = ck.r[it];
      float x[L::EPC], p1[L::EPC], p2[L::EPC];
      if constexpr (sizeof(T) == 2) {
        const uint16_t* e = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
        for (int i = 0; i < L::EPC; ++i) x[i] = bf16_to_f32(e[i]);
      } else {
        const float* e = reinterpret_cast<const float*>(&raw);
#pragma unroll
        for (int i = 0; i < L::EPC; ++i) x[i] = e[i];
      }
      const bool ok = k0 + key < N;
#pragma unroll
      for (int i = 0; i < L::EPC; ++i) {
        phi12(x[i], p1[i], p2[i]);
        if (!ok) { p1[i] = 0.f; p2[i] = 0.f; }
      }
#pragma unroll
      for (int l = 0; l < R; ++l) {
        const float* p = l == 0 ? p1 : p2;
        if constexpr (sizeof(T) == 2) {
          v[l][it] = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
        } else {
          v[l][it] = make_uint4(__float_as_uint(p[0]), __float_as_uint(p[1]),
                                __float_as_uint(p[2]), __float_as_uint(p[3]));
        }
      }
    }
  }
  __device__ __forceinline__ void store(T* pk, int ST) const {
#pragma unroll
    for (int it = 0; it < RC::IT; ++it) {
      const int t = threadIdx.x + it * NT;
      if (t >= TM * RC::CPR) continue;
      const int key = t / RC::CPR, c = t % RC::CPR;
#pragma unroll
      for (int l = 0; l < R; ++l)
        *reinterpret_cast<uint4*>(pk + l * TM * ST + key * ST + c * L::EPC) = v[l][it];
    }
  }
};

// Intra-tile far part of the strip of wave w for map l: keys [t0, row] of the
// tile, A = tril(phi_l(K_t) phi_l(q)^T) from pk, num[nb] += V^T A and the row
// sums of A into num[NB].  vt0 / vt1: LDS rows of the tile's two V units.
template <typename T, int D, int R>
__device__ __forceinline__ void causal_intra(const T* pk, const T* vt0, const T* vt1, int ST,
                                             int t0, int w, int l,
                                             const typename QuadOf<T>::type* pql,
                                             f32x4* num) {
  using Q = typename QuadOf<T>::type;
  constexpr int NB = D / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int row = t0 + 16 * w + r;
  const Q ones = quad_fill<T>(1.f);
  const T* pkl = pk + l * TM * ST;
  for (int u = 0; u <= (w >> 1); ++u) {
    const T* vx = u == 0 ? vt0 : vt1;
    const bool diag = u == (w >> 1);
    float a[2][4];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      Q ka[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) ka[cb] = ld_quad(pkl, 32 * u + 16 * b + r, 16 * cb + 4 * g, ST);
      const f32x4 at = contract<NB>(ka, pql, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = t0 + 32 * u + 16 * b + 4 * g + i;
        a[b][i] = (!diag || j <= row) ? at[i] : 0.f;
      }
    }
    const Q p0 = f32_to_quad<T>(a[0]), p1 = f32_to_quad<T>(a[1]);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      num[nb] = mma_step2(ld_tquad(vx, 0, 16 * nb, ST), ld_tquad(vx, 16, 16 * nb, ST), p0, p1,
                          num[nb]);
    num[NB] = mma_step2(ones, ones, p0, p1, num[NB]);
  }
}

// ------------------------------------------------------------------ state tiles
// A wave's share of the running state T_l = phi_l(K)^T [V | 1] in the causal
// walk: groups ag = w + NW*a (l = ag / NB, cb = ag % NB), every value block
// eb < NB plus the ones column eb = NB that yields z_l.
template <typename T, int D, int R>
struct StateTiles {
  using Q = typename QuadOf<T>::type;
  static constexpr int NB = D / 16;
  static constexpr int AG = R * NB;
  static constexpr int AGPW = AG >= NW ? AG / NW : 1;
  static_assert(AG < NW || AG % NW == 0, "group split");
  f32x4 acc[AGPW][NB + 1];

  __device__ __forceinline__ static bool active(int w) { return w < AG; }
  __device__ __forceinline__ static int group(int w, int a) { return w + NW * a; }

  // acc += phi_l(K)^T [V | 1] over one 32-key unit: phi rows from pk (rows
  // pr .. pr+31 of map l's buffer), V rows at vx.
  __device__ __forceinline__ void add_unit(int w, const T* pk, int pr, const T* vx, int ST) {
    const int lane = threadIdx.x & 63, r = lane & 15;
    Q vb0[NB + 1], vb1[NB + 1];
#pragma unroll
    for (int eb = 0; eb < NB; ++eb) {
      vb0[eb] = ld_tquad(vx, 0, 16 * eb, ST);
      vb1[eb] = ld_tquad(vx, 16, 16 * eb, ST);
    }
    vb0[NB] = quad_fill<T>(r == 0 ? 1.f : 0.f);
    vb1[NB] = vb0[NB];
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
      const T* pkl = pk + l * TM * ST;
      const Q a0 = ld_tquad(pkl, pr, 16 * cb, ST), a1 = ld_tquad(pkl, pr + 16, 16 * cb, ST);
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb) acc[a][eb] = mma_step2(a0, a1, vb0[eb], vb1[eb], acc[a][eb]);
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
  // This wave's tiles as operand quads, ready to store with store_frags.
  struct Frags {
    Q s[AGPW][NB];
    Q z[AGPW];
  };
  __device__ __forceinline__ Frags pack() const {
    Frags f;
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
#pragma unroll
      for (int eb = 0; eb <= NB; ++eb) {
        const float x[4] = {acc[a][eb][0], acc[a][eb][1], acc[a][eb][2], acc[a][eb][3]};
        if (eb < NB) f.s[a][eb] = f32_to_quad<T>(x);
        else f.z[a] = f32_to_quad<T>(x);
      }
    }
    return f;
  }
  __device__ __forceinline__ static void store_frags(int w, const Frags& f, Q* sf, Q* szq) {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int a = 0; a < AGPW; ++a) {
      const int ag = group(w, a);
      const int l = ag / NB, cb = ag % NB;
#pragma unroll
      for (int eb = 0; eb < NB; ++eb) sf[((l * NB + eb) * NB + cb) * 64 + lane] = f.s[a][eb];
      if (r == 0) szq[(l * NB + cb) * 4 + g] = f.z[a];
    }
  }
  // Write this wave's tiles as apply fragments (sf, szq) for the prefix far part.
  __device__ __forceinline__ void to_frags(int w, Q* sf, Q* szq) const {
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
      if (r == 0) {
        const float f[4] = {acc[a][NB][0], acc[a][NB][1], acc[a][NB][2], acc[a][NB][3]};
        szq[(l * NB + cb) * 4 + g] = f32_to_quad<T>(f);
      }
    }
  }
};

// ------------------------------------------------------------------ k_seg_state
// grid.x = nseg * BH (segment fastest), 8 waves.  Segment s of head bh covers
// rows [s*L, min(N, s*L + L)), walked in chunks of TK keys double-buffered in
// LDS, the next chunk's loads in flight during compute.  Waves sharing a
// feature block split the 32-key units and are summed in a fixed tree at the
// end.  Output: the segment's tile-order state record.  TK is 64 or, for long
// segments, 32 units per wave sharing a feature block (128 keys at d = 32,
// 256 at d = 16), which keeps every wave busy and more bytes in flight.
constexpr int SW = 8;          // waves in k_seg_state
constexpr int SNT = SW * 64;
template <typename T, int D, int R, int TK>
__global__ __launch_bounds__(SNT) void k_seg_state(const T* __restrict__ k,
                                                   const T* __restrict__ v,
                                                   float* __restrict__ part, int N, int L,
                                                   int nseg) {
  constexpr int NB = D / 16;
  constexpr int ST = D + Lay<T>::PAD;
  // waves are laid out as (rs, cb): cb = w % NB, rs = w / NB splits the units
  constexpr int RS = SW / NB;
  __shared__ __attribute__((aligned(16))) T s_kv[2][2][TK * ST];  // [buffer][K, V]

  const int seg = blockIdx.x % nseg, bh = blockIdx.x / nseg;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
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

  // the first two chunks' loads are issued together (a second chunk past the
  // segment's end has no rows: its loads return zeros without memory access)
  RowCopy<T, D, SNT, TK> ck, cv, ck0, cv0;
  auto ident = [](int i) { return i; };
  ck0.load(kh, r0, min(TK, r1 - r0), r1);
  cv0.load(vh, r0, min(TK, r1 - r0), r1);
  ck.load(kh, r0 + TK, min(TK, r1 - r0 - TK), r1);
  cv.load(vh, r0 + TK, min(TK, r1 - r0 - TK), r1);
  ck0.store(s_kv[0][0], ST, TK, ident);
  cv0.store(s_kv[0][1], ST, TK, ident);
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
      float p[2][R][4];  // [b][map][i]
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float kf[4];
        quad_to_f32(ld_tquad(kx, 32 * u + 16 * b, 16 * cbw, ST), kf);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float pm[R];
          phi_maps<R>(kf[i], pm);
          const bool valid = 16 * b + 4 * g + i < kvalid;
#pragma unroll
          for (int l = 0; l < R; ++l) p[b][l][i] = valid ? pm[l] : 0.f;
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
                                                       int rec, int nchunk) {
  // the causal scan keeps the first CACHE values of its range in registers
  // between the two passes, so each record is read from memory once
  constexpr int CACHE = CAUSAL ? 32 : 1;
  __shared__ float tot[4][64];
  const int el = threadIdx.x & 63, qr = threadIdx.x >> 6;
  // one-dimensional grid: (batch, head) slice major, 64-element chunk minor
  const int bh = blockIdx.x / nchunk;
  const int e = (blockIdx.x - bh * nchunk) * 64 + el;
  const int per = (nseg + 3) / 4;
  const int s0 = min(nseg, qr * per), s1 = min(nseg, s0 + per);
  float* p = part + (size_t)bh * nseg * rec + e;
  float s = 0.f;
  float keep[CACHE];
  if (e < rec) {
    if constexpr (CAUSAL) {
#pragma unroll
      for (int jj = 0; jj < CACHE; ++jj) {
        keep[jj] = s0 + jj < s1 ? p[(size_t)(s0 + jj) * rec] : 0.f;
        if (s0 + jj < s1) s += keep[jj];
      }
      for (int j = s0 + CACHE; j < s1; ++j) s += p[(size_t)j * rec];
    } else {
      int j = s0;
      for (; j + 4 <= s1; j += 4) {
        const float a0 = p[(size_t)j * rec], a1 = p[(size_t)(j + 1) * rec];
        const float a2 = p[(size_t)(j + 2) * rec], a3 = p[(size_t)(j + 3) * rec];
        s += a0; s += a1; s += a2; s += a3;
      }
      for (; j < s1; ++j) s += p[(size_t)j * rec];
    }
  }
  tot[qr][el] = s;
  __syncthreads();
  if (e >= rec) return;
  if constexpr (!CAUSAL) {
    if (qr == 0) fin[(size_t)bh * rec + e] = ((tot[0][el] + tot[1][el]) + tot[2][el]) + tot[3][el];
  } else {
    float run = 0.f;
    for (int q2 = 0; q2 < qr; ++q2) run += tot[q2][el];
#pragma unroll
    for (int jj = 0; jj < CACHE; ++jj) {
      if (s0 + jj < s1) {
        p[(size_t)(s0 + jj) * rec] = run;
        run += keep[jj];
      }
    }
    for (int j = s0 + CACHE; j < s1; ++j) {
      const float t = p[(size_t)j * rec];
      p[(size_t)j * rec] = run;
      run += t;
    }
  }
}

// ------------------------------------------------------------------ apply LDS
// One workgroup's LDS: key and value rows (ring or round), state fragments,
// z, and for the causal form the tile's phi_l(K) rows.
template <typename T, int D, int R>
struct ApplyLds {
  using Q = typename QuadOf<T>::type;
  static constexpr int ST = D + Lay<T>::PAD, NB = D / 16;
  T* k;
  T* v;
  Q* sf;
  Q* sz;  // z quads, see far_terms
  T* pk;
  __device__ __forceinline__ ApplyLds(unsigned char* base, int rows) {
    k = reinterpret_cast<T*>(base);
    v = k + rows * ST;
    sf = reinterpret_cast<Q*>(v + rows * ST);
    sz = sf + R * NB * NB * 64;
    pk = reinterpret_cast<T*>(sz + R * NB * 4);
  }
};

// Copy absolute units [ua, ua + n) of K and V into the ring (synchronously).
template <typename T, int D, int R>
__device__ __forceinline__ void ring_fill(const ApplyLds<T, D, R>& sm, const T* kh, const T* vh,
                                          int ua, int n, RingMap map, int N) {
  constexpr int ST = ApplyLds<T, D, R>::ST;
  for (int x = 0; x < n; x += 2) {
    const int m = min(2, n - x);
    RowCopy<T, D, NT, 64> ck, cv;
    ck.load(kh, (ua + x) * 32, 32 * m, N);
    cv.load(vh, (ua + x) * 32, 32 * m, N);
    auto row = [&](int i) { return map(ua + x + (i >> 5)) + (i & 31); };
    ck.store(sm.k, ST, 32 * m, row);
    cv.store(sm.v, ST, 32 * m, row);
  }
}

// ------------------------------------------------------------------ k_band_ring
// Non-causal.  grid.x = BH * nseg (XCD-aware remap); the workgroup walks the
// 64-row tiles of rows [s*L, min(N, s*L + L)).  Window of a tile starting at
// t0: keys [t0 - 32*ceil(k/32), t0 + 64 + 32*ceil(k/32)) = U = 2 + 2*ceil(k/32)
// units; it slides by two units per tile.
template <typename T, int D, int R>
__global__ __launch_bounds__(NT) void k_band_ring(const T* __restrict__ q,
                                                  const T* __restrict__ k,
                                                  const T* __restrict__ v, T* __restrict__ out,
                                                  const float* __restrict__ fin,
                                                  const float* __restrict__ w_near,
                                                  const float* __restrict__ w_far, int H, int N,
                                                  int band_k, int L, int nseg, float scale2) {
  using Q = typename QuadOf<T>::type;
  using SM = ApplyLds<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  const int kc = (band_k + 31) >> 5;  // band half-width in units (rounded up)
  const int U = 2 + 2 * kc;
  const SM sm(dyn_smem, U * 32);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const T* qh = q + base;
  const T* kh = k + base;
  const T* vh = v + base;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + TM - 1) / TM;
  const RingMap map{(s0 >> 5) - kc, U};

  load_state_frags<T, D, R, NT>(fin + (size_t)bh * R * D * (D + 1), sm.sf, sm.sz);
  ring_fill<T, D, R>(sm, kh, vh, map.ua0, U, map, N);
  Q qq[NB];
  load_q<T, D>(qh, s0 + 16 * w + r, N, qq);
  RowCopy<T, D, NT, 64> pk, pv;
  pk.load(kh, (map.ua0 + U) * 32, ntile > 1 ? 64 : 0, N);
  pv.load(vh, (map.ua0 + U) * 32, ntile > 1 ? 64 : 0, N);
  for (int t = 0; t < ntile; ++t) {
    __syncthreads();  // ring holds the window of tile t
    const int t0 = s0 + t * TM, i0 = t0 + 16 * w, row = i0 + r;
    NearState<D> st;
    st.init();
    const int lo = max(0, i0 - band_k), hi = min(N - 1, i0 + 15 + band_k);
    if (fixed_strip<false, 5>(i0, N, band_k))
      near_fixed<T, D, false, 5>(st, qq, sm.k, sm.v, ST, map, (i0 - band_k) >> 5, i0, N, band_k,
                                 scale2);
    else
      near_units<T, D, false, 6>(st, qq, sm.k, sm.v, ST, map, lo >> 5, hi >> 5, i0, N, band_k,
                                 scale2);
    Q pq[R][NB];
    phi_q<T, D, R>(qq, pq);
    // the query quads are dead: load the next tile's rows into them (a copy
    // from separate prefetch registers would make the loop wait for every
    // outstanding load at its head)
    load_q<T, D>(qh, t0 + TM + 16 * w + r, t + 1 < ntile ? N : 0, qq);
    f32x4 num[R][NB + 1];
    far_terms<T, D, R, false>(sm.sf, sm.sz, pq, num);
    blend_store<T, D, R>(out + base, row, N, sn, sfw, st, num);
    // slide the ring (after the last tile this stores zeros nobody reads;
    // prefetches past the walk are empty row ranges, so there is no branch
    // around any global load)
    __syncthreads();  // every wave is done with the window of tile t
    const int ua_new = map.ua0 + 2 * t + U;  // the two units tile t+1 adds
    const int ra = map(ua_new), rb = map(ua_new + 1);
    auto rowmap = [=](int i) { return (i < 32 ? ra : rb) + (i & 31); };
    pk.store(sm.k, ST, 64, rowmap);
    pv.store(sm.v, ST, 64, rowmap);
    const bool pf = t + 2 < ntile;
    pk.load(kh, (ua_new + 2) * 32, pf ? 64 : 0, N);
    pv.load(vh, (ua_new + 2) * 32, pf ? 64 : 0, N);
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
  using SM = ApplyLds<T, D, R>;
  using Tiles = StateTiles<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  const int kc = (band_k + 31) >> 5;
  const int U = 2 + kc;
  const SM sm(dyn_smem, U * 32);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const T* qh = q + base;
  const T* kh = k + base;
  const T* vh = v + base;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const int s0 = seg * L, s1 = min(N, s0 + L);
  const int ntile = (s1 - s0 + TM - 1) / TM;
  const RingMap map{(s0 >> 5) - kc, U};
  const bool has_ag = Tiles::active(w);

  Tiles tiles;
  if (has_ag) tiles.load(w, prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1));
  ring_fill<T, D, R>(sm, kh, vh, map.ua0, U, map, N);
  if (has_ag) tiles.to_frags(w, sm.sf, sm.sz);
  Q qq[NB];
  load_q<T, D>(qh, s0 + 16 * w + r, N, qq);
  RowCopy<T, D, NT, 64> pk, pv;
  pk.load(kh, (map.ua0 + U) * 32, ntile > 1 ? 64 : 0, N);
  pv.load(vh, (map.ua0 + U) * 32, ntile > 1 ? 64 : 0, N);
  __syncthreads();  // ring filled
  stage_phi_tile<T, D, R>(sm.k, map(s0 >> 5), map((s0 >> 5) + 1), ST, s0, N, sm.pk);
  for (int t = 0; t < ntile; ++t) {
    const int t0 = s0 + t * TM, i0 = t0 + 16 * w, row = i0 + r;
    const int rt0 = map(t0 >> 5), rt1 = map((t0 >> 5) + 1);  // ring rows of the tile
    __syncthreads();  // window, phi rows and prefix fragments of tile t are in LDS
    NearState<D> st;
    st.init();
    const int lo = max(0, i0 - band_k), hi = min(N - 1, i0 + 15);
    if (fixed_strip<true, 3>(i0, N, band_k))
      near_fixed<T, D, true, 3>(st, qq, sm.k, sm.v, ST, map, (i0 - band_k) >> 5, i0, N, band_k,
                                scale2);
    else
      near_units<T, D, true, 4>(st, qq, sm.k, sm.v, ST, map, lo >> 5, hi >> 5, i0, N, band_k,
                                scale2);
    f32x4 fo[NB];
    near_out<D>(st, sn, fo);
    Q pq[R][NB];
    phi_q<T, D, R>(qq, pq);
    // the query quads are dead: load the next tile's rows into them
    load_q<T, D>(qh, t0 + TM + 16 * w + r, t + 1 < ntile ? N : 0, qq);
#pragma unroll
    for (int l = 0; l < R; ++l) {
      f32x4 num[NB + 1];
#pragma unroll
      for (int nb = 0; nb <= NB; ++nb) num[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      causal_intra<T, D, R>(sm.pk, sm.v + rt0 * ST, sm.v + rt1 * ST, ST, t0, w, l, pq[l], num);
      far_terms_map<T, D>(sm.sf, sm.sz, l, pq[l], num);
      add_far_map<D>(num, sfw, fo);
    }
    store_row<T, D>(out + base, row, N, fo);
    // everything tile t+1 needs in LDS is prepared in registers first, so
    // that only plain stores sit between the two barriers (the scheduling
    // fence keeps this work from being hoisted into the compute above, where
    // it would raise register pressure).  After the last tile this advances
    // a state nobody reads; prefetches past the walk are empty row ranges, so
    // there is no branch around any global load.
    __builtin_amdgcn_sched_barrier(0);
    if (has_ag) {
      tiles.add_unit(w, sm.pk, 0, sm.v + rt0 * ST, ST);
      tiles.add_unit(w, sm.pk, 32, sm.v + rt1 * ST, ST);
    }
    typename Tiles::Frags fr;
    if (has_ag) fr = tiles.pack();
    PhiRows<T, D, R> ph;
    ph.compute(pk, t0 + TM, N);  // the prefetched rows are the keys of tile t+1
    __syncthreads();  // every wave is done with tile t's LDS
    const int ua_new = map.ua0 + 2 * t + U;
    const int ra = map(ua_new), rb = map(ua_new + 1);
    auto rowmap = [=](int i) { return (i < 32 ? ra : rb) + (i & 31); };
    pk.store(sm.k, ST, 64, rowmap);
    pv.store(sm.v, ST, 64, rowmap);
    ph.store(sm.pk, ST);
    if (has_ag) Tiles::store_frags(w, fr, sm.sf, sm.sz);
    const bool pf = t + 2 < ntile;
    pk.load(kh, (ua_new + 2) * 32, pf ? 64 : 0, N);
    pv.load(vh, (ua_new + 2) * 32, pf ? 64 : 0, N);
  }
}

// ------------------------------------------------------------------ rounds variants
// Bands too wide for the ring: every tile stages its window in rounds of up to
// 32 * Ring::UR keys (row-major K and V, like the ring).
template <typename T, int D, int R>
__device__ __forceinline__ void round_stage(const ApplyLds<T, D, R>& sm, const T* kh,
                                            const T* vh, int ks, int nk, int kend) {
  constexpr int ST = ApplyLds<T, D, R>::ST;
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
  using SM = ApplyLds<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  constexpr int WK = 32 * Ring<T, D, R>::UR;
  const SM sm(dyn_smem, WK);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / ntile, tile = lin % ntile, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15;
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
    if (lo <= hi)
      near_units<T, D, false, 6>(st, qq, sm.k, sm.v, ST, RoundMap{ks}, lo >> 5, hi >> 5, i0, N,
                              band_k, scale2);
  }
  Q pq[R][NB];
  phi_q<T, D, R>(qq, pq);
  f32x4 num[R][NB + 1];
  far_terms<T, D, R, false>(sm.sf, sm.sz, pq, num);
  blend_store<T, D, R>(out + base, row, N, sn, sfw, st, num);
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
  using SM = ApplyLds<T, D, R>;
  using Tiles = StateTiles<T, D, R>;
  constexpr int NB = D / 16, ST = SM::ST;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn_smem[];
  constexpr int WK = 32 * Ring<T, D, R>::UR;
  const SM sm(dyn_smem, WK);
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = lin / nseg, seg = lin % nseg, h = bh % H;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, r = lane & 15;
  const size_t base = (size_t)bh * N * D;
  const float sn = sigmoidf_exact(w_near[h]), sfw = sigmoidf_exact(w_far[h]);
  const bool has_ag = Tiles::active(w);
  Tiles tiles;
  if (has_ag) tiles.load(w, prefix + ((size_t)bh * nseg + seg) * R * D * (D + 1));
  const int s0 = seg * L, s1 = min(N, s0 + L);
  for (int t0 = s0; t0 < s1; t0 += TM) {
    const int i0 = t0 + 16 * w, row = i0 + r;
    Q qq[NB];
    load_q<T, D>(q + base, row, N, qq);
    Q pq[R][NB];
    phi_q<T, D, R>(qq, pq);
    NearState<D> st;
    st.init();
    f32x4 num[R][NB + 1];
#pragma unroll
    for (int l = 0; l < R; ++l)
#pragma unroll
      for (int nb = 0; nb <= NB; ++nb) num[l][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ka = (max(0, t0 - band_k) >> 5) << 5;
    const int hi = t0 + TM;
    for (int ke = hi; ke > ka; ke -= WK) {
      const int ks = max(ka, ke - WK), nk = ke - ks;
      __syncthreads();  // every wave is done with the previous round / tile
      round_stage<T, D, R>(sm, k + base, v + base, ks, nk, min(N, ke));
      if (ke == hi) {
        if (has_ag) tiles.to_frags(w, sm.sf, sm.sz);
        __syncthreads();  // the tile's keys are staged
        stage_phi_tile<T, D, R>(sm.k, t0 - ks, t0 - ks + 32, ST, t0, N, sm.pk);
      }
      __syncthreads();
      const int lo = max(max(0, i0 - band_k), ks), hj = min(min(N - 1, i0 + 15), ks + nk - 1);
      if (lo <= hj)
        near_units<T, D, true, 4>(st, qq, sm.k, sm.v, ST, RoundMap{ks}, lo >> 5, hj >> 5, i0, N,
                               band_k, scale2);
      if (ke != hi) continue;
      const int tk = t0 - ks;
#pragma unroll
      for (int l = 0; l < R; ++l)
        causal_intra<T, D, R>(sm.pk, sm.v + tk * ST, sm.v + (tk + 32) * ST, ST, t0, w, l, pq[l],
                              num[l]);
      if (has_ag && t0 + TM < s1) {
        tiles.add_unit(w, sm.pk, 0, sm.v + tk * ST, ST);
        tiles.add_unit(w, sm.pk, 32, sm.v + (tk + 32) * ST, ST);
      }
    }
    far_terms<T, D, R, true>(sm.sf, sm.sz, pq, num);
    blend_store<T, D, R>(out + base, row, N, sn, sfw, st, num);
  }
}

// ------------------------------------------------------------------ launchers
// The tuned apply kernels (widths up to 64, one or two maps, per-map
// normalisation): strip kernels for bf16 at d = 32 / 64 with bands up to 64,
// ring kernels while the band fits the LDS ring, rounds kernels beyond.
template <typename T, int D, int R>
static hipError_t launch_tuned(const LaunchArgs& a, Launcher& L, float* part, float* fin) {
  using RG = Ring<T, D, R>;
  const int BH = a.B * a.H;
  const float scale2 = 1.4426950408889634f / sqrtf((float)D);
  hipStream_t s = (hipStream_t)a.stream;
  const T* q = (const T*)a.q;
  const T* k = (const T*)a.k;
  const T* v = (const T*)a.v;
  T* o = (T*)a.out;
  const int kc = (a.band_k + 31) / 32;
  const int U = a.causal ? 2 + kc : 2 + 2 * kc;
  const bool ring = U <= (a.causal ? RG::U_C : RG::U_NC);
  const size_t lds = RG::bytes(ring ? U : RG::UR, a.causal != 0);
  {
    static std::atomic<unsigned long long> set_band{0}, set_causal{0}, set_brounds{0},
        set_crounds{0};
    if (L.note(lds_limit_once((const void*)k_band_ring<T, D, R>, (int)RG::bytes(RG::U_NC, false),
                              set_band)) != hipSuccess ||
        L.note(lds_limit_once((const void*)k_causal_ring<T, D, R>, (int)RG::bytes(RG::U_C, true),
                              set_causal)) != hipSuccess ||
        L.note(lds_limit_once((const void*)k_band_rounds<T, D, R>, (int)RG::bytes(RG::UR, false),
                              set_brounds)) != hipSuccess ||
        L.note(lds_limit_once((const void*)k_causal_rounds<T, D, R>,
                              (int)RG::bytes(RG::UR, true), set_crounds)) != hipSuccess)
      return L.err;
  }
  if (a.causal) {
    if (causal_strip_applies(a.dtype, a.d, a.band_k, a.causal, a.N))
      return launch_causal_strip(a, L, part);
    if (ring)
      L(FMM_KERNEL_CAUSAL_APPLY, k_causal_ring<T, D, R>, dim3(BH * a.nseg), dim3(NT), lds, s, q,
        k, v, o, (const float*)part, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg, scale2);
    else
      L(FMM_KERNEL_CAUSAL_APPLY, k_causal_rounds<T, D, R>, dim3(BH * a.nseg), dim3(NT), lds, s,
        q, k, v, o, (const float*)part, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L, a.nseg,
        scale2);
  } else {
    if (band_pair_applies(a.dtype, a.d, a.band_k, a.causal, a.N)) {
      return launch_band_pair(a, L, fin);
    } else if (ring) {
      L(FMM_KERNEL_BAND_APPLY, k_band_ring<T, D, R>, dim3(BH * a.nseg_apply), dim3(NT), lds, s,
        q, k, v, o, (const float*)fin, a.w_near, a.w_far, a.H, a.N, a.band_k, a.L_apply,
        a.nseg_apply, scale2);
    } else {
      const long long ntile = (a.N + TM - 1) / TM;
      if ((long long)BH * ntile > 0x7FFFFFFFLL) return L.note(hipErrorInvalidConfiguration);
      L(FMM_KERNEL_BAND_APPLY, k_band_rounds<T, D, R>, dim3((unsigned)(BH * ntile)), dim3(NT),
        lds, s, q, k, v, o, (const float*)fin, a.w_near, a.w_far, a.H, a.N, a.band_k,
        (int)ntile, scale2);
    }
  }
  return L.err;
}

// The far-field state: per-segment records T_l = phi_l(K)^T [V | 1], then the
// fixed-order sum (non-causal, into the final records) or the exclusive scan
// over segments (causal, in place).
template <typename T, int D, int R>
static hipError_t launch_state(const LaunchArgs& a, Launcher& L) {
  const int BH = a.B * a.H;
  const int REC = R * D * (D + 1);
  hipStream_t s = (hipStream_t)a.stream;
  const T* k = (const T*)a.k;
  const T* v = (const T*)a.v;
  float* part = a.ws;
  // (integer arithmetic: the dry pass runs with no workspace yet)
  float* fin = reinterpret_cast<float*>(reinterpret_cast<uintptr_t>(a.ws) +
                                        (size_t)BH * a.nseg * REC * sizeof(float));

  // long chunks once a segment spans at least four of them; fp32 at d = 128
  // stages 32-key chunks (a 64-key double buffer would take 135 KiB)
  constexpr int TKL = 32 * (SW / (D / 16));
  constexpr int TKS = (D == 128 && sizeof(T) == 4) ? 32 : 64;
  bool long_chunks = false;
  if constexpr (TKL > 64) {
    long_chunks = a.L >= 4 * TKL;
    if (long_chunks)
      L(FMM_KERNEL_SEG_STATE, k_seg_state<T, D, R, TKL>, dim3(a.nseg * BH), dim3(SNT), 0, s, k,
        v, part, a.N, a.L, a.nseg);
  }
  if (!long_chunks)
    L(FMM_KERNEL_SEG_STATE, k_seg_state<T, D, R, TKS>, dim3(a.nseg * BH), dim3(SNT), 0, s, k, v,
      part, a.N, a.L, a.nseg);

  const int nchunk = (REC + 63) / 64;
  // (clamped: a grid this large fails the dry pass's dispatch-limit check)
  const dim3 cgrid((unsigned)std::min<long long>((long long)nchunk * BH, 0xFFFFFFFFll));
  if (a.causal)
    L(FMM_KERNEL_STATE_COMBINE, k_state_combine<true>, cgrid, dim3(256), 0, s, part, fin, a.nseg,
      REC, nchunk);
  else
    L(FMM_KERNEL_STATE_COMBINE, k_state_combine<false>, cgrid, dim3(256), 0, s, part, fin,
      a.nseg, REC, nchunk);
  return L.err;
}

template <typename T, int D, int R>
static hipError_t launch_all(const LaunchArgs& a, Launcher& L) {
  // widths above 64 and three feature maps take the general apply kernel
  constexpr bool tuned = D <= 64 && R <= 2;
  if constexpr (tuned && sizeof(T) == 2) {
    if (a.fused_g > 0 && !a.causal && a.far_norm == FMM_FAR_NORM_PER_MAP)
      return launch_band_fused(a, L);
  }
  if (launch_state<T, D, R>(a, L) != hipSuccess) return L.err;
  float* part = a.ws;
  float* fin = reinterpret_cast<float*>(reinterpret_cast<uintptr_t>(a.ws) +
                                        (size_t)a.B * a.H * a.nseg * R * D * (D + 1) *
                                            sizeof(float));
  if constexpr (tuned) {
    if (a.far_norm == FMM_FAR_NORM_PER_MAP) return launch_tuned<T, D, R>(a, L, part, fin);
  }
  return launch_wide(a, L, a.causal ? part : fin);
}

template <typename T, bool STATE_ONLY>
static hipError_t dispatch_d(const LaunchArgs& a, Launcher& L) {
#define FMM_CASE(DD, RR)                                                          \
  case DD * 4 + RR:                                                              \
    return STATE_ONLY ? launch_state<T, DD, RR>(a, L) : launch_all<T, DD, RR>(a, L);
  switch (a.d * 4 + a.rank) {
    FMM_CASE(16, 1) FMM_CASE(16, 2) FMM_CASE(16, 3)
    FMM_CASE(32, 1) FMM_CASE(32, 2) FMM_CASE(32, 3)
    FMM_CASE(64, 1) FMM_CASE(64, 2) FMM_CASE(64, 3)
    FMM_CASE(128, 1) FMM_CASE(128, 2) FMM_CASE(128, 3)
    default: return L.note(hipErrorInvalidValue);
  }
#undef FMM_CASE
}

hipError_t launch_forward(const LaunchArgs& a, Launcher& L) {
  return a.dtype == FMM_DTYPE_BF16 ? dispatch_d<bf16_t, false>(a, L)
                                   : dispatch_d<float, false>(a, L);
}

hipError_t launch_state_only(const LaunchArgs& a, Launcher& L) {
  return a.dtype == FMM_DTYPE_BF16 ? dispatch_d<bf16_t, true>(a, L)
                                   : dispatch_d<float, true>(a, L);
}

hipError_t launch_state_sum(Launcher& L, float* part, float* fin, int nseg, int rec, int BH,
                            hipStream_t s) {
  const int nchunk = (rec + 63) / 64;
  const dim3 cgrid((unsigned)std::min<long long>((long long)nchunk * BH, 0xFFFFFFFFll));
  L(FMM_KERNEL_STATE_COMBINE, k_state_combine<false>, cgrid, dim3(256), 0, s, part, fin, nseg,
    rec, nchunk);
  return L.err;
}

int tile_rows() { return TM; }

}  // namespace fmm
