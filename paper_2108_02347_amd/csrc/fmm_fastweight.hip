// Fast-weight far field (Appendix D): the linear transformer with the delta-
// rule fast weight update of the cited fast-weight-programmer work, causal.
// Per (batch, head), with p(x) = phi_1(x) / sum_c phi_1(x)_c (phi_1 = elu + 1):
//   u_i = W_{i-1} p(k_i);  W_i = W_{i-1} + beta_i (v_i - u_i) p(k_i)^T
//   z_i = z_{i-1} + p(k_i);  fw_i = W_i p(q_i) / (z_i . p(q_i))
// The recurrence is sequential in i; one workgroup runs one (batch, head)
// slice with one thread per row r of W (row r of W and z_r in registers), so
// a step is two length-d dot products per thread and the rank-one update of
// its row, plus three sums over the threads (sum of phi(k), sum of phi(q), the
// denominator), by DPP within the wave; for d = 16 and 32, 64 / d lanes share
// a row (k_fast_weight_narrow), which fills the wave and needs no LDS, and a
// parallel pass (k_fw_normalise) forms p(k) and p(q) of every position first,
// so that the sequential step does not normalise.  Each
// step's q, k, v, beta and output row are loaded a few steps ahead (memory
// latency is longer than a step, and a load issued in the step that needs it
// would hold up every later load: the memory counter is waited for in
// order).  The kernel adds
// sigmoid(w_far[h]) fw_i to `out`, which already holds the rest of the
// operator (near field and, for the two-kernel variant, the linear far part).
#include <hip/hip_runtime.h>

#include <atomic>
#include <type_traits>

#include "fmm_device.h"
#include "fmm_launch.h"
#include "fmm_fw.h"

namespace fmm {
namespace {

template <typename T> __device__ __forceinline__ float ld_elem(const T* p);
template <> __device__ __forceinline__ float ld_elem<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_elem<bf16_t>(const bf16_t* p) {
  return bf16_to_f32(*p);
}
template <typename T> __device__ __forceinline__ void st_elem(T* p, float x);
template <> __device__ __forceinline__ void st_elem<float>(float* p, float x) { *p = x; }
template <> __device__ __forceinline__ void st_elem<bf16_t>(bf16_t* p, float x) {
  *p = (bf16_t)f32_to_bf16_bits(x);
}

// x plus lane (lane ^ ...) of x as a DPP move: quad_perm(1,0,3,2) (0xB1),
// quad_perm(2,3,0,1) (0x4E), row_half_mirror (0x141), row_mirror (0x140).
template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                           0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the first 16 * ROWS lanes of the wave, in every lane: within each
// 16-lane row by four DPP steps (pairs, quads, halves, the row), then the
// rows' sums read out of lanes 0, 16, 32, 48.
template <int ROWS>
__device__ __forceinline__ float wave_sum(float x) {
  x = dpp_add<0xB1>(x);
  x = dpp_add<0x4E>(x);
  x = dpp_add<0x141>(x);
  x = dpp_add<0x140>(x);
  float s = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
#pragma unroll
  for (int rr = 1; rr < ROWS; ++rr)
    s += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16 * rr));
  return s;
}

// Sum over the workgroup's NWV waves (each lane contributes x; lanes past d
// contribute 0); every thread gets the total.  `red` holds NWV floats per
// parity slot, so consecutive calls alternate slots.
template <int NWV, int ROWS>
__device__ __forceinline__ float block_sum(float x, float* red, int slot) {
  x = wave_sum<ROWS>(x);
  if constexpr (NWV == 1) {
    return x;
  } else {
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[slot * NWV + w] = x;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NWV; ++i) s += red[slot * NWV + i];
    return s;
  }
}

// a . b over D features with four interleaved partial sums: a dependent chain
// of D / 4 + 2 operations instead of D, which is what each sequential step
// waits on
template <int D>
__device__ __forceinline__ float dot_split(const float* a, const float* b) {
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
  for (int c = 0; c < D; c += 4) {
    s0 = fmaf(a[c], b[c], s0);
    s1 = fmaf(a[c + 1], b[c + 1], s1);
    s2 = fmaf(a[c + 2], b[c + 2], s2);
    s3 = fmaf(a[c + 3], b[c + 3], s3);
  }
  return (s0 + s1) + (s2 + s3);
}

// Takes x out of its ring slot here: the register allocator then reuses the
// slot for the load issued next instead of copying the slot at the loop's
// back edge (a copy of a register whose load is in flight waits for it).
__device__ __forceinline__ void take(float& x) { asm volatile("" : "+v"(x)); }

// steps between loading a step's inputs and running it (even: the LDS
// buffers alternate by step parity; two for the widest heads, whose rows
// already fill the registers)
template <int D>
constexpr int ahead_steps() { return D >= 128 ? 2 : 4; }

template <typename T, int D>
__global__ __launch_bounds__(D > 64 ? D : 64) void k_fast_weight(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ beta, T* __restrict__ out, const float* __restrict__ w_far, int H,
    int N) {
  constexpr int NWV = D > 64 ? D / 64 : 1;
  constexpr int kAhead = ahead_steps<D>();
  constexpr int ROWS = D >= 64 ? 4 : D / 16;  // 16-lane rows holding features
  __shared__ float pk_s[2][D], pq_s[2][D];
  __shared__ float red[2 * 3 * NWV];
  const int bh = blockIdx.x, h = bh % H;
  const int r = threadIdx.x;
  const bool act = r < D;
  const size_t base = (size_t)bh * N * D;
  const float sf = sigmoidf_exact(w_far[h]);
  float wrow[D];
#pragma unroll
  for (int c = 0; c < D; ++c) wrow[c] = 0.f;
  float zr = 0.f;
  // a step's inputs are loaded kAhead steps before it runs (register ring,
  // slot t for the steps i = t mod kAhead), so that no step waits on memory
  // latency, which is longer than a step (row j of out is not written before
  // step j)
  // The loads are unconditional (positions past the end and idle lanes read a
  // valid element that is then ignored), so that every path issues the same
  // loads and each step waits only for its own.
  const int rl = act ? r : 0;
  float rk[kAhead], rq[kAhead], rv[kAhead], ro[kAhead], rb[kAhead];
  auto fetch = [&](int j, int t) {
    const int jc = j < N ? j : N - 1;
    const size_t o = base + (size_t)jc * D + rl;
    rk[t] = ld_elem<T>(k + o);
    rq[t] = ld_elem<T>(q + o);
    rv[t] = ld_elem<T>(v + o);
    ro[t] = ld_elem<T>(out + o);
    rb[t] = beta[(size_t)bh * N + jc];
  };
#pragma unroll
  for (int t = 0; t < kAhead; ++t) fetch(t, t);
  for (int i0 = 0; i0 < N; i0 += kAhead)
#pragma unroll
  for (int t = 0; t < kAhead; ++t) {
    const int i = i0 + t;
    if (i >= N) break;
    const int par = t & 1;
    float xk = act ? rk[t] : 0.f, xq = act ? rq[t] : 0.f, xv = act ? rv[t] : 0.f;
    float xo = act ? ro[t] : 0.f, bt = rb[t];
    take(xk), take(xq), take(xv), take(xo), take(bt);
    fetch(i + kAhead, t);
    const float fk = act ? phi_l(xk, 0) : 0.f;
    const float fq = act ? phi_l(xq, 0) : 0.f;
    const float sk = block_sum<NWV, ROWS>(fk, red, 0);
    const float sq = block_sum<NWV, ROWS>(fq, red + 2 * NWV, 0);
    const float pk = fk / sk, pq = fq / sq;
    if (act) {
      pk_s[par][r] = pk;
      pq_s[par][r] = pq;
    }
    // (one wave: its own LDS writes are seen by its later reads)
    if constexpr (NWV > 1) __syncthreads();
    // u_r = W_r . p(k); W_r += beta (v_r - u_r) p(k); num_r = W_r . p(q)
    const float u = dot_split<D>(wrow, pk_s[par]);
    const float coef = bt * (xv - u);
#pragma unroll
    for (int c = 0; c < D; ++c) wrow[c] = fmaf(coef, pk_s[par][c], wrow[c]);
    const float num = dot_split<D>(wrow, pq_s[par]);
    zr += pk;
    const float den = block_sum<NWV, ROWS>(act ? zr * pq : 0.f, red + 4 * NWV, par);
    if (act && sf > 0.f) st_elem<T>(out + base + (size_t)i * D + r, xo + sf * (num / den));
  }
}

// Narrow heads (d = 16, 32): 64 / d lanes share a row of W, each holding
// d / (64 / d) of its columns and the same columns of z, so that the wave has
// no idle lanes and a step needs no LDS: every lane forms p(k) and p(q) for
// its own columns (the sums over the features by DPP within the row's
// lanes), and the three length-d dot products (W_r . p(k), W_r . p(q),
// z . p(q)) are partial sums over the lane's columns plus the same DPP steps.
// Lane 0 of each row's group writes that row's output.
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
  if constexpr (LPR >= 2) x = dpp_add<0xB1>(x);
  if constexpr (LPR >= 4) x = dpp_add<0x4E>(x);
  return x;
}

template <typename T, int D, bool PRE>
__global__ __launch_bounds__(64) void k_fast_weight_narrow(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ beta, T* __restrict__ out, const float* __restrict__ w_far,
    const float* __restrict__ pre, int H, int N) {
  static_assert(D == 16 || D == 32, "rows shared by 64 / d lanes");
  constexpr int LPR = 64 / D;    // lanes per row of W
  constexpr int CPL = D / LPR;   // columns per lane
  constexpr int NQ = CPL / 4;    // quads per lane
  constexpr int kAhead = D <= 16 ? 8 : ahead_steps<D>();  // (d = 16: registers to spare)
  // PRE: p(k) and p(q) of every position already formed by k_fw_normalise
  // (pre holds p(k), then p(q), fp32 in the layout of k); else from k and q
  typedef typename std::conditional<PRE, float4, typename QuadOf<T>::type>::type quad_t;
  const int bh = blockIdx.x, h = bh % H;
  const int lane = threadIdx.x;
  const int r = lane / LPR, c0 = (lane % LPR) * CPL;
  const size_t base = (size_t)bh * N * D;
  const size_t pq_off = (size_t)gridDim.x * N * D;
  const float sf = sigmoidf_exact(w_far[h]);
  float w[CPL], z[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) w[c] = z[c] = 0.f;
  // inputs kAhead steps ahead in a register ring, as in k_fast_weight
  quad_t rk[kAhead][NQ], rq[kAhead][NQ];
  float rv[kAhead], ro[kAhead], rb[kAhead];
  auto fetch = [&](int j, int t) {
    const int jc = j < N ? j : N - 1;
    const size_t o = base + (size_t)jc * D;
#pragma unroll
    for (int m = 0; m < NQ; ++m) {
      if constexpr (PRE) {
        rk[t][m] = *reinterpret_cast<const float4*>(pre + o + c0 + 4 * m);
        rq[t][m] = *reinterpret_cast<const float4*>(pre + pq_off + o + c0 + 4 * m);
      } else {
        rk[t][m] = *reinterpret_cast<const quad_t*>(k + o + c0 + 4 * m);
        rq[t][m] = *reinterpret_cast<const quad_t*>(q + o + c0 + 4 * m);
      }
    }
    rv[t] = ld_elem<T>(v + o + r);
    ro[t] = ld_elem<T>(out + o + r);
    rb[t] = beta[(size_t)bh * N + jc];
  };
#pragma unroll
  for (int t = 0; t < kAhead; ++t) fetch(t, t);
  for (int i0 = 0; i0 < N; i0 += kAhead)
#pragma unroll
  for (int t = 0; t < kAhead; ++t) {
    const int i = i0 + t;
    if (i >= N) break;
    float xk[CPL], xq[CPL];
#pragma unroll
    for (int m = 0; m < NQ; ++m) {
      quad_to_f32(rk[t][m], xk + 4 * m);
      quad_to_f32(rq[t][m], xq + 4 * m);
    }
    float xv = rv[t], xo = ro[t], bt = rb[t];
#pragma unroll
    for (int c = 0; c < CPL; ++c) take(xk[c]), take(xq[c]);
    take(xv), take(xo), take(bt);
    fetch(i + kAhead, t);
    float pk[CPL], pq[CPL];
    if constexpr (PRE) {
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        pk[c] = xk[c];
        pq[c] = xq[c];
      }
    } else {
      float fk[CPL], fq[CPL];
      float sk = 0.f, sq = 0.f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        fk[c] = phi_l(xk[c], 0);
        fq[c] = phi_l(xq[c], 0);
        sk += fk[c];
        sq += fq[c];
      }
      sk = row_sum<LPR>(sk);
      sq = row_sum<LPR>(sq);
      // one division per sum, then products (within an ulp or so of the
      // quotients, and a quarter of the instructions)
      const float ik = 1.f / sk, iq = 1.f / sq;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        pk[c] = fk[c] * ik;
        pq[c] = fq[c] * iq;
      }
    }
    // u_r = W_r . p(k); W_r += beta (v_r - u_r) p(k); num_r = W_r . p(q);
    // z += p(k); den = z . p(q)
    const float u = row_sum<LPR>(dot_split<CPL>(w, pk));
    const float coef = bt * (xv - u);
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      w[c] = fmaf(coef, pk[c], w[c]);
      z[c] += pk[c];
    }
    const float num = row_sum<LPR>(dot_split<CPL>(w, pq));
    const float den = row_sum<LPR>(dot_split<CPL>(z, pq));
    // (the hardware reciprocal, within an ulp: the division's refinement
    // would lengthen every step)
    if (lane % LPR == 0 && sf > 0.f)
      st_elem<T>(out + base + (size_t)i * D + r, xo + sf * (num * __builtin_amdgcn_rcpf(den)));
  }
}

// p(k) and p(q) of every position (fp32, in the layout of k), one thread per
// (slice, position): the normalisation the narrow scan would otherwise redo
// on its sequential path
template <typename T, int D>
__global__ __launch_bounds__(256) void k_fw_normalise(const T* __restrict__ k,
                                                      const T* __restrict__ q,
                                                      float* __restrict__ pre, size_t rows,
                                                      float* __restrict__ inv_sums) {
  const size_t row = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= rows) return;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    const T* x = (which ? q : k) + row * D;
    float* p = pre + (which ? rows * D : 0) + row * D;
    float f[D];
    float s = 0.f;
#pragma unroll
    for (int m = 0; m < D / 4; ++m) {
      quad_to_f32(*reinterpret_cast<const typename QuadOf<T>::type*>(x + 4 * m), f + 4 * m);
#pragma unroll
      for (int c = 4 * m; c < 4 * m + 4; ++c) {
        f[c] = phi_l(f[c], 0);
        s += f[c];
      }
    }
    const float inv = 1.f / s;
    if (inv_sums) inv_sums[which * rows + row] = inv;
#pragma unroll
    for (int c = 0; c < D; c += 4)
      *reinterpret_cast<float4*>(p + c) =
          make_float4(f[c] * inv, f[c + 1] * inv, f[c + 2] * inv, f[c + 3] * inv);
  }
}

// ------------------------------------------------------------------ backward
// Gradients of sum(f . fw) for f_i = sigmoid(w_far[h]) g_i, per (b, h), by the
// recurrence differentiated and run backwards (G_i: the gradient with respect
// to W_i including every later use, Zs_i: with respect to z_i):
//   n_i = W_i p(q_i),  s_i = z_i . p(q_i),  fw_i = n_i / s_i
//   dn_i = f_i / s_i,  ds_i = -(f_i . fw_i) / s_i
//   G_i = dn_i p(q_i)^T + G_{i+1} (I - beta_{i+1} p(k_{i+1}) p(k_{i+1})^T)
//   Zs_i = ds_i p(q_i) + Zs_{i+1}
//   dp(q_i) = W_i^T dn_i + ds_i z_i
//   e_i = v_i - W_{i-1} p(k_i),  gp_i = G_i p(k_i)
//   dv_i = beta_i gp_i,  dbeta_i = e_i . gp_i
//   dp(k_i) = beta_i (G_i^T e_i - W_{i-1}^T gp_i) + Zs_i
// then through p = phi_1 / sum(phi_1): dx = phi_1'(x) (dp - dp . p) / sum(phi_1).
// A forward sweep first stores W_i and z_i (thread r: row r of W_i, z_i[r]) in
// the workspace; the backward sweep keeps row r of G and Zs[r] in registers,
// forms the two column sums (W_i^T dn and G^T e - W_{i-1}^T gp) through LDS and
// adds its dq, dk, dv to the gradients already in place (the near field and
// the linear part, from the operator's backward); it writes dbeta and, per
// slice, sum_i g_i . fw_i for dw_far.
// PRE (d <= 32): p(k), p(q) and the inverse sums 1 / sum(phi_1(k)),
// 1 / sum(phi_1(q)) of every position already formed by k_fw_normalise in
// `pre` (p(k), p(q), then the two inverse sums); the narrow sweeps read them
// in place of k and q.
template <typename T, int D, bool PRE>
__global__ __launch_bounds__(D > 64 ? D : 64) void k_fast_weight_bwd(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ beta, const T* __restrict__ dout, T* __restrict__ dq,
    T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ dbeta,
    float* __restrict__ wst, float* __restrict__ zst, float* __restrict__ gfw,
    const float* __restrict__ w_far, const float* __restrict__ pre, int H, int N) {
  constexpr int NWV = D > 64 ? D / 64 : 1;
  const size_t prow = (size_t)gridDim.x * N;  // rows of pre
  const float* pre_q = PRE ? pre + prow * D : nullptr;
  const float* pre_ik = PRE ? pre + 2 * prow * D : nullptr;
  const float* pre_iq = PRE ? pre + 2 * prow * D + prow : nullptr;
  constexpr int kAhead = ahead_steps<D>();
  constexpr int ROWS = D >= 64 ? 4 : D / 16;
  constexpr int LD = D + 1;  // padded rows of the column-sum buffers
  __shared__ float pk_s[2][D], pq_s[2][D];
  __shared__ float red[2 * 3 * NWV];
  extern __shared__ __align__(16) float colbuf[];  // the two column-sum buffers
  float* cb1 = colbuf;
  float* cb2 = colbuf + D * LD;
  const int bh = blockIdx.x, h = bh % H;
  const int r = threadIdx.x;
  const bool act = r < D;
  const int rl = act ? r : 0;  // the row an idle lane reads (and ignores)
  const size_t base = (size_t)bh * N * D;
  float* ws = wst + (size_t)bh * N * D * D;
  float* zs = zst + (size_t)bh * N * D;
  const float sf = sigmoidf_exact(w_far[h]);
  int slot = 0;  // parity of the block sums' scratch
  auto bsum = [&](float x, int which) {
    const float t = block_sum<NWV, ROWS>(x, red + 2 * which * NWV, slot);
    return t;
  };
  auto norm_phi = [&](float x, float* p_s, float& p, float& sum) {
    const float f = act ? phi_l(x, 0) : 0.f;
    sum = bsum(f, 0);
    p = f / sum;
    if (act) p_s[r] = p;
  };

  // ---- forward sweep: W_i and z_i of every step into the workspace
  if constexpr (D <= 32) {
    // narrow heads: 64 / d lanes per row of W, each with d / (64 / d) of its
    // columns (and the same columns of z), as in k_fast_weight_narrow
    constexpr int LPR = 64 / D, CPL = D / LPR, NQ = CPL / 4;
    constexpr int kAheadF = D <= 16 ? 8 : kAhead;  // (d = 16: registers to spare)
    typedef typename std::conditional<PRE, float4, typename QuadOf<T>::type>::type quad_t;
    const int rn = r / LPR, c0 = (r % LPR) * CPL;
    float w[CPL], z[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) w[c] = z[c] = 0.f;
    quad_t rkq[kAheadF][NQ];
    float rv[kAheadF], rb[kAheadF];
    auto fetch = [&](int j, int t) {
      const int jc = j < N ? j : N - 1;
      const size_t o = base + (size_t)jc * D;
#pragma unroll
      for (int m = 0; m < NQ; ++m)
        rkq[t][m] = PRE ? *reinterpret_cast<const quad_t*>(pre + o + c0 + 4 * m)
                        : *reinterpret_cast<const quad_t*>(k + o + c0 + 4 * m);
      rv[t] = ld_elem<T>(v + o + rn);
      rb[t] = beta[(size_t)bh * N + jc];
    };
#pragma unroll
    for (int t = 0; t < kAheadF; ++t) fetch(t, t);
    for (int i0 = 0; i0 < N; i0 += kAheadF)
#pragma unroll
    for (int t = 0; t < kAheadF; ++t) {
      const int i = i0 + t;
      if (i >= N) break;
      float xk[CPL];
#pragma unroll
      for (int m = 0; m < NQ; ++m) quad_to_f32(rkq[t][m], xk + 4 * m);
      float xv = rv[t], bt = rb[t];
#pragma unroll
      for (int c = 0; c < CPL; ++c) take(xk[c]);
      take(xv), take(bt);
      fetch(i + kAheadF, t);
      float pk[CPL];
      if constexpr (PRE) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) pk[c] = xk[c];
      } else {
        float fk[CPL], sk = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          fk[c] = phi_l(xk[c], 0);
          sk += fk[c];
        }
        const float ik = 1.f / row_sum<LPR>(sk);
#pragma unroll
        for (int c = 0; c < CPL; ++c) pk[c] = fk[c] * ik;
      }
      const float u = row_sum<LPR>(dot_split<CPL>(w, pk));
      const float coef = bt * (xv - u);
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        w[c] = fmaf(coef, pk[c], w[c]);
        z[c] += pk[c];
      }
      float* dst = ws + ((size_t)i * D + rn) * D + c0;
#pragma unroll
      for (int c = 0; c < CPL; c += 4)
        *reinterpret_cast<float4*>(dst + c) = make_float4(w[c], w[c + 1], w[c + 2], w[c + 3]);
      if (rn == 0) {
#pragma unroll
        for (int c = 0; c < CPL; c += 4)
          *reinterpret_cast<float4*>(zs + (size_t)i * D + c0 + c) =
              make_float4(z[c], z[c + 1], z[c + 2], z[c + 3]);
      }
    }
  } else {
    float wrow[D];
#pragma unroll
    for (int c = 0; c < D; ++c) wrow[c] = 0.f;
    float zr = 0.f;
    // step i's inputs, loaded kAhead steps earlier (ring slot i mod kAhead)
    // (unconditional loads: past the end and on idle lanes a valid element
    // is read and ignored)
    float rk[kAhead], rv[kAhead], rb[kAhead];
    auto fetch = [&](int j, int t) {
      const int jc = j < N ? j : N - 1;
      const size_t oj = base + (size_t)jc * D + rl;
      rk[t] = ld_elem<T>(k + oj);
      rv[t] = ld_elem<T>(v + oj);
      rb[t] = beta[(size_t)bh * N + jc];
    };
#pragma unroll
    for (int t = 0; t < kAhead; ++t) fetch(t, t);
    for (int i0 = 0; i0 < N; i0 += kAhead)
#pragma unroll
    for (int t = 0; t < kAhead; ++t) {
      const int i = i0 + t;
      if (i >= N) break;
      const int par = t & 1;
      slot = par;
      float xk = act ? rk[t] : 0.f, xv = act ? rv[t] : 0.f, bt = rb[t];
      take(xk), take(xv), take(bt);
      fetch(i + kAhead, t);
      float pk, sk;
      norm_phi(xk, pk_s[par], pk, sk);
      if constexpr (NWV > 1) __syncthreads();
      const float u = dot_split<D>(wrow, pk_s[par]);
      const float coef = bt * (xv - u);
#pragma unroll
      for (int c = 0; c < D; ++c) wrow[c] = fmaf(coef, pk_s[par][c], wrow[c]);
      zr += pk;
      if (act) {
        float* dst = ws + ((size_t)i * D + r) * D;
#pragma unroll
        for (int c = 0; c < D; c += 4)
          *reinterpret_cast<float4*>(dst + c) =
              make_float4(wrow[c], wrow[c + 1], wrow[c + 2], wrow[c + 3]);
        zs[(size_t)i * D + r] = zr;
      }
    }
  }
  // the stores above are read back below by other threads of the workgroup
  __threadfence_block();
  __syncthreads();

  // ---- backward sweep
  float acc_gfw = 0.f;   // this thread's share of sum_i g_i . fw_i
  if constexpr (D == 16) {
    // d = 16: the row-wise work (G carried and updated, the row dot products,
    // the terms of the column sums) with four lanes per row of W, each on
    // four of its columns; the per-feature work (p at one feature, Zs, the
    // column sums read back, dq and dk) on lanes 0..15, one feature each.
    constexpr int LPR = 64 / D, CPL = D / LPR;
    constexpr int LDN = D + 4;  // padded, 16-byte aligned rows of the column-sum buffers
    static_assert(D * LPR == 64 && D % 8 == 0, "four quarters of the wave, two rows at a time");
    constexpr int kRingW = kAhead;
    typedef typename std::conditional<PRE, float4, typename QuadOf<T>::type>::type quad_t;
    static_assert(CPL == 4, "one quad of columns per lane");
    float* cn1 = colbuf;
    float* cn2 = colbuf + D * LDN;
    const int rn = r / LPR, g = r % LPR, c0 = g * CPL;
    const bool col = r < D;  // the lane of feature r
    float gr[CPL], pkn[CPL];  // row rn of G, p(k_{i+1}), at the lane's columns
#pragma unroll
    for (int c = 0; c < CPL; ++c) gr[c] = pkn[c] = 0.f;
    float zs_col = 0.f;  // Zs at feature r
    float bt_next = 0.f;
    // ring of W rows: slot (N - 1 - i) mod kRingW holds row rn of W_i at the
    // lane's columns; rows before the first read as W_0 and are ignored
    float wr[kRingW][CPL];
    auto ld_wrow = [&](int j, float* w) {
      const float4 a =
          *reinterpret_cast<const float4*>(ws + ((size_t)(j < 0 ? 0 : j) * D + rn) * D + c0);
      w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    };
    // step inputs kAhead steps ahead (unconditional loads, as above)
    quad_t rk[kAhead], rq[kAhead];
    float4 rz[kAhead];
    float rv[kAhead], rg[kAhead], rdv[kAhead], rb[kAhead];
    float rkc[kAhead], rqc[kAhead], rzc[kAhead], rdq[kAhead], rdk[kAhead];
    float rik[kAhead], riq[kAhead];  // PRE: the row's inverse sums
    auto fetch = [&](int j, int t) {
      const int jc = j < 0 ? 0 : j;
      const size_t o = base + (size_t)jc * D;
      if constexpr (PRE) {
        rk[t] = *reinterpret_cast<const quad_t*>(pre + o + c0);
        rq[t] = *reinterpret_cast<const quad_t*>(pre_q + o + c0);
        rkc[t] = pre[o + rl];
        rqc[t] = pre_q[o + rl];
        rik[t] = pre_ik[(size_t)bh * N + jc];
        riq[t] = pre_iq[(size_t)bh * N + jc];
      } else {
        rk[t] = *reinterpret_cast<const quad_t*>(k + o + c0);
        rq[t] = *reinterpret_cast<const quad_t*>(q + o + c0);
        rkc[t] = ld_elem<T>(k + o + rl);
        rqc[t] = ld_elem<T>(q + o + rl);
      }
      rz[t] = *reinterpret_cast<const float4*>(zs + (size_t)jc * D + c0);
      rv[t] = ld_elem<T>(v + o + rn);
      rg[t] = ld_elem<T>(dout + o + rn);
      rdv[t] = ld_elem<T>(dv + o + rn);
      rzc[t] = zs[(size_t)jc * D + rl];
      rdq[t] = ld_elem<T>(dq + o + rl);
      rdk[t] = ld_elem<T>(dk + o + rl);
      rb[t] = beta[(size_t)bh * N + jc];
    };
#pragma unroll
    for (int t = 0; t < kRingW; ++t) ld_wrow(N - 1 - t, wr[t]);
#pragma unroll
    for (int t = 0; t < kAhead; ++t) fetch(N - 1 - t, t);
    for (int i0 = N - 1; i0 >= 0; i0 -= kAhead)
#pragma unroll
    for (int t = 0; t < kAhead; ++t) {
      const int i = i0 - t;
      if (i < 0) break;
      float xk[CPL], xq[CPL];
      quad_to_f32(rk[t], xk);
      quad_to_f32(rq[t], xq);
      float zi[CPL] = {rz[t].x, rz[t].y, rz[t].z, rz[t].w};
      float xv = rv[t], xg = rg[t], odv = rdv[t], bt = rb[t];
      float xkc = rkc[t], xqc = rqc[t], zic = rzc[t], odq = rdq[t], odk = rdk[t];
      float xik = 0.f, xiq = 0.f;
      if constexpr (PRE) {
        xik = rik[t];
        xiq = riq[t];
        take(xik), take(xiq);
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) take(xk[c]), take(xq[c]), take(zi[c]);
      take(xv), take(xg), take(odv), take(bt);
      take(xkc), take(xqc), take(zic), take(odq), take(odk);
      fetch(i - kAhead, t);
      const float* wi = wr[t % kRingW];
      const float* wp = wr[(t + 1) % kRingW];  // W_{i-1} (W_0 at i = 0, ignored)
      const float wm = i > 0 ? 1.f : 0.f;
      // G_{i+1} carried back through step i + 1's write
      if (i + 1 < N) {
        const float gp1 = row_sum<LPR>(dot_split<CPL>(gr, pkn));
        const float m = bt_next * gp1;
#pragma unroll
        for (int c = 0; c < CPL; ++c) gr[c] = fmaf(-m, pkn[c], gr[c]);
      }
      // p(k_i), p(q_i) at the lane's columns and at feature r
      float pk[CPL], pq[CPL], ik, iq, pkc, pqc;
      if constexpr (PRE) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          pk[c] = xk[c];
          pq[c] = xq[c];
        }
        ik = xik;
        iq = xiq;
        pkc = xkc;
        pqc = xqc;
      } else {
        float fk[CPL], fq[CPL], sk = 0.f, sq = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          fk[c] = phi_l(xk[c], 0);
          fq[c] = phi_l(xq[c], 0);
          sk += fk[c];
          sq += fq[c];
        }
        sk = row_sum<LPR>(sk);
        sq = row_sum<LPR>(sq);
        ik = 1.f / sk;
        iq = 1.f / sq;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          pk[c] = fk[c] * ik;
          pq[c] = fq[c] * iq;
        }
        pkc = phi_l(xkc, 0) * ik;
        pqc = phi_l(xqc, 0) * iq;
      }
      // n_r, s, fw_r; dn_r, ds
      const float nr = row_sum<LPR>(dot_split<CPL>(wi, pq));
      const float s_i = row_sum<LPR>(dot_split<CPL>(zi, pq));
      const float is = __builtin_amdgcn_rcpf(s_i);  // (the hardware reciprocal, within an ulp)
      const float fw = nr * is;
      const float gdot = wave_sum<4>(g == 0 ? xg * fw : 0.f);  // g_i . fw_i
      acc_gfw += r == 0 ? gdot : 0.f;
      const float dn = sf * xg * is;
      const float ds = -sf * gdot * is;
      // G_i, Zs_i
#pragma unroll
      for (int c = 0; c < CPL; ++c) gr[c] = fmaf(dn, pq[c], gr[c]);
      zs_col = fmaf(ds, pqc, zs_col);
      // e_r, gp_r, dbeta
      const float u = wm * row_sum<LPR>(dot_split<CPL>(wp, pk));
      const float gp = row_sum<LPR>(dot_split<CPL>(gr, pk));
      const float gpw = wm * gp;
      const float e = xv - u;
      const float db = wave_sum<4>(g == 0 ? e * gp : 0.f);
      // the column sums W_i^T dn and G_i^T e - W_{i-1}^T gp through LDS
      *reinterpret_cast<float4*>(cn1 + rn * LDN + c0) =
          make_float4(wi[0] * dn, wi[1] * dn, wi[2] * dn, wi[3] * dn);
      *reinterpret_cast<float4*>(cn2 + rn * LDN + c0) =
          make_float4(fmaf(gr[0], e, -wp[0] * gpw), fmaf(gr[1], e, -wp[1] * gpw),
                      fmaf(gr[2], e, -wp[2] * gpw), fmaf(gr[3], e, -wp[3] * gpw));
      __syncthreads();
      // each quarter of the wave sums four rows of feature r mod 16, then the
      // quarters' sums are added across the wave (lanes 16 and 32 apart)
      float c1, c2;
      {
        const int cc = r % D, r0 = (r / D) * (D / 4);
        float a0 = 0.f, a1 = 0.f, b0 = 0.f, b1 = 0.f;
#pragma unroll
        for (int rr = 0; rr < D / 4; rr += 2) {
          a0 += cn1[(r0 + rr) * LDN + cc];
          a1 += cn1[(r0 + rr + 1) * LDN + cc];
          b0 += cn2[(r0 + rr) * LDN + cc];
          b1 += cn2[(r0 + rr + 1) * LDN + cc];
        }
        c1 = a0 + a1;
        c2 = b0 + b1;
        c1 += __shfl_xor(c1, 16);
        c2 += __shfl_xor(c2, 16);
        c1 += __shfl_xor(c1, 32);
        c2 += __shfl_xor(c2, 32);
      }
      __syncthreads();  // the buffers are rewritten next step
      const float dpq = c1 + ds * zic;
      const float dpk = bt * c2 + zs_col;
      const float tq = wave_sum<1>(col ? dpq * pqc : 0.f);
      const float tk = wave_sum<1>(col ? dpk * pkc : 0.f);
      const size_t o = base + (size_t)i * D;
      if (col) {
        // phi_1'(x) / S = min(1, phi_1(x)) / S = min(1 / S, p(x))
        const float gq = (PRE ? fminf(iq, pqc) : (xqc > 0.f ? 1.f : __expf(xqc)) * iq) * (dpq - tq);
        const float gk = (PRE ? fminf(ik, pkc) : (xkc > 0.f ? 1.f : __expf(xkc)) * ik) * (dpk - tk);
        st_elem<T>(dq + o + r, odq + gq);
        st_elem<T>(dk + o + r, odk + gk);
      }
      if (g == 0) st_elem<T>(dv + o + rn, odv + bt * gp);
      if (r == 0) dbeta[(size_t)bh * N + i] = db;
      bt_next = bt;
#pragma unroll
      for (int c = 0; c < CPL; ++c) pkn[c] = pk[c];
      // W_i's slot takes W_{i-kRingW}
      ld_wrow(i - kRingW, wr[t % kRingW]);
    }
  } else {
  float grow[D];
#pragma unroll
  for (int c = 0; c < D; ++c) grow[c] = 0.f;
  float zsr = 0.f;       // Zs[r]
  float bt_next = 0.f;   // beta_{i+1}
  // row r of W_j (of W_0 for j < 0, which the step then ignores)
  auto ld_row = [&](int j, float* w) {
    const float* src = ws + ((size_t)(j < 0 ? 0 : j) * D + rl) * D;
#pragma unroll
    for (int c = 0; c < D; c += 4) {
      const float4 a = *reinterpret_cast<const float4*>(src + c);
      w[c] = a.x; w[c + 1] = a.y; w[c + 2] = a.z; w[c + 3] = a.w;
    }
  };
  // step i's inputs (and the gradients already in place at position i) are
  // loaded kAhead steps earlier (ring slot (N - 1 - i) mod kAhead); the rows
  // of W sit in a ring of kRingW slots (slot (N - 1 - i) mod kRingW holds W_i
  // at step i), refilled as soon as a step is done with its W_i, so W_j is
  // loaded kRingW - 1 steps before its first use (as many as the registers
  // allow)
  constexpr int kRingW = D <= 16 ? 4 : 2;
  static_assert(kAhead % kRingW == 0, "the W ring's slot must follow the step ring's");
  float wr[kRingW][D];
  float rk[kAhead], rq[kAhead], rv[kAhead], rg[kAhead], rb[kAhead], rz[kAhead];
  float rdq[kAhead], rdk[kAhead], rdv[kAhead];
  // (unconditional loads: before the start and on idle lanes a valid
  // element is read and ignored)
  auto fetch = [&](int j, int t) {
    const int jc = j < 0 ? 0 : j;
    const size_t oj = base + (size_t)jc * D + rl;
    rk[t] = ld_elem<T>(k + oj);
    rq[t] = ld_elem<T>(q + oj);
    rv[t] = ld_elem<T>(v + oj);
    rg[t] = ld_elem<T>(dout + oj);
    rb[t] = beta[(size_t)bh * N + jc];
    rz[t] = zs[(size_t)jc * D + rl];
    rdq[t] = ld_elem<T>(dq + oj);
    rdk[t] = ld_elem<T>(dk + oj);
    rdv[t] = ld_elem<T>(dv + oj);
  };
#pragma unroll
  for (int t = 0; t < kRingW; ++t) ld_row(N - 1 - t, wr[t]);
#pragma unroll
  for (int t = 0; t < kAhead; ++t) fetch(N - 1 - t, t);
  for (int i0 = N - 1; i0 >= 0; i0 -= kAhead)
#pragma unroll
  for (int t = 0; t < kAhead; ++t) {
    const int i = i0 - t;
    if (i < 0) break;
    const int par = i & 1;
    slot = par;
    const size_t o = base + (size_t)i * D + r;
    float xk = act ? rk[t] : 0.f, xq = act ? rq[t] : 0.f, xv = act ? rv[t] : 0.f;
    float xg = act ? rg[t] : 0.f, zi = act ? rz[t] : 0.f, bt = rb[t];
    float odq = rdq[t], odk = rdk[t], odv = rdv[t];
    take(xk), take(xq), take(xv), take(xg), take(zi), take(bt);
    take(odq), take(odk), take(odv);
    fetch(i - kAhead, t);
    const float* wi = wr[t % kRingW];
    const float* wp = wr[(t + 1) % kRingW];  // W_{i-1} (W_0 at i = 0, where W_{-1} = 0)
    const float wm = i > 0 ? 1.f : 0.f;
    // G_{i+1} carried back through step i + 1's write (p(k_{i+1}) still in
    // pk_s[par ^ 1], written last iteration)
    if (i + 1 < N) {
      const float gp1 = dot_split<D>(grow, pk_s[par ^ 1]);
      const float m = bt_next * gp1;
#pragma unroll
      for (int c = 0; c < D; ++c) grow[c] = fmaf(-m, pk_s[par ^ 1][c], grow[c]);
    }
    if constexpr (NWV > 1) __syncthreads();  // pk_s[par ^ 1] read before rewrite below
    float pk, sk, pq, sq;
    norm_phi(xk, pk_s[par], pk, sk);
    slot ^= 1;
    norm_phi(xq, pq_s[par], pq, sq);
    slot ^= 1;
    if constexpr (NWV > 1) __syncthreads();
    // n_r, s, fw_r; dn_r, ds
    const float nr = dot_split<D>(wi, pq_s[par]);
    const float s_i = bsum(act ? zi * pq : 0.f, 1);
    const float fw = nr / s_i;
    const float gdot = bsum(act ? xg * fw : 0.f, 2);  // g_i . fw_i
    acc_gfw += r == 0 ? gdot : 0.f;
    const float dn = act ? sf * xg / s_i : 0.f;
    const float ds = -sf * gdot / s_i;
    // G_i, Zs_i
#pragma unroll
    for (int c = 0; c < D; ++c) grow[c] = fmaf(dn, pq_s[par][c], grow[c]);
    zsr = fmaf(ds, pq, zsr);
    // e_r, gp_r, dv, dbeta
    const float u = wm * dot_split<D>(wp, pk_s[par]);
    const float gp = dot_split<D>(grow, pk_s[par]);
    const float gpw = wm * gp;
    const float e = act ? xv - u : 0.f;
    slot ^= 1;
    const float db = bsum(e * gp, 1);
    slot ^= 1;
    // the two column sums through LDS: W_i^T dn and G_i^T e - W_{i-1}^T gp
    if (act) {
#pragma unroll
      for (int c = 0; c < D; ++c) {
        cb1[r * LD + c] = wi[c] * dn;
        cb2[r * LD + c] = fmaf(grow[c], e, -wp[c] * gpw);
      }
    }
    __syncthreads();
    float c1 = 0.f, c2 = 0.f;
    if (act) {
      float a0 = 0.f, a1 = 0.f, b0 = 0.f, b1 = 0.f;
#pragma unroll
      for (int rr = 0; rr < D; rr += 2) {
        a0 += cb1[rr * LD + r];
        a1 += cb1[(rr + 1) * LD + r];
        b0 += cb2[rr * LD + r];
        b1 += cb2[(rr + 1) * LD + r];
      }
      c1 = a0 + a1;
      c2 = b0 + b1;
    }
    __syncthreads();  // the buffers are rewritten next step
    const float dpq = c1 + ds * zi;
    const float dpk = bt * c2 + zsr;
    const float tq = bsum(act ? dpq * pq : 0.f, 2);
    slot ^= 1;
    const float tk = bsum(act ? dpk * pk : 0.f, 2);
    slot ^= 1;
    if (act) {
      const float gq = (xq > 0.f ? 1.f : __expf(xq)) * (dpq - tq) / sq;
      const float gk = (xk > 0.f ? 1.f : __expf(xk)) * (dpk - tk) / sk;
      st_elem<T>(dq + o, odq + gq);
      st_elem<T>(dk + o, odk + gk);
      st_elem<T>(dv + o, odv + bt * gp);
    }
    if (r == 0) dbeta[(size_t)bh * N + i] = db;
    bt_next = bt;
    // W_i's slot takes W_{i-kRingW}
    ld_row(i - kRingW, wr[t % kRingW]);
  }
  }
  if (r == 0) gfw[bh] = acc_gfw;
}

// dw_far[h] += c (1 - c) sum_b sum_i g . fw over the slices of head h, in
// batch order
__global__ void k_fw_dw(const float* __restrict__ gfw, const float* __restrict__ w_far,
                        float* __restrict__ dw_far, int B, int H) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= H) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s += gfw[(size_t)b * H + h];
  const float c = sigmoidf_exact(w_far[h]);
  dw_far[h] += c * (1.f - c) * s;
}

template <typename T, int D, bool PRE>
void launch_fw_bwd_k(Launcher& L, const FwBwdArgs& a, float* pre) {
  // two D x (D + 4) buffers (rows padded by one float, or by four where
  // they are written as quads)
  const size_t lds = (size_t)2 * D * (D + 4) * sizeof(float);
  static std::atomic<unsigned long long> lds_set{0};
  if (L.note(lds_limit_once((const void*)k_fast_weight_bwd<T, D, PRE>, (int)lds, lds_set)) !=
      hipSuccess)
    return;
  L(FMM_KERNEL_FAST_WEIGHT, k_fast_weight_bwd<T, D, PRE>, dim3(a.B * a.H),
    dim3(D > 64 ? D : 64), lds, (hipStream_t)a.stream, (const T*)a.q, (const T*)a.k,
    (const T*)a.v, a.beta, (const T*)a.dout, (T*)a.dq, (T*)a.dk, (T*)a.dv, a.dbeta, a.wst, a.zst,
    a.gfw, a.w_far, (const float*)pre, a.H, a.N);
}

template <typename T, int D>
void launch_fw_bwd_d(Launcher& L, const FwBwdArgs& a, float* pre) {
  if constexpr (D <= 32) {
    if (pre) {
      const size_t rows = (size_t)a.B * a.H * a.N;
      L(FMM_KERNEL_FAST_WEIGHT, k_fw_normalise<T, D>, dim3((unsigned)((rows + 255) / 256)),
        dim3(256), 0, (hipStream_t)a.stream, (const T*)a.k, (const T*)a.q, pre, rows,
        pre + 2 * rows * D);
      launch_fw_bwd_k<T, D, true>(L, a, pre);
    } else {
      launch_fw_bwd_k<T, D, false>(L, a, nullptr);
    }
  } else {
    launch_fw_bwd_k<T, D, false>(L, a, nullptr);
  }
  L(FMM_KERNEL_FAST_WEIGHT, k_fw_dw, dim3((a.H + 63) / 64), dim3(64), 0, (hipStream_t)a.stream,
    (const float*)a.gfw, a.w_far, a.dw_far, a.B, a.H);
}

template <typename T>
hipError_t launch_fw_bwd_t(Launcher& L, const FwBwdArgs& a, float* pre) {
  switch (a.d) {
    case 16: launch_fw_bwd_d<T, 16>(L, a, pre); break;
    case 32: launch_fw_bwd_d<T, 32>(L, a, pre); break;
    case 64: launch_fw_bwd_d<T, 64>(L, a, pre); break;
    case 128: launch_fw_bwd_d<T, 128>(L, a, pre); break;
    default: return L.note(hipErrorInvalidValue);
  }
  return L.err;
}

template <typename T, int D>
void launch_fw_d(Launcher& L, const FwArgs& a, float* pre) {
  if constexpr (D <= 32) {
    if (pre) {
      const size_t rows = (size_t)a.B * a.H * a.N;
      L(FMM_KERNEL_FAST_WEIGHT, k_fw_normalise<T, D>, dim3((unsigned)((rows + 255) / 256)),
        dim3(256), 0, (hipStream_t)a.stream, (const T*)a.k, (const T*)a.q, pre, rows,
        (float*)nullptr);
      L(FMM_KERNEL_FAST_WEIGHT, k_fast_weight_narrow<T, D, true>, dim3(a.B * a.H), dim3(64), 0,
        (hipStream_t)a.stream, (const T*)a.q, (const T*)a.k, (const T*)a.v, a.beta, (T*)a.out,
        a.w_far, (const float*)pre, a.H, a.N);
    } else {
      L(FMM_KERNEL_FAST_WEIGHT, k_fast_weight_narrow<T, D, false>, dim3(a.B * a.H), dim3(64), 0,
        (hipStream_t)a.stream, (const T*)a.q, (const T*)a.k, (const T*)a.v, a.beta, (T*)a.out,
        a.w_far, (const float*)nullptr, a.H, a.N);
    }
  } else {
    L(FMM_KERNEL_FAST_WEIGHT, k_fast_weight<T, D>, dim3(a.B * a.H), dim3(D > 64 ? D : 64), 0,
      (hipStream_t)a.stream, (const T*)a.q, (const T*)a.k, (const T*)a.v, a.beta, (T*)a.out,
      a.w_far, a.H, a.N);
  }
}

template <typename T>
hipError_t launch_fw_t(Launcher& L, const FwArgs& a, float* pre) {
  switch (a.d) {
    case 16: launch_fw_d<T, 16>(L, a, pre); break;
    case 32: launch_fw_d<T, 32>(L, a, pre); break;
    case 64: launch_fw_d<T, 64>(L, a, pre); break;
    case 128: launch_fw_d<T, 128>(L, a, pre); break;
    default: return L.note(hipErrorInvalidValue);
  }
  return L.err;
}

__global__ void k_fill(float* __restrict__ p, int n, float x) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = x;
}

}  // namespace

hipError_t launch_fast_weight(Launcher& L, const FwArgs& a) {
  return launch_fast_weight_pre(L, a, nullptr);
}

size_t fast_weight_pre_bytes(int B, int H, int N, int d) {
  return d <= 32 ? (size_t)2 * B * H * N * d * sizeof(float) : 0;
}

hipError_t launch_fast_weight_pre(Launcher& L, const FwArgs& a, float* pre) {
  return a.dtype == FMM_DTYPE_BF16 ? launch_fw_t<bf16_t>(L, a, pre)
                                   : launch_fw_t<float>(L, a, pre);
}

hipError_t launch_fast_weight_backward(Launcher& L, const FwBwdArgs& a) {
  return launch_fast_weight_backward_pre(L, a, nullptr);
}

size_t fast_weight_backward_pre_bytes(int B, int H, int N, int d) {
  return d <= 32 ? (size_t)2 * B * H * N * (d + 1) * sizeof(float) : 0;
}

hipError_t launch_fast_weight_backward_pre(Launcher& L, const FwBwdArgs& a, float* pre) {
  return a.dtype == FMM_DTYPE_BF16 ? launch_fw_bwd_t<bf16_t>(L, a, pre)
                                   : launch_fw_bwd_t<float>(L, a, pre);
}

hipError_t launch_fill(Launcher& L, float* p, int n, float x, void* stream) {
  L(FMM_KERNEL_FAST_WEIGHT, k_fill, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream, p,
    n, x);
  return L.err;
}

}  // namespace fmm
