// Fast-weight far field (Appendix D): the linear transformer with the delta-
// rule fast weight update of the cited fast-weight-programmer work, causal.
// Per (batch, head), with p(x) = phi_1(x) / sum_c phi_1(x)_c (phi_1 = elu + 1):
//   u_i = W_{i-1} p(k_i);  W_i = W_{i-1} + beta_i (v_i - u_i) p(k_i)^T
//   z_i = z_{i-1} + p(k_i);  fw_i = W_i p(q_i) / (z_i . p(q_i))
// The recurrence is sequential in i; one workgroup runs one (batch, head)
// slice with one thread per row r of W (row r of W and z_r in registers), so
// a step is two length-d dot products per thread and the rank-one update of
// its row, plus three sums over the threads (sum of phi(k), sum of phi(q), the
// denominator), by DPP within the wave.  The next step's
// q, k, v, beta and output row are loaded while the current one computes (a
// load issued in the step that needs it would hold up every later load: the
// memory counter is waited for in order).  The kernel adds
// sigmoid(w_far[h]) fw_i to `out`, which already holds the rest of the
// operator (near field and, for the two-kernel variant, the linear far part).
#include <hip/hip_runtime.h>

#include "fmm_device.h"
#include "fmm_launch.h"

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

template <typename T, int D>
__global__ __launch_bounds__(D > 64 ? D : 64) void k_fast_weight(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ beta, T* __restrict__ out, const float* __restrict__ w_far, int H,
    int N) {
  constexpr int NWV = D > 64 ? D / 64 : 1;
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
  // the first step's inputs
  float xk = 0.f, xq = 0.f, xv = 0.f, bt = 0.f, xo = 0.f;
  if (N > 0) {
    if (act) {
      xk = ld_elem<T>(k + base + r);
      xq = ld_elem<T>(q + base + r);
      xv = ld_elem<T>(v + base + r);
      xo = ld_elem<T>(out + base + r);
    }
    bt = beta[(size_t)bh * N];
  }
  for (int i = 0; i < N; ++i) {
    const int par = i & 1;
    // prefetch step i + 1 (row i + 1 of out is not written before step i + 1)
    float nk = 0.f, nq = 0.f, nv = 0.f, nb = 0.f, no = 0.f;
    if (i + 1 < N) {
      const size_t o = base + (size_t)(i + 1) * D + r;
      if (act) {
        nk = ld_elem<T>(k + o);
        nq = ld_elem<T>(q + o);
        nv = ld_elem<T>(v + o);
        no = ld_elem<T>(out + o);
      }
      nb = beta[(size_t)bh * N + i + 1];
    }
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
    float u = 0.f;
#pragma unroll
    for (int c = 0; c < D; ++c) u = fmaf(wrow[c], pk_s[par][c], u);
    const float coef = bt * (xv - u);
    float num = 0.f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      wrow[c] = fmaf(coef, pk_s[par][c], wrow[c]);
      num = fmaf(wrow[c], pq_s[par][c], num);
    }
    zr += pk;
    const float den = block_sum<NWV, ROWS>(act ? zr * pq : 0.f, red + 4 * NWV, par);
    if (act && sf > 0.f) st_elem<T>(out + base + (size_t)i * D + r, xo + sf * (num / den));
    xk = nk;
    xq = nq;
    xv = nv;
    xo = no;
    bt = nb;
  }
}

template <typename T, int D>
void launch_fw_d(Launcher& L, const FwArgs& a) {
  L(FMM_KERNEL_FAST_WEIGHT, k_fast_weight<T, D>, dim3(a.B * a.H), dim3(D > 64 ? D : 64), 0,
    (hipStream_t)a.stream, (const T*)a.q, (const T*)a.k, (const T*)a.v, a.beta, (T*)a.out,
    a.w_far, a.H, a.N);
}

template <typename T>
hipError_t launch_fw_t(Launcher& L, const FwArgs& a) {
  switch (a.d) {
    case 16: launch_fw_d<T, 16>(L, a); break;
    case 32: launch_fw_d<T, 32>(L, a); break;
    case 64: launch_fw_d<T, 64>(L, a); break;
    case 128: launch_fw_d<T, 128>(L, a); break;
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
  return a.dtype == FMM_DTYPE_BF16 ? launch_fw_t<bf16_t>(L, a) : launch_fw_t<float>(L, a);
}

hipError_t launch_fill(Launcher& L, float* p, int n, float x, void* stream) {
  L(FMM_KERNEL_FAST_WEIGHT, k_fill, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream, p,
    n, x);
  return L.err;
}

}  // namespace fmm
