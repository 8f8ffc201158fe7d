// The attention layer around the operator: the Step-1 projections of Sec. 1.1
// ([q | k | v] = x W_qkv per token), the FMMformer operator per head, and the
// output projection (heads concatenated per token, times W_out).
//
//   x [B, N, E] --GEMM--> qkv [B*N, 3E] --k_split_heads--> q, k, v [B, H, N, d]
//     --operator--> o [B, H, N, d] --k_merge_heads--> m [B*N, E] --GEMM--> y [B, N, E]
//
// The two projections are plain GEMMs and go to rocBLAS (gemm_ex, fp32
// accumulation, the storage type in and out); the head split and merge are
// coalesced 16-byte copies; the operator is this library's.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include "fmm_device.h"
#include "fmm_launch.h"

namespace fmm {
namespace {

// One 16-byte chunk per thread.  qkv row t = b*N + n holds [q | k | v], each
// part E = H*d wide with the heads in order; chunk c of the row covers
// columns 8c .. 8c+7 (bf16) or 4c .. 4c+3 (fp32), which never straddle a head
// since d is a multiple of 16.
template <typename T>
__global__ __launch_bounds__(256) void k_split_heads(const T* __restrict__ qkv,
                                                     T* __restrict__ q, T* __restrict__ k,
                                                     T* __restrict__ v, long long nchunk, int N,
                                                     int H, int d) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= nchunk) return;
  const int E = H * d, cpr = 3 * E / EPC;
  const long long t = i / cpr;
  const int col = (int)(i - t * cpr) * EPC;
  const int part = col / E, h = (col % E) / d, c = col % d;
  const long long b = t / N, n = t - b * N;
  T* dst = part == 0 ? q : (part == 1 ? k : v);
  const uint4 val = *reinterpret_cast<const uint4*>(qkv + t * 3 * E + col);
  *reinterpret_cast<uint4*>(dst + (((b * H + h) * N + n) * d + c)) = val;
}

// o [B, H, N, d] -> m [B*N, E] (the heads of a token side by side).
template <typename T>
__global__ __launch_bounds__(256) void k_merge_heads(const T* __restrict__ o, T* __restrict__ m,
                                                     long long nchunk, int N, int H, int d) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= nchunk) return;
  const int E = H * d, cpr = E / EPC;
  const long long t = i / cpr;
  const int col = (int)(i - t * cpr) * EPC;
  const int h = col / d, c = col % d;
  const long long b = t / N, n = t - b * N;
  const uint4 val = *reinterpret_cast<const uint4*>(o + (((b * H + h) * N + n) * d + c));
  *reinterpret_cast<uint4*>(m + t * E + col) = val;
}

template <typename T>
void launch_split(Launcher& L, const void* qkv, void* q, void* k, void* v, int B, int N, int H,
                  int d, hipStream_t s) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long nchunk = (long long)B * N * 3 * H * d / EPC;
  const long long nb = (nchunk + 255) / 256;
  L(FMM_KERNEL_LAYER_COPY, k_split_heads<T>, dim3((unsigned)std::min<long long>(nb, 0xFFFFFFFFll)),
    dim3(256), 0, s, (const T*)qkv, (T*)q, (T*)k, (T*)v, nchunk, N, H, d);
}

template <typename T>
void launch_merge(Launcher& L, const void* o, void* m, int B, int N, int H, int d,
                  hipStream_t s) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long nchunk = (long long)B * N * H * d / EPC;
  const long long nb = (nchunk + 255) / 256;
  L(FMM_KERNEL_LAYER_COPY, k_merge_heads<T>, dim3((unsigned)std::min<long long>(nb, 0xFFFFFFFFll)),
    dim3(256), 0, s, (const T*)o, (T*)m, nchunk, N, H, d);
}

// Row-major C [M, Nc] = A [M, K] B [K, Nc] as the column-major product
// C^T = B^T A^T.
hipError_t gemm_rm(rocblas_handle hdl, int dtype, const void* A, const void* Bm, void* C, int M,
                   int K, int Nc) {
  const rocblas_datatype t =
      dtype == FMM_DTYPE_BF16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const float one = 1.f, zero = 0.f;
  const rocblas_status st = rocblas_gemm_ex(
      hdl, rocblas_operation_none, rocblas_operation_none, Nc, M, K, &one, Bm, t, Nc, A, t, K,
      &zero, C, t, Nc, C, t, Nc, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  return st == rocblas_status_success ? hipSuccess : hipErrorLaunchFailure;
}

}  // namespace

hipError_t launch_layer_copy(Launcher& L, bool split, int dtype, const void* src, void* d0,
                             void* d1, void* d2, int B, int N, int H, int d, hipStream_t s) {
  if (dtype == FMM_DTYPE_BF16) {
    if (split) launch_split<bf16_t>(L, src, d0, d1, d2, B, N, H, d, s);
    else launch_merge<bf16_t>(L, src, d0, B, N, H, d, s);
  } else {
    if (split) launch_split<float>(L, src, d0, d1, d2, B, N, H, d, s);
    else launch_merge<float>(L, src, d0, B, N, H, d, s);
  }
  return L.err;
}

hipError_t layer_gemm(void* handle, void* stream, int dtype, const void* A, const void* Bm,
                      void* C, int M, int K, int Nc) {
  rocblas_handle hdl = (rocblas_handle)handle;
  if (rocblas_set_stream(hdl, (hipStream_t)stream) != rocblas_status_success)
    return hipErrorLaunchFailure;
  return gemm_rm(hdl, dtype, A, Bm, C, M, K, Nc);
}

void* layer_blas_handle_create() {
  rocblas_handle h = nullptr;
  if (rocblas_create_handle(&h) != rocblas_status_success) return nullptr;
  return (void*)h;
}

}  // namespace fmm
