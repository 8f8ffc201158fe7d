// The attention layer around the operator: the Step-1 projections of Sec. 1.1
// ([q | k | v] = x W_qkv per token), the FMMformer operator per head, and the
// output projection (heads concatenated per token, times W_out).
//
//   x [B, N, E] --GEMM--> qkv [B*N, 3E] --k_split_heads--> q, k, v [B, H, N, d]
//     --operator--> o [B, H, N, d] --k_merge_heads--> m [B*N, E] --GEMM--> y [B, N, E]
//
// bf16 with E a multiple of 32 up to 128 (the long-range models' 64-wide
// embedding among them): each projection is one kernel of this file that
// reads its input rows once and writes its output in the layout the next
// step reads (k_proj: x -> q, k, v per head; heads -> y), matrix-core
// products with fp32 accumulation.  Otherwise the projections go to rocBLAS
// (gemm_ex, fp32 accumulation, the storage type in and out) with the head
// split and merge as coalesced 16-byte copies.  The operator is this
// library's either way.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include "fmm_device.h"
#include "fmm_launch.h"
#include "fmm_oct.h"

namespace fmm {
namespace {

// One 16-byte chunk per thread.  qkv row t = b*N + n holds [q | k | v], each
// part E = H*d wide with the heads in order; chunk c of the row covers
// columns 8c .. 8c+7 (bf16) or 4c .. 4c+3 (fp32), which never straddle a head
// since d is a multiple of 16.
// (parts = 1: rows of one E-wide part, into q only)
template <typename T>
__global__ __launch_bounds__(256) void k_split_heads(const T* __restrict__ qkv,
                                                     T* __restrict__ q, T* __restrict__ k,
                                                     T* __restrict__ v, long long nchunk, int N,
                                                     int H, int d, int parts) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= nchunk) return;
  const int E = H * d, cpr = parts * E / EPC;
  const long long t = i / cpr;
  const int col = (int)(i - t * cpr) * EPC;
  const int part = col / E, h = (col % E) / d, c = col % d;
  const long long b = t / N, n = t - b * N;
  T* dst = part == 0 ? q : (part == 1 ? k : v);
  const uint4 val = *reinterpret_cast<const uint4*>(qkv + t * parts * E + col);
  *reinterpret_cast<uint4*>(dst + (((b * H + h) * N + n) * d + c)) = val;
}

// o [B, H, N, d] -> m [B*N, E] (the heads of a token side by side), in rows
// of row_len elements from column col0 (E and 0 for the layer's forward).
template <typename T>
__global__ __launch_bounds__(256) void k_merge_heads(const T* __restrict__ o, T* __restrict__ m,
                                                     long long nchunk, int N, int H, int d,
                                                     int row_len, int col0) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= nchunk) return;
  const int E = H * d, cpr = E / EPC;
  const long long t = i / cpr;
  const int col = (int)(i - t * cpr) * EPC;
  const int h = col / d, c = col % d;
  const long long b = t / N, n = t - b * N;
  const uint4 val = *reinterpret_cast<const uint4*>(o + (((b * H + h) * N + n) * d + c));
  *reinterpret_cast<uint4*>(m + t * row_len + col0 + col) = val;
}

template <typename T>
void launch_split(Launcher& L, const void* qkv, void* q, void* k, void* v, int B, int N, int H,
                  int d, hipStream_t s, int parts = 3) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long nchunk = (long long)B * N * parts * H * d / EPC;
  const long long nb = (nchunk + 255) / 256;
  L(FMM_KERNEL_LAYER_COPY, k_split_heads<T>, dim3((unsigned)std::min<long long>(nb, 0xFFFFFFFFll)),
    dim3(256), 0, s, (const T*)qkv, (T*)q, (T*)k, (T*)v, nchunk, N, H, d, parts);
}

template <typename T>
void launch_merge(Launcher& L, const void* o, void* m, int B, int N, int H, int d,
                  hipStream_t s, int row_len = 0, int col0 = 0) {
  constexpr int EPC = 16 / (int)sizeof(T);
  const long long nchunk = (long long)B * N * H * d / EPC;
  const long long nb = (nchunk + 255) / 256;
  L(FMM_KERNEL_LAYER_COPY, k_merge_heads<T>, dim3((unsigned)std::min<long long>(nb, 0xFFFFFFFFll)),
    dim3(256), 0, s, (const T*)o, (T*)m, nchunk, N, H, d, row_len > 0 ? row_len : H * d, col0);
}

// ------------------------------------------------------------------ k_proj
// One projection of the layer for bf16, E = K = 32 KB (KB = 1 .. 4):
// out[t][c] = sum_e in[t][e] W[e][c], c < OUTC (3E for QKV, E for the
// output).  MODE 0 (QKV): in = x rows [T, E]; column c goes to q, k or v
// (c / E), head (c % E) / d, feature c % d of [B, H, N, d].  MODE 1 (output):
// in row t = the heads' outputs of token t side by side (gathered from
// [B, H, N, d]); out = y rows [T, E].
//
// A workgroup (4 waves) takes 64 tokens, a wave 16.  W is staged in LDS
// (rows padded by 8 elements); the product is formed transposed, D[c][t] =
// sum_e W[e][c] in[t][e]: the W operand comes from transposed LDS reads
// (keys 4g.. and 16 + 4g.. of each 32-wide block, as the P V product reads V),
// the token operand straight from memory in the same order, and each lane
// ends with four consecutive columns of one token, stored as 8 bytes.
template <int E, int MODE>
__global__ __launch_bounds__(256) void k_proj(const bf16_t* __restrict__ in,
                                              const bf16_t* __restrict__ w,
                                              bf16_t* __restrict__ o0, bf16_t* __restrict__ o1,
                                              bf16_t* __restrict__ o2, int T, int N, int H,
                                              int d) {
  constexpr int OUTC = MODE == 0 ? 3 * E : E;
  constexpr int KB = E / 32, NCB = OUTC / 16;
  constexpr int WS = OUTC + 8;  // padded LDS row (elements)
  static_assert(E % 32 == 0 && E <= 128, "E = 32, 64, 96 or 128");
  __shared__ __attribute__((aligned(16))) bf16_t wl[E * WS];
  for (int i = threadIdx.x; i < E * (OUTC / 8); i += 256) {
    const int row = i / (OUTC / 8), c8 = i % (OUTC / 8);
    *reinterpret_cast<uint4*>(wl + row * WS + 8 * c8) =
        *reinterpret_cast<const uint4*>(w + (size_t)row * OUTC + 8 * c8);
  }
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const long long tok = (long long)blockIdx.x * 64 + 16 * wv + r;  // this lane's token
  const bool ok = tok < T;
  const long long b = ok ? tok / N : 0, n = ok ? tok - b * N : 0;
  // in[tok][k .. k+3] as 8 bytes (zero past T)
  auto piece = [&](int kk) -> uint2 {
    if (!ok) return make_uint2(0u, 0u);
    if constexpr (MODE == 0) {
      return *reinterpret_cast<const uint2*>(in + tok * E + kk);
    } else {
      const int hh = kk / d, f = kk - hh * d;
      return *reinterpret_cast<const uint2*>(in + (((b * H + hh) * N + n) * d + f));
    }
  };
  Oct xo[KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) xo[kb] = oct_of(piece(32 * kb + 4 * g), piece(32 * kb + 16 + 4 * g));
  __syncthreads();
  // lane (t, g) of a transposed read: W row 4g + t/4, columns 16cb + 4(t%4) .. +3
  const int tr_off = (4 * g + (r >> 2)) * WS + 4 * (r & 3);
#pragma unroll 4
  for (int cb = 0; cb < NCB; ++cb) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const unsigned char* p =
          reinterpret_cast<const unsigned char*>(wl + (32 * kb) * WS + 16 * cb + tr_off);
      const Oct wo = oct_of(ld_tr16(p), ld_tr16(p + 16 * WS * 2));
      acc = mma8(wo, xo[kb], acc);
    }
    if (!ok) continue;
    // lane (r, g): columns 16cb + 4g .. +3 of token tok
    const int c = 16 * cb + 4 * g;
    const uint2 val = quad_pack(acc);
    if constexpr (MODE == 0) {
      const int part = c / E, hc = c - part * E, hh = hc / d, f = hc - hh * d;
      bf16_t* dst = part == 0 ? o0 : (part == 1 ? o1 : o2);
      *reinterpret_cast<uint2*>(dst + (((b * H + hh) * N + n) * d + f)) = val;
    } else {
      *reinterpret_cast<uint2*>(o0 + tok * E + c) = val;
    }
  }
}

template <int E>
void launch_proj_e(Launcher& L, bool qkv, const void* in, const void* w, void* o0, void* o1,
                   void* o2, int B, int N, int H, int d, hipStream_t s) {
  const long long T = (long long)B * N;
  const dim3 grid((unsigned)std::min<long long>((T + 63) / 64, 0xFFFFFFFFll));
  if (qkv)
    L(FMM_KERNEL_LAYER_COPY, k_proj<E, 0>, grid, dim3(256), 0, s, (const bf16_t*)in,
      (const bf16_t*)w, (bf16_t*)o0, (bf16_t*)o1, (bf16_t*)o2, (int)T, N, H, d);
  else
    L(FMM_KERNEL_LAYER_COPY, k_proj<E, 1>, grid, dim3(256), 0, s, (const bf16_t*)in,
      (const bf16_t*)w, (bf16_t*)o0, (bf16_t*)nullptr, (bf16_t*)nullptr, (int)T, N, H, d);
}

// Row-major C [M, Nc] = A [M, K] B [K, Nc] as the column-major product
// C^T = B^T A^T.
// With ta (tb): A (B) is stored transposed, i.e. A is [K, M] (B is [Nc, K])
// row-major and the product uses its transpose.
hipError_t gemm_rm(rocblas_handle hdl, int dtype, const void* A, const void* Bm, void* C, int M,
                   int K, int Nc, bool ta = false, bool tb = false) {
  const rocblas_datatype t =
      dtype == FMM_DTYPE_BF16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const float one = 1.f, zero = 0.f;
  const rocblas_status st = rocblas_gemm_ex(
      hdl, tb ? rocblas_operation_transpose : rocblas_operation_none,
      ta ? rocblas_operation_transpose : rocblas_operation_none, Nc, M, K, &one, Bm, t,
      tb ? K : Nc, A, t, ta ? M : K, &zero, C, t, Nc, C, t, Nc, rocblas_datatype_f32_r,
      rocblas_gemm_algo_standard, 0, 0);
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

bool layer_proj_applies(int dtype, int E) {
  return dtype == FMM_DTYPE_BF16 && E % 32 == 0 && E >= 32 && E <= 128;
}

hipError_t launch_layer_proj(Launcher& L, bool qkv, const void* in, const void* w, void* o0,
                             void* o1, void* o2, int B, int N, int H, int d, hipStream_t s) {
  switch (H * d) {
    case 32: launch_proj_e<32>(L, qkv, in, w, o0, o1, o2, B, N, H, d, s); break;
    case 64: launch_proj_e<64>(L, qkv, in, w, o0, o1, o2, B, N, H, d, s); break;
    case 96: launch_proj_e<96>(L, qkv, in, w, o0, o1, o2, B, N, H, d, s); break;
    case 128: launch_proj_e<128>(L, qkv, in, w, o0, o1, o2, B, N, H, d, s); break;
    default: return L.note(hipErrorInvalidValue);
  }
  return L.err;
}

hipError_t layer_gemm(void* handle, void* stream, int dtype, const void* A, const void* Bm,
                      void* C, int M, int K, int Nc, bool ta, bool tb) {
  rocblas_handle hdl = (rocblas_handle)handle;
  if (rocblas_set_stream(hdl, (hipStream_t)stream) != rocblas_status_success)
    return hipErrorLaunchFailure;
  return gemm_rm(hdl, dtype, A, Bm, C, M, K, Nc, ta, tb);
}

// Weight gradients C [E, Nc] = A^T B with A [M, E] and B [M, Nc] row-major and
// M (the tokens) far larger than E and Nc: one product per chunk of KC tokens
// (a strided batch, fp32 results), then the chunks summed in order into C (the
// storage type).  A single product would leave most of the GPU idle (a few
// output tiles, each walking all M tokens).
namespace {
template <typename T>
__global__ __launch_bounds__(256) void k_sum_chunks(const float* __restrict__ part,
                                                    T* __restrict__ c, int n, int nchunk) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int j = 0; j < nchunk; ++j) s += part[(size_t)j * n + i];
  if constexpr (sizeof(T) == 2) c[i] = (T)f32_to_bf16_bits(s);
  else c[i] = s;
}
}  // namespace

size_t layer_wgrad_scratch_bytes(int M, int E, int Nc) {
  const int nchunk = (M + kWgradChunk - 1) / kWgradChunk;
  return (size_t)nchunk * E * Nc * sizeof(float);
}

hipError_t layer_wgrad(void* handle, Launcher& L, void* stream, int dtype, const void* A,
                       const void* Bm, void* C, int M, int E, int Nc, float* scratch) {
  const int nchunk = (M + kWgradChunk - 1) / kWgradChunk;
  const int n = E * Nc;
  hipStream_t s = (hipStream_t)stream;
  if (!L.dry) {
    rocblas_handle hdl = (rocblas_handle)handle;
    if (rocblas_set_stream(hdl, s) != rocblas_status_success) return L.note(hipErrorLaunchFailure);
    const rocblas_datatype t =
        dtype == FMM_DTYPE_BF16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
    const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
    const float one = 1.f, zero = 0.f;
    // column-major: C^T [Nc, E] = B^T [Nc, K] A [K, E] per chunk of K tokens;
    // the full chunks as one strided batch, a shorter last chunk as one more
    // product
    const int full = M / kWgradChunk, rem = M - full * kWgradChunk;
    auto batch = [&](int k, int count, const void* a0, const void* b0, float* c0) {
      return rocblas_gemm_strided_batched_ex(
          hdl, rocblas_operation_none, rocblas_operation_transpose, Nc, E, k, &one, b0, t, Nc,
          (rocblas_stride)k * Nc, a0, t, E, (rocblas_stride)k * E, &zero, c0,
          rocblas_datatype_f32_r, Nc, (rocblas_stride)n, c0, rocblas_datatype_f32_r, Nc,
          (rocblas_stride)n, count, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    };
    if (full > 0 && batch(kWgradChunk, full, A, Bm, scratch) != rocblas_status_success)
      return L.note(hipErrorLaunchFailure);
    if (rem > 0) {
      const size_t off = (size_t)full * kWgradChunk;
      const void* a1 = static_cast<const unsigned char*>(A) + off * E * es;
      const void* b1 = static_cast<const unsigned char*>(Bm) + off * Nc * es;
      if (batch(rem, 1, a1, b1, scratch + (size_t)full * n) != rocblas_status_success)
        return L.note(hipErrorLaunchFailure);
    }
  }
  const dim3 grid((n + 255) / 256);
  if (dtype == FMM_DTYPE_BF16)
    L(FMM_KERNEL_LAYER_COPY, k_sum_chunks<bf16_t>, grid, dim3(256), 0, s,
      (const float*)scratch, (bf16_t*)C, n, nchunk);
  else
    L(FMM_KERNEL_LAYER_COPY, k_sum_chunks<float>, grid, dim3(256), 0, s,
      (const float*)scratch, (float*)C, n, nchunk);
  return L.err;
}

hipError_t launch_layer_split1(Launcher& L, int dtype, const void* src, void* dst, int B, int N,
                               int H, int d, hipStream_t s) {
  if (dtype == FMM_DTYPE_BF16)
    launch_split<bf16_t>(L, src, dst, nullptr, nullptr, B, N, H, d, s, 1);
  else
    launch_split<float>(L, src, dst, nullptr, nullptr, B, N, H, d, s, 1);
  return L.err;
}

hipError_t launch_layer_merge_part(Launcher& L, int dtype, const void* src, void* dst, int part,
                                   int B, int N, int H, int d, hipStream_t s) {
  if (dtype == FMM_DTYPE_BF16)
    launch_merge<bf16_t>(L, src, dst, B, N, H, d, s, 3 * H * d, part * H * d);
  else
    launch_merge<float>(L, src, dst, B, N, H, d, s, 3 * H * d, part * H * d);
  return L.err;
}

void* layer_blas_handle_create() {
  rocblas_handle h = nullptr;
  if (rocblas_create_handle(&h) != rocblas_status_success) return nullptr;
  return (void*)h;
}

}  // namespace fmm
