// fmm_attn_forward_noalloc: the forward operator for callers that cannot
// allocate device memory (code under stream capture, tight serving loops).
// Its far-field segment records live in a fixed device array of this file,
// one copy per GPU, instead of a library- or caller-owned workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/fmm_attn.h"
#include "fmm_launch.h"

namespace {

// Room for the segment records of every workload the library is tuned for
// (2^16 tokens x 8 heads of width 64, rank 2, needs 16.5 MiB).  Each GPU the
// library runs on holds one copy until the process ends.
constexpr size_t kScratchBytes = (size_t)32 << 20;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

// Device address of `scratch` per GPU, looked up once with that GPU current.
// In host code the name `scratch` is only a host-side handle: it is never
// passed to a kernel or a copy; the looked-up address is.
std::mutex& scratch_mutex() {
  static std::mutex* m = new std::mutex();
  return *m;
}
void* scratch_addr[kMaxDevices] = {};

int scratch_for_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return FMM_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return FMM_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> g(scratch_mutex());
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return FMM_ERR_HIP;
    }
    scratch_addr[dev] = p;
  }
  *out = scratch_addr[dev];
  return FMM_OK;
}

}  // namespace

extern "C" {

size_t fmm_attn_noalloc_max_bytes(void) { return kScratchBytes; }

int fmm_attn_forward_noalloc(const void* q, const void* k, const void* v, void* out, int B,
                             int H, int N, int d, int band_k, int rank, int causal,
                             const float* w_near, const float* w_far, int dtype,
                             void* stream) {
  // argument errors first, so they are reported as such whatever the size
  int st = fmm::validate_forward(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far,
                                 dtype);
  if (st != FMM_OK) return st;
  const size_t need = fmm::forward_workspace_bytes(B, H, N, d, band_k, rank, causal, dtype);
  if (need == 0) return FMM_ERR_UNSUPPORTED;
  if (need > kScratchBytes) return FMM_ERR_SCRATCH;
  void* ws = nullptr;
  st = scratch_for_current_device(&ws);
  if (st != FMM_OK) return st;
  // every record the kernels read is written earlier in the same call, so
  // nothing in the array needs clearing between calls
  return fmm::forward_with_workspace(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near,
                                     w_far, dtype, ws, kScratchBytes, stream);
}

}  // extern "C"
