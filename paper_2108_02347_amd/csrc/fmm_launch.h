// Host-side interface between the C ABI and the kernel launchers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>

#include <algorithm>
#include <atomic>

#include "../../include/fmm_attn.h"

namespace fmm {

struct LaunchArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  const float* w_near;
  const float* w_far;
  int B, H, N, d, band_k, rank, causal, dtype;
  int far_norm;    // FMM_FAR_NORM_PER_MAP or FMM_FAR_NORM_JOINT
  void* stream;
  float* ws;   // segment states (+ final state for the non-causal form)
  int nseg;        // state segments per (batch, head)
  int L;           // rows per state segment (multiple of the tile height)
  int nseg_apply;  // row segments walked by one non-causal apply workgroup
  int L_apply;     // rows per apply segment (multiple of the tile height)
  // one-launch path for short non-causal slices (k_band_fused): workgroups
  // per slice (0: the three-launch path), the call's epoch for its stamps,
  // and whether the workgroups exchange partial states (0: each computes its
  // slice's state itself)
  int fused_g = 0;
  unsigned long long epoch = 0;
  int exchange = 1;
};

// Supplies a start/stop HIP event pair per kernel launch when timing is
// enabled; the events are attached to the kernel's own dispatch
// (hipExtLaunchKernel), so they bracket exactly the kernel's execution.
struct LaunchTimer {
  virtual bool take(int kernel, hipEvent_t* start, hipEvent_t* stop) = 0;
  virtual void commit(int kernel, hipEvent_t start, hipEvent_t stop) = 0;
  virtual ~LaunchTimer() {}
};

// Launch `kern` on stream s; with timing enabled, the timer's events are
// attached to this dispatch.
template <typename F, typename... Args>
inline void launch_timed(LaunchTimer* t, int id, F kern, dim3 grid, dim3 block, size_t shm,
                         hipStream_t s, Args... args) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (t && t->take(id, &e0, &e1)) {
    hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)shm, s, e0, e1, 0, args...);
    t->commit(id, e0, e1);
  } else {
    hipLaunchKernelGGL(kern, grid, block, shm, s, args...);
  }
}

// Runs the launch sequence of one forward call in two passes over the same
// code: a dry pass that only checks every grid against the dispatch limits
// (work-items per dimension below 2^32) and raises the kernels' LDS limits,
// then the real pass that enqueues.  A call that fails the dry pass therefore
// enqueues nothing.  The first error stops every later launch.
struct Launcher {
  LaunchTimer* timer = nullptr;
  bool dry = false;
  hipError_t err = hipSuccess;

  template <typename F, typename... Args>
  void operator()(int id, F kern, dim3 grid, dim3 block, size_t shm, hipStream_t s,
                  Args... args) {
    if (err != hipSuccess) return;
    if (dry) {
      const unsigned long long lim = 0xFFFFFFFFull;
      if (grid.x == 0 || grid.y == 0 || grid.z == 0 ||
          (unsigned long long)grid.x * block.x > lim ||
          (unsigned long long)grid.y * block.y > lim ||
          (unsigned long long)grid.z * block.z > lim)
        err = hipErrorInvalidConfiguration;
      return;
    }
    launch_timed(timer, id, kern, grid, block, shm, s, args...);
    err = hipGetLastError();
  }
  // records the result of a host-side step (an LDS attribute, a dispatch)
  hipError_t note(hipError_t e) {
    if (err == hipSuccess) err = e;
    return err;
  }
};

// Raises a kernel's dynamic LDS limit to `bytes` on the current device, once
// per device (HIP keeps the attribute per device); `done` is the caller's
// per-kernel record of the devices already set (devices 0..63; others are set
// on every call).
inline hipError_t lds_limit_once(const void* kern, int bytes,
                                 std::atomic<unsigned long long>& done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return hipErrorNoDevice;
  }
  const unsigned long long bit = dev >= 0 && dev < 64 ? 1ull << dev : 0ull;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  const hipError_t e =
      hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  (void)hipGetLastError();
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
  return e;
}

// Enqueues the forward operator (or, with L.dry, only checks and prepares it).
hipError_t launch_forward(const LaunchArgs& a, Launcher& L);
int tile_rows();

// Non-causal apply with two 16-row strips per wavefront (fmm_pair.hip): bf16,
// d = 32 or 64, band half-width <= 64.  Its row segments are multiples of
// pair_tile_rows().
bool band_pair_applies(int dtype, int d, int band_k, int causal, long long n);
int pair_tile_rows();
hipError_t launch_band_pair(const LaunchArgs& a, Launcher& L, const float* fin);

// One launch for short non-causal slices (fmm_pair.hip, k_band_fused): the
// workgroups per slice G (one per 128-row tile) when the shape qualifies and
// B*H*G <= max_workgroups, else 0.
int fused_groups(int dtype, int d, int band_k, int rank, int causal, long long bh, long long n,
                 int max_workgroups);
hipError_t launch_band_fused(const LaunchArgs& a, Launcher& L);
// Its workspace: G partial records per slice, one total record per slice,
// two 8-byte stamps per workgroup.
struct FusedLayout {
  size_t off_part, off_tot, off_stamp, total;
};
inline FusedLayout fused_layout(long long bh, int G, long long rec) {
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  FusedLayout f;
  f.off_part = 0;
  f.off_tot = al((size_t)bh * G * rec * sizeof(float));
  f.off_stamp = f.off_tot + al((size_t)bh * rec * sizeof(float));
  f.total = f.off_stamp + al((size_t)bh * G * 2 * sizeof(unsigned long long));
  return f;
}
// polls of a stamp wait before a workgroup computes its slice's state itself
constexpr int kFusedSpinLimit = 20000;

// Causal apply with one 16-row strip per wavefront (fmm_causal.hip): bf16,
// d = 32 or 64, band half-width <= 64; walks the state segments (a.L rows,
// a multiple of tile_rows()) from their exclusive prefix records.
bool causal_strip_applies(int dtype, int d, int band_k, int causal, long long n);
hipError_t launch_causal_strip(const LaunchArgs& a, Launcher& L, const float* prefix);

// General apply kernel (fmm_wide.hip): any supported width, one to three
// feature maps, both far-field normalisations, both forms.  recs: the final
// records (non-causal) or the exclusive prefix records per state segment
// (causal, advanced in place).
hipError_t launch_wide(const LaunchArgs& a, Launcher& L, float* recs);

// Backward pass (fmm_bwd.hip).  The forward state (k_seg_state +
// k_state_combine into part / fin) is launched first by launch_state_only;
// launch_backward_tail then runs the row pass, the dS combine, the key pass
// and the blend-logit reduction.
struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  float* dw_near;
  float* dw_far;
  const float* w_near;
  const float* w_far;
  int B, H, N, d, band_k, rank, causal, dtype;
  void* stream;
  int nseg, L;      // state segments (as the forward plan)
  float* part;      // forward segment records (causal: exclusive prefix)
  float* fin;       // forward final records (non-causal)
  float* dpart;     // dS partial records per segment (causal: exclusive suffix)
  float* dfin;      // dS totals per slice (non-causal)
  float* rowstat;   // [B*H*N][3]: scaled row maximum, 1/l, D
  float* rowfar;    // [B*H*N][rank][2]: 1/den, dden
  float* dwpart;    // [B*H*nseg][2]: sums of g . near, g . far
  int far_norm = FMM_FAR_NORM_PER_MAP;  // of the forward whose gradients these are
};
hipError_t launch_state_only(const LaunchArgs& a, Launcher& L);
hipError_t launch_state_sum(Launcher& L, float* part, float* fin, int nseg, int rec, int BH,
                            hipStream_t s);
hipError_t launch_backward_tail(const BwdArgs& a, Launcher& L);

// Attention layer pieces (fmm_layer.hip): the head split / merge copies, the
// projections through rocBLAS (row-major C [M, Nc] = A [M, K] B [K, Nc] on
// `stream`), and a rocBLAS handle (nullptr on failure).
hipError_t launch_layer_copy(Launcher& L, bool split, int dtype, const void* src, void* d0,
                             void* d1, void* d2, int B, int N, int H, int d, hipStream_t s);
// The layer's projections as kernels of this library (fmm_layer.hip, k_proj):
// bf16 with E = 32, 64, 96 or 128.  qkv: x [B N, E] -> q, k, v [B, H, N, d]
// (o0, o1, o2); otherwise the heads [B, H, N, d] -> y [B N, E] (o0).
bool layer_proj_applies(int dtype, int E);
hipError_t launch_layer_proj(Launcher& L, bool qkv, const void* in, const void* w, void* o0,
                             void* o1, void* o2, int B, int N, int H, int d, hipStream_t s);
// ta (tb): A (B) stored transposed ([K, M] and [Nc, K] row-major).
hipError_t layer_gemm(void* handle, void* stream, int dtype, const void* A, const void* Bm,
                      void* C, int M, int K, int Nc, bool ta = false, bool tb = false);
void* layer_blas_handle_create();
// The layer's weight gradients C [E, Nc] = A^T B (A [M, E], B [M, Nc] of the
// storage type, C too): per chunk of kWgradChunk tokens into `scratch`
// (layer_wgrad_scratch_bytes), then summed in chunk order.
constexpr int kWgradChunk = 1024;
size_t layer_wgrad_scratch_bytes(int M, int E, int Nc);
hipError_t layer_wgrad(void* handle, Launcher& L, void* stream, int dtype, const void* A,
                       const void* Bm, void* C, int M, int E, int Nc, float* scratch);
// The layer's backward copies: [B N, E] rows -> [B, H, N, d] (split1), and
// [B, H, N, d] -> part `part` (E columns from part * E) of [B N, 3E] rows.
hipError_t launch_layer_split1(Launcher& L, int dtype, const void* src, void* dst, int B, int N,
                               int H, int d, hipStream_t s);
hipError_t launch_layer_merge_part(Launcher& L, int dtype, const void* src, void* dst, int part,
                                   int B, int N, int H, int d, hipStream_t s);

// Fast-weight far field (fmm_fastweight.hip): adds sigmoid(w_far) fw to out.
struct FwArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  void* out;
  const float* w_far;
  int B, H, N, d, dtype;
  void* stream;
};
hipError_t launch_fast_weight(Launcher& L, const FwArgs& a);
// Its backward (fmm_fastweight.hip): adds the fast-weight part's dq, dk, dv to
// the gradients in place, writes dbeta, and adds its share to dw_far; wst and
// zst hold W_i and z_i of every step (B*H*N*d*d and B*H*N*d floats), gfw one
// float per (batch, head).
struct FwBwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  float* dbeta;
  float* dw_far;
  const float* w_far;
  float* wst;
  float* zst;
  float* gfw;
  int B, H, N, d, dtype;
  void* stream;
};
hipError_t launch_fast_weight_backward(Launcher& L, const FwBwdArgs& a);
// n floats at p set to x (on `stream`)
hipError_t launch_fill(Launcher& L, float* p, int n, float x, void* stream);

// The C ABI's host logic (fmm_api.cpp), shared with the no-allocation entry
// point (fmm_noalloc.hip): argument checks, the workspace size of the call's
// segment plan, and the checked launch with a given workspace.
int validate_forward(const void* q, const void* k, const void* v, void* out, int B, int H,
                     int N, int d, int band_k, int rank, int causal, const float* w_near,
                     const float* w_far, int dtype);
size_t forward_workspace_bytes(int B, int H, int N, int d, int band_k, int rank, int causal,
                               int dtype);
int forward_with_workspace(const void* q, const void* k, const void* v, void* out, int B, int H,
                           int N, int d, int band_k, int rank, int causal, const float* w_near,
                           const float* w_far, int dtype, void* ws, size_t ws_bytes,
                           void* stream);

}  // namespace fmm
