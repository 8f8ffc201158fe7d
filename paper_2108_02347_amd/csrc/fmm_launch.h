// Host-side interface between the C ABI and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

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
  void* stream;
  float* ws;   // segment states (+ final state for the non-causal form)
  int nseg;        // state segments per (batch, head)
  int L;           // rows per state segment (multiple of the tile height)
  int nseg_apply;  // row segments walked by one non-causal apply workgroup
  int L_apply;     // rows per apply segment (multiple of the tile height)
};

// Supplies a start/stop HIP event pair per kernel launch when timing is
// enabled; the events are attached to the kernel's own dispatch
// (hipExtLaunchKernel), so they bracket exactly the kernel's execution.
struct LaunchTimer {
  virtual bool take(int kernel, hipEvent_t* start, hipEvent_t* stop) = 0;
  virtual void commit(int kernel, hipEvent_t start, hipEvent_t stop) = 0;
  virtual ~LaunchTimer() {}
};

hipError_t launch_forward(const LaunchArgs& a, LaunchTimer* timer);
int tile_rows();

}  // namespace fmm
