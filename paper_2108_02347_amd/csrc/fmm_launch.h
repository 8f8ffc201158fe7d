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

// Records HIP events around kernel launches when timing is enabled.
struct LaunchTimer {
  virtual void begin(int kernel, hipStream_t s) = 0;
  virtual void end(int kernel, hipStream_t s) = 0;
  virtual ~LaunchTimer() {}
};

hipError_t launch_forward(const LaunchArgs& a, LaunchTimer* timer);
int tile_rows();

}  // namespace fmm
