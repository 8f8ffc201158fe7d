// The fast-weight forward and backward with the normalisation of k and q
// taken off their sequential paths: a parallel pass writes p(k) and p(q) of every position
// (fp32, in the layout of k) into caller-provided scratch, which the narrow
// scan (d = 16, 32) then reads in place of k and q.
#pragma once

#include <cstddef>

#include "fmm_launch.h"

namespace fmm {

// Bytes of scratch launch_fast_weight_pre uses (0 where the head width has no
// narrow scan: the scan then normalises in place).
size_t fast_weight_pre_bytes(int B, int H, int N, int d);

// launch_fast_weight with `pre` (fast_weight_pre_bytes bytes, 16-byte
// aligned, or null to normalise inside the scan) as the scratch for p(k) and
// p(q).
hipError_t launch_fast_weight_pre(Launcher& L, const FwArgs& a, float* pre);

// The same for the fast-weight backward: p(k), p(q) and the inverse sums
// 1 / sum(phi_1(k)), 1 / sum(phi_1(q)) of every position, read by its narrow
// sweeps.
size_t fast_weight_backward_pre_bytes(int B, int H, int N, int d);
hipError_t launch_fast_weight_backward_pre(Launcher& L, const FwBwdArgs& a, float* pre);

}  // namespace fmm
