// Host-side launchers of the Q-Delta kernels (internal to libqdelta.so).
#pragma once

#include <hip/hip_runtime.h>

#include "qd_common.h"

namespace qd {

// Chunk preparation (UT solve, WY factors) over all slots, then, if
// with_scan, the sequential forward state scan (+ chunk outputs when p.o is
// set).  bwd_prep also stores T and P^T for the backward kernels.
hipError_t launch_fwd(const Params& p, int dtype, int Dk, int Dv, int bwd_prep, int with_scan,
                      hipStream_t st);

// Backward after the preparation and the saved states are in place: reverse
// state scan, then the two intra-chunk gradient kernels.
hipError_t launch_bwd(const Params& p, int dtype, int Dk, int Dv, hipStream_t st);

// One token of the recurrence for N sequences.
hipError_t launch_step(int N, int H, int Dk, int Dv, int dtype, const void* q, const void* k,
                       const void* v, const float* beta, const float* lam, const float* la,
                       float* state, void* o, hipStream_t st);

}  // namespace qd
