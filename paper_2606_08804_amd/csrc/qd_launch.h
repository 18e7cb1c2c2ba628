// Host-side launchers of the Q-Delta kernels (internal to libqdelta.so).
#pragma once

#include <hip/hip_runtime.h>

#include "qd_common.h"

namespace qd {

enum Stage {
  ST_PREP_FWD = 0,
  ST_SCAN_FWD = 1,
  ST_PREP_BWD = 2,
  ST_SCAN_BWD = 3,
  ST_INTRA = 4,
  ST_STEP = 5,
  ST_REC_FWD = 6,
  ST_SEG_MAPS = 7,
  ST_SEG_COMPOSE = 8,
  ST_SEG_OUT = 9,
  ST_REC_BWD = 10,
  ST_COUNT = 11
};

// Records a HIP event on `st` before (after == 0) or after (after == 1) a
// kernel launch of `stage` while the measurement facility is active.
void prof_mark(int stage, int after, hipStream_t st);

// Chunk preparation (UT solve, WY factors) over all slots, then, if
// with_scan, the sequential forward state scan (+ chunk outputs when p.o is
// set).  in_bwd only labels the launches for the measurement facility (a
// backward that recomputes the saved context).
hipError_t launch_fwd(const Params& p, int dtype, int Dk, int Dv, int in_bwd, int with_scan,
                      hipStream_t st);

// Segment-parallel forward of a dense batch (p.n_seg segments of
// p.seg_chunks chunks per sequence; p.wSegOut, p.wSegIn set): preparation,
// segment maps, composition, outputs.
hipError_t launch_fwd_seg(const Params& p, int dtype, int Dk, int Dv, hipStream_t st);

// Backward once the saved context (states, D, b, W, P, M) is in place:
// reverse state scan, then the intra-chunk gradient kernel.
hipError_t launch_bwd(const Params& p, int dtype, int Dk, int Dv, hipStream_t st);

// Writes 0 to one device float (a gradient with nothing to sum).
hipError_t launch_zero(float* x, hipStream_t st);

// One token of the recurrence for N sequences.
hipError_t launch_step(int N, int H, int Dk, int Dv, int dtype, const void* q, const void* k,
                       const void* v, const float* beta, const float* lam, float lam_c, const float* la,
                       float* state, void* o, hipStream_t st);

// Fully recurrent forward over whole sequences: dense (cu == nullptr, N
// sequences of T tokens) or packed (cu[N+1] on the device, T_total tokens).
hipError_t launch_rec_fwd(int N, int T, const int* cu, int T_total, int H, int Dk, int Dv,
                          int dtype, const void* q, const void* k, const void* v,
                          const float* beta, const float* lam, float lam_c, const float* la,
                          const float* S0, float* Sfin, void* o, hipStream_t st);

// Arguments of the fully recurrent backward (one workgroup per (sequence,
// head) unit).
struct RecBwdArgs {
  int T;                    // dense: tokens per sequence
  const int* cu;            // varlen: cu_seqlens[N+1] (device), clamped to [0, T_total]
  int T_total;
  int H, DV;
  const void *q, *k, *v, *dO;
  const float *beta, *lam, *la, *S0, *dSfin;
  float lam_c;              // lambda when lam is nullptr
  void *dq, *dk, *dv;
  float *dbeta, *dlam, *dla, *dS0;
  float* wDL;               // per token-head gradient of a constant lambda (else nullptr)
  float *wP, *wZ, *wDP, *wWK, *wF;   // workspace: [tok][H][DV] x3 and [tok][H][DK] fp32, [unit][DV] fp32
};

// Fully recurrent backward over `units` (sequence, head) units; when
// dlam_sum is set, the constant lambda's gradient (sum of a.wDL over
// n_tok_heads entries) is written there.
hipError_t launch_rec_bwd(const RecBwdArgs& a, int units, int dtype, int Dk, float* dlam_sum, long long n_tok_heads,
                          hipStream_t st);

// Row L2 normalisation (bwd == 0: x -> out, rn_out) or its backward
// (bwd == 1: y, rn_in, dy -> out).
hipError_t launch_l2norm(int bwd, long rows, int D, long ldx, int dtype, const void* x,
                         const void* y, const float* rn_in, float* rn_out, const void* dy, void* out,
                         hipStream_t st);

}  // namespace qd
