// Single-token Q-Delta update for N sequences (decode), Sec. 3.3
// Eq. (qdelta_decay) applied once per (sequence, head):
//
//   x = k + lambda q;  p = S x;  S <- alpha S + beta (v - alpha p) k^T;  o = S q
//
// Each state row S[v, :] is independent, so a row is owned by a group of
// Dk/4 lanes (one float4 each): the state is read once and written once with
// fully coalesced 16-byte accesses, and the two row dot products are reduced
// with cross-lane shuffles.  The kernel is bound by HBM (or MALL) bandwidth.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

// Each lane group owns RPT state rows RPB apart (RPB = rows per workgroup
// pass), so a wave has RPT independent 16-byte loads in flight instead of
// one; the per-row dot products are reduced side by side.
constexpr int STEP_RPT = 4;

template <typename E, int DK>
__global__ __launch_bounds__(NTHREADS) void k_step(int DV, int nrb, const E* __restrict__ q,
                                                  const E* __restrict__ k, const E* __restrict__ v,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ lam,
                                                  const float* __restrict__ la, float* __restrict__ S,
                                                  E* __restrict__ o) {
  constexpr int LPR = DK / 4;            // lanes per state row
  constexpr int RPB = NTHREADS / LPR;    // rows per workgroup pass
  constexpr int RPT = STEP_RPT;          // passes (rows per lane group)
  const size_t u = blockIdx.x / nrb;     // (sequence, head) unit
  const int rb = blockIdx.x % nrb;       // block of RPB * RPT state rows
  const int tid = threadIdx.x;
  const int row0 = rb * RPB * RPT + tid / LPR;
  const int c0 = (tid % LPR) * 4;
  float qv[4], kv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    qv[j] = tof(q[u * DK + c0 + j]);
    kv[j] = tof(k[u * DK + c0 + j]);
  }
  const float lm = lam[u], bt = beta[u];
  const float al = la ? __expf(la[u]) : 1.f;
  float xv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) xv[j] = kv[j] + lm * qv[j];
  f4 s[RPT];
  float vr[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {        // rows past DV: the whole lane group skips them
    const int row = row0 + i * RPB;
    s[i] = row < DV ? *(const f4*)(S + (u * DV + row) * DK + c0) : zero4();
    vr[i] = row < DV ? tof(v[u * DV + row]) : 0.f;
  }
  float px[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    px[i] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) px[i] += s[i][j] * xv[j];
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
    for (int i = 0; i < RPT; ++i) px[i] += __shfl_xor(px[i], off, 64);
  float oq[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const float e = bt * (vr[i] - al * px[i]);
    oq[i] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      s[i][j] = al * s[i][j] + e * kv[j];
      oq[i] += s[i][j] * qv[j];
    }
    const int row = row0 + i * RPB;
    if (row < DV) *(f4*)(S + (u * DV + row) * DK + c0) = s[i];
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1)
#pragma unroll
    for (int i = 0; i < RPT; ++i) oq[i] += __shfl_xor(oq[i], off, 64);
  if ((tid % LPR) == 0) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int row = row0 + i * RPB;
      if (row < DV) o[u * DV + row] = fromf<E>(oq[i]);
    }
  }
}

hipError_t launch_step(int N, int H, int Dk, int Dv, int dtype, const void* q, const void* k,
                       const void* v, const float* beta, const float* lam, const float* la,
                       float* state, void* o, hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int RPB = NTHREADS / (Dk / 4) * STEP_RPT;   // state rows per workgroup
  const int nrb = (Dv + RPB - 1) / RPB;
  dim3 grid((unsigned)((size_t)N * H * nrb));
#define QD_STEP(ET, DKV)                                                                        \
  hipLaunchKernelGGL((k_step<ET, DKV>), grid, dim3(NTHREADS), 0, st, Dv, nrb, (const ET*)q,     \
                     (const ET*)k, (const ET*)v, beta, lam, la, state, (ET*)o)
  if (!((dtype == 1 || dtype == 0) && (Dk == 128 || Dk == 64))) return hipErrorInvalidValue;
  prof_mark(ST_STEP, 0, st);
  if (dtype == 1 && Dk == 128) QD_STEP(__bf16, 128);
  else if (dtype == 1 && Dk == 64) QD_STEP(__bf16, 64);
  else if (dtype == 0 && Dk == 128) QD_STEP(float, 128);
  else QD_STEP(float, 64);
  prof_mark(ST_STEP, 1, st);
#undef QD_STEP
  return hipGetLastError();
}

}  // namespace qd
