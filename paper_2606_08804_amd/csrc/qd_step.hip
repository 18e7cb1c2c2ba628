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

template <int LPR>
__device__ inline float group_sum(float x) {
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

template <typename E, int DK>
__global__ __launch_bounds__(NTHREADS) void k_step(int DV, int nrb, const E* __restrict__ q,
                                                  const E* __restrict__ k, const E* __restrict__ v,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ lam,
                                                  const float* __restrict__ la, float* __restrict__ S,
                                                  E* __restrict__ o) {
  constexpr int LPR = DK / 4;            // lanes per state row
  constexpr int RPB = NTHREADS / LPR;    // rows per workgroup
  const size_t u = blockIdx.x / nrb;     // (sequence, head) unit
  const int rb = blockIdx.x % nrb;       // block of RPB state rows
  const int tid = threadIdx.x;
  const int row = rb * RPB + tid / LPR;
  const int c0 = (tid % LPR) * 4;
  if (row >= DV) return;                 // whole lane group leaves together
  float qv[4], kv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    qv[j] = tof(q[u * DK + c0 + j]);
    kv[j] = tof(k[u * DK + c0 + j]);
  }
  const float lm = lam[u], bt = beta[u];
  const float al = la ? __expf(la[u]) : 1.f;
  float* Sr = S + (u * DV + row) * DK + c0;
  f4 s = *(const f4*)Sr;
  float px = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) px += s[j] * (kv[j] + lm * qv[j]);
  px = group_sum<LPR>(px);
  const float e = bt * (tof(v[u * DV + row]) - al * px);
  float oq = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    s[j] = al * s[j] + e * kv[j];
    oq += s[j] * qv[j];
  }
  *(f4*)Sr = s;
  oq = group_sum<LPR>(oq);
  if ((tid % LPR) == 0) o[u * DV + row] = fromf<E>(oq);
}

hipError_t launch_step(int N, int H, int Dk, int Dv, int dtype, const void* q, const void* k,
                       const void* v, const float* beta, const float* lam, const float* la,
                       float* state, void* o, hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int RPB = NTHREADS / (Dk / 4);
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
