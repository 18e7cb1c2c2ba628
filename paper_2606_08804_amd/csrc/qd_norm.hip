// Per-row L2 normalisation of q and k for the layer (the condition of Sec. 3.4
// Lemma 1, under which the update contracts), forward and backward, one HBM
// pass each:
//
//   forward   y = x / max(|x|, eps),  r = 1 / max(|x|, eps)   (r stored as -r when clamped)
//   backward  dx = r (dy - y (y . dy)),  or dx = r dy for a clamped row
//
// A row is owned by L = D * sizeof(E) / 16 lanes (16 bytes each); the input
// rows may be strided (views into a fused projection), the outputs are
// contiguous [rows, D].  Row sums use DPP lane moves.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

typedef unsigned int nu32x4 __attribute__((ext_vector_type(4)));

template <int L>
__device__ inline float lane_group_sum(float x) {
  static_assert(L == 8 || L == 16 || L == 32, "lane group of 8, 16 or 32");
  x += dpp_mov<0xB1>(x);                    // quad_perm [1,0,3,2]
  x += dpp_mov<0x4E>(x);                    // quad_perm [2,3,0,1]
  if (L == 8) return x + dpp_mov<0x141>(x); // row_half_mirror: the other quad of 8
  x += dpp_mov<0x124>(x);                   // row_ror:4
  x += dpp_mov<0x128>(x);                   // row_ror:8
  if (L == 32) x += __shfl_xor(x, 16, 64);
  return x;
}

template <typename E>
struct Piece {                              // 16 bytes of a row, widened to fp32
  static constexpr int N = 16 / (int)sizeof(E);
  float v[N];
  __device__ void load(const E* p) {
    const nu32x4 raw = *(const nu32x4*)p;
    const E* e = (const E*)&raw;
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = tof(e[i]);
  }
  __device__ void store(E* p) const {
    nu32x4 raw;
    E* e = (E*)&raw;
#pragma unroll
    for (int i = 0; i < N; ++i) e[i] = fromf<E>(v[i]);
    *(nu32x4*)p = raw;
  }
};

constexpr float NORM_EPS = 1e-12f;

template <typename E, int D>
__global__ __launch_bounds__(NTHREADS) void k_l2norm_fwd(long rows, long ldx, const E* __restrict__ x,
                                                        E* __restrict__ y, float* __restrict__ rn) {
  constexpr int L = D * (int)sizeof(E) / 16;
  constexpr int RPB = NTHREADS / L;
  const long row = (long)blockIdx.x * RPB + threadIdx.x / L;
  const int c = (threadIdx.x % L) * Piece<E>::N;
  if (row >= rows) return;                  // whole lane groups leave together
  Piece<E> a;
  a.load(x + row * ldx + c);
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < Piece<E>::N; ++i) ss += a.v[i] * a.v[i];
  ss = lane_group_sum<L>(ss);
  const float n = sqrtf(ss);
  const bool clamped = !(n > NORM_EPS);
  const float r = 1.f / (clamped ? NORM_EPS : n);
#pragma unroll
  for (int i = 0; i < Piece<E>::N; ++i) a.v[i] *= r;
  a.store(y + row * D + c);
  if (threadIdx.x % L == 0) rn[row] = clamped ? -r : r;
}

template <typename E, int D>
__global__ __launch_bounds__(NTHREADS) void k_l2norm_bwd(long rows, const E* __restrict__ y,
                                                        const float* __restrict__ rn,
                                                        const E* __restrict__ dy, E* __restrict__ dx) {
  constexpr int L = D * (int)sizeof(E) / 16;
  constexpr int RPB = NTHREADS / L;
  const long row = (long)blockIdx.x * RPB + threadIdx.x / L;
  const int c = (threadIdx.x % L) * Piece<E>::N;
  if (row >= rows) return;
  Piece<E> a, g;
  a.load(y + row * D + c);
  g.load(dy + row * D + c);
  float yd = 0.f;
#pragma unroll
  for (int i = 0; i < Piece<E>::N; ++i) yd += a.v[i] * g.v[i];
  yd = lane_group_sum<L>(yd);
  const float rs = rn[row];
  const float r = fabsf(rs);
  const float proj = rs > 0.f ? yd : 0.f;   // a clamped row scales only
#pragma unroll
  for (int i = 0; i < Piece<E>::N; ++i) g.v[i] = r * (g.v[i] - a.v[i] * proj);
  g.store(dx + row * D + c);
}

hipError_t launch_l2norm(int bwd, long rows, int D, long ldx, int dtype, const void* x,
                         const void* y, const float* rn_in, float* rn_out, const void* dy, void* out,
                         hipStream_t st) {
  if (rows == 0) return hipSuccess;
#define QD_NORM(ET, DV)                                                                          \
  do {                                                                                         \
    constexpr int RPB = NTHREADS / (DV * (int)sizeof(ET) / 16);                                \
    dim3 grid((unsigned)((rows + RPB - 1) / RPB));                                             \
    if (bwd)                                                                                   \
      hipLaunchKernelGGL((k_l2norm_bwd<ET, DV>), grid, dim3(NTHREADS), 0, st, rows,            \
                         (const ET*)y, rn_in, (const ET*)dy, (ET*)out);                        \
    else                                                                                       \
      hipLaunchKernelGGL((k_l2norm_fwd<ET, DV>), grid, dim3(NTHREADS), 0, st, rows, ldx,       \
                         (const ET*)x, (ET*)out, rn_out);                                      \
  } while (0)
  if (dtype == 1 && D == 128) QD_NORM(__bf16, 128);
  else if (dtype == 1 && D == 64) QD_NORM(__bf16, 64);
  else if (dtype == 0 && D == 128) QD_NORM(float, 128);
  else if (dtype == 0 && D == 64) QD_NORM(float, 64);
  else return hipErrorInvalidValue;
#undef QD_NORM
  return hipGetLastError();
}

}  // namespace qd
