// Q-Delta chunkwise forward kernels for gfx950.
//
// Per chunk of C tokens with entry state S (Dv x Dk), following Sec. 3.3
// ("Chunkwise parallel form") and App. D.1/D.2 (WY representation, UT
// transform), with the readings listed in the design notes (decay ratios on
// the intra-chunk output term, inclusive causal mask, products read as W S^T):
//
//   b_r = sum_{j<=r} log alpha_j,  g_r = exp(b_r),  Gam_ri = exp(b_r - b_i)
//   X   = K + diag(lambda) Q
//   A   = strictLower(diag(beta) (Gam * X K^T)),   T = (I + A)^{-1} diag(beta)
//   U   = T V,   W = T diag(g) X
//   D   = U - W S^T
//   O   = diag(g) Q S^T + (Gam * M * Q K^T) D     (M includes the diagonal)
//   S'  = g_C S + D^T diag(g_C / g) K
//
// k_prep   (one workgroup per chunk and head, fully parallel): b, X, the two
//          Gram products, A, the UT solve, U and W; writes them to workspace.
// k_scan_fwd (one workgroup per sequence, head and Dv tile): the sequential
//          pass over chunks; the state tile stays in MFMA accumulators in fp32;
//          D, the chunk output and the state update are computed on chip.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

template <typename E, int DK, int DV>
struct PrepSmem {
  static constexpr int P = Pad<E>::v;
  float b[C], beta[C], lam[C];
  union {
    struct {
      E K[C][DK + P];
      E Q[C][DK + P];
      E X[C][DK + P];
    } a;
    E Vt[DV][C + P];
  } u;
  E GXt[DK][C + P];
  float A[C][C + 4];
  float M[C][C + 4];
  float tmp[NWAVES * 16 * 17];
  E Tm[C][C + P];
};

// BWD: additionally write P^T and T for the backward kernels.
template <typename E, int DK, int DV, bool BWD>
__global__ __launch_bounds__(NTHREADS) void k_prep(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P;
  __shared__ PrepSmem<E, DK, DV> sm;
  const int g = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int n, t0, len;
  if (!locate(p, g, n, t0, len)) return;
  const int H = p.H;
  const size_t gi = (size_t)g * H + h;

  if (tid < C) {
    const bool ok = tid < len;
    const size_t gt = (size_t)(t0 + tid) * H + h;
    const float la = (ok && p.la) ? p.la[gt] : 0.f;
    const float b = wave_incl_scan(la, lane);
    sm.b[tid] = b;
    sm.beta[tid] = ok ? p.beta[gt] : 0.f;
    sm.lam[tid] = ok ? p.lam[gt] : 0.f;
    p.wb[gi * C + tid] = b;
  }
  const E* qg = (const E*)p.q + ((size_t)t0 * H + h) * DK;
  const E* kg = (const E*)p.k + ((size_t)t0 * H + h) * DK;
  const E* vg = (const E*)p.v + ((size_t)t0 * H + h) * DV;
  load_rows<E, DK>(&sm.u.a.K[0][0], LK, kg, (size_t)H * DK, len, tid);
  load_rows<E, DK>(&sm.u.a.Q[0][0], LK, qg, (size_t)H * DK, len, tid);
  __syncthreads();

  // mixed inputs X = K + lambda Q and the transposed decayed copy (g X)^T
  for (int idx = tid; idx < C * DK; idx += NTHREADS) {
    const int r = idx % C, c = idx / C;
    const float x = tof(sm.u.a.K[r][c]) + sm.lam[r] * tof(sm.u.a.Q[r][c]);
    sm.u.a.X[r][c] = fromf<E>(x);
    sm.GXt[c][r] = fromf<E>(__expf(sm.b[r]) * x);
  }
  __syncthreads();

  // Gram products X K^T and Q K^T; A (fp32, LDS) and P (workspace)
  E* wP = (E*)p.wP + gi * C * C;
  E* wPT = BWD ? (E*)p.wT + gi * 2 * C * C + C * C : nullptr;
  for (int t = w; t < 16; t += NWAVES) {
    const int m0 = (t >> 2) * 16, n0 = (t & 3) * 16;
    const f4 gx = mma_k<E, DK>(kmaj(&sm.u.a.X[0][0], LK), kmaj(&sm.u.a.K[0][0], LK), m0, n0, zero4(), lane);
    const f4 qk = mma_k<E, DK>(kmaj(&sm.u.a.Q[0][0], LK), kmaj(&sm.u.a.K[0][0], LK), m0, n0, zero4(), lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + frow(lane, j), i = n0 + fcol(lane);
      const float gam = (r >= i) ? __expf(sm.b[r] - sm.b[i]) : 0.f;
      sm.A[r][i] = (r > i) ? sm.beta[r] * gam * gx[j] : 0.f;
      const E pv = fromf<E>(gam * qk[j]);
      wP[r * C + i] = pv;
      if (BWD) wPT[i * C + r] = pv;
    }
  }
  __syncthreads();

  // UT solve: M = (I + A)^{-1}, T = M diag(beta)
  unit_lower_inverse(&sm.A[0][0], C + 4, &sm.M[0][0], C + 4, sm.tmp, tid);
  E* wT = BWD ? (E*)p.wT + gi * 2 * C * C : nullptr;
  for (int idx = tid; idx < C * C; idx += NTHREADS) {
    const int r = idx / C, i = idx % C;
    const E tv = fromf<E>(sm.M[r][i] * sm.beta[i]);
    sm.Tm[r][i] = tv;
    if (BWD) wT[idx] = tv;
  }
  // V^T (K, Q, X are dead: all Gram reads finished before the solve's barriers)
  load_rows_t<E, DV>(&sm.u.Vt[0][0], LC, vg, (size_t)H * DV, len, tid, One());
  __syncthreads();

  // U = T V, stored C-fragment tiled: tile (mt, nt) at ((mt*(DV/16)+nt)*64 + lane)*4
  E* wU = (E*)p.wU + gi * C * DV;
  for (int t = w; t < (C / 16) * (DV / 16); t += NWAVES) {
    const int m0 = (t / (DV / 16)) * 16, n0 = (t % (DV / 16)) * 16;
    const f4 u = mma_k<E, C>(kmaj(&sm.Tm[0][0], LC), kmaj(&sm.u.Vt[0][0], LC), m0, n0, zero4(), lane);
    E* dst = wU + ((size_t)t * 64 + lane) * 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) dst[j] = fromf<E>(u[j]);
  }
  // W = T diag(g) X, row-major C x DK
  E* wW = (E*)p.wW + gi * C * DK;
  for (int t = w; t < (C / 16) * (DK / 16); t += NWAVES) {
    const int m0 = (t / (DK / 16)) * 16, n0 = (t % (DK / 16)) * 16;
    const f4 wv = mma_k<E, C>(kmaj(&sm.Tm[0][0], LC), kmaj(&sm.GXt[0][0], LC), m0, n0, zero4(), lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) wW[(m0 + frow(lane, j)) * DK + n0 + fcol(lane)] = fromf<E>(wv[j]);
  }
}

template <typename E, int DK, int BV>
struct ScanFwdSmem {
  static constexpr int P = Pad<E>::v;
  float b[C];
  E W[C][DK + P];
  E Q[C][DK + P];
  E Kt[DK][C + P];
  E Pm[C][C + P];
  E S[BV][DK + P];
  E Dt[BV][C + P];
};

// One workgroup per (sequence, head, Dv tile of BV columns).  The state tile
// S^T (Dk x BV) lives in fp32 MFMA accumulators across the whole sequence.
// When p.o is null only the states are produced (saved / final).
template <typename E, int DK, int DV, int BV>
__global__ __launch_bounds__(NTHREADS) void k_scan_fwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P;
  constexpr int NVT = DV / BV;
  constexpr int SPW = (DK / 16) * (BV / 16) / NWAVES;   // state tiles per wave
  constexpr int DPW = (C / 16) * (BV / 16) / NWAVES;    // D / O tiles per wave
  static_assert(SPW >= 1 && DPW >= 1, "tile split");
  __shared__ ScanFwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int unit, vt;
  if (!xcd_unit_tile(blockIdx.x, p.N * p.H, NVT, unit, vt)) return;
  const int H = p.H, n = unit / H, h = unit % H, v0 = vt * BV;
  int s, e;
  if (!seq_range(p, n, s, e)) return;
  const int nch = (e - s + C - 1) / C;
  const int base = slot_base(p, n, s);

  f4 acc[SPW];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int t = w * SPW + i, kt = t / (BV / 16), nt = t % (BV / 16);
    if (p.S0) {
      const float* src = p.S0 + ((size_t)unit * DV + v0 + nt * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0);
      acc[i] = *(const f4*)src;
    } else {
      acc[i] = zero4();
    }
  }

  const E* qbase = (const E*)p.q;
  const E* kbase = (const E*)p.k;
  for (int c = 0; c < nch; ++c) {
    const int slot = base + c;
    if (slot >= p.n_slots) break;
    const int t0 = s + c * C, len = min(C, e - t0);
    const size_t gi = (size_t)slot * H + h;
    __syncthreads();
    if (tid < C) sm.b[tid] = p.wb[gi * C + tid];
    load_rows<E, DK>(&sm.W[0][0], LK, (const E*)p.wW + gi * C * DK, DK, C, tid);
    if (p.o) {
      load_rows<E, DK>(&sm.Q[0][0], LK, qbase + ((size_t)t0 * H + h) * DK, (size_t)H * DK, len, tid);
      load_rows<E, C>(&sm.Pm[0][0], LC, (const E*)p.wP + gi * C * C, C, C, tid);
    }
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int t = w * SPW + i, kt = t / (BV / 16), nt = t % (BV / 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.S[nt * 16 + fcol(lane)][kt * 16 + frow(lane, j)] = fromf<E>(acc[i][j]);
      if (p.saved)
        *(f4*)(p.saved + (gi * DV + v0 + nt * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) = acc[i];
    }
    __syncthreads();
    const float bl = sm.b[C - 1];
    load_rows_t<E, DK>(&sm.Kt[0][0], LC, kbase + ((size_t)t0 * H + h) * DK, (size_t)H * DK, len, tid,
                       [&](int r) { return __expf(bl - sm.b[r]); });
    // D = U - W S^T
    f4 dfr[DPW];
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const int t = w * DPW + i, mt = t / (BV / 16), nt = t % (BV / 16);
      const E* us = (const E*)p.wU + gi * C * DV +
                    ((size_t)(mt * (DV / 16) + vt * (BV / 16) + nt) * 64 + lane) * 4;
      f4 d = mma_k<E, DK>(kmaj(&sm.W[0][0], LK), kmaj(&sm.S[0][0], LK), mt * 16, nt * 16, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        d[j] = tof(us[j]) - d[j];
        sm.Dt[nt * 16 + fcol(lane)][mt * 16 + frow(lane, j)] = fromf<E>(d[j]);
      }
      dfr[i] = d;
    }
    __syncthreads();
    if (p.o) {
      E* obase = (E*)p.o;
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        const int t = w * DPW + i, mt = t / (BV / 16), nt = t % (BV / 16);
        const f4 o1 = mma_k<E, DK>(kmaj(&sm.Q[0][0], LK), kmaj(&sm.S[0][0], LK), mt * 16, nt * 16, zero4(), lane);
        const f4 o2 = mma_k<E, C>(kmaj(&sm.Pm[0][0], LC), kmaj(&sm.Dt[0][0], LC), mt * 16, nt * 16, zero4(), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = mt * 16 + frow(lane, j);
          if (r < len)
            obase[((size_t)(t0 + r) * H + h) * DV + v0 + nt * 16 + fcol(lane)] =
                fromf<E>(__expf(sm.b[r]) * o1[j] + o2[j]);
        }
      }
    }
    (void)dfr;
    const float gC = __expf(bl);
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int t = w * SPW + i, kt = t / (BV / 16), nt = t % (BV / 16);
      acc[i] = mma_k<E, C>(kmaj(&sm.Kt[0][0], LC), kmaj(&sm.Dt[0][0], LC), kt * 16, nt * 16, gC * acc[i], lane);
    }
  }
  if (p.Sfin) {
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int t = w * SPW + i, kt = t / (BV / 16), nt = t % (BV / 16);
      *(f4*)(p.Sfin + ((size_t)unit * DV + v0 + nt * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) = acc[i];
    }
  }
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_fwd_t(const Params& p, int bwd_prep, int with_scan, hipStream_t st) {
  constexpr int BV = 32;
  if (p.n_slots > 0) {
    dim3 gp(p.n_slots, p.H);
    const int stage = bwd_prep ? ST_PREP_BWD : ST_PREP_FWD;
    prof_mark(stage, 0, st);
    if (bwd_prep)
      hipLaunchKernelGGL((k_prep<E, DK, DV, true>), gp, dim3(NTHREADS), 0, st, p);
    else
      hipLaunchKernelGGL((k_prep<E, DK, DV, false>), gp, dim3(NTHREADS), 0, st, p);
    prof_mark(stage, 1, st);
  }
  if (with_scan) {
    const int units = p.N * p.H;
    const int nb = ((units + 7) / 8) * 8 * (DV / BV);
    if (nb > 0) {
      prof_mark(ST_SCAN_FWD, 0, st);
      hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, BV>), dim3(nb), dim3(NTHREADS), 0, st, p);
      prof_mark(ST_SCAN_FWD, 1, st);
    }
  }
  return hipGetLastError();
}

hipError_t launch_fwd(const Params& p, int dtype, int Dk, int Dv, int bwd_prep, int with_scan,
                      hipStream_t st) {
#define QD_CASE(ET, DKV, DVV) \
  if (Dk == DKV && Dv == DVV) return launch_fwd_t<ET, DKV, DVV>(p, bwd_prep, with_scan, st);
  if (dtype == 1) {
    QD_CASE(__bf16, 64, 64) QD_CASE(__bf16, 64, 128) QD_CASE(__bf16, 64, 256)
    QD_CASE(__bf16, 128, 64) QD_CASE(__bf16, 128, 128) QD_CASE(__bf16, 128, 256)
  } else {
    QD_CASE(float, 64, 64) QD_CASE(float, 64, 128) QD_CASE(float, 64, 256)
  }
#undef QD_CASE
  return hipErrorInvalidValue;
}

}  // namespace qd
