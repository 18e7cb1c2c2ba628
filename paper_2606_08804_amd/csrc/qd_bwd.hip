// Q-Delta chunkwise backward kernels for gfx950.
//
// The paper states no backward pass.  These kernels apply the chain rule to
// the chunk steps of the forward (see qd_fwd.hip), per chunk with entry state
// S, exit-state gradient dS' and output gradient dO:
//
//   inter-chunk (sequential, reverse):
//     dD   = P^T dO + Kbar dS'^T                  Kbar = diag(g_C / g) K
//     dS   = g_C dS' + dO^T diag(g) Q - dD^T W    (gradient w.r.t. the entry state)
//   intra-chunk (parallel over chunks):
//     D    = U - W S^T
//     dQ   = diag(g) dO S + dQK K + diag(lambda) dX,      dQK = Gam * M * (dO D^T)
//     dK   = diag(g_C/g) D dS' + dQK^T Q + dG^T X + dX
//     dV   = T^T dD,   dW = -dD S
//     dT   = dD V^T + dW (diag(g) X)^T
//     dbeta_i  = sum_r dT_ri Minv_ri + sum_{i'<i} dA_ii' Gam_ii' G_ii'
//     dA   = strictLower(-Minv^T (dT diag(beta)) Minv^T),  Minv = (I + A)^{-1}
//     dG   = diag(beta) dA * Gam,   G = X K^T
//     dX   = diag(g) T^T dW + dG K,  dlambda_r = q_r . dX_r
//     dlog alpha = reverse chunk-local cumulative sum of db, where db collects
//     every term through g, Gam, Kbar and g_C.
//
// k_scan_bwd : one workgroup per (sequence, head, Dv tile); dS^T tile in fp32
//              accumulators; writes dD and dS' per chunk.
// k_intra_a  : per (chunk, head); the products that contract over Dv
//              (dO S, D dS', dD S, dO D^T, dD V^T) and dV.
// k_intra_b  : per (chunk, head); UT-solve backward and the remaining
//              products over Dk, in halves of KH columns; final gradients.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

// ------------------------------------------------------------------ scan
template <typename E, int DK, int BV>
struct ScanBwdSmem {
  static constexpr int P = Pad<E>::v;
  float b[C];
  E dS[BV][DK + P];   // dS' tile [v][k]
  E dDn[BV][C + P];   // -dD tile, transposed [v][r]
};

// Operands of one chunk for one wave of the backward scan, prefetched from
// global memory straight into MFMA fragments.
template <typename E, int DK, int KPW, int NB>
struct ScanBwdPre {
  AFrag<E, C> PT;          // rows 16w.. of P^T
  AFrag<E, DK> K;          // rows 16w.. of K
  AFrag<E, C> Qg[KPW];     // rows of (diag(g) Q)^T for this wave's key blocks
  AFrag<E, C> Wt[KPW];     // rows of W^T for this wave's key blocks
  AFrag<E, C> dO[NB];      // B fragments of dO^T for the tile's value blocks
  float b;
};

// One workgroup per (sequence, head, Dv tile of BV = 32); reverse pass over
// the chunks with the next (earlier) chunk's operands prefetched.
template <typename E, int DK, int DV, int BV>
__global__ __launch_bounds__(NTHREADS) void k_scan_bwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P;
  constexpr int NVT = DV / BV;
  constexpr int NB = BV / 16;
  constexpr int KS = Mma<E>::KS;
  constexpr int KPW = DK / 16 / NWAVES;
  static_assert(KPW >= 1 && KPW * 16 * NWAVES == DK, "key blocks per wave");
  typedef typename Quad<E>::raw QR;
  typedef typename Mma<E>::frag FR;
  __shared__ ScanBwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int unit, vt;
  if (!xcd_unit_tile(blockIdx.x, p.N * p.H, NVT, unit, vt)) return;
  const int H = p.H, n = unit / H, h = unit % H, v0 = vt * BV;
  int s, e;
  if (!seq_range(p, n, s, e)) return;
  const int base = slot_base(p, n, s);
  const int nch = max(0, min((e - s + C - 1) / C, p.n_slots - base));

  f4 acc[KPW][NB];
#pragma unroll
  for (int i = 0; i < KPW; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int kt = KPW * w + i;
      acc[i][nb] = p.dSfin ? *(const f4*)(p.dSfin + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK +
                                          kt * 16 + frow(lane, 0))
                           : zero4();
    }
  const E* kb = (const E*)p.k;
  ScanBwdPre<E, DK, KPW, NB> pre;
  auto prefetch = [&](int c) {
    const int t0 = s + c * C, len = min(C, e - t0);
    const size_t gi = (size_t)(base + c) * H + h;
    pre.b = tid < C ? p.wb[gi * C + tid] : 0.f;
    pre.PT.load((const E*)p.wT + gi * 2 * C * C + C * C + (size_t)(16 * w) * C, C, 16, lane);
    pre.K.load(kb + ((size_t)(t0 + 16 * w) * H + h) * DK, (size_t)H * DK, len - 16 * w, lane);
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const size_t row = (size_t)16 * (KPW * w + i) * C;
      pre.Qg[i].load((const E*)p.wQgt + gi * DK * C + row, C, 16, lane);
      pre.Wt[i].load((const E*)p.wWt + gi * DK * C + row, C, 16, lane);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      pre.dO[nb].load((const E*)p.wdOt + gi * DV * C + (size_t)(v0 + 16 * nb) * C, C, 16, lane);
  };
  if (nch > 0) prefetch(nch - 1);

  for (int c = nch - 1; c >= 0; --c) {
    const size_t gi = (size_t)(base + c) * H + h;
    const ScanBwdPre<E, DK, KPW, NB> cur = pre;
    block_sync_lds();
    if (tid < C) sm.b[tid] = cur.b;
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int kt = KPW * w + i;
        *(QR*)&sm.dS[nb * 16 + fcol(lane)][kt * 16 + frow(lane, 0)] = Quad<E>::pack(acc[i][nb]);
        *(f4*)(p.w_dSo + (gi * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) = acc[i][nb];
      }
    block_sync_lds();
    if (c > 0) prefetch(c - 1);
    const float bl = sm.b[C - 1];
    // dD = P^T dO + diag(g_C/g) K dS'^T   (rows 16w..)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f4 d1 = zero4(), d2 = zero4();
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) d1 = Mma<E>::mma(cur.PT.f[ks], cur.dO[nb].f[ks], d1);
#pragma unroll
      for (int ks = 0; ks < DK / KS; ++ks)
        d2 = Mma<E>::mma(cur.K.f[ks], Frag<E>::load(kmaj(&sm.dS[0][0], LK), nb * 16, ks * KS, lane), d2);
      f4 dn;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 16 * w + frow(lane, j);
        const float d = d1[j] + __expf(bl - sm.b[r]) * d2[j];
        dn[j] = -d;
        p.w_dD[(gi * C + r) * DV + v0 + nb * 16 + fcol(lane)] = d;
      }
      *(QR*)&sm.dDn[nb * 16 + fcol(lane)][16 * w + frow(lane, 0)] = Quad<E>::pack(dn);
    }
    block_sync_lds();
    // dS_entry^T = g_C dS'^T + (g Q)^T dO - W^T dD
    const float gC = __expf(bl);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int i = 0; i < KPW; ++i) acc[i][nb] = gC * acc[i][nb];
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) {
        const FR bd = Frag<E>::load(kmaj(&sm.dDn[0][0], LC), nb * 16, ks * KS, lane);
#pragma unroll
        for (int i = 0; i < KPW; ++i) {
          acc[i][nb] = Mma<E>::mma(cur.Qg[i].f[ks], cur.dO[nb].f[ks], acc[i][nb]);
          acc[i][nb] = Mma<E>::mma(cur.Wt[i].f[ks], bd, acc[i][nb]);
        }
      }
    }
  }
  if (p.dS0) {
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int kt = KPW * w + i;
        *(f4*)(p.dS0 + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) =
            acc[i][nb];
      }
  }
}

// ------------------------------------------------------------------ intra A
template <typename E, int DK, int BV>
struct IntraASmem {
  static constexpr int P = Pad<E>::v;
  float b[C], g[C], kb[C], rq[C], rk[C];
  float sdot[NWAVES];
  E W[C][DK + P];
  E Tm[C][C + P];
  E Q[C][DK + P];
  E K[C][DK + P];
  E S[BV][DK + P];
  E dS[BV][DK + P];
  E dO[C][BV + P];
  E dD[C][BV + P];
  E V[C][BV + P];
  E D[C][BV + P];
};

template <typename E, int DK, int DV, int BV>
__global__ __launch_bounds__(NTHREADS) void k_intra_a(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P, LB = BV + P;
  constexpr int QT = (C / 16) * (DK / 16) / NWAVES;   // C x DK tiles per wave (one row block)
  constexpr int PT = 16 / NWAVES;                      // C x C tiles per wave
  constexpr int DT = (C / 16) * (BV / 16) / NWAVES;    // C x BV tiles per wave
  static_assert(QT == DK / 16, "each wave owns one 16-row block of the C x Dk accumulators");
  __shared__ IntraASmem<E, DK, BV> sm;
  const int g = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int n, t0, len;
  if (!locate(p, g, n, t0, len)) return;
  const int H = p.H;
  const size_t gi = (size_t)g * H + h;

  if (tid < C) {
    const float b = p.wb[gi * C + tid];
    sm.b[tid] = b;
    sm.g[tid] = __expf(b);
  }
  load_rows<E, DK>(&sm.W[0][0], LK, (const E*)p.wW + gi * C * DK, DK, C, tid);
  load_rows<E, C>(&sm.Tm[0][0], LC, (const E*)p.wT + gi * 2 * C * C, C, C, tid);
  load_rows<E, DK>(&sm.Q[0][0], LK, (const E*)p.q + ((size_t)t0 * H + h) * DK, (size_t)H * DK, len, tid);
  load_rows<E, DK>(&sm.K[0][0], LK, (const E*)p.k + ((size_t)t0 * H + h) * DK, (size_t)H * DK, len, tid);

  f4 aQ[QT], aK[QT], aW[QT], aP[PT], aT[PT];
#pragma unroll
  for (int i = 0; i < QT; ++i) aQ[i] = aK[i] = aW[i] = zero4();
#pragma unroll
  for (int i = 0; i < PT; ++i) aP[i] = aT[i] = zero4();
  float sdot = 0.f;

  const float* Sg = p.saved + gi * DV * DK;
  const float* dSg = p.w_dSo + gi * DV * DK;
  const E* dOg = (const E*)p.dO + ((size_t)t0 * H + h) * DV;
  const E* Vg = (const E*)p.v + ((size_t)t0 * H + h) * DV;
  const float* dDg = p.w_dD + gi * C * DV;
  E* dvout = (E*)p.dv;

  for (int vt = 0; vt < DV / BV; ++vt) {
    const int v0 = vt * BV;
    __syncthreads();
    for (int idx = tid; idx < BV * DK / 4; idx += NTHREADS) {
      const int vv = idx / (DK / 4), kk = (idx % (DK / 4)) * 4;
      const f4 sv = *(const f4*)(Sg + (size_t)(v0 + vv) * DK + kk);
      const f4 dv = *(const f4*)(dSg + (size_t)(v0 + vv) * DK + kk);
      sdot += sv[0] * dv[0] + sv[1] * dv[1] + sv[2] * dv[2] + sv[3] * dv[3];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sm.S[vv][kk + j] = fromf<E>(sv[j]);
        sm.dS[vv][kk + j] = fromf<E>(dv[j]);
      }
    }
    load_rows<E, BV>(&sm.dO[0][0], LB, dOg + v0, (size_t)H * DV, len, tid);
    load_rows<E, BV>(&sm.V[0][0], LB, Vg + v0, (size_t)H * DV, len, tid);
    for (int idx = tid; idx < C * BV / 4; idx += NTHREADS) {
      const int r = idx / (BV / 4), vv = (idx % (BV / 4)) * 4;
      const f4 d = *(const f4*)(dDg + (size_t)r * DV + v0 + vv);
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.dD[r][vv + j] = fromf<E>(d[j]);
    }
    __syncthreads();
    // D = U - W S^T (tile) and dV = T^T dD (tile)
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      const int t = w * DT + i, mt = t / (BV / 16), nt = t % (BV / 16);
      const E* us = (const E*)p.wU + gi * C * DV +
                    ((size_t)(mt * (DV / 16) + vt * (BV / 16) + nt) * 64 + lane) * 4;
      f4 d = mma_k<E, DK>(kmaj(&sm.W[0][0], LK), kmaj(&sm.S[0][0], LK), mt * 16, nt * 16, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        sm.D[mt * 16 + frow(lane, j)][nt * 16 + fcol(lane)] = fromf<E>(tof(us[j]) - d[j]);
      const f4 dv = mma_k<E, C>(imaj(&sm.Tm[0][0], LC), imaj(&sm.dD[0][0], LB), mt * 16, nt * 16, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = mt * 16 + frow(lane, j);
        if (r < len) dvout[((size_t)(t0 + r) * H + h) * DV + v0 + nt * 16 + fcol(lane)] = fromf<E>(dv[j]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < QT; ++i) {
      const int t = w * QT + i, mt = t / (DK / 16), nt = t % (DK / 16);
      aQ[i] = mma_k<E, BV>(kmaj(&sm.dO[0][0], LB), imaj(&sm.S[0][0], LK), mt * 16, nt * 16, aQ[i], lane);
      aK[i] = mma_k<E, BV>(kmaj(&sm.D[0][0], LB), imaj(&sm.dS[0][0], LK), mt * 16, nt * 16, aK[i], lane);
      aW[i] = mma_k<E, BV>(kmaj(&sm.dD[0][0], LB), imaj(&sm.S[0][0], LK), mt * 16, nt * 16, aW[i], lane);
    }
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int t = w * PT + i, mt = t / 4, nt = t % 4;
      aP[i] = mma_k<E, BV>(kmaj(&sm.dO[0][0], LB), kmaj(&sm.D[0][0], LB), mt * 16, nt * 16, aP[i], lane);
      aT[i] = mma_k<E, BV>(kmaj(&sm.dD[0][0], LB), kmaj(&sm.V[0][0], LB), mt * 16, nt * 16, aT[i], lane);
    }
  }

  // <dS', S> over the whole state
  sdot = wave_sum(sdot);
  if (lane == 0) sm.sdot[w] = sdot;

  // epilogue: dq part, dk part, dW, dP, dT_part and the db terms
  float* wq = p.w_dq + gi * C * DK;
  float* wk = p.w_dk + gi * C * DK;
  float* ww = p.w_dW + gi * C * DK;
  float rq[4] = {0.f, 0.f, 0.f, 0.f}, rk[4] = {0.f, 0.f, 0.f, 0.f};
  const int mt = w;   // this wave's row block
#pragma unroll
  for (int i = 0; i < QT; ++i) {
    const int nt = (w * QT + i) % (DK / 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = mt * 16 + frow(lane, j), kk = nt * 16 + fcol(lane);
      rq[j] += tof(sm.Q[r][kk]) * aQ[i][j];
      rk[j] += tof(sm.K[r][kk]) * aK[i][j];
      wq[r * DK + kk] = sm.g[r] * aQ[i][j];
      wk[r * DK + kk] = __expf(sm.b[C - 1] - sm.b[r]) * aK[i][j];
      ww[r * DK + kk] = -aW[i][j];
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    rq[j] = sum16(rq[j]);
    rk[j] = sum16(rk[j]);
  }
  if (fcol(lane) == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = mt * 16 + frow(lane, j);
      sm.rq[r] = rq[j];
      sm.rk[r] = rk[j];
    }
  }
  float* wPd = p.w_dP + gi * C * C;
  float* wTd = p.w_dT + gi * C * C;
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const int t = w * PT + i, m0 = (t / 4) * 16, n0 = (t % 4) * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + frow(lane, j), c = n0 + fcol(lane);
      wPd[r * C + c] = aP[i][j];
      wTd[r * C + c] = aT[i][j];
    }
  }
  __syncthreads();
  if (tid < C) {
    const int r = tid;
    const float bl = sm.b[C - 1];
    const float tr = __expf(bl - sm.b[r]) * sm.rk[r];   // Kbar row term
    float db = sm.g[r] * sm.rq[r] - tr;
    float tot = tr;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) tot += __shfl_xor(tot, off, 64);
    if (r == C - 1) {
      const float sd = sm.sdot[0] + sm.sdot[1] + sm.sdot[2] + sm.sdot[3];
      db += tot + __expf(bl) * sd;
    }
    p.w_db[gi * C + r] = db;
  }
}

// ------------------------------------------------------------------ intra B
template <typename E, int KH>
struct IntraBSmem {
  static constexpr int P = Pad<E>::v;
  float b[C], g[C], beta[C], lam[C], db[C], dbeta[C], dlam[C];
  union {
    struct {
      E Q[C][KH + P];
      E K[C][KH + P];
      E X[C][KH + P];
      E GX[C][KH + P];
      E dW[C][KH + P];
      float dX[C][KH + 4];
    } h;
    struct {
      float G[C][C + 4];
      float QK[C][C + 4];
      float dT[C][C + 4];
      float A[C][C + 4];
      float M[C][C + 4];
      float Y[C][C + 4];
      float tmp[NWAVES * 16 * 17];
    } c;
  } u;
  E Tm[C][C + P];
  E dG[C][C + P];
  E dQK[C][C + P];
};

template <typename E, int DK, int KH>
__global__ __launch_bounds__(NTHREADS) void k_intra_b(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LH = KH + P, LC = C + P, LF = C + 4;
  constexpr int HT = (C / 16) * (KH / 16);   // C x KH tiles
  __shared__ IntraBSmem<E, KH> sm;
  const int g = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int n, t0, len;
  if (!locate(p, g, n, t0, len)) return;
  const int H = p.H;
  const size_t gi = (size_t)g * H + h;

  if (tid < C) {
    const bool ok = tid < len;
    const size_t gt = (size_t)(t0 + tid) * H + h;
    const float b = p.wb[gi * C + tid];
    sm.b[tid] = b;
    sm.g[tid] = __expf(b);
    sm.beta[tid] = ok ? p.beta[gt] : 0.f;
    sm.lam[tid] = ok ? p.lam[gt] : 0.f;
    sm.dlam[tid] = 0.f;
  }
  const E* qg = (const E*)p.q + ((size_t)t0 * H + h) * DK;
  const E* kg = (const E*)p.k + ((size_t)t0 * H + h) * DK;
  const float* dWg = p.w_dW + gi * C * DK;

  auto load_half = [&](int k0) {
    load_rows<E, KH>(&sm.u.h.Q[0][0], LH, qg + k0, (size_t)H * DK, len, tid);
    load_rows<E, KH>(&sm.u.h.K[0][0], LH, kg + k0, (size_t)H * DK, len, tid);
    for (int idx = tid; idx < C * KH / 4; idx += NTHREADS) {
      const int r = idx / (KH / 4), kk = (idx % (KH / 4)) * 4;
      const f4 d = *(const f4*)(dWg + (size_t)r * DK + k0 + kk);
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.u.h.dW[r][kk + j] = fromf<E>(d[j]);
    }
  };
  auto make_x = [&]() {
    for (int idx = tid; idx < C * KH; idx += NTHREADS) {
      const int r = idx / KH, c = idx % KH;
      const float x = tof(sm.u.h.K[r][c]) + sm.lam[r] * tof(sm.u.h.Q[r][c]);
      sm.u.h.X[r][c] = fromf<E>(x);
      sm.u.h.GX[r][c] = fromf<E>(sm.g[r] * x);
    }
  };

  // ---- phase 1: G = X K^T, QK = Q K^T, dT2 = dW (g X)^T over Dk halves
  f4 aG[4], aQK[4], adT[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) aG[i] = aQK[i] = adT[i] = zero4();
  for (int k0 = 0; k0 < DK; k0 += KH) {
    __syncthreads();
    load_half(k0);
    __syncthreads();
    make_x();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = w * 4 + i, m0 = (t / 4) * 16, n0 = (t % 4) * 16;
      aG[i] = mma_k<E, KH>(kmaj(&sm.u.h.X[0][0], LH), kmaj(&sm.u.h.K[0][0], LH), m0, n0, aG[i], lane);
      aQK[i] = mma_k<E, KH>(kmaj(&sm.u.h.Q[0][0], LH), kmaj(&sm.u.h.K[0][0], LH), m0, n0, aQK[i], lane);
      adT[i] = mma_k<E, KH>(kmaj(&sm.u.h.dW[0][0], LH), kmaj(&sm.u.h.GX[0][0], LH), m0, n0, adT[i], lane);
    }
  }
  __syncthreads();

  // ---- phase 2: UT-solve backward and the C x C gradient terms
  const float* dTg = p.w_dT + gi * C * C;
  const float* dPg = p.w_dP + gi * C * C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = w * 4 + i, m0 = (t / 4) * 16, n0 = (t % 4) * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + frow(lane, j), c = n0 + fcol(lane);
      sm.u.c.G[r][c] = aG[i][j];
      sm.u.c.QK[r][c] = aQK[i][j];
      sm.u.c.dT[r][c] = dTg[r * C + c] + adT[i][j];
      sm.u.c.A[r][c] = (r > c) ? sm.beta[r] * __expf(sm.b[r] - sm.b[c]) * aG[i][j] : 0.f;
    }
  }
  __syncthreads();
  unit_lower_inverse(&sm.u.c.A[0][0], LF, &sm.u.c.M[0][0], LF, sm.u.c.tmp, tid);
  // Four lanes share one row (or column) of the C x C element-wise passes:
  // lane quad q4 = tid >> 2 owns row/column q4, segment (tid & 3) * 16 .. +16.
  const int q4 = tid >> 2, seg = (tid & 3) * 16;
  // dbeta (T = Minv diag(beta)): column sums of dT * Minv;  T into LDS
  {
    float s4 = 0.f;
#pragma unroll 4
    for (int r = seg; r < seg + 16; ++r) s4 += sm.u.c.dT[r][q4] * sm.u.c.M[r][q4];
    s4 += __shfl_xor(s4, 1, 64);
    s4 += __shfl_xor(s4, 2, 64);
    if ((tid & 3) == 0) sm.dbeta[q4] = s4;
  }
  for (int idx = tid; idx < C * C; idx += NTHREADS) {
    const int r = idx / C, i = idx % C;
    sm.Tm[r][i] = fromf<E>(sm.u.c.M[r][i] * sm.beta[i]);
  }
  __syncthreads();
  // dMinv = dT diag(beta), in place
  for (int idx = tid; idx < C * C; idx += NTHREADS) {
    const int r = idx / C, i = idx % C;
    sm.u.c.dT[r][i] *= sm.beta[i];
  }
  __syncthreads();
  // Y = Minv^T dMinv
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = w * 4 + i, m0 = (t / 4) * 16, n0 = (t % 4) * 16;
    const f4 y = mma_k<E, C>(imaj(&sm.u.c.M[0][0], LF), imaj(&sm.u.c.dT[0][0], LF), m0, n0, zero4(), lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) sm.u.c.Y[m0 + frow(lane, j)][n0 + fcol(lane)] = y[j];
  }
  __syncthreads();
  // dA = strictLower(-Y Minv^T)   (A is dead after the solve: reuse its storage)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = w * 4 + i, m0 = (t / 4) * 16, n0 = (t % 4) * 16;
    const f4 y = mma_k<E, C>(kmaj(&sm.u.c.Y[0][0], LF), kmaj(&sm.u.c.M[0][0], LF), m0, n0, zero4(), lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + frow(lane, j), c = n0 + fcol(lane);
      sm.u.c.A[r][c] = (r > c) ? -y[j] : 0.f;
    }
  }
  __syncthreads();
  // dP (from intra A) into the dead Y buffer, coalesced
  for (int idx = tid; idx < C * C / 4; idx += NTHREADS) {
    const int r = idx / (C / 4), c = (idx % (C / 4)) * 4;
    *(f4*)&sm.u.c.Y[r][c] = *(const f4*)(dPg + r * C + c);
  }
  __syncthreads();
  // element-wise, by rows: dbeta row part, dG, dQK, and the row sums of
  // dGam * Gam (decay gradient), with dGam = dA beta G + dP QK on r >= i
  const float* dbg = p.w_db + gi * C;
  {
    const int r = q4;
    const float br = sm.b[r], betar = sm.beta[r];
    float dbr = 0.f, er = 0.f;
#pragma unroll 4
    for (int i = seg; i < seg + 16; ++i) {
      float dg = 0.f, dqk = 0.f;
      if (i <= r) {
        const float gam = __expf(br - sm.b[i]);
        const float dA = sm.u.c.A[r][i];
        const float Gv = sm.u.c.G[r][i];
        const float dP = sm.u.c.Y[r][i];
        dbr += dA * gam * Gv;
        dg = dA * betar * gam;
        dqk = dP * gam;
        er += (dA * betar * Gv + dP * sm.u.c.QK[r][i]) * gam;
      }
      sm.dG[r][i] = fromf<E>(dg);
      sm.dQK[r][i] = fromf<E>(dqk);
    }
    dbr += __shfl_xor(dbr, 1, 64);
    dbr += __shfl_xor(dbr, 2, 64);
    er += __shfl_xor(er, 1, 64);
    er += __shfl_xor(er, 2, 64);
    __syncthreads();   // dbeta column part written above (other lanes) is complete
    if ((tid & 3) == 0) {
      sm.dbeta[r] += dbr;
      sm.db[r] = dbg[r] + er;
    }
  }
  __syncthreads();
  // element-wise, by columns: subtract the column sums of dGam * Gam
  {
    const int i = q4;
    const float bi = sm.b[i];
    float ec = 0.f;
#pragma unroll 4
    for (int r = seg; r < seg + 16; ++r) {
      if (r >= i) {
        const float gam = __expf(sm.b[r] - bi);
        ec += (sm.u.c.A[r][i] * sm.beta[r] * sm.u.c.G[r][i] + sm.u.c.Y[r][i] * sm.u.c.QK[r][i]) * gam;
      }
    }
    ec += __shfl_xor(ec, 1, 64);
    ec += __shfl_xor(ec, 2, 64);
    if ((tid & 3) == 0) sm.db[i] -= ec;
  }
  __syncthreads();

  // ---- phase 3: dX, dQ, dK over Dk halves
  E* dqo = (E*)p.dq;
  E* dko = (E*)p.dk;
  const float* wq = p.w_dq + gi * C * DK;
  const float* wk = p.w_dk + gi * C * DK;
  for (int k0 = 0; k0 < DK; k0 += KH) {
    __syncthreads();
    load_half(k0);
    __syncthreads();
    make_x();
    // dgX = T^T dW
    for (int t = w; t < HT; t += NWAVES) {
      const int m0 = (t / (KH / 16)) * 16, n0 = (t % (KH / 16)) * 16;
      const f4 d = mma_k<E, C>(imaj(&sm.Tm[0][0], LC), imaj(&sm.u.h.dW[0][0], LH), m0, n0, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.u.h.dX[m0 + frow(lane, j)][n0 + fcol(lane)] = d[j];
    }
    __syncthreads();
    {
      const int r = q4, c0 = (tid & 3) * (KH / 4);
      float s4 = 0.f;
#pragma unroll
      for (int c = c0; c < c0 + KH / 4; ++c) s4 += tof(sm.u.h.X[r][c]) * sm.u.h.dX[r][c];
      s4 += __shfl_xor(s4, 1, 64);
      s4 += __shfl_xor(s4, 2, 64);
      if ((tid & 3) == 0) sm.db[r] += sm.g[r] * s4;
    }
    __syncthreads();
    // dX = g dgX + dG K
    for (int t = w; t < HT; t += NWAVES) {
      const int m0 = (t / (KH / 16)) * 16, n0 = (t % (KH / 16)) * 16;
      const f4 d = mma_k<E, C>(kmaj(&sm.dG[0][0], LC), imaj(&sm.u.h.K[0][0], LH), m0, n0, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = m0 + frow(lane, j), c = n0 + fcol(lane);
        sm.u.h.dX[r][c] = sm.g[r] * sm.u.h.dX[r][c] + d[j];
      }
    }
    __syncthreads();
    {
      const int r = q4, c0 = (tid & 3) * (KH / 4);
      float s4 = 0.f;
#pragma unroll
      for (int c = c0; c < c0 + KH / 4; ++c) s4 += tof(sm.u.h.Q[r][c]) * sm.u.h.dX[r][c];
      s4 += __shfl_xor(s4, 1, 64);
      s4 += __shfl_xor(s4, 2, 64);
      if ((tid & 3) == 0) sm.dlam[r] += s4;
    }
    // dQ = dq_part + dQK K + lambda dX ;  dK = dk_part + dQK^T Q + dG^T X + dX
    for (int t = w; t < HT; t += NWAVES) {
      const int m0 = (t / (KH / 16)) * 16, n0 = (t % (KH / 16)) * 16;
      const f4 a = mma_k<E, C>(kmaj(&sm.dQK[0][0], LC), imaj(&sm.u.h.K[0][0], LH), m0, n0, zero4(), lane);
      f4 bk = mma_k<E, C>(imaj(&sm.dQK[0][0], LC), imaj(&sm.u.h.Q[0][0], LH), m0, n0, zero4(), lane);
      bk = mma_k<E, C>(imaj(&sm.dG[0][0], LC), imaj(&sm.u.h.X[0][0], LH), m0, n0, bk, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = m0 + frow(lane, j), c = n0 + fcol(lane);
        if (r < len) {
          const float dx = sm.u.h.dX[r][c];
          const size_t o = ((size_t)(t0 + r) * H + h) * DK + k0 + c;
          dqo[o] = fromf<E>(wq[r * DK + k0 + c] + a[j] + sm.lam[r] * dx);
          dko[o] = fromf<E>(wk[r * DK + k0 + c] + bk[j] + dx);
        }
      }
    }
  }
  __syncthreads();
  if (tid < C) {
    // dlog alpha_j = sum_{r >= j} db_r  (chunk-local reverse cumulative sum)
    const int j = tid;
    float x = sm.db[C - 1 - j];
    x = wave_incl_scan(x, lane);     // lane j holds sum_{r >= C-1-j} db_r
    const float suffix = __shfl(x, C - 1 - j, 64);
    if (j < len) {
      const size_t gt = (size_t)(t0 + j) * H + h;
      p.dbeta[gt] = sm.dbeta[j];
      p.dlam[gt] = sm.dlam[j];
      if (p.dla) p.dla[gt] = suffix;
    }
  }
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_bwd_t(const Params& p, hipStream_t st) {
  constexpr int BV = 32;
  constexpr int SBV = 32;   // value columns per backward-scan workgroup
  constexpr int KH = 32;
  const int units = p.N * p.H;
  const int nb = ((units + 7) / 8) * 8 * (DV / SBV);
  if (nb > 0) {
    prof_mark(ST_SCAN_BWD, 0, st);
    hipLaunchKernelGGL((k_scan_bwd<E, DK, DV, SBV>), dim3(nb), dim3(NTHREADS), 0, st, p);
    prof_mark(ST_SCAN_BWD, 1, st);
  }
  if (p.n_slots > 0) {
    dim3 gp(p.n_slots, p.H);
    prof_mark(ST_INTRA_A, 0, st);
    hipLaunchKernelGGL((k_intra_a<E, DK, DV, BV>), gp, dim3(NTHREADS), 0, st, p);
    prof_mark(ST_INTRA_A, 1, st);
    prof_mark(ST_INTRA_B, 0, st);
    hipLaunchKernelGGL((k_intra_b<E, DK, KH>), gp, dim3(NTHREADS), 0, st, p);
    prof_mark(ST_INTRA_B, 1, st);
  }
  return hipGetLastError();
}

hipError_t launch_bwd(const Params& p, int dtype, int Dk, int Dv, hipStream_t st) {
#define QD_CASE(ET, DKV, DVV) \
  if (Dk == DKV && Dv == DVV) return launch_bwd_t<ET, DKV, DVV>(p, st);
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
