// Q-Delta chunkwise backward kernels for gfx950.
//
// The paper states no backward pass.  These kernels apply the chain rule to
// the chunk steps of the forward (see qd_fwd.hip), per chunk with entry state
// S, exit-state gradient dS' and output gradient dO:
//
//   inter-chunk (sequential, reverse):
//     dD   = P^T dO + Kbar dS'^T                  Kbar = diag(g_C / g) K
//     dV   = T^T dD = diag(beta) M^T dD
//     dS   = g_C dS' + dO^T diag(g) Q - dD^T W    (gradient w.r.t. the entry state)
//          = g_C dS' + (dO - diag(lambda) dV)^T diag(g) Q - dV^T diag(g) K
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
// k_scan_bwd  : one workgroup per (sequence, head, Dv tile); dS^T tile in fp32
//               accumulators; per chunk writes dD and dS' and produces dV.
// k_bwd_intra : per (chunk, head); the products that contract over Dv
//               (dO S, D dS', dD S, dO D^T, dD V^T), then the UT-solve backward
//               and the products over Dk; final dq, dk, dbeta, dlambda, dlog alpha.
#include "qd_common.h"
#include "qd_launch.h"

#include <type_traits>

namespace qd {

// ------------------------------------------------------------------ scan
// Backward-scan operands of one chunk, filled by direct global->LDS loads as
// swizzled row-major tiles, in sets by the phases that read them:
//   set X (phases 2-4): Q, K (C x Dk), this tile's columns of dO (C x BV) and
//                       the gate block (b, beta, lambda);
//   P (phase 2):        the output operator Gam * M_causal * Q K^T (C x C);
//   M (phase 3):        (I + A)^{-1} (C x C).
// The transposed operands (P, M^T, Q^T, K^T, dO^T) are LDS transpose reads
// of these tiles.  Set X has a ring of NA chunks, P of NP and M one buffer.
// The four producer waves split every tile's 1 KB instructions evenly;
// producers 0-2 also load one gate vector each.
template <typename E, int DK, int BV>
struct ScanBwdRing {
  static constexpr int RK = DK * (int)sizeof(E), RC = C * (int)sizeof(E), RO = BV * (int)sizeof(E);
  static constexpr int XQ = 0, XK = XQ + C * RK, XO = XK + C * RK, XG = XO + C * RO, XBYTES = XG + 3 * C * 4;
  static constexpr int MBYTES = C * RC;
  static constexpr int NA = sizeof(E) == 2 ? 3 : 2;
  static constexpr int NP = sizeof(E) == 2 ? 2 : 1;         // P buffers
  static constexpr int LQ = C * RK / 1024 / 4;              // loads per producer: Q
  static constexpr int LK = (C * RK + C * RO) / 1024 / 4;   // K and dO (plus one gate vector for producers 0-2)
  static constexpr int LM = C * RC / 1024 / 4;              // M, and P
  static_assert((C * RK / 1024) % 4 == 0 && (C * RC / 1024) % 4 == 0 && (C * RO / 1024) % 4 == 0, "even split");
  static_assert(2 * LM + LQ + LK + 1 <= 63, "outstanding-load counter range");
};

template <typename E, int DK, int BV>
struct alignas(16) ScanBwdSmem {
  static constexpr int P = Pad<E>::v;
  typedef ScanBwdRing<E, DK, BV> R;
  alignas(16) char ringX[R::NA][R::XBYTES];
  alignas(16) char ringM[R::MBYTES];
  alignas(16) char ringP[R::NP][R::MBYTES];
  E dS[BV][DK + P];   // dS' tile (row v, column k): MFMA operand and output source
  E dD[C][BV + P];    // dD (row i, column v)
  E z1[C][BV + P];    // diag(g) (dO - diag(lambda) dV)  (row r, column v)
  E z2[C][BV + P];    // -diag(g) dV
};

// One workgroup per (sequence, head, Dv tile of BV = 32): four compute waves
// and four producer waves; reverse pass over the chunks.  The exit-state
// gradient tile dS'^T (Dk x BV) lives in fp32 MFMA accumulators; compute wave
// w owns its key rows 16 KPW w.. and the chunk rows 16w.. of every C-row
// operand.
//
// W is not read: with W^T = X^T diag(g) diag(beta) M^T the entry-state
// gradient is
//   dS = g_C dS' + Q^T diag(g) (dO - diag(lambda) dV) - K^T diag(g) dV,
// dV = diag(beta) M^T dD being an output anyway.  Per chunk the compute
// waves pass three barriers:
//   B_a  dS' staged, set X, P       phase 2: dS' output; dD = P^T dO +
//        visible                    Kbar dS'^T (as its transpose); dD staged;
//   B_b  dD staged, set M visible   phase 3: dD output; dV = diag(beta) M^T dD
//                                   (as its transpose), stored; the gated
//                                   operands z1, z2 of the state gradient
//                                   formed elementwise from dV and dO;
//   B_c  z1, z2 staged              phase 4: entry-state gradient
//                                   Q^T z1 + K^T z2; dS' of the next chunk staged.
// Producers: Q of the chunk NA-1 steps ahead in phase 2, K, dO and gates of
// that chunk in phase 3, P of the next chunk in phase 2 (two buffers) or 3
// (one), M of the next chunk in phase 4; they wait for M in phase 2 and for
// set X and P of the next chunk in phase 4.
template <typename E, int DK, int DV, int BV>
__global__ __launch_bounds__(NTHREADS + 256) void k_scan_bwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LV = BV + P;
  constexpr int NVT = DV / BV;
  constexpr int NB = BV / 16;
  constexpr int KS = Mma<E>::KS, KPL = Mma<E>::KPL;
  constexpr int NKS = DK / KS;
  constexpr int KPW = DK / 16 / NWAVES;
  static_assert(KPW >= 1 && KPW * 16 * NWAVES == DK, "key blocks per wave");
  typedef typename Quad<E>::raw QR;
  typedef typename Mma<E>::frag FR;
  typedef ScanBwdRing<E, DK, BV> R;
  constexpr int NA = R::NA;
  // fp32 operands take 4-deep k-steps; their long k loops are only partly unrolled
  constexpr int UKD = NKS > 4 ? 4 : NKS;
  __shared__ ScanBwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int prod = w - NWAVES;               // 0-3 for the producer waves, negative otherwise
  const bool producer = prod >= 0;
  int unit, vt;
  if (!xcd_unit_tile(blockIdx.x, p.N * p.H, NVT, unit, vt)) return;
  const int H = p.H, n = unit / H, h = unit % H, v0 = vt * BV;
  int s, e;
  if (!seq_range(p, n, s, e)) return;
  const int base = slot_base(p, n, s);
  const int nch = max(0, min((e - s + C - 1) / C, p.n_slots - base));

  auto chunk_at = [&](int c, size_t& gi, size_t& arow, int& len) {
    const int t0 = s + c * C;
    len = min(C, e - t0);
    gi = (size_t)(base + c) * H + h;
    arow = (size_t)t0 * H + h;
  };
  // producers: Q of the chunk of iteration it (rows past the chunk re-read
  // its last row: they only meet zero dO rows and zero gates)
  auto issueQ = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    const char* Qg = (const char*)((const E*)p.q + arow * DK);
    dma_rows<R::RK, C, 4, true>(sm.ringX[it % NA] + R::XQ, Qg, (size_t)H * R::RK, len,
                                Qg + (size_t)(len - 1) * H * R::RK, 0, prod, lane);
  };
  // producers: K, dO (rows past the chunk from D, zero there) and the gates
  auto issueK = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    char* r = sm.ringX[it % NA];
    const char* Kg = (const char*)((const E*)p.k + arow * DK);
    const char* Og = (const char*)((const E*)p.dO + arow * DV + v0);
    const char* Dg = (const char*)((const E*)p.savedD + gi * C * DV + v0);
    dma_rows<R::RK, C, 4, true>(r + R::XK, Kg, (size_t)H * R::RK, len, Kg + (size_t)(len - 1) * H * R::RK, 0,
                                prod, lane);
    dma_rows<R::RO, C, 4, true>(r + R::XO, Og, (size_t)H * DV * sizeof(E), len, Dg, DV * sizeof(E), prod, lane);
    if (prod < 3) dma4_asm(p.wb + gi * 3 * C + prod * C + lane, r + R::XG + prod * C * 4);
  };
  auto issueP = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    const char* Pg = (const char*)((const E*)p.wP + gi * C * C);
    dma_rows<R::RC, C, 4, true>(sm.ringP[it % R::NP], Pg, R::RC, C, Pg, 0, prod, lane);
  };
  auto issueM = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    const char* Mg = (const char*)((const E*)p.wM + gi * C * C);
    dma_rows<R::RC, C, 4, true>(sm.ringM, Mg, R::RC, C, Mg, 0, prod, lane);
  };

  f4 acc[KPW][NB];
#pragma unroll
  for (int i = 0; i < KPW; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int kt = KPW * w + i;
      acc[i][nb] = (p.dSfin && !producer)
                       ? *(const f4*)(p.dSfin + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 +
                                      frow(lane, 0))
                       : zero4();
    }
  auto stage_dS = [&]() {
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        *(QR*)&sm.dS[nb * 16 + fcol(lane)][(KPW * w + i) * 16 + frow(lane, 0)] = Quad<E>::pack(acc[i][nb]);
  };

  if (nch > 0) {
    if (producer) {
      for (int it = 0; it < NA - 1 && it < nch; ++it) {
        issueQ(it);
        issueK(it);
      }
      issueP(0);
      issueM(0);
      wait_vm<0>();
    } else {
      stage_dS();
    }
  }
  for (int it = 0; it < nch; ++it) {
    const int c = nch - 1 - it;
    const size_t gi = (size_t)(base + c) * H + h;
    const int t0 = s + c * C, len = min(C, e - t0);
    const char* rx = sm.ringX[it % NA];
    const float* gb = (const float*)(rx + R::XG);   // b, then beta, then lambda
    const int rr = 16 * w + fcol(lane);             // chunk row of this lane's result columns
    block_sync_lds();                      // B_a: dS' staged; set X of this chunk visible
    // ---- phase 2
    if (!producer) {
      {
        // dS' of this chunk for the intra-chunk kernel (row v, column k), 16-byte stores
        constexpr int VEC = 16 / sizeof(E), PR = DK / VEC;
        E* dst = (E*)p.w_dSo + gi * DV * DK + (size_t)v0 * DK;
        for (int idx = tid; idx < BV * PR; idx += NTHREADS) {
          const int r = idx / PR, cc = (idx % PR) * VEC;
          *(uint4*)(dst + (size_t)r * DK + cc) = *(const uint4*)&sm.dS[r][cc];
        }
      }
      // dD^T (value rows, key columns 16w..) = dS' Kbar^T + dO^T P
      const float bi = gb[rr], kbi = __expf(gb[C - 1] - bi);
      f4 dt[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) dt[nb] = zero4();
#pragma unroll UKD
      for (int ks = 0; ks < NKS; ++ks) {
        const FR kB = tile_frag<E, R::RK>(rx + R::XK, 16 * w, ks * KS, lane);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          dt[nb] = Mma<E>::mma(Frag<E>::load(kmaj(&sm.dS[0][0], LK), nb * 16, ks * KS, lane), kB, dt[nb]);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 4; ++j) dt[nb][j] *= kbi;
      // + dO^T P (P causal: k blocks before this wave's key rows are skipped)
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks)
        if (ks * KS + KS > 16 * w) {
          const FR pB = tile_tr_frag<E, R::RC>(sm.ringP[it % R::NP], ks * KS, 16 * w, lane);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            dt[nb] = Mma<E>::mma(tile_tr_frag<E, R::RO>(rx + R::XO, ks * KS, nb * 16, lane), pB, dt[nb]);
        }
      // key rows past the chunk carry no gradient
      const float keep = rr < len ? 1.f : 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) *(QR*)&sm.dD[rr][nb * 16 + frow(lane, 0)] = Quad<E>::pack(keep * dt[nb]);
    } else {
      // Q of the chunk NA-1 steps ahead (its ring slot was freed at B_a) and,
      // with two P buffers, P of the next chunk (its buffer was last read in
      // the previous phase 2); then M of this chunk must have landed
      const bool q_next = it + NA - 1 < nch, p_next = R::NP == 2 && it + 1 < nch;
      if (q_next) issueQ(it + NA - 1);
      if (p_next) issueP(it + 1);
      if (q_next && p_next) wait_vm<R::LQ + R::LM>();
      else if (q_next) wait_vm<R::LQ>();
      else if (p_next) wait_vm<R::LM>();
      else wait_vm<0>();
    }
    block_sync_lds();                      // B_b: dD staged; M of this chunk visible
    // ---- phase 3
    if (!producer) {
      {
        // dD rows for the intra-chunk kernel
        constexpr int VEC = 16 / sizeof(E), PR = BV / VEC;
        E* ddst = (E*)p.w_dDb + gi * C * DV + v0;
        for (int idx = tid; idx < C * PR; idx += NTHREADS) {
          const int r = idx / PR, cc = (idx % PR) * VEC;
          *(uint4*)(ddst + (size_t)r * DV + cc) = *(const uint4*)&sm.dD[r][cc];
        }
      }
      // dV^T (value rows, chunk columns 16w..) = beta_r (dD^T M); M is lower
      // triangular, so k blocks before this wave's rows are skipped.  Each
      // lane holds four consecutive values of row rr: dV goes out directly,
      // and z1 = g_r (dO - lambda_r dV), z2 = -g_r dV are formed here, where
      // the wave's own rows cover the tile once.
      const float betar = gb[C + rr], gr = __expf(gb[rr]), lr = gb[2 * C + rr];
      E* vrow = (E*)p.dv + ((size_t)(t0 + rr) * H + h) * DV + v0;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f4 dv = zero4();
#pragma unroll
        for (int ks = 0; ks < C / KS; ++ks)
          if (ks * KS + KS > 16 * w)
            dv = Mma<E>::mma(tr_frag<E>(&sm.dD[0][0], LV, ks * KS, nb * 16, lane),
                             tile_tr_frag<E, R::RC>(sm.ringM, ks * KS, 16 * w, lane), dv);
        const int v = nb * 16 + frow(lane, 0);
        const QR doq = *(const QR*)(rx + R::XO + tile_off<R::RO>(rr, v * (int)sizeof(E)));
        f4 a, b;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dv[j] *= betar;
          a[j] = gr * (Quad<E>::get(doq, j) - lr * dv[j]);
          b[j] = -gr * dv[j];
        }
        if (rr < len) *(QR*)(vrow + v) = Quad<E>::pack(dv);
        *(QR*)&sm.z1[rr][v] = Quad<E>::pack(a);
        *(QR*)&sm.z2[rr][v] = Quad<E>::pack(b);
      }
    } else {
      if (it + NA - 1 < nch) issueK(it + NA - 1);
      if (R::NP == 1 && it + 1 < nch) issueP(it + 1);   // its buffer was last read in phase 2
    }
    block_sync_lds();                      // B_c: z1, z2 staged; M of this chunk free
    // ---- phase 4
    if (!producer) {
      // dS_entry^T = g_C dS'^T + Q^T z1 + K^T z2
      const float gC = __expf(gb[C - 1]);
#pragma unroll
      for (int i = 0; i < KPW; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[i][nb] = gC * acc[i][nb];
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) {
        FR qa[KPW], ka[KPW];
#pragma unroll
        for (int i = 0; i < KPW; ++i) {
          qa[i] = tile_tr_frag<E, R::RK>(rx + R::XQ, ks * KS, 16 * (KPW * w + i), lane);
          ka[i] = tile_tr_frag<E, R::RK>(rx + R::XK, ks * KS, 16 * (KPW * w + i), lane);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const FR z1 = tr_frag<E>(&sm.z1[0][0], LV, ks * KS, nb * 16, lane);
          const FR z2 = tr_frag<E>(&sm.z2[0][0], LV, ks * KS, nb * 16, lane);
#pragma unroll
          for (int i = 0; i < KPW; ++i) {
            acc[i][nb] = Mma<E>::mma(qa[i], z1, acc[i][nb]);
            acc[i][nb] = Mma<E>::mma(ka[i], z2, acc[i][nb]);
          }
        }
      }
      stage_dS();
    } else if (it + 1 < nch) {
      issueM(it + 1);
      // set X and P of the next chunk complete: what was issued after the
      // later of their last parts may still be in flight
      if constexpr (NA == 2) {
        wait_vm<R::LM>();                  // K and P were issued last before M
      } else {
        if (it + 2 < nch) {                // P issued after K of the next chunk: K ahead and M follow
          if (prod < 3) wait_vm<R::LK + 1 + R::LM>();
          else wait_vm<R::LK + R::LM>();
        } else {
          wait_vm<R::LM>();
        }
      }
    }
  }
  if (producer) {
    wait_vm<0>();
  } else if (p.dS0) {
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

// ------------------------------------------------------------------ intra
// Fused intra-chunk backward, one workgroup per (chunk, head) unit.
//
// Phase A walks the value dimension in tiles of 32 columns, streamed into LDS
// by direct global->LDS loads through a ring of three tiles (two in flight
// while one is consumed), and accumulates, for rows 16w.. of wave w,
//   aQ = dO S,  aK = D dS',  aW = dD S   (C x Dk)   and   aP = dO D^T, aT = dD V^T (C x C).
// Phase B1 forms the Gram products G = X K^T, Q K^T and the second part of
// dT; B2 back-propagates through the UT solve with the saved (I + A)^{-1} and
// forms dG, dQK and the beta and decay terms in MFMA-layout registers; B3
// produces dX, dq and dk.  The tail turns the decay terms into d log alpha.

// Phase-A tile of 32 value columns: S, dS' (32 value rows of Dk), D, V, dO,
// dD (C rows of 32), each in the swizzled direct-load layout; a ring of NBUF
// tiles keeps two in flight.
template <typename E, int DK>
struct TileA {
  static constexpr int BV = 32;
  static constexpr int RE = BV * (int)sizeof(E);    // row bytes of the C-row tiles
  static constexpr int RK = DK * (int)sizeof(E);    // row bytes of the state tiles
  static constexpr int S = 0, DS = S + BV * RK, D = DS + BV * RK, V = D + C * RE, DO = V + C * RE,
                       DD = DO + C * RE, BYTES = DD + C * RE;
  static constexpr int NBUF = sizeof(E) == 2 ? 3 : 2;   // fp32 tiles are twice as large
  static constexpr int LOADS = BYTES / 1024 / NWAVES;   // direct loads per wave and tile
};

template <typename E, int DK>
struct alignas(16) BwdSmem {
  static constexpr int P = Pad<E>::v;
  float b[C], g[C], kb[C], beta[C], lam[C], db[C], dbeta[C];
  float rsum[5][2][C];      // per-row partial sums of the two column halves:
                            // dbeta rows, decay rows (B2); decay, Kbar, dlambda rows (B3)
  float sdot[8];            // per-wave parts of <dS', S>
  union {
    alignas(16) char tiles[TileA<E, DK>::NBUF][TileA<E, DK>::BYTES];   // phase A
    struct {
      struct {
        E K[C][DK + P];       // chunk keys (r, k)
        E Q[C][DK + P];       // chunk queries (r, k)
        E dW[C][DK + P];      // dW = -dD S (r, k)
      } b1;                   // from phase B1 to the end of phase B3
      union {
        struct {
          union {
            struct {
              E MT[C][C + P];     // M^T (i, r)
              E dMt[C][C + P];    // (dT diag(beta))^T (i, r)
            } m;
            struct {
              E dG[C][C + P];     // dG (r, i), after M^T and dMinv^T are dead
              E dQK[C][C + P];    // dQK (r, i)
              E dGl[C][C + P];    // dQK + diag(lambda) dG (r, i)
            } g;
          } v;
          E Y[C][C + P];          // M^T dT diag(beta) (r, i)
          float dbc[16][C];       // column partial sums of dT (.) M, per row block and lane group
          float ecc[16][C];       // column partial sums of the decay-gradient terms
        } b2;
        struct {
          E keep[3][C][C + P];    // dG, dQK, dQK + diag(lambda) dG (phase-B3 A operands)
          E oq[C][DK + P];        // dq staging, over the dead Y and column sums
          E ok[C][DK + P];        // dk staging
        } b3;
      } u;
    } s;
  } x;
  // M = (I + A)^{-1} (r, i), direct-loaded at the start (swizzled rows of C
  // elements, outside the phase-A ring)
  alignas(16) char Mm[C * C * sizeof(E)];
};

// Eight waves: wave w takes rows 16 rb.. (rb = w & 3) of every C-row operand
// and one half (ch = w >> 2) of the Dk column blocks and of the C x C column
// blocks; two waves share each SIMD and hide each other's latency.
constexpr int INTRA_THREADS = 2 * NTHREADS;

template <typename E, int DK, int DV>
__global__ __launch_bounds__(INTRA_THREADS) void k_bwd_intra(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int BV = 32;
  constexpr int LC = C + P;
  constexpr int KS = Mma<E>::KS;
  constexpr int NKB = DK / 16;        // 16-column blocks of Dk
  constexpr int HK = NKB / 2;         // Dk blocks per column half
  constexpr int NVT = DV / BV;
  constexpr int IT = INTRA_THREADS;
  typedef typename Mma<E>::frag FR;
  typedef typename Quad<E>::raw QR;
  __shared__ BwdSmem<E, DK> sm;
  if ((int)blockIdx.x < p.lead) {
    // a leading workgroup holds its CU for about half a unit, so that half of
    // the CUs run phase-shifted and their value-dimension loads overlap the
    // other half's compute phases
    const long long t0c = clock64();
    while (clock64() - t0c < p.lead_cycles) __builtin_amdgcn_s_sleep(32);
    return;
  }
  const int bid = (int)blockIdx.x - p.lead;
  const int g = bid % p.n_slots, h = bid / p.n_slots, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int rb = w & 3, ch = w >> 2;
  const int kb0 = ch * HK, ib0 = 2 * ch;
  int n, t0, len;
  if (!locate(p, g, n, t0, len)) return;
  const int H = p.H;
  const size_t gi = (size_t)g * H + h;
  const size_t arow = (size_t)t0 * H + h;   // first activation row of the chunk


  // ---------------- phase A: contractions over the value dimension
  typedef TileA<E, DK> TA;
  f4 aQ[HK], aK[HK], aW[HK], aP[2], aT[2], asd = zero4();
#pragma unroll
  for (int i = 0; i < HK; ++i) aQ[i] = aK[i] = aW[i] = zero4();
#pragma unroll
  for (int i = 0; i < 2; ++i) aP[i] = aT[i] = zero4();
  constexpr size_t ES = sizeof(E);
  const char* Sg = (const char*)((const E*)p.saved + gi * DK * DV);
  const char* dSg = (const char*)((const E*)p.w_dSo + gi * DK * DV);
  const char* Dg = (const char*)((const E*)p.savedD + gi * C * DV);
  const char* dDg = (const char*)((const E*)p.w_dDb + gi * C * DV);
  const char* dOg = (const char*)((const E*)p.dO + arow * DV);
  const char* Vg = (const char*)((const E*)p.v + arow * DV);
  // direct loads are issued by waves 0-3 only; the others' waits are no-ops
  const bool loader = w < NWAVES;
  constexpr int RBC = C * (int)sizeof(E);
  // rows of V and dO past the chunk come from D, whose rows there are zero
  auto issue = [&](int vt) {
    char* t = &sm.x.tiles[vt % TA::NBUF][0];
    const size_t vb = (size_t)vt * BV;
    dma_rows<TA::RK, BV>(t + TA::S, Sg + vb * TA::RK, TA::RK, BV, Sg, 0, w, lane);
    dma_rows<TA::RK, BV>(t + TA::DS, dSg + vb * TA::RK, TA::RK, BV, dSg, 0, w, lane);
    dma_rows<TA::RE, C>(t + TA::D, Dg + vb * ES, DV * ES, C, Dg, 0, w, lane);
    dma_rows<TA::RE, C>(t + TA::DD, dDg + vb * ES, DV * ES, C, dDg, 0, w, lane);
    dma_rows<TA::RE, C>(t + TA::V, Vg + vb * ES, (size_t)H * DV * ES, len, Dg + vb * ES, DV * ES, w, lane);
    dma_rows<TA::RE, C>(t + TA::DO, dOg + vb * ES, (size_t)H * DV * ES, len, Dg + vb * ES, DV * ES, w, lane);
  };
  // the first tiles and M = (I + A)^{-1} go out first; the gates and the
  // chunk's K, Q rows (registers, needed from phase B on) follow once the
  // first tile has landed, so that they do not compete with it
  constexpr int NB0 = NVT < TA::NBUF ? NVT : TA::NBUF;
  if (loader) {
#pragma unroll
    for (int vt = 0; vt < NB0; ++vt) issue(vt);
    const char* Mg = (const char*)((const E*)p.wM + gi * C * C);
    dma_rows<RBC, C>(sm.Mm, Mg, RBC, C, Mg, 0, w, lane);
  }
  const int ti = tid & (C - 1);
  float gb, gbeta, glam;
  TileRegs<E, C, DK, IT> rKf, rQf;
  // vector-memory operations a loading wave has issued after tile vt's, at
  // the wait for tile vt: later tiles, and M and the register loads when
  // tile vt is one of the first NB0
  constexpr int ML = C * RBC / 1024 / NWAVES;
  constexpr int KQN = 3 + 2 * TileRegs<E, C, DK, IT>::N;
  static_assert((NB0 - 1) * TA::LOADS + ML <= 63 && 2 * TA::LOADS + ML + KQN <= 63, "outstanding-load counter range");
  constexpr int UVT = NVT > 4 ? 1 : NVT;   // full unroll only for short tile loops
#pragma unroll UVT
  for (int vt = 0; vt < NVT; ++vt) {
    // tile vt is complete once at most `pending` later operations are outstanding
    const int after = (vt == 0 ? NB0 : min(NVT, vt + TA::NBUF - 1)) - 1 - vt;
    const int extra = vt < NB0 ? ML + (vt >= 1 ? KQN : 0) : 0;
    const int pending = after * TA::LOADS + extra;
    if (vt == 0) wait_vm<(NB0 - 1) * TA::LOADS + ML>();
    else if (pending >= 2 * TA::LOADS + ML + KQN) wait_vm<2 * TA::LOADS + ML + KQN>();
    else if (pending >= TA::LOADS + ML + KQN) wait_vm<TA::LOADS + ML + KQN>();
    else if (pending >= ML + KQN) wait_vm<ML + KQN>();
    else if (pending >= 2 * TA::LOADS) wait_vm<2 * TA::LOADS>();
    else if (pending >= TA::LOADS) wait_vm<TA::LOADS>();
    else wait_vm<0>();
    block_sync_lds();                 // tile vt visible; tile vt-1's buffer is free
    if (vt == 0) {
      asm volatile("" ::: "memory");
      gb = p.wb[gi * 3 * C + ti];
      gbeta = p.wb[gi * 3 * C + C + ti];
      glam = p.wb[gi * 3 * C + 2 * C + ti];
      rKf.load_clamped((const E*)p.k + arow * DK, (size_t)H * DK, len, tid);
      rQf.load_clamped((const E*)p.q + arow * DK, (size_t)H * DK, len, tid);
      asm volatile("" ::: "memory");
    }
    if (loader && vt >= 1 && vt + TA::NBUF - 1 < NVT) issue(vt + TA::NBUF - 1);
    const char* t = &sm.x.tiles[vt % TA::NBUF][0];
#pragma unroll
    for (int ks = 0; ks < BV / KS; ++ks) {
      const FR aO = tile_frag<E, TA::RE>(t + TA::DO, 16 * rb, ks * KS, lane);
      const FR adD = tile_frag<E, TA::RE>(t + TA::DD, 16 * rb, ks * KS, lane);
      const FR aD = tile_frag<E, TA::RE>(t + TA::D, 16 * rb, ks * KS, lane);
#pragma unroll
      for (int i = 0; i < HK; ++i) {
        const int kb = kb0 + i;
        const FR bS = tile_tr_frag<E, TA::RK>(t + TA::S, ks * KS, kb * 16, lane);
        const FR bdS = tile_tr_frag<E, TA::RK>(t + TA::DS, ks * KS, kb * 16, lane);
        aQ[i] = Mma<E>::mma(aO, bS, aQ[i]);
        aW[i] = Mma<E>::mma(adD, bS, aW[i]);
        aK[i] = Mma<E>::mma(aD, bdS, aK[i]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ib = ib0 + i;
        const FR bD = tile_frag<E, TA::RE>(t + TA::D, ib * 16, ks * KS, lane);
        const FR bV = tile_frag<E, TA::RE>(t + TA::V, ib * 16, ks * KS, lane);
        aP[i] = Mma<E>::mma(aO, bD, aP[i]);
        aT[i] = Mma<E>::mma(adD, bV, aT[i]);
      }
    }
    // <dS', S> = trace(S dS'^T): wave w adds the diagonal 16 x 16 block
    // (w & 1) of this tile's S dS'^T over the key steps w >> 1, +4, ...
#pragma unroll
    for (int ks = 0; ks < DK / KS; ks += 4)
      if (ks + (w >> 1) < DK / KS)
        asd = Mma<E>::mma(tile_frag<E, TA::RK>(t + TA::S, 16 * (w & 1), (ks + (w >> 1)) * KS, lane),
                          tile_frag<E, TA::RK>(t + TA::DS, 16 * (w & 1), (ks + (w >> 1)) * KS, lane), asd);
  }
  {
    // diagonal elements of the accumulated block: row 4 (l >> 4) + j == column l & 15
    const int j = (lane & 15) - 4 * (lane >> 4);
    float sdot = 0.f;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      if (jj == j) sdot = asd[jj];
    sdot = wave_sum(sdot);
    if (lane == 0) sm.sdot[w] = sdot;
  }
  if (tid < C) {
    sm.b[tid] = gb;
    sm.g[tid] = __expf(gb);
    sm.beta[tid] = gbeta;   // zero past the chunk in the gate block
    sm.lam[tid] = glam;
  }

  // ---------------- phase B1: G = X K^T, QK = Q K^T, dT2 = dW (g X)^T
  constexpr int LKD = DK + P;
  block_sync_lds();
  rKf.store_rows(&sm.x.s.b1.K[0][0], LKD, len, tid);
  rQf.store_rows(&sm.x.s.b1.Q[0][0], LKD, len, tid);
#pragma unroll
  for (int i = 0; i < HK; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      sm.x.s.b1.dW[16 * rb + frow(lane, j)][(kb0 + i) * 16 + fcol(lane)] = fromf<E>(-aW[i][j]);
  if (tid < C) sm.kb[tid] = __expf(sm.b[C - 1] - sm.b[tid]);
  block_sync_lds();
  // G = X K^T = K K^T + diag(lambda) Q K^T and dT2 = dW (diag(g) X)^T =
  // (dW K^T + dW Q^T diag(lambda)) diag(g): four products of the stored
  // operands, the gates applied to the fp32 results
  f4 aG[2], aQK[2], adT[2];
  {
    f4 aKK[2], aDK[2], aDQ[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) aKK[i] = aQK[i] = aDK[i] = aDQ[i] = zero4();
#pragma unroll
    for (int ks = 0; ks < DK / KS; ++ks) {
      const FR kA = Frag<E>::load(kmaj(&sm.x.s.b1.K[0][0], LKD), 16 * rb, ks * KS, lane);
      const FR qA = Frag<E>::load(kmaj(&sm.x.s.b1.Q[0][0], LKD), 16 * rb, ks * KS, lane);
      const FR dwA = Frag<E>::load(kmaj(&sm.x.s.b1.dW[0][0], LKD), 16 * rb, ks * KS, lane);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ib = ib0 + i;
        const FR kB = Frag<E>::load(kmaj(&sm.x.s.b1.K[0][0], LKD), ib * 16, ks * KS, lane);
        const FR qB = Frag<E>::load(kmaj(&sm.x.s.b1.Q[0][0], LKD), ib * 16, ks * KS, lane);
        aKK[i] = Mma<E>::mma(kA, kB, aKK[i]);
        aQK[i] = Mma<E>::mma(qA, kB, aQK[i]);
        aDK[i] = Mma<E>::mma(dwA, kB, aDK[i]);
        aDQ[i] = Mma<E>::mma(dwA, qB, aDQ[i]);
      }
    }
    const int r0 = 16 * rb + frow(lane, 0);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = (ib0 + i) * 16 + fcol(lane);
      const float gc = sm.g[c], lc = sm.lam[c];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        aG[i][j] = aKK[i][j] + sm.lam[r0 + j] * aQK[i][j];
        adT[i][j] = gc * (aDK[i][j] + lc * aDQ[i][j]);
      }
    }
  }

  // ---------------- phase B2: UT-solve backward and the C x C gradient terms.
  // Lane (w, lane) holds element (r, c) = (16 rb + frow(lane, j), 16 ib + fcol(lane))
  // of every C x C accumulator, for the two column blocks ib of its half.
  const int rw = 16 * rb + frow(lane, 0), cl = fcol(lane);
  {
    // dT = dD V^T + dW (g X)^T: column sums of dT (.) M feed dbeta; M^T and
    // (dT diag(beta))^T become the operands of Y = M^T dT diag(beta)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = (ib0 + i) * 16 + cl;
      const float bc = sm.beta[c];
      f4 mv, dm;
      float cs = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float m = tof(*(const E*)(sm.Mm + tile_off<RBC>(rw + j, c * (int)sizeof(E))));
        const float dt = aT[i][j] + adT[i][j];
        cs += dt * m;
        mv[j] = m;
        dm[j] = dt * bc;
      }
      *(QR*)&sm.x.s.u.b2.v.m.MT[c][rw] = Quad<E>::pack(mv);
      *(QR*)&sm.x.s.u.b2.v.m.dMt[c][rw] = Quad<E>::pack(dm);
      sm.x.s.u.b2.dbc[4 * rb + (lane >> 4)][c] = cs;
    }
  }
  block_sync_lds();
  f4 adA[2];
  {
    // Y = M^T dMinv: rows 16 rb.., this half's column blocks
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int ib = ib0 + i;
      const f4 y = mma_k<E, C>(kmaj(&sm.x.s.u.b2.v.m.MT[0][0], LC), kmaj(&sm.x.s.u.b2.v.m.dMt[0][0], LC), 16 * rb,
                               ib * 16, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.x.s.u.b2.Y[rw + j][ib * 16 + cl] = fromf<E>(y[j]);
    }
    block_sync_lds();                  // Y complete; M^T and dMinv^T dead after this point
#pragma unroll
    for (int i = 0; i < 2; ++i) {           // dA = strictLower(-Y M^T)
      adA[i] = zero4();
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks)
        adA[i] = Mma<E>::mma(Frag<E>::load(kmaj(&sm.x.s.u.b2.Y[0][0], LC), 16 * rb, ks * KS, lane),
                             tile_frag<E, RBC>(sm.Mm, (ib0 + i) * 16, ks * KS, lane), adA[i]);
    }
  }
  {
    // dG = diag(beta) dA (.) Gamma, dQK = dP (.) Gamma (causal, inclusive),
    // the decay-gradient terms t = (dG (.) G + dQK (.) QK) and the rows of
    // dbeta from A = strictLower(diag(beta) Gamma (.) G)
    float br[4], betar[4], lamr[4], dbr[4] = {0.f, 0.f, 0.f, 0.f}, er[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      br[j] = sm.b[rw + j];
      betar[j] = sm.beta[rw + j];
      lamr[j] = sm.lam[rw + j];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = (ib0 + i) * 16 + cl;
      const float bc = sm.b[c];
      float ec = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = rw + j;
        const float gam = (r >= c) ? __expf(br[j] - bc) : 0.f;
        const float dA = (r > c) ? -adA[i][j] : 0.f;
        const float dAg = dA * gam;
        const float dg = dAg * betar[j];
        const float dqk = aP[i][j] * gam;
        const float t = dg * aG[i][j] + dqk * aQK[i][j];
        dbr[j] += dAg * aG[i][j];
        er[j] += t;
        ec += t;
        sm.x.s.u.b2.v.g.dG[r][c] = fromf<E>(dg);
        sm.x.s.u.b2.v.g.dQK[r][c] = fromf<E>(dqk);
        sm.x.s.u.b2.v.g.dGl[r][c] = fromf<E>(dqk + lamr[j] * dg);
      }
      sm.x.s.u.b2.ecc[4 * rb + (lane >> 4)][c] = ec;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dbr[j] = sum16(dbr[j]);
      er[j] = sum16(er[j]);
    }
    if (cl == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sm.rsum[0][ch][rw + j] = dbr[j];
        sm.rsum[1][ch][rw + j] = er[j];
      }
    }
  }
  block_sync_lds();
  if (tid < C) {
    // dbeta = row parts + colsum(dT (.) M); db = row parts - column parts of the decay terms
    float cb = 0.f, ce = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      cb += sm.x.s.u.b2.dbc[v][tid];
      ce += sm.x.s.u.b2.ecc[v][tid];
    }
    sm.dbeta[tid] = sm.rsum[0][0][tid] + sm.rsum[0][1][tid] + cb;
    sm.db[tid] = sm.rsum[1][0][tid] + sm.rsum[1][1][tid] - ce;
  }
  block_sync_lds();                    // the b2 buffers are dead past here

  // ---------------- phase B3: dX, dq, dk (rows 16 rb.., Dk blocks of this half)
  // K^T, Q^T and dW^T fragments are transpose reads of the row-major K, Q, dW
  // kept since phase B1; dG^T, (dQK + diag(lambda) dG)^T and M^T likewise
  // (T^T dW = diag(beta) M^T dW; dQK^T Q + dG^T X = dG^T K + (dQK + diag(lambda) dG)^T Q)
  {
    constexpr int NTK = C / KS;
    FR tA[NTK], gA[NTK], qkA[NTK], gltA[NTK], gtA[NTK];
    const E* dGp = &sm.x.s.u.b2.v.g.dG[0][0];
    const E* dQKp = &sm.x.s.u.b2.v.g.dQK[0][0];
    const E* dGlp = &sm.x.s.u.b2.v.g.dGl[0][0];
#pragma unroll
    for (int ks = 0; ks < NTK; ++ks) {
      tA[ks] = tile_tr_frag<E, RBC>(sm.Mm, ks * KS, 16 * rb, lane);
      gA[ks] = Frag<E>::load(kmaj(dGp, LC), 16 * rb, ks * KS, lane);
      qkA[ks] = Frag<E>::load(kmaj(dQKp, LC), 16 * rb, ks * KS, lane);
      gltA[ks] = tr_frag<E>(dGlp, LC, ks * KS, 16 * rb, lane);
      gtA[ks] = tr_frag<E>(dGp, LC, ks * KS, 16 * rb, lane);
    }
    const int r0 = 16 * rb + frow(lane, 0);
    float rdb[4] = {0.f, 0.f, 0.f, 0.f}, rtk[4] = {0.f, 0.f, 0.f, 0.f}, rdl[4] = {0.f, 0.f, 0.f, 0.f};
    float gr4[4], lr4[4], kbr4[4], br4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      gr4[j] = sm.g[r0 + j];
      lr4[j] = sm.lam[r0 + j];
      kbr4[j] = sm.kb[r0 + j];
      br4[j] = sm.beta[r0 + j];
    }
    const E* Kp = &sm.x.s.b1.K[0][0];
    const E* Qp = &sm.x.s.b1.Q[0][0];
    const E* dWp = &sm.x.s.b1.dW[0][0];
#pragma unroll
    for (int i = 0; i < HK; ++i) {
      const int kb = kb0 + i;
      f4 dgx = zero4(), dxp = zero4(), dqp = zero4(), dkp = zero4();
#pragma unroll
      for (int ks = 0; ks < NTK; ++ks) {
        const FR ktB = tr_frag<E>(Kp, LKD, ks * KS, kb * 16, lane);
        const FR qtB = tr_frag<E>(Qp, LKD, ks * KS, kb * 16, lane);
        const FR dwB = tr_frag<E>(dWp, LKD, ks * KS, kb * 16, lane);
        dgx = Mma<E>::mma(tA[ks], dwB, dgx);      // M^T dW
        dxp = Mma<E>::mma(gA[ks], ktB, dxp);      // dG K
        dqp = Mma<E>::mma(qkA[ks], ktB, dqp);     // dQK K
        dkp = Mma<E>::mma(gtA[ks], ktB, dkp);     // dG^T K
        dkp = Mma<E>::mma(gltA[ks], qtB, dkp);    // (dQK + diag(lambda) dG)^T Q
      }
      const int kc = kb * 16 + fcol(lane);
      const f4 kv = tr_col4(Kp, LKD, r0, kb * 16, lane);
      const f4 qv = tr_col4(Qp, LKD, r0, kb * 16, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + j;
        const float Kv = kv[j], Qv = qv[j];
        const float gr = gr4[j], lr = lr4[j], kbr = kbr4[j];
        const float X = Kv + lr * Qv, tdw = br4[j] * dgx[j];   // (T^T dW)_r
        rdb[j] += gr * (X * tdw + Qv * aQ[i][j]);
        rtk[j] += kbr * Kv * aK[i][j];
        const float dX = gr * tdw + dxp[j];
        rdl[j] += Qv * dX;
        sm.x.s.u.b3.oq[r][kc] = fromf<E>(gr * aQ[i][j] + dqp[j] + lr * dX);
        sm.x.s.u.b3.ok[r][kc] = fromf<E>(kbr * aK[i][j] + dkp[j] + dX);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      rdb[j] = sum16(rdb[j]);
      rtk[j] = sum16(rtk[j]);
      rdl[j] = sum16(rdl[j]);
    }
    if (fcol(lane) == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sm.rsum[2][ch][r0 + j] = rdb[j];
        sm.rsum[3][ch][r0 + j] = rtk[j];
        sm.rsum[4][ch][r0 + j] = rdl[j];
      }
    }
  }
  block_sync_lds();
  {
    constexpr int VEC = 16 / sizeof(E), PR = DK / VEC;
    E* dqo = (E*)p.dq + arow * DK;
    E* dko = (E*)p.dk + arow * DK;
    for (int idx = tid; idx < C * PR; idx += IT) {
      const int r = idx / PR, cc = (idx % PR) * VEC;
      if (r < len) {
        *(uint4*)(dqo + (size_t)r * H * DK + cc) = *(const uint4*)&sm.x.s.u.b3.oq[r][cc];
        *(uint4*)(dko + (size_t)r * H * DK + cc) = *(const uint4*)&sm.x.s.u.b3.ok[r][cc];
      }
    }
  }
  if (tid < C) {
    // Kbar terms: db_r -= t_r, db_{C-1} += sum_r t_r + g_C <dS', S>;
    // then dlog alpha_j = sum_{r >= j} db_r (chunk-local reverse cumulative sum)
    const int j = tid;
    const float tk = sm.rsum[3][0][j] + sm.rsum[3][1][j];
    float tot = tk;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) tot += __shfl_xor(tot, off, 64);
    float dbj = sm.db[j] + sm.rsum[2][0][j] + sm.rsum[2][1][j] - tk;
    if (j == C - 1) {
      float sd = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) sd += sm.sdot[q];
      dbj += tot + sm.g[C - 1] * sd;
    }
    float x = __shfl(dbj, C - 1 - j, 64);
    x = wave_incl_scan(x, lane);
    const float suffix = __shfl(x, C - 1 - j, 64);
    if (j < len) {
      const size_t gt = arow + (size_t)j * H;
      p.dbeta[gt] = sm.dbeta[j];
      p.dlam[gt] = sm.rsum[4][0][j] + sm.rsum[4][1][j];
      if (p.dla) p.dla[gt] = suffix;
    }
  }
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_bwd_t(const Params& p, hipStream_t st) {
  constexpr int SBV = 32;   // value columns per backward-scan workgroup
  const int units = p.N * p.H;
  const int nb = ((units + 7) / 8) * 8 * (DV / SBV);
  if (nb > 0) {
    prof_mark(ST_SCAN_BWD, 0, st);
    hipLaunchKernelGGL((k_scan_bwd<E, DK, DV, SBV>), dim3(nb), dim3(NTHREADS + 256), 0, st, p);
    prof_mark(ST_SCAN_BWD, 1, st);
  }
  if (p.n_slots > 0) {
    // Every unit costs the same, so without an offset all CUs would load
    // their value-dimension tiles together and then compute together, leaving
    // HBM idle half the time.  Half of the CUs start about half a unit later.
    Params q = p;
    const int total = p.n_slots * p.H, cus = device_cu_count();
    q.lead = total >= 4 * cus ? cus / 2 : 0;
    q.lead_cycles = 15000;
    prof_mark(ST_INTRA, 0, st);
    hipLaunchKernelGGL((k_bwd_intra<E, DK, DV>), dim3(total + q.lead), dim3(INTRA_THREADS), 0, st, q);
    prof_mark(ST_INTRA, 1, st);
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
