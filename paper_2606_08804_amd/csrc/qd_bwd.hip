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
//     dD   (formed again from dS', dO and P, exactly as the scan formed it)
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
//               accumulators; per chunk writes dS' and produces dV.
// k_bwd_intra : per (chunk, head); dD, then the products that contract over Dv
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
  // ring depths: fp32 tiles and 64-column value tiles leave room for two
  // chunks of set X and one P buffer
  static constexpr bool DEEP = sizeof(E) == 2 && BV == 32;
  static constexpr int NA = DEEP ? 3 : 2;
  static constexpr int NP = DEEP ? 2 : 1;                   // P buffers
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

// One workgroup per (sequence, head, Dv tile of BV value rows): NCW compute
// waves (eight for bf16, two per SIMD, as in the forward scan) and four
// producer waves; reverse pass over the chunks.  The exit-state gradient tile
// dS'^T (Dk x BV) lives in fp32 MFMA accumulators, split over the compute
// waves by key blocks (and value blocks when there are more waves than key
// blocks); compute wave w owns chunk rows 16 (w & 3).. of every C-row result
// and a range of its value blocks.
//
// W is not read: with W^T = X^T diag(g) diag(beta) M^T the entry-state
// gradient is
//   dS = g_C dS' + Q^T diag(g) (dO - diag(lambda) dV) - K^T diag(g) dV,
// dV = diag(beta) M^T dD being an output anyway.  Per chunk the compute
// waves pass three barriers:
//   B_a  dS' staged, set X, P       phase 2: dS' output; dD = P^T dO +
//        visible                    Kbar dS'^T (as its transpose); dD staged;
//   B_b  dD staged, set M visible   phase 3: dV = diag(beta) M^T dD
//                                   (as its transpose), stored; the gated
//                                   operands z1, z2 of the state gradient
//                                   formed elementwise from dV and dO;
//   B_c  z1, z2 staged              phase 4: entry-state gradient
//                                   Q^T z1 + K^T z2; dS' of the next chunk staged.
// Producers: Q of the chunk NA-1 steps ahead in phase 2, K, dO and gates of
// that chunk in phase 3, P of the next chunk in phase 2 (two buffers) or 3
// (one), M of the next chunk in phase 4; they wait for M in phase 2 and for
// set X and P of the next chunk in phase 4.
template <typename E, int DK, int DV, int BV, int NCW>
__global__ __launch_bounds__(NCW * 64 + 256) void k_scan_bwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LV = BV + P;
  constexpr int NVT = DV / BV;
  constexpr int NB = BV / 16;
  constexpr int KS = Mma<E>::KS;
  constexpr int NKS = DK / KS;
  constexpr int NCT = NCW * 64;               // compute threads
  constexpr int NBW = NB / (NCW / 4);         // value blocks per wave in phases 2-3
  constexpr int KB = DK / 16;
  constexpr int KPW = KB >= NCW ? KB / NCW : 1;   // key blocks of dS'^T per wave
  constexpr int SG = KB >= NCW ? 1 : NCW / KB;    // waves that share a key block
  constexpr int NBS = NB / SG;                    // value blocks of dS'^T per wave
  static_assert(NCW % 4 == 0 && NBW >= 1 && NBS >= 1 && KPW * (NCW / SG) == KB, "wave mapping");
  typedef typename Quad<E>::raw QR;
  typedef typename Mma<E>::frag FR;
  typedef ScanBwdRing<E, DK, BV> R;
  constexpr int NA = R::NA;
  // fp32 operands take 4-deep k-steps; their long k loops are only partly unrolled
  constexpr int UKD = NKS > 4 ? 4 : NKS;
  __shared__ ScanBwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id(tid);
  const int prod = w - NCW;                  // 0-3 for the producer waves, negative otherwise
  const bool producer = prod >= 0;
  const int cb = w & 3, nb0 = (w >> 2) * NBW;
  const int kb0 = (w % (NCW / SG)) * KPW, ns0 = (w / (NCW / SG)) * NBS;
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
  // producers: K, dO (rows past the chunk from the preparation's zero block)
  // and the gates
  auto issueK = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    char* r = sm.ringX[it % NA];
    const char* Kg = (const char*)((const E*)p.k + arow * DK);
    const char* Og = (const char*)((const E*)p.dO + arow * DV + v0);
    static_assert(R::RO <= 1024, "a row of dO within the zero block");
    dma_rows<R::RK, C, 4, true>(r + R::XK, Kg, (size_t)H * R::RK, len, Kg + (size_t)(len - 1) * H * R::RK, 0,
                                prod, lane);
    dma_rows<R::RO, C, 4, true>(r + R::XO, Og, (size_t)H * DV * sizeof(E), len, (const char*)p.wZ, 0, prod, lane);
    if (prod < 3) dma4_asm(p.wb + gi * 3 * C + prod * C + lane, r + R::XG + prod * C * 4);
  };
  auto issueP = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    dma_lbt<E, 4>(sm.ringP[it % R::NP], (const char*)((const E*)p.wP + gi * LBT_ELEMS), prod, lane);
  };
  auto issueM = [&](int it) {
    size_t gi, arow;
    int len;
    chunk_at(nch - 1 - it, gi, arow, len);
    dma_lbt<E, 4>(sm.ringM, (const char*)((const E*)p.wM + gi * LBT_ELEMS), prod, lane);
  };

  f4 acc[KPW][NBS];
#pragma unroll
  for (int i = 0; i < KPW; ++i)
#pragma unroll
    for (int j = 0; j < NBS; ++j) {
      const int kt = kb0 + i, nb = ns0 + j;
      acc[i][j] = (p.dSfin && !producer)
                      ? *(const f4*)(p.dSfin + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 +
                                     frow(lane, 0))
                      : zero4();
    }
  auto stage_dS = [&]() {
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int j = 0; j < NBS; ++j)
        *(QR*)&sm.dS[(ns0 + j) * 16 + fcol(lane)][(kb0 + i) * 16 + frow(lane, 0)] = Quad<E>::pack(acc[i][j]);
  };

  // P and M arrive packed: the chunks above their diagonal blocks are zeroed
  // once here and never loaded (the first barrier of the loop orders these
  // stores before any read)
  zero_upper_chunks<E>(sm.ringM, tid, NCT + 256);
#pragma unroll
  for (int i = 0; i < R::NP; ++i) zero_upper_chunks<E>(sm.ringP[i], tid, NCT + 256);
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
    const int rr = 16 * cb + fcol(lane);            // chunk row of this lane's result columns
    block_sync_lds();                      // B_a: dS' staged; set X of this chunk visible
    // ---- phase 2
    if (!producer) {
      {
        // dS' of this chunk for the intra-chunk kernel (row v, column k), 16-byte stores
        constexpr int VEC = 16 / sizeof(E), PR = DK / VEC;
        E* dst = (E*)p.w_dSo + gi * DV * DK + (size_t)v0 * DK;
        for (int idx = tid; idx < BV * PR; idx += NCT) {
          const int r = idx / PR, cc = (idx % PR) * VEC;
          *(uint4*)(dst + (size_t)r * DK + cc) = *(const uint4*)&sm.dS[r][cc];
        }
      }
      // dD^T (value rows, chunk columns 16 cb..) = dS' Kbar^T + dO^T P
      const float bi = gb[rr], kbi = __expf(gb[C - 1] - bi);
      f4 dt[NBW];
#pragma unroll
      for (int j = 0; j < NBW; ++j) dt[j] = zero4();
#pragma unroll UKD
      for (int ks = 0; ks < NKS; ++ks) {
        const FR kB = tile_frag<E, R::RK>(rx + R::XK, 16 * cb, ks * KS, lane);
#pragma unroll
        for (int j = 0; j < NBW; ++j)
          dt[j] = Mma<E>::mma(Frag<E>::load(kmaj(&sm.dS[0][0], LK), (nb0 + j) * 16, ks * KS, lane), kB, dt[j]);
      }
#pragma unroll
      for (int j = 0; j < NBW; ++j)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) dt[j][jj] *= kbi;
      // + dO^T P (P causal: k blocks before this wave's chunk rows are zero)
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks)
        if (keep_kblock<E>(ks * KS + KS > 16 * cb)) {
          const FR pB = tile_tr_frag<E, R::RC>(sm.ringP[it % R::NP], ks * KS, 16 * cb, lane);
#pragma unroll
          for (int j = 0; j < NBW; ++j)
            dt[j] = Mma<E>::mma(tile_tr_frag<E, R::RO>(rx + R::XO, ks * KS, (nb0 + j) * 16, lane), pB, dt[j]);
        }
      // key rows past the chunk carry no gradient
      const float keep = rr < len ? 1.f : 0.f;
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        *(QR*)&sm.dD[rr][(nb0 + j) * 16 + frow(lane, 0)] = Quad<E>::pack(keep * dt[j]);
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
      // dV^T (value rows, chunk columns 16 cb..) = beta_r (dD^T M); M is lower
      // triangular (k blocks before this wave's rows are zero).  Each
      // lane holds four consecutive values of row rr: dV goes out directly,
      // and z1 = g_r (dO - lambda_r dV), z2 = -g_r dV are formed here, where
      // the wave's own rows cover the tile once.
      const float betar = gb[C + rr], gr = __expf(gb[rr]), lr = gb[2 * C + rr];
      E* vrow = (E*)p.dv + ((size_t)(t0 + rr) * H + h) * DV + v0;
#pragma unroll
      for (int jn = 0; jn < NBW; ++jn) {
        const int nb = nb0 + jn;
        f4 dv = zero4();
#pragma unroll
        for (int ks = 0; ks < C / KS; ++ks)
          if (keep_kblock<E>(ks * KS + KS > 16 * cb))
            dv = Mma<E>::mma(tr_frag<E>(&sm.dD[0][0], LV, ks * KS, nb * 16, lane),
                             tile_tr_frag<E, R::RC>(sm.ringM, ks * KS, 16 * cb, lane), dv);
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
        for (int j = 0; j < NBS; ++j) acc[i][j] = gC * acc[i][j];
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) {
        FR qa[KPW], ka[KPW];
#pragma unroll
        for (int i = 0; i < KPW; ++i) {
          qa[i] = tile_tr_frag<E, R::RK>(rx + R::XQ, ks * KS, 16 * (kb0 + i), lane);
          ka[i] = tile_tr_frag<E, R::RK>(rx + R::XK, ks * KS, 16 * (kb0 + i), lane);
        }
#pragma unroll
        for (int j = 0; j < NBS; ++j) {
          const FR z1 = tr_frag<E>(&sm.z1[0][0], LV, ks * KS, (ns0 + j) * 16, lane);
          const FR z2 = tr_frag<E>(&sm.z2[0][0], LV, ks * KS, (ns0 + j) * 16, lane);
#pragma unroll
          for (int i = 0; i < KPW; ++i) {
            acc[i][j] = Mma<E>::mma(qa[i], z1, acc[i][j]);
            acc[i][j] = Mma<E>::mma(ka[i], z2, acc[i][j]);
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
      for (int j = 0; j < NBS; ++j) {
        const int kt = kb0 + i, nb = ns0 + j;
        *(f4*)(p.dS0 + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) =
            acc[i][j];
      }
  }
}

// ------------------------------------------------------------------ intra
// Fused intra-chunk backward, one four-wave workgroup per (chunk, head) unit.
// Two workgroups share a CU (under 80 KB of LDS and 256 VGPRs each), so that
// one streams its value-dimension tiles (bound by the CU's memory pipeline)
// while the other computes (bound by VALU work).  Wave w owns chunk rows
// 16w.. of every C-row operand.
//
// Phase A walks the value dimension in tiles of 32 columns through a ring of
// two LDS tiles.  The tile's dD rows are not read from memory: each wave
// forms its own rows as the backward scan does (dD^T = dS' Kbar^T + dO^T P,
// the same operands in the same order, so the values are the scan's own),
// from its rows of K held in registers and P, which sits in the M buffer
// until the last tile.  Then it accumulates
//   (dO S)^T, (D dS')^T, (dD S)^T   (Dk x 16 blocks: key rows, this wave's chunk columns)
//   dO D^T, dD V^T                  (this wave's chunk rows x C)
// and <dS', S> from diagonal blocks of S dS'^T.
// Phase B1: K K^T, Q K^T, dW K^T, dW Q^T (dW = -dD S) and (T^T dW)^T;
// B2: UT-solve backward with the saved M, dG, dQK, dQK + diag(lambda) dG, the
// beta and decay terms; B3: dX, dq, dk as transposes, stored from registers.
// The tail turns the decay terms into d log alpha.
//
// Wherever a result is needed in the other orientation the transposed
// product is computed instead, so that a lane holds four consecutive values
// of one row and writes them to LDS (or global memory) as one store.

// Phase-A tile of 32 value columns: S, dS' (32 value rows of Dk), D, V, dO
// (C rows of 32), each in the swizzled direct-load layout, and room for the
// tile's dD (C rows of 32), which the kernel forms itself.
template <typename E, int DK>
struct TileA {
  static constexpr int BV = 32;
  static constexpr int RE = BV * (int)sizeof(E);    // row bytes of the C-row tiles
  static constexpr int RK = DK * (int)sizeof(E);    // row bytes of the state tiles
  static constexpr int S = 0, DS = S + BV * RK, D = DS + BV * RK, V = D + C * RE, DO = V + C * RE,
                       DD = DO + C * RE, BYTES = DD + C * RE;
  static constexpr int LOADS = (BYTES - C * RE) / 1024 / NWAVES;   // direct loads per wave and tile
};

template <typename E, int DK>
struct alignas(16) IntraSmem {
  typedef TileA<E, DK> TA;
  static constexpr int RK = DK * (int)sizeof(E), RC = C * (int)sizeof(E);
  // phase-B placement inside the ring (swizzled tiles): K, Q in slot 0; dW,
  // (dT diag(beta))^T and Y in slot 1; dG over dW, dQK after it (or after K
  // and Q in slot 0), dQK + diag(lambda) dG over Y
  static constexpr int OK = 0, OQ = C * RK, OW = TA::BYTES, ODT = OW + C * RK, OY = ODT + C * RC, OG = OW;
  static constexpr int OQK = 2 * C * RC <= C * RK ? OW + C * RC : 2 * C * RK;
  static_assert(OY + C * RC <= 2 * TA::BYTES, "slot 1 holds dW, (dT diag(beta))^T and Y");
  static_assert(2 * C * RC <= C * RK || 2 * C * RK + C * RC <= TA::BYTES, "room for dQK");
  alignas(16) char ring[2][TA::BYTES];
  alignas(16) char Mm[C * RC];    // P (phase A), then M = (I + A)^{-1} (r, i), swizzled rows
  float b[C], g[C], beta[C], lam[C];
  float rdbeta[C], rer[C], rdb[C], rtk[C], rdl[C];   // row parts (each row owned by one wave)
  float colp[2][NWAVES][C];                          // column parts per wave: dT (.) M, decay terms
  float sdot[NWAVES];
};

constexpr int INTRA_THREADS = NTHREADS;

// Two workgroups per CU with bf16 operands; fp32 tiles take more than half
// of the LDS, so one, with the whole register file.
template <typename E>
constexpr int intra_per_cu() { return sizeof(E) == 2 ? 2 : 1; }

template <typename E, int DK, int DV>
__global__ __launch_bounds__(INTRA_THREADS) __attribute__((amdgpu_waves_per_eu(intra_per_cu<E>(), intra_per_cu<E>()))) void k_bwd_intra(Params p) {
  constexpr int KS = Mma<E>::KS;
  constexpr int NKB = DK / 16;        // 16-column blocks of Dk
  constexpr int NKK = DK / KS;        // k steps over Dk
  constexpr int NKC = C / KS;         // k steps over the chunk
  constexpr int BV = 32;
  constexpr int NVT = DV / BV;
  constexpr size_t ES = sizeof(E);
  typedef typename Mma<E>::frag FR;
  typedef typename Quad<E>::raw QR;
  typedef TileA<E, DK> TA;
  typedef IntraSmem<E, DK> SM;
  constexpr int RK = SM::RK, RC = SM::RC;
  static_assert(NVT >= 2, "at least two value tiles");
  __shared__ SM sm;
  if ((int)blockIdx.x < p.lead) {
    // leading workgroups hold their slot for about half a unit, so that the
    // workgroups run phase-shifted and the value-dimension loads of some
    // overlap the compute phases of others
    const long long t0c = clock64();
    while (clock64() - t0c < p.lead_cycles) __builtin_amdgcn_s_sleep(32);
    return;
  }
  // Workgroup -> (slot, head), slot-grouped: the H heads of eight slots
  // take H * 8 consecutive workgroups, slot g on XCD g mod 8 (workgroups go
  // to XCD blockIdx.x mod 8, and the sleepers number a multiple of 8).  A
  // token's gate gradients (dbeta, dlambda, dlog alpha: H x 4 bytes each)
  // share cache lines across the heads, so the heads of a slot write them
  // into one L2 at about the same time and the lines leave it whole; and
  // the heads of one token read adjacent rows of q, k, v and dO.  Slots past
  // the last multiple of 8 follow in plain order.
  const int bid = (int)blockIdx.x - p.lead;
  const int H8 = p.H * 8, ns8 = (p.n_slots / 8) * 8, tot8 = ns8 * p.H;
  int g, h;
  if (bid < tot8) {
    const int r = bid % H8;
    g = 8 * (bid / H8) + (r & 7);
    h = r >> 3;
  } else {
    const int idx = bid - tot8, nt = p.n_slots - ns8;
    g = ns8 + idx % nt;
    h = idx / nt;
  }
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id(tid);
  int n, t0, len;
  if (!locate(p, g, n, t0, len)) return;
  const int H = p.H;
  const size_t gi = (size_t)g * H + h;
  const size_t arow = (size_t)t0 * H + h;   // first activation row of the chunk
  const int rr = 16 * w + fcol(lane);       // chunk row of this lane's transposed results

  // ---------------- phase A: contractions over the value dimension
  f4 aQt[NKB], aKt[NKB], aWt[NKB], aP[4], aT[4], asd = zero4();
#pragma unroll
  for (int i = 0; i < NKB; ++i) aQt[i] = aKt[i] = aWt[i] = zero4();
#pragma unroll
  for (int i = 0; i < 4; ++i) aP[i] = aT[i] = zero4();
  const char* Sg = (const char*)((const E*)p.saved + gi * DK * DV);
  const char* dSg = (const char*)((const E*)p.w_dSo + gi * DK * DV);
  const char* Dg = (const char*)((const E*)p.savedD + gi * C * DV);   // 32-column tiles, C x 32 each
  const char* dOg = (const char*)((const E*)p.dO + arow * DV);
  const char* Vg = (const char*)((const E*)p.v + arow * DV);
  // the gate block (b, beta, lambda; waves 0-2 one vector each, straight
  // into LDS) and this wave's rows of K as B operands of Kbar dS'^T (k = key;
  // rows past the chunk re-read its last row: their dD rows are zeroed),
  // ahead of the first tile
  if (w < 3) dma4_asm(p.wb + gi * 3 * C + w * C + lane, (char*)(w == 0 ? sm.b : w == 1 ? sm.beta : sm.lam));
  FR kf[NKK];
  {
    const E* kr = (const E*)p.k + (arow + (size_t)min(rr, len - 1) * H) * DK + (lane >> 4) * Mma<E>::KPL;
#pragma unroll
    for (int ks = 0; ks < NKK; ++ks) kf[ks] = *(const FR*)(kr + ks * KS);
  }
  // rows of V and dO past the chunk come from D, whose rows there are zero
  static_assert(BV == 32, "one saved-D tile per value tile");
  auto issue = [&](int vt) {
    const int ln = lane;
    char* t = sm.ring[vt & 1];
    const size_t vb = (size_t)vt * BV;
    const char* Dt = Dg + vb * C * ES;   // this value tile's C x 32 block of D
    dma_rows<RK, BV, NWAVES, true>(t + TA::S, Sg + vb * RK, RK, BV, Sg, 0, w, ln);
    dma_rows<RK, BV, NWAVES, true>(t + TA::DS, dSg + vb * RK, RK, BV, dSg, 0, w, ln);
    dma_rows<TA::RE, C, NWAVES, true>(t + TA::D, Dt, TA::RE, C, Dt, 0, w, ln);
    dma_rows<TA::RE, C, NWAVES, true>(t + TA::V, Vg + vb * ES, (size_t)H * DV * ES, len, Dt, TA::RE, w, ln);
    dma_rows<TA::RE, C, NWAVES, true>(t + TA::DO, dOg + vb * ES, (size_t)H * DV * ES, len, Dt, TA::RE, w, ln);
  };
  // this wave's rows of the tile's dD, as their transpose (value rows, chunk
  // columns 16w..): dS' Kbar^T + dO^T P, P causal; rows past the chunk carry
  // no gradient
  float kbi = 0.f;                                // g_C / g of this lane's row
  auto form_dD = [&](char* t, int la) {
    const float keep = rr < len ? 1.f : 0.f;
#pragma unroll
    for (int nb = 0; nb < BV / 16; ++nb) {
      f4 dt = zero4();
#pragma unroll
      for (int ks = 0; ks < NKK; ++ks) dt = Mma<E>::mma(tile_frag<E, RK>(t + TA::DS, nb * 16, ks * KS, la), kf[ks], dt);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) dt[jj] *= kbi;
#pragma unroll
      for (int ks = 0; ks < NKC; ++ks)
        if (keep_kblock<E>(ks * KS + KS > 16 * w))
          dt = Mma<E>::mma(tile_tr_frag<E, TA::RE>(t + TA::DO, ks * KS, nb * 16, la),
                           tile_tr_frag<E, RC>(sm.Mm, ks * KS, 16 * w, la), dt);
      *(QR*)(t + TA::DD + tile_off<TA::RE>(rr, (nb * 16 + frow(la, 0)) * (int)ES)) = Quad<E>::pack(keep * dt);
    }
    // the wave reads back only its own rows: its LDS accesses complete in order
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  };
  // the tile's products: WITH_DD selects those that take dD (dD S, dD V^T),
  // WITHOUT_DD the others (dO S, D dS', dO D^T and <dS', S>)
  enum { WITHOUT_DD = 1, WITH_DD = 2 };
  auto products = [&](const char* t, int la, int which) {
#pragma unroll
    for (int ks = 0; ks < BV / KS; ++ks) {
      const FR aO = tile_frag<E, TA::RE>(t + TA::DO, 16 * w, ks * KS, la);
      const FR aD = tile_frag<E, TA::RE>(t + TA::D, 16 * w, ks * KS, la);
      FR adD = aD;
      if (which & WITH_DD) adD = tile_frag<E, TA::RE>(t + TA::DD, 16 * w, ks * KS, la);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const FR bS = tile_tr_frag<E, RK>(t + TA::S, ks * KS, kb * 16, la);
        if (which & WITHOUT_DD) {
          const FR bdS = tile_tr_frag<E, RK>(t + TA::DS, ks * KS, kb * 16, la);
          aQt[kb] = Mma<E>::mma(bS, aO, aQt[kb]);
          aKt[kb] = Mma<E>::mma(bdS, aD, aKt[kb]);
        }
        if (which & WITH_DD) aWt[kb] = Mma<E>::mma(bS, adD, aWt[kb]);
      }
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        if (which & WITHOUT_DD) aP[cb] = Mma<E>::mma(aO, tile_frag<E, TA::RE>(t + TA::D, cb * 16, ks * KS, la), aP[cb]);
        if (which & WITH_DD) aT[cb] = Mma<E>::mma(adD, tile_frag<E, TA::RE>(t + TA::V, cb * 16, ks * KS, la), aT[cb]);
      }
    }
    if (which & WITHOUT_DD) {
      // <dS', S> = trace(S dS'^T): wave w adds the diagonal 16 x 16 block
      // (w & 1) of this tile's S dS'^T over the key steps w >> 1, +2, ...
#pragma unroll
      for (int ks = 0; ks < NKK; ks += 2)
        if (ks + (w >> 1) < NKK)
          asd = Mma<E>::mma(tile_frag<E, RK>(t + TA::S, 16 * (w & 1), (ks + (w >> 1)) * KS, la),
                            tile_frag<E, RK>(t + TA::DS, 16 * (w & 1), (ks + (w >> 1)) * KS, la), asd);
    }
  };

  // First tile, P (into the M buffer) and the second tile; every later tile
  // once the one before it has landed; with the last tile the chunk's Q rows
  // into the free slot 0 (for phase B; rows past the chunk re-read its last
  // row and are zeroed afterwards) beside the K rows the waves write from
  // their registers, and once the last tile's dD is formed, M over P.
  constexpr int ML = C * RC / 1024 / NWAVES;
  // P and M arrive packed: the chunks above their diagonal blocks are zeroed
  // once here and never loaded (ordered before any read by the barrier after
  // the first tile)
  zero_upper_chunks<E>(sm.Mm, tid, INTRA_THREADS);
  issue(0);
  {
    dma_lbt<E, NWAVES>(sm.Mm, (const char*)((const E*)p.wP + gi * LBT_ELEMS), w, lane);
  }
  issue(1);
  static_assert(NVT % 2 == 0, "the last tile uses slot 1");
  wait_vm<TA::LOADS>();                           // all but tile 1 landed
  block_sync_lds();
  kbi = __expf(sm.b[C - 1] - sm.b[rr]);
  {
    // The first tile runs the products without dD first.  The K rows are the
    // compiler's own loads, and at their first use (forming dD) it waits with
    // a count of its own loads only, so for the second tile as well, which
    // has had that time to land.
    char* t = sm.ring[0];
    int la = lane;
    asm volatile("" : "+v"(la));
    products(t, la, WITHOUT_DD);
    form_dD(t, la);
    products(t, la, WITH_DD);
  }
#pragma unroll 1
  for (int vt = 1; vt < NVT; ++vt) {
    wait_vm<0>();                                 // tile vt (issued during tile vt-1)
    block_sync_lds();                             // tile vt visible; tile vt-1's slot is free
    if (vt + 1 < NVT) issue(vt + 1);
    if (vt == NVT - 1) {
      // phase B's K rows come from the waves' registers (rows past the
      // chunk written as zero), its Q rows from memory
      const char* Qg = (const char*)((const E*)p.q + arow * DK);
      dma_rows<RK, C, NWAVES, true>(sm.ring[0] + SM::OQ, Qg, (size_t)H * RK, len, Qg + (size_t)(len - 1) * H * RK, 0, w, lane);
      const float kz = rr < len ? 1.f : 0.f;
#pragma unroll
      for (int ks = 0; ks < NKK; ++ks) {
        const int kbyte = (ks * KS + (lane >> 4) * Mma<E>::KPL) * (int)ES;
        if constexpr (sizeof(E) == 2) {
          const uint4 z = make_uint4(0, 0, 0, 0);
          *(uint4*)(sm.ring[0] + SM::OK + tile_off<RK>(rr, kbyte)) = kz != 0.f ? __builtin_bit_cast(uint4, kf[ks]) : z;
        } else {
          *(float*)(sm.ring[0] + SM::OK + tile_off<RK>(rr, kbyte)) = kz * kf[ks];
        }
      }
    }
    char* t = sm.ring[vt & 1];
    int la = lane;                        // laundered: addresses formed per tile
    asm volatile("" : "+v"(la));
    form_dD(t, la);
    if (vt == NVT - 1) {
      // every wave is past its last read of P: M goes over it
      block_sync_lds();
      dma_lbt<E, NWAVES>(sm.Mm, (const char*)((const E*)p.wM + gi * LBT_ELEMS), w, lane);
    }
    products(t, la, WITHOUT_DD | WITH_DD);
  }
  {
    // diagonal elements of the accumulated block: row 4 (l >> 4) + j == column l & 15
    const int j = (lane & 15) - 4 * (lane >> 4);
    float sdot = 0.f;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      if (jj == j) sdot = asd[jj];
    int ls = lane;
    asm volatile("" : "+v"(ls));
    sdot = wave_sum_l(sdot, ls);
    if (lane == 0) sm.sdot[w] = sdot;
  }
  if (w == 0) sm.g[lane] = __expf(sm.b[lane]);   // (beta, lambda: zero past the chunk in the gate block)

  // ---------------- phase B1
  // The lane index is laundered at each phase so that per-lane LDS addresses
  // are formed where they are used rather than hoisted into long-lived
  // registers (the compiler would spill them).
  char* const ring = &sm.ring[0][0];
  int lb = lane;
  asm volatile("" : "+v"(lb));
  wait_vm<ML>();                           // this wave's Q rows landed (M may be in flight)
  if (len < C) {
    // rows of Q past the chunk are zero; each wave clears the rows its own
    // loads filled (rows of instruction i belong to wave i mod NWAVES)
    constexpr int PR = RK / 16, RPI = 1024 / RK;
    for (int idx = lane; idx < (C - len) * PR; idx += 64) {
      const int r = len + idx / PR, c = (idx % PR) * 16;
      if ((r / RPI) % NWAVES == w) *(uint4*)(ring + SM::OQ + tile_off<RK>(r, c)) = make_uint4(0, 0, 0, 0);
    }
  }
  block_sync_lds();                        // phase-A tiles consumed; gates, K, Q visible; slot 1 free
  // dW = -dD S rows of this wave from (dD S)^T: four consecutive keys per lane
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
    *(QR*)(ring + SM::OW + tile_off<RK>(rr, (kb * 16 + frow(lb, 0)) * (int)ES)) = Quad<E>::pack(-aWt[kb]);
  block_sync_lds();
  const int r0 = 16 * w + frow(lb, 0);
  float lamr[4], betr[4], br4[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    lamr[j] = sm.lam[r0 + j];
    betr[j] = sm.beta[r0 + j];
    br4[j] = sm.b[r0 + j];
  }
  f4 aG[4], aQK[4], dT[4];
  {
    // dT = dD V^T + dW (diag(g) X)^T, the second part as
    // (dW K^T + dW Q^T diag(lambda)) diag(g)
    f4 aDK[4], aDQ[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) aDK[cb] = aDQ[cb] = zero4();
#pragma unroll
    for (int ks = 0; ks < NKK; ++ks) {
      const FR dwA = tile_frag<E, RK>(ring + SM::OW, 16 * w, ks * KS, lb);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        aDK[cb] = Mma<E>::mma(dwA, tile_frag<E, RK>(ring + SM::OK, cb * 16, ks * KS, lb), aDK[cb]);
        aDQ[cb] = Mma<E>::mma(dwA, tile_frag<E, RK>(ring + SM::OQ, cb * 16, ks * KS, lb), aDQ[cb]);
      }
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int c = cb * 16 + fcol(lb);
      const float gc = sm.g[c], lc = sm.lam[c];
#pragma unroll
      for (int j = 0; j < 4; ++j) dT[cb][j] = aT[cb][j] + gc * (aDK[cb][j] + lc * aDQ[cb][j]);
    }
  }
  {
    // G = X K^T = K K^T + diag(lambda) Q K^T (rows 16w.., all columns)
    f4 aKK[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) aKK[cb] = aQK[cb] = zero4();
#pragma unroll
    for (int ks = 0; ks < NKK; ++ks) {
      const FR kA = tile_frag<E, RK>(ring + SM::OK, 16 * w, ks * KS, lb);
      const FR qA = tile_frag<E, RK>(ring + SM::OQ, 16 * w, ks * KS, lb);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const FR kB = tile_frag<E, RK>(ring + SM::OK, cb * 16, ks * KS, lb);
        aKK[cb] = Mma<E>::mma(kA, kB, aKK[cb]);
        aQK[cb] = Mma<E>::mma(qA, kB, aQK[cb]);
      }
    }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int j = 0; j < 4; ++j) aG[cb][j] = aKK[cb][j] + lamr[j] * aQK[cb][j];
  }
  // (T^T dW)^T = (diag(beta) M^T dW)^T: key rows, this wave's chunk columns;
  // M is lower triangular, so k blocks before this wave's rows are skipped
  wait_vm<0>();
  block_sync_lds();                        // M visible
  f4 tdwt[NKB];
  {
    const float betc = sm.beta[rr];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      f4 x = zero4();
#pragma unroll
      for (int ks = 0; ks < NKC; ++ks)
        if (keep_kblock<E>(ks * KS + KS > 16 * w))
          x = Mma<E>::mma(tile_tr_frag<E, RK>(ring + SM::OW, ks * KS, kb * 16, lb),
                          tile_tr_frag<E, RC>(sm.Mm, ks * KS, 16 * w, lb), x);
#pragma unroll
      for (int j = 0; j < 4; ++j) tdwt[kb][j] = betc * x[j];
    }
  }

  // ---------------- phase B2: UT-solve backward and the C x C gradient terms
  asm volatile("" : "+v"(lb));
  // dT = dD V^T + dW (g X)^T; the column sums of dT (.) M feed dbeta;
  // (dT diag(beta))^T is the operand of Y = M^T dT diag(beta)
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    const int c = cb * 16 + fcol(lb);
    const float bc = sm.beta[c];
    f4 dm;
    float cs = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      cs += dT[cb][j] * tof(*(const E*)(sm.Mm + tile_off<RC>(r0 + j, c * (int)ES)));
      dm[j] = dT[cb][j] * bc;
    }
    *(QR*)(ring + SM::ODT + tile_off<RC>(c, r0 * (int)ES)) = Quad<E>::pack(dm);
    cs += lane_xor(cs, 16, lb);
    cs += lane_xor(cs, 32, lb);
    if (lane < 16) sm.colp[0][w][c] = cs;
  }
  block_sync_lds();                        // (dT diag(beta))^T complete; dW no longer read
  f4 adA[4];
  {
    // Y^T = (dT diag(beta))^T M (chunk columns, this wave's rows), stored as Y rows
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      f4 y = zero4();
#pragma unroll
      for (int ks = 0; ks < NKC; ++ks)
        if (keep_kblock<E>(ks * KS + KS > 16 * w))
          y = Mma<E>::mma(tile_frag<E, RC>(ring + SM::ODT, cb * 16, ks * KS, lb),
                          tile_tr_frag<E, RC>(sm.Mm, ks * KS, 16 * w, lb), y);
      *(QR*)(ring + SM::OY + tile_off<RC>(rr, (cb * 16 + frow(lb, 0)) * (int)ES)) = Quad<E>::pack(y);
    }
    // dA = strictLower(-Y M^T) (this wave's rows; M lower triangular)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      adA[cb] = zero4();
#pragma unroll
      for (int ks = 0; ks < NKC; ++ks)
        if (keep_kblock<E>(ks * KS <= cb * 16 + 15))
          adA[cb] = Mma<E>::mma(tile_frag<E, RC>(ring + SM::OY, 16 * w, ks * KS, lb),
                                tile_frag<E, RC>(sm.Mm, cb * 16, ks * KS, lb), adA[cb]);
    }
  }
  {
    // dG = diag(beta) dA (.) Gamma, dQK = dP (.) Gamma (causal, inclusive),
    // dQK + diag(lambda) dG (over Y: own rows), the decay-gradient terms
    // t = dG (.) G + dQK (.) QK and the row parts of dbeta from
    // A = strictLower(diag(beta) Gamma (.) G)
    float dbr[4] = {0.f, 0.f, 0.f, 0.f}, er[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int c = cb * 16 + fcol(lb);
      const float bc = sm.b[c];
      float ec = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + j;
        const float gam = (r >= c) ? __expf(br4[j] - bc) : 0.f;
        const float dA = (r > c) ? -adA[cb][j] : 0.f;
        const float dAg = dA * gam;
        const float dg = dAg * betr[j];
        const float dqk = aP[cb][j] * gam;
        const float t = dg * aG[cb][j] + dqk * aQK[cb][j];
        dbr[j] += dAg * aG[cb][j];
        er[j] += t;
        ec += t;
        *(E*)(ring + SM::OG + tile_off<RC>(r, c * (int)ES)) = fromf<E>(dg);
        *(E*)(ring + SM::OQK + tile_off<RC>(r, c * (int)ES)) = fromf<E>(dqk);
        *(E*)(ring + SM::OY + tile_off<RC>(r, c * (int)ES)) = fromf<E>(dqk + lamr[j] * dg);
      }
      ec += lane_xor(ec, 16, lb);
      ec += lane_xor(ec, 32, lb);
      if (lane < 16) sm.colp[1][w][c] = ec;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dbr[j] = sum16(dbr[j]);
      er[j] = sum16(er[j]);
    }
    if (fcol(lb) == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sm.rdbeta[r0 + j] = dbr[j];
        sm.rer[r0 + j] = er[j];
      }
    }
  }
  block_sync_lds();                        // dG, dQK, dQK + diag(lambda) dG complete

  asm volatile("" : "+v"(lb));
  // ---------------- phase B3: dX, dq, dk as transposes (key rows, this
  // wave's chunk columns); the K^T, Q^T operands are transpose reads of the
  // row-major K, Q tiles
  {
    FR gB[NKC], qkB[NKC], gtB[NKC], gltB[NKC];
#pragma unroll
    for (int ks = 0; ks < NKC; ++ks) {
      gB[ks] = tile_frag<E, RC>(ring + SM::OG, 16 * w, ks * KS, lb);       // dG rows, as (r, c)
      qkB[ks] = tile_frag<E, RC>(ring + SM::OQK, 16 * w, ks * KS, lb);     // dQK rows
      gtB[ks] = tile_tr_frag<E, RC>(ring + SM::OG, ks * KS, 16 * w, lb);   // dG columns, as (r, c) of dG^T
      gltB[ks] = tile_tr_frag<E, RC>(ring + SM::OY, ks * KS, 16 * w, lb);  // (dQK + diag(lambda) dG) columns
    }
    const float gr = sm.g[rr], lr = sm.lam[rr], kbr = __expf(sm.b[C - 1] - sm.b[rr]);
    float s1 = 0.f, s2 = 0.f, s3 = 0.f;
    E* dqo = (E*)p.dq + (arow + (size_t)rr * H) * DK;
    E* dko = (E*)p.dk + (arow + (size_t)rr * H) * DK;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      f4 dxp = zero4(), dqp = zero4(), dkp = zero4();
#pragma unroll
      for (int ks = 0; ks < NKC; ++ks) {
        const FR kT = tile_tr_frag<E, RK>(ring + SM::OK, ks * KS, kb * 16, lb);
        const FR qT = tile_tr_frag<E, RK>(ring + SM::OQ, ks * KS, kb * 16, lb);
        dxp = Mma<E>::mma(kT, gB[ks], dxp);        // (dG K)^T
        dqp = Mma<E>::mma(kT, qkB[ks], dqp);       // (dQK K)^T
        dkp = Mma<E>::mma(kT, gtB[ks], dkp);       // (dG^T K)^T
        dkp = Mma<E>::mma(qT, gltB[ks], dkp);      // ((dQK + diag(lambda) dG)^T Q)^T
      }
      const int kc = kb * 16 + frow(lb, 0);
      const QR kq = *(const QR*)(ring + SM::OK + tile_off<RK>(rr, kc * (int)ES));
      const QR qq = *(const QR*)(ring + SM::OQ + tile_off<RK>(rr, kc * (int)ES));
      f4 oq, ok;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float Kv = Quad<E>::get(kq, j), Qv = Quad<E>::get(qq, j);
        const float X = Kv + lr * Qv, tdw = tdwt[kb][j], aq = aQt[kb][j], ak = aKt[kb][j];
        s1 += X * tdw + Qv * aq;
        s2 += Kv * ak;
        const float dX = gr * tdw + dxp[j];
        s3 += Qv * dX;
        oq[j] = gr * aq + dqp[j] + lr * dX;
        ok[j] = kbr * ak + dkp[j] + dX;
      }
      if (rr < len) {
        *(QR*)(dqo + kc) = Quad<E>::pack(oq);
        *(QR*)(dko + kc) = Quad<E>::pack(ok);
      }
    }
    s1 += lane_xor(s1, 16, lb);
    s1 += lane_xor(s1, 32, lb);
    s2 += lane_xor(s2, 16, lb);
    s2 += lane_xor(s2, 32, lb);
    s3 += lane_xor(s3, 16, lb);
    s3 += lane_xor(s3, 32, lb);
    if (lane < 16) {
      sm.rdb[rr] = gr * s1;
      sm.rtk[rr] = kbr * s2;
      sm.rdl[rr] = s3;
    }
  }
  block_sync_lds();
  if (w == 0) {
    // dbeta = row parts + column sums of dT (.) M; db = decay row parts -
    // column parts + the B3 terms; Kbar terms: db_r -= t_r,
    // db_{C-1} += sum_r t_r + g_C <dS', S>; then dlog alpha_j = sum_{r >= j} db_r
    // (chunk-local reverse cumulative sum)
    const int j = lane;
    float cb_ = 0.f, ce = 0.f;
#pragma unroll
    for (int q = 0; q < NWAVES; ++q) {
      cb_ += sm.colp[0][q][j];
      ce += sm.colp[1][q][j];
    }
    const float tk = sm.rtk[j];
    float tot = tk;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) tot += lane_xor(tot, off, lb);
    float dbj = sm.rer[j] - ce + sm.rdb[j] - tk;
    if (j == C - 1) {
      float sd = 0.f;
#pragma unroll
      for (int q = 0; q < NWAVES; ++q) sd += sm.sdot[q];
      dbj += tot + sm.g[C - 1] * sd;
    }
    float x = lane_from(dbj, C - 1 - j);
    x = wave_incl_scan_dpp(x);
    const float suffix = lane_from(x, C - 1 - j);
    if (j < len) {
      const size_t gt = arow + (size_t)j * H;
      p.dbeta[gt] = sm.rdbeta[j] + cb_;
      if (p.dlam) p.dlam[gt] = sm.rdl[j];
      if (p.dla) p.dla[gt] = suffix;
    }
    if (p.w_dlam) {
      // constant lambda: this unit's share of its gradient
      const float part = wave_sum_l(j < len ? sm.rdl[j] : 0.f, lb);
      if (j == 0) p.w_dlam[gi] = part;
    }
  }
}

// Gradient of a constant lambda: the sum of the per-unit partials of every
// unit a chunk maps to, in a fixed order (one workgroup: strided per-thread
// sums, then a tree), so the result is the same on every run.
__global__ __launch_bounds__(NTHREADS) void k_sum_units(Params p) {
  __shared__ float part[NTHREADS];
  const int tid = threadIdx.x;
  const int total = p.n_slots * p.H;
  float acc = 0.f;
  for (int u = tid; u < total; u += NTHREADS) {
    int n, t0, len;
    if (locate(p, u / p.H, n, t0, len)) acc += p.w_dlam[u];
  }
  part[tid] = acc;
  __syncthreads();
#pragma unroll
  for (int off = NTHREADS / 2; off >= 1; off >>= 1) {
    if (tid < off) part[tid] += part[tid + off];
    __syncthreads();
  }
  if (tid == 0) *p.dlam_sum = part[0];
}

__global__ void k_zero1(float* x) {
  if (threadIdx.x == 0) *x = 0.f;
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_bwd_t(const Params& p, hipStream_t st) {
  const int units = p.N * p.H;
  const int bv = scan_bv<E, DV>(units);
  const int nb = ((units + 7) / 8) * 8 * (DV / bv);
  if (nb > 0) {
    prof_mark(ST_SCAN_BWD, 0, st);
    constexpr int NCW = sizeof(E) == 2 ? 8 : 4;   // compute waves: two per SIMD for bf16
    if constexpr (scan_bv_max<E, DV>() == 64) {
      if (bv == 64)
        hipLaunchKernelGGL((k_scan_bwd<E, DK, DV, 64, NCW>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
      else
        hipLaunchKernelGGL((k_scan_bwd<E, DK, DV, 32, NCW>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
    } else {
      hipLaunchKernelGGL((k_scan_bwd<E, DK, DV, 32, NCW>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
    }
    prof_mark(ST_SCAN_BWD, 1, st);
  }
  if (p.n_slots > 0) {
    // Every unit costs the same, so without an offset all CUs would load
    // their value-dimension tiles together and then compute together, leaving
    // HBM idle half the time.  Half of the CUs start about half a unit later.
    Params q = p;
    const int total = p.n_slots * p.H, cus = device_cu_count();
    q.lead = total >= 8 * cus ? cus / 8 * 8 : 0;   // two workgroups per CU: half of the slots (a multiple of 8)
    q.lead_cycles = 20000;
    prof_mark(ST_INTRA, 0, st);
    hipLaunchKernelGGL((k_bwd_intra<E, DK, DV>), dim3(total + q.lead), dim3(INTRA_THREADS), 0, st, q);
    prof_mark(ST_INTRA, 1, st);
  }
  if (p.dlam_sum) {
    if (p.n_slots > 0) hipLaunchKernelGGL(k_sum_units, dim3(1), dim3(NTHREADS), 0, st, p);
    else hipLaunchKernelGGL(k_zero1, dim3(1), dim3(64), 0, st, p.dlam_sum);
  }
  return hipGetLastError();
}

hipError_t launch_zero(float* x, hipStream_t st) {
  hipLaunchKernelGGL(k_zero1, dim3(1), dim3(64), 0, st, x);
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
