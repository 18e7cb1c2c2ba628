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
// k_prep   (persistent over chunk-head units, fully parallel): b, the Gram
//          products, A, the UT solve, U and W; writes b, U, W, P and M.
// k_scan_fwd (one workgroup per sequence, head and Dv tile): the sequential
//          pass over chunks; the state tile stays in MFMA accumulators in fp32;
//          D, the chunk output and the state update are computed on chip.
#include "qd_common.h"
#include "qd_launch.h"

#include <type_traits>

namespace qd {

template <typename E, int DK, int DV>
struct alignas(16) PrepSmem {
  static constexpr int P = Pad<E>::v;
  alignas(16) float b[C], g[C], gl[C], beta[C], lam[C];   // gl = g lambda
  union {
    struct {
      E K[C][DK + P];
      E Q[C][DK + P];
    } a;
    E V[C][DV + P];           // after W, the last reader of K and Q
  } u;
  E Ws[C][DK + P];            // W staging for 16-byte stores
  union {
    float A[C][C + 4];        // strictly lower A, consumed by the solve
    struct {
      E Tg[C][C + P];         // T diag(g)
      E Tgl[C][C + P];        // T diag(g lambda)
    } t;                      // after the solve
  } am;
  alignas(16) float M[C][C + 4];
  E Tm[C][C + P];             // P staging during the Gram products, then T
};

// Raw inputs of one (chunk, head) unit, staged in registers one unit ahead.
constexpr int PREP_THREADS = 512;   // 8 waves: two per SIMD hide each other's latency

template <typename E, int DK, int DV>
struct PrepPre {
  TileRegs<E, C, DK, PREP_THREADS> K, Q;
  TileRegs<E, C, DV, PREP_THREADS> V;
  float la, beta, lam;
  int t0, len, g, h;
  bool valid;
};

// Copies a C x D LDS tile (row stride ld elements) to a dense row-major
// global block with 16-byte stores.
template <typename E, int D, int NT>
__device__ inline void store_tile(E* dst, const E* src, int ld, int tid) {
  constexpr int VEC = 16 / sizeof(E), PR = D / VEC;
  for (int idx = tid; idx < C * PR; idx += NT) {
    const int r = idx / PR, c = (idx % PR) * VEC;
    *(uint4*)(dst + (size_t)r * D + c) = *(const uint4*)(src + (size_t)r * ld + c);
  }
}

// Writes b, U, W, P and, when p.wM is set, M = (I + A)^{-1} for every unit.
// Persistent: each workgroup walks units blockIdx.x, +gridDim.x, ... and
// prefetches the next unit's inputs into registers while computing the
// current one.
template <typename E, int DK, int DV>
__global__ __launch_bounds__(PREP_THREADS) void k_prep(Params p) {
  constexpr int NT = PREP_THREADS, NW = NT / 64;
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P;
  constexpr int KS = Mma<E>::KS;
  typedef PrepPre<E, DK, DV> Pre;
  __shared__ PrepSmem<E, DK, DV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int H = p.H;
  const int total = p.n_slots * H;

  auto fetch = [&](int u, Pre& x) {
    x.valid = false;
    if (u >= total) return;
    x.g = u / H;
    x.h = u % H;
    int n;
    if (!locate(p, x.g, n, x.t0, x.len)) return;
    x.valid = true;
    const size_t row = (size_t)x.t0 * H + x.h;
    x.K.load((const E*)p.k + row * DK, (size_t)H * DK, x.len, tid);
    x.Q.load((const E*)p.q + row * DK, (size_t)H * DK, x.len, tid);
    x.V.load((const E*)p.v + row * DV, (size_t)H * DV, x.len, tid);
    if (tid < C) {
      const bool ok = tid < x.len;
      const size_t gt = row + (size_t)tid * H;
      x.la = (ok && p.la) ? p.la[gt] : 0.f;
      x.beta = ok ? p.beta[gt] : 0.f;
      x.lam = ok ? p.lam[gt] : 0.f;
    }
  };

  Pre pre;
  fetch(blockIdx.x, pre);
  for (int u = blockIdx.x; u < total; u += gridDim.x) {
    const Pre x = pre;
    fetch(u + gridDim.x, pre);
    if (!x.valid) continue;                 // uniform across the workgroup
    const int h = x.h;
    const size_t gi = (size_t)x.g * H + h;
    block_sync_lds();                        // previous unit's LDS use is over
    x.K.store(&sm.u.a.K[0][0], LK, tid);
    x.Q.store(&sm.u.a.Q[0][0], LK, tid);
    if (tid < C) {
      const float b = wave_incl_scan(x.la, lane), g = __expf(b);
      sm.b[tid] = b;
      sm.g[tid] = g;
      sm.gl[tid] = g * x.lam;
      sm.beta[tid] = x.beta;
      sm.lam[tid] = x.lam;
      p.wb[gi * C + tid] = b;
    }
    block_sync_lds();

    // Gram products K K^T and Q K^T, with X K^T = K K^T + diag(lambda) Q K^T;
    // A (fp32) and P (staged in Tm)
#pragma unroll
    for (int tk = 0; tk < 16 / NW; ++tk) {
      const int t = w + tk * NW;
      const int m0 = (t >> 2) * 16, n0 = (t & 3) * 16, i = n0 + fcol(lane);
      const float bi = sm.b[i];
      float br[4], betr[4], lr[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = m0 + frow(lane, j);
        br[j] = sm.b[r];
        betr[j] = sm.beta[r];
        lr[j] = sm.lam[r];
      }
      const f4 kk = mma_k<E, DK>(kmaj(&sm.u.a.K[0][0], LK), kmaj(&sm.u.a.K[0][0], LK), m0, n0, zero4(), lane);
      const f4 qk = mma_k<E, DK>(kmaj(&sm.u.a.Q[0][0], LK), kmaj(&sm.u.a.K[0][0], LK), m0, n0, zero4(), lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = m0 + frow(lane, j);
        const float gam = (r >= i) ? __expf(br[j] - bi) : 0.f;
        sm.am.A[r][i] = (r > i) ? betr[j] * gam * (kk[j] + lr[j] * qk[j]) : 0.f;
        sm.Tm[r][i] = fromf<E>(gam * qk[j]);
      }
    }
    block_sync_lds();
    // P out before the solve (whose barriers order the later T writes to Tm)
    store_tile<E, C, NT>((E*)p.wP + gi * C * C, &sm.Tm[0][0], LC, tid);

    // UT solve: M = (I + A)^{-1}, T = M diag(beta)
    unit_lower_inverse<NT>(&sm.am.A[0][0], C + 4, &sm.M[0][0], C + 4, tid);
    {
      // T, T diag(g) and T diag(g lambda) into LDS (A is dead: the solve ends
      // with a barrier) and M to global; a thread takes VEC consecutive
      // columns of one row
      constexpr int VEC = 16 / sizeof(E);
      E* wM = (E*)p.wM;
      for (int idx = tid; idx < C * C / VEC; idx += NT) {
        const int r = idx / (C / VEC), i0 = (idx % (C / VEC)) * VEC;
        const bool upper = (i0 >> 4) > (r >> 4);   // strictly-upper block: zero
        uint4 tr, tgr, tglr, mr;
        E* te = (E*)&tr;
        E* tge = (E*)&tgr;
        E* tgle = (E*)&tglr;
        E* me = (E*)&mr;
        float mv[VEC], bv[VEC], gv[VEC], glv[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j += 4) {
          *(f4*)&mv[j] = *(const f4*)&sm.M[r][i0 + j];
          *(f4*)&bv[j] = *(const f4*)&sm.beta[i0 + j];
          *(f4*)&gv[j] = *(const f4*)&sm.g[i0 + j];
          *(f4*)&glv[j] = *(const f4*)&sm.gl[i0 + j];
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const float m = upper ? 0.f : mv[j];
          const float tv = m * bv[j];
          te[j] = fromf<E>(tv);
          tge[j] = fromf<E>(tv * gv[j]);
          tgle[j] = fromf<E>(tv * glv[j]);
          me[j] = fromf<E>(m);
        }
        *(uint4*)&sm.Tm[r][i0] = tr;
        *(uint4*)&sm.am.t.Tg[r][i0] = tgr;
        *(uint4*)&sm.am.t.Tgl[r][i0] = tglr;
        if (wM) *(uint4*)(wM + gi * C * C + r * C + i0) = mr;
      }
    }
    block_sync_lds();

    // W = T diag(g) X = T diag(g) K + T diag(g lambda) Q (B operands: transpose
    // reads of K and Q), staged row-major for 16-byte stores
#pragma unroll
    for (int tk = 0; tk < (C / 16) * (DK / 16) / NW; ++tk) {
      const int t = w + tk * NW;
      const int m0 = (t / (DK / 16)) * 16, n0 = (t % (DK / 16)) * 16;
      f4 wv = zero4();
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) {
        wv = Mma<E>::mma(Frag<E>::load(kmaj(&sm.am.t.Tg[0][0], LC), m0, ks * KS, lane),
                         tr_frag<E>(&sm.u.a.K[0][0], LK, ks * KS, n0, lane), wv);
        wv = Mma<E>::mma(Frag<E>::load(kmaj(&sm.am.t.Tgl[0][0], LC), m0, ks * KS, lane),
                         tr_frag<E>(&sm.u.a.Q[0][0], LK, ks * KS, n0, lane), wv);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) sm.Ws[m0 + frow(lane, j)][n0 + fcol(lane)] = fromf<E>(wv[j]);
    }
    block_sync_lds();
    store_tile<E, DK, NT>((E*)p.wW + gi * C * DK, &sm.Ws[0][0], LK, tid);
    // V (K and Q are dead: W, their last reader, ended at the barrier above)
    x.V.store(&sm.u.V[0][0], DV + P, tid);
    block_sync_lds();

    // U = T V (the B operand is a transpose read of V), stored C-fragment
    // tiled: tile (mt, nt) at ((mt*(DV/16)+nt)*64 + lane)*4
    E* wU = (E*)p.wU + gi * C * DV;
#pragma unroll
    for (int tk = 0; tk < (C / 16) * (DV / 16) / NW; ++tk) {
      const int t = w + tk * NW;
      const int m0 = (t / (DV / 16)) * 16, n0 = (t % (DV / 16)) * 16;
      f4 uu = zero4();
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks)
        uu = Mma<E>::mma(Frag<E>::load(kmaj(&sm.Tm[0][0], LC), m0, ks * KS, lane),
                         tr_frag<E>(&sm.u.V[0][0], DV + P, ks * KS, n0, lane), uu);
      *(typename Quad<E>::raw*)(wU + ((size_t)t * 64 + lane) * 4) = Quad<E>::pack(uu);
    }
  }
}

// Forward-scan operands of one chunk, filled by direct global->LDS loads as
// swizzled row-major tiles, in two sets by the phase that reads them:
//   set A (D = U - W S^T):            W (C x Dk), this tile's U fragments (byte
//                                     copy of the C-fragment-ordered layout), b;
//   set B (output and state update):  Q, K (C x Dk), P (C x C), b.
// Each set has its own ring of NBUF chunks and its own producer wave.
template <typename E, int DK, int BV>
struct ScanFwdRing {
  static constexpr int RK = DK * (int)sizeof(E), RC = C * (int)sizeof(E);   // row bytes
  static constexpr int NB = BV / 16;
  static constexpr int UM = NB * 64 * 4 * (int)sizeof(E);   // U bytes per 16-row block
  static constexpr int AW = 0, AU = AW + C * RK, AB = AU + 4 * UM, ABYTES = AB + C * 4;
  static constexpr int BQ = 0, BK = BQ + C * RK, BP = BK + C * RK, BB = BP + C * RC, BBYTES = BB + C * 4;
  static constexpr int NBUF = sizeof(E) == 2 ? 2 : 1;      // fp32 tiles are twice as large
  // direct loads per chunk of each of the two producers of a set (the 1 KB
  // instructions of every tile split evenly; producer 1 also loads b)
  static constexpr int IA = (AB - AW) / 1024, IB = (BB - BQ) / 1024;
  static constexpr int LOADS_A0 = IA / 2, LOADS_A1 = IA / 2 + 1, LOADS_B0 = IB / 2, LOADS_B1 = IB / 2 + 1;
  static_assert((C * RK / 1024) % 2 == 0 && (4 * UM / 1024) % 2 == 0 && (C * RC / 1024) % 2 == 0, "even split");
  static_assert(NBUF == 1 || (LOADS_A1 <= 63 && LOADS_B1 <= 63), "outstanding-load counter range");
};

template <typename E, int DK, int BV>
struct alignas(16) ScanFwdSmem {
  static constexpr int P = Pad<E>::v;
  typedef ScanFwdRing<E, DK, BV> R;
  alignas(16) char ringA[R::NBUF][R::ABYTES];
  alignas(16) char ringB[R::NBUF][R::BBYTES];
  E Dt[BV][C + P];    // D^T
  E Dkt[BV][C + P];   // (diag(g_C / g) D)^T
  union {
    struct {
      E S[BV][DK + P];        // state tile (MFMA operand copy)
      E Sf[DK][BV + P];       // entry-state tile staging for the saved context ([k][v])
    } s;
    E O[C][BV + P];           // output tile staging (after the state copies are dead)
  } u;
};

// One workgroup per (sequence, head, Dv tile of BV = 32 value rows): four
// compute waves and four producer waves (two per operand set; one wave alone
// issues direct loads at only about 12 bytes per clock).  Compute wave w owns rows 16w.. of
// the chunk's D and O tiles and key rows 16 KPW w.. of the state tile S^T
// (Dk x BV), which lives in fp32 MFMA accumulators across the whole sequence.
//
// Per chunk the compute waves pass four barriers: B1 (start), B2 (S staged),
// B3 (D staged), B4 (outputs staged).  Producers 0-1 stream set A, 2-3 set
// B; each issues a chunk's loads while the compute waves work on phases
// that no longer read the buffer being refilled, so that issuing (which
// stalls the issuing wave while the memory pipeline is busy) overlaps compute
// instead of delaying a barrier:
//   set A of chunk c+2 is issued after B3 of chunk c (its last reader, phase
//   2, is over) and waited for before B2 of chunk c+2;
//   set B of chunk c+1 is issued in two parts between B1, B2 and B3 of chunk
//   c (its buffer was released at B4 of chunk c-1) and waited for before B3
//   of chunk c+1.
// The producers issue no other memory operations, so their outstanding-load
// counts are exact.  With one buffer per set (fp32) the refills follow the
// last reader's barrier.  When p.o is null only the states are produced.
template <typename E, int DK, int DV, int BV>
__global__ __launch_bounds__(NTHREADS + 256) void k_scan_fwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LC = C + P;
  constexpr int NVT = DV / BV;
  constexpr int NB = BV / 16;                 // 16-column blocks per tile
  constexpr int KS = Mma<E>::KS;
  static_assert(DK / 16 == 2 * NWAVES || DK / 16 == NWAVES, "key blocks per wave");
  constexpr int KPW = DK / 16 / NWAVES;       // key row blocks of S^T per wave (1 or 2)
  typedef typename Quad<E>::raw QR;
  typedef typename Mma<E>::frag FR;
  typedef ScanFwdRing<E, DK, BV> R;
  constexpr bool DB = R::NBUF == 2;
  __shared__ ScanFwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int prod = w - NWAVES;                // 0-3 for the producer waves, negative otherwise
  const bool producer = prod >= 0;
  const bool prodA = prod == 0 || prod == 1, prodB = prod >= 2;
  const int wp = prod & 1;                    // producer index within its set
  int unit, vt;
  if (!xcd_unit_tile(blockIdx.x, p.N * p.H, NVT, unit, vt)) return;
  const int H = p.H, n = unit / H, h = unit % H, v0 = vt * BV;
  int s, e;
  if (!seq_range(p, n, s, e)) return;
  const int base = slot_base(p, n, s);
  const int nch = max(0, min((e - s + C - 1) / C, p.n_slots - base));
  const bool with_o = p.o != nullptr;

  auto chunk_ptrs = [&](int c, size_t& gi, const char*& Wg, int& len, size_t& arow) {
    const int t0 = s + c * C;
    len = min(C, e - t0);
    gi = (size_t)(base + c) * H + h;
    arow = (size_t)t0 * H + h;
    Wg = (const char*)((const E*)p.wW + gi * C * DK);
  };
  // producers 0-1: their share of set A of chunk c into buffer buf
  auto issueA = [&](int c, int buf) {
    size_t gi, arow;
    const char* Wg;
    int len;
    chunk_ptrs(c, gi, Wg, len, arow);
    char* r = sm.ringA[buf];
    dma_rows<R::RK, C, 2, true>(r + R::AW, Wg, R::RK, C, Wg, 0, wp, lane);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
      if ((mt & 1) == wp)
        dma_block_asm<R::UM>(r + R::AU + mt * R::UM,
                             (const char*)((const E*)p.wU + gi * C * DV + (size_t)(mt * (DV / 16) + vt * NB) * 256),
                             lane);
    if (wp == 1) dma4_asm(p.wb + gi * C + lane, r + R::AB);
  };
  // producers 2-3: their share of part `part` (0: Q, P; 1: K, b; 2: both)
  // of set B of chunk c into buffer buf; rows of Q and K past the chunk come
  // from W, whose rows there are zero
  auto issueB = [&](int c, int buf, int part) {
    size_t gi, arow;
    const char* Wg;
    int len;
    chunk_ptrs(c, gi, Wg, len, arow);
    char* r = sm.ringB[buf];
    if (part != 1) {
      const char* Qg = (const char*)((const E*)p.q + arow * DK);
      const char* Pg = (const char*)((const E*)p.wP + gi * C * C);
      dma_rows<R::RK, C, 2, true>(r + R::BQ, Qg, (size_t)H * R::RK, len, Wg, R::RK, wp, lane);
      dma_rows<R::RC, C, 2, true>(r + R::BP, Pg, R::RC, C, Pg, 0, wp, lane);
    }
    if (part != 0) {
      const char* Kg = (const char*)((const E*)p.k + arow * DK);
      dma_rows<R::RK, C, 2, true>(r + R::BK, Kg, (size_t)H * R::RK, len, Wg, R::RK, wp, lane);
      if (wp == 1) dma4_asm(p.wb + gi * C + lane, r + R::BB);
    }
  };

  // state: acc[i][nb] = S^T rows 16*(KPW*w+i).., columns 16*nb.. of this tile
  f4 acc[KPW][NB];
#pragma unroll
  for (int i = 0; i < KPW; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int kt = KPW * w + i;
      acc[i][nb] = (p.S0 && !producer)
                       ? *(const f4*)(p.S0 + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 +
                                      frow(lane, 0))
                       : zero4();
    }

  if (nch > 0) {
    if (prodA) {
      issueA(0, 0);
      if (DB && nch > 1) issueA(1, 1);
    } else if (prodB) {
      issueB(0, 0, 2);
    }
  }
  for (int c = 0; c < nch; ++c) {
    const int t0 = s + c * C, len = min(C, e - t0);
    const size_t gi = (size_t)(base + c) * H + h;
    const int buf = DB ? (c & 1) : 0;
    const char* ra = sm.ringA[buf];
    const char* rb = sm.ringB[buf];
    FR sf[NB][DK / KS];                    // S fragments (B operand of D and O)
    block_sync_lds();                      // B1: chunk c-1 done
    // ---- phase 1: stage S (compute); producer 1 issues the first part of set B of chunk c+1
    if (!producer) {
#pragma unroll
      for (int i = 0; i < KPW; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int kt = KPW * w + i;
          *(QR*)&sm.u.s.S[nb * 16 + fcol(lane)][kt * 16 + frow(lane, 0)] = Quad<E>::pack(acc[i][nb]);
          if (p.saved) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
              sm.u.s.Sf[kt * 16 + frow(lane, j)][nb * 16 + fcol(lane)] = fromf<E>(acc[i][nb][j]);
          }
        }
    } else if (prodB) {
      if (DB && c + 1 < nch) issueB(c + 1, (c + 1) & 1, 0);
    } else {
      // set A of chunk c must have landed (set A of chunk c+1 may be in flight)
      if (DB && c + 1 < nch) {
        if (wp == 0) wait_vm<DB ? R::LOADS_A0 : 0>();
        else wait_vm<DB ? R::LOADS_A1 : 0>();
      } else {
        wait_vm<0>();
      }
    }
    block_sync_lds();                      // B2: S staged; set A of chunk c visible
    // ---- phase 2: saved S, D = U - W S^T (compute); producer 1 finishes set B
    if (!producer) {
      if (p.saved) {
        // saved entry state, transposed (element (k, v) at [k][v]), 16-byte stores
        constexpr int VEC = 16 / sizeof(E), PR = BV / VEC;
        E* dst = (E*)p.saved + gi * DK * DV + v0;
        for (int idx = tid; idx < DK * PR; idx += NTHREADS) {
          const int r = idx / PR, cc = (idx % PR) * VEC;
          *(uint4*)(dst + (size_t)r * DV + cc) = *(const uint4*)&sm.u.s.Sf[r][cc];
        }
      }
      const float* bch = (const float*)(ra + R::AB);
      const float bl = bch[C - 1];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int ks = 0; ks < DK / KS; ++ks)
          sf[nb][ks] = Frag<E>::load(kmaj(&sm.u.s.S[0][0], LK), nb * 16, ks * KS, lane);
      // D = U - W S^T (rows 16w..), to LDS as D^T and (diag(g_C/g) D)^T
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f4 d = zero4();
#pragma unroll
        for (int ks = 0; ks < DK / KS; ++ks)
          d = Mma<E>::mma(tile_frag<E, R::RK>(ra + R::AW, 16 * w, ks * KS, lane), sf[nb][ks], d);
        const QR uq = *(const QR*)(ra + R::AU + ((w * NB + nb) * 64 + lane) * 4 * sizeof(E));
        f4 dk;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          d[j] = Quad<E>::get(uq, j) - d[j];
          dk[j] = __expf(bl - bch[16 * w + frow(lane, j)]) * d[j];
        }
        *(QR*)&sm.Dt[nb * 16 + fcol(lane)][16 * w + frow(lane, 0)] = Quad<E>::pack(d);
        *(QR*)&sm.Dkt[nb * 16 + fcol(lane)][16 * w + frow(lane, 0)] = Quad<E>::pack(dk);
      }
    } else if (prodB) {
      if (DB && c + 1 < nch) {
        issueB(c + 1, (c + 1) & 1, 1);
        // set B of chunk c landed; chunk c+1's in flight
        if (wp == 0) wait_vm<DB ? R::LOADS_B0 : 0>();
        else wait_vm<DB ? R::LOADS_B1 : 0>();
      } else {
        wait_vm<0>();
      }
    }
    block_sync_lds();                      // B3: D staged; set B of chunk c visible; set A of chunk c free
    // ---- phase 3: saved D, O, state update (compute); producer 0 refills set A
    if (!producer) {
      if (p.saved) {
        // D rows of this tile into the saved context (rows past the chunk are zero),
        // read back from D^T; one thread per (row, 8-column group)
        constexpr int VEC = 16 / sizeof(E), PR = BV / VEC;
        E* dbase = (E*)p.savedD + gi * C * DV + v0;
        for (int idx = tid; idx < C * PR; idx += NTHREADS) {
          const int r = idx % C, cc = (idx / C) * VEC;
          uint4 o;
          E* oe = (E*)&o;
#pragma unroll
          for (int j = 0; j < VEC; ++j) oe[j] = sm.Dt[cc + j][r];
          *(uint4*)(dbase + (size_t)r * DV + cc) = o;
        }
      }
      const float* bch = (const float*)(rb + R::BB);
      const float gC = __expf(bch[C - 1]);
      if (with_o) {
        // O = diag(g) Q S^T + P D   (rows 16w..)
        f4 oo[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          f4 o1 = zero4(), o2 = zero4();
#pragma unroll
          for (int ks = 0; ks < DK / KS; ++ks)
            o1 = Mma<E>::mma(tile_frag<E, R::RK>(rb + R::BQ, 16 * w, ks * KS, lane), sf[nb][ks], o1);
#pragma unroll
          for (int ks = 0; ks < C / KS; ++ks)
            o2 = Mma<E>::mma(tile_frag<E, R::RC>(rb + R::BP, 16 * w, ks * KS, lane),
                             Frag<E>::load(kmaj(&sm.Dt[0][0], LC), nb * 16, ks * KS, lane), o2);
#pragma unroll
          for (int j = 0; j < 4; ++j) oo[nb][j] = __expf(bch[16 * w + frow(lane, j)]) * o1[j] + o2[j];
        }
        // the state copies aliased by O were last read before B3
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int j = 0; j < 4; ++j) sm.u.O[16 * w + frow(lane, j)][nb * 16 + fcol(lane)] = fromf<E>(oo[nb][j]);
      }
      // S^T <- g_C S^T + K^T diag(g_C/g) D  (K^T fragments are transpose reads of the K tile)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int i = 0; i < KPW; ++i) acc[i][nb] = gC * acc[i][nb];
#pragma unroll
        for (int ks = 0; ks < C / KS; ++ks) {
          const FR bf = Frag<E>::load(kmaj(&sm.Dkt[0][0], LC), nb * 16, ks * KS, lane);
#pragma unroll
          for (int i = 0; i < KPW; ++i)
            acc[i][nb] = Mma<E>::mma(tile_tr_frag<E, R::RK>(rb + R::BK, ks * KS, 16 * (KPW * w + i), lane), bf,
                                     acc[i][nb]);
        }
      }
    } else if (prodA) {
      if (DB && c + 2 < nch) issueA(c + 2, c & 1);
      if (!DB && c + 1 < nch) issueA(c + 1, 0);
    }
    block_sync_lds();                      // B4: O staged; set B of chunk c free
    if (prodB) {
      if (!DB && c + 1 < nch) issueB(c + 1, 0, 2);
    } else if (!producer && with_o) {
      constexpr int VEC = 16 / sizeof(E), PR = BV / VEC;
      E* obase = (E*)p.o + ((size_t)t0 * H + h) * DV + v0;
      for (int idx = tid; idx < C * PR; idx += NTHREADS) {
        const int r = idx / PR, cc = (idx % PR) * VEC;
        if (r < len) *(uint4*)(obase + (size_t)r * H * DV + cc) = *(const uint4*)&sm.u.O[r][cc];
      }
    }
  }
  if (p.Sfin && !producer) {
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int kt = KPW * w + i;
        *(f4*)(p.Sfin + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) =
            acc[i][nb];
      }
  }
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_fwd_t(const Params& p, int in_bwd, int with_scan, hipStream_t st) {
  constexpr int BV = 32;   // value columns per forward-scan workgroup
  if (p.n_slots > 0) {
    const int units = p.n_slots * p.H;
    dim3 gp(min(units, device_cu_count()));
    const int stage = in_bwd ? ST_PREP_BWD : ST_PREP_FWD;
    prof_mark(stage, 0, st);
    hipLaunchKernelGGL((k_prep<E, DK, DV>), gp, dim3(PREP_THREADS), 0, st, p);
    prof_mark(stage, 1, st);
  }
  if (with_scan) {
    const int units = p.N * p.H;
    const int nb = ((units + 7) / 8) * 8 * (DV / BV);
    if (nb > 0) {
      prof_mark(ST_SCAN_FWD, 0, st);
      hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, BV>), dim3(nb), dim3(NTHREADS + 256), 0, st, p);
      prof_mark(ST_SCAN_FWD, 1, st);
    }
  }
  return hipGetLastError();
}

hipError_t launch_fwd(const Params& p, int dtype, int Dk, int Dv, int in_bwd, int with_scan,
                      hipStream_t st) {
#define QD_CASE(ET, DKV, DVV) \
  if (Dk == DKV && Dv == DVV) return launch_fwd_t<ET, DKV, DVV>(p, in_bwd, with_scan, st);
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
