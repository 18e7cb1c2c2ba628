// Q-Delta chunkwise forward kernels for gfx950.
//
// Per chunk of C tokens with entry state S (Dv x Dk), following Sec. 3.3
// ("Chunkwise parallel form") and App. D.1/D.2 (WY representation, UT
// transform), with the readings listed in the design notes (decay ratios on
// the intra-chunk output term, inclusive causal mask, products read as W S^T):
//
//   b_r = sum_{j<=r} log alpha_j,  g_r = exp(b_r),  Gam_ri = exp(b_r - b_i)
//   X   = K + diag(lambda) Q
//   A   = strictLower(diag(beta) (Gam * X K^T)),   M = (I + A)^{-1},  T = M diag(beta)
//   U   = T V,   W = T diag(g) X
//   D   = U - W S^T = U - M Y,   Y = diag(beta g) (K S^T + diag(lambda) Q S^T)
//   O   = diag(g) Q S^T + (Gam * M_causal * Q K^T) D     (the mask includes the diagonal)
//   S'  = g_C S + D^T diag(g_C / g) K
//
// k_prep   (persistent over chunk-head units, fully parallel): b, the Gram
//          products, A, the UT solve; writes the gate block (b, beta,
//          lambda), the output operator P = Gam * M_causal * Q K^T,
//          T = M diag(beta) and, when a saved context is kept, M.
// k_scan_fwd (one workgroup per sequence, head and Dv tile): the sequential
//          pass over chunks; the state tile stays in MFMA accumulators in fp32;
//          D = T V + T Y, the chunk output and the state update are computed
//          on chip from Q, K, V, T, P and the gates (U and W are never formed
//          in memory).
#include "qd_common.h"
#include "qd_launch.h"

#include <type_traits>

namespace qd {

// 16 x 16 fp32 blocks of A and M in the preparation kernel: row stride 20
// floats (16-byte rows for vector stores; the 16 rows of a fragment read fall
// in distinct banks).  Twelve slots: 0-3 the diagonal blocks (A_ww, then
// M_ww over it: only the inverse of that block reads A_ww); 4-9 the blocks
// A_10, A_20, A_21, A_30, A_31, A_32 (then A~ in place); M_10 and M_21 in 10
// and 11; M_32, M_31, M_20 and M_30 over A~_32, A~_31, A~_30 and A~_20, each
// written once the solve has read that A~ block for the last time.
constexpr int PREP_LB = 20;
constexpr int PREP_SLOTS = 12;
__device__ inline int prep_slot_a(int i, int j) {
  if (i == j) return i;
  return i == 1 ? 4 : i == 2 ? 5 + j : 7 + j;
}
__device__ inline int prep_slot_m(int i, int j) {
  if (i == j) return i;
  const int ij = 4 * i + j;
  return ij == 4 ? 10 : ij == 9 ? 11 : ij == 14 ? 9 : ij == 13 ? 8 : ij == 8 ? 7 : 5;
}

template <typename E, int DK>
struct alignas(16) PrepSmem {
  static constexpr int RK = DK * (int)sizeof(E);
  alignas(16) char Kt[C * RK];      // K and Q of a unit (swizzled direct-load tiles); the
  alignas(16) char Qt[C * RK];      // next unit's land here once the Gram products are done
  alignas(16) float rla[C], rbeta[C], rlam[C];   // raw gate vectors of the next unit
  alignas(16) float b[C], beta[C], lam[C];       // the gate block
  alignas(16) float blk[PREP_SLOTS][16][PREP_LB];   // A and M blocks on and below the diagonal
};

// Four waves per workgroup; with bf16 inputs three workgroups share a CU
// (under 54 KB of LDS and 168 registers each), so that the latency chains of
// one (UT solve, Gram) run beside the others'.  fp32 operands take more
// registers: at most two per CU (one when the LDS allows no more).
constexpr int PREP_THREADS = 256;
template <typename E, int DK>
constexpr int prep_per_cu() {
  constexpr int fit = sizeof(PrepSmem<E, DK>) * 3 <= 160 * 1024 ? 3 : sizeof(PrepSmem<E, DK>) * 2 <= 160 * 1024 ? 2 : 1;
  return sizeof(E) == 2 ? fit : (fit < 2 ? fit : 2);
}

// Writes, for every unit, the gate block (b, beta, lambda), the intra-chunk
// output operator P = Gam * M_causal * Q K^T, M = (I + A)^{-1} (when p.wM is
// set) and T = M diag(beta).  Persistent: each workgroup walks units
// blockIdx.x, +gridDim.x, ...: the gate block and the Gram products K K^T,
// Q K^T of the 16 x 16 blocks on and below the diagonal, A and P (P stored
// straight from registers, its blocks above the diagonal as zeros), the UT
// solve (the blocked inverse below, the products of each level spread over
// the four waves), M and T.  The Gram blocks are formed as their transposes
// (operands swapped), so that a lane holds four consecutive columns of one
// row: one vector store into A and one into P.  Once the Gram products are
// done the next unit's K, Q and raw gates go straight into LDS (direct loads
// in assembly form) and land during the solve; the only memory operations
// issued after them are this unit's P, M and T stores, which fixes the wait
// count at the top of the next unit (the compiler's wait for register loads
// would also cover every store still in flight).
template <typename E, int DK, int DV>
__global__ __launch_bounds__(PREP_THREADS) __attribute__((amdgpu_waves_per_eu(prep_per_cu<E, DK>(), prep_per_cu<E, DK>()))) void k_prep(Params p) {
  constexpr int NT = PREP_THREADS, NW = NT / 64;
  constexpr int LB = PREP_LB;
  constexpr int RK = DK * (int)sizeof(E), KS = Mma<E>::KS, NKK = DK / KS;
  constexpr int VEC = 16 / sizeof(E);
  constexpr int BCH = 16 / VEC;                 // M/T stores per block row
  constexpr int MT_STORES = 10 * 16 * BCH;      // M/T stores per matrix (packed)
  constexpr int MT_ROUNDS = (MT_STORES + NT - 1) / NT;
  static_assert(C == 64 && NW == 4 && MT_STORES % 64 == 0, "four waves; whole-wave store rounds");
  typedef typename Mma<E>::frag FR;
  __shared__ PrepSmem<E, DK> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;   // vector wave index: measured faster here than the scalar one
  const int H = p.H;
  const int total = p.n_slots * H;
  const bool keep_m = p.wM != nullptr;

  struct Unit {
    int g, h, t0, len;
    bool valid;
  };
  // Work item u -> (slot, head).  Workgroups sit on XCD blockIdx.x mod 8
  // and step by a multiple of 8, so item u runs on XCD u mod 8; every head
  // of a slot is given to the same XCD, because the raw gate vectors of the
  // H heads of a token share cache lines (H x 4 bytes per token), which each
  // XCD's L2 would otherwise fetch again.  Slots past the last multiple of 8
  // keep the plain order.
  const int total8 = (p.n_slots / 8) * 8 * H;
  auto find = [&](int u, Unit& x) {
    x.valid = false;
    if (u >= total) return;
    if (u < total8) {
      const int k = u >> 3;
      x.g = 8 * (k / H) + (u & 7);
      x.h = k % H;
    } else {
      x.g = u / H;
      x.h = u % H;
    }
    int n;
    x.valid = locate(p, x.g, n, x.t0, x.len);
  };
  // K, Q rows past the chunk re-read its last row: they meet only zero
  // gates, or masked entries of P; so do the raw gates, masked when read
  auto issue = [&](const Unit& x) {
    if (!x.valid) return;
    const size_t row = (size_t)x.t0 * H + x.h;
    const char* Kg = (const char*)((const E*)p.k + row * DK);
    const char* Qg = (const char*)((const E*)p.q + row * DK);
    dma_rows<RK, C, NW, true>(sm.Kt, Kg, (size_t)H * RK, x.len, Kg + (size_t)(x.len - 1) * H * RK, 0, w, lane);
    dma_rows<RK, C, NW, true>(sm.Qt, Qg, (size_t)H * RK, x.len, Qg + (size_t)(x.len - 1) * H * RK, 0, w, lane);
    if (w == 0) {
      const size_t gt = row + (size_t)min(lane, x.len - 1) * H;
      if (p.la) dma4_asm(p.la + gt, (char*)sm.rla);
      dma4_asm(p.beta + gt, (char*)sm.rbeta);
      if (p.lam) dma4_asm(p.lam + gt, (char*)sm.rlam);
    }
  };

  // UT solve, M = (I + A)^{-1} blocked 16 x 16: A~_mj = A_mj M_jj,
  // M_ij = -sum_{m=j+1..i} M_im A~_mj
  auto blkA = [&](int i, int j) { return &sm.blk[prep_slot_a(i, j)][0][0]; };
  auto blkM = [&](int i, int j) { return &sm.blk[prep_slot_m(i, j)][0][0]; };
  auto put = [&](float* dst, f4 v, float sc) {
#pragma unroll
    for (int j = 0; j < 4; ++j) dst[frow(lane, j) * LB + fcol(lane)] = sc * v[j];
  };
  auto prod = [&](const float* a, const float* m, f4 acc) {
    return mma_k<float, 16>(kmaj(a, LB), imaj(m, LB), 0, 0, acc, lane);
  };

  // the zero block that the kernels reading this launch's outputs take as
  // zero rows (covered by the wait below)
  if (blockIdx.x == 0 && w == 0) *(uint4*)((char*)p.wZ + lane * 16) = make_uint4(0, 0, 0, 0);
  Unit cur;
  find(blockIdx.x, cur);
  issue(cur);
  wait_vm<0>();
  for (int u = blockIdx.x; u < total; u += gridDim.x) {
    const Unit x = cur;
    Unit nx;
    find(u + gridDim.x, nx);
    block_sync_lds();                        // x's inputs landed in every wave; the previous unit's LDS use is over
    if (!x.valid) {                          // uniform across the workgroup
      issue(nx);
      wait_vm<0>();
      cur = nx;
      continue;
    }
    const size_t gi = (size_t)x.g * H + x.h;
    const int ws = wave_id(tid);             // scalar: the branches below are uniform
    // the ten 16 x 16 blocks on and below the diagonal (the others are zero in
    // A and P): wave 0 (0,0) (1,0) (1,1), wave 1 (2,0) (2,1) (2,2), wave 2
    // (3,0) (3,1) and the gate block, wave 3 (3,2) (3,3)
    if (ws == 2) {
      // gates past the chunk's end are zero; NULL lambda: the constant
      const bool ok = lane < x.len;
      const float la = (ok && p.la) ? sm.rla[lane] : 0.f, be = ok ? sm.rbeta[lane] : 0.f;
      const float lm = ok ? (p.lam ? sm.rlam[lane] : p.lam_c) : 0.f;
      const float b = wave_incl_scan_dpp(la);
      sm.b[lane] = b;
      sm.beta[lane] = be;
      sm.lam[lane] = lm;
      float* gblk = p.wb + gi * 3 * C;
      gblk[lane] = b;
      gblk[C + lane] = be;
      gblk[2 * C + lane] = lm;
    }
    // K K^T and Q K^T of the wave's blocks (row, column), each as its
    // transpose: K_c K_r^T and K_c Q_r^T; operand fragments shared within a
    // wave are read once
    f4 kk[3], qk[3];
#pragma unroll
    for (int n = 0; n < 3; ++n) kk[n] = qk[n] = zero4();
    auto gram = [&](auto... blk) {
      constexpr int NBK = sizeof...(blk);
      constexpr int br[NBK] = {(decltype(blk)::value / 4)...}, bc[NBK] = {(decltype(blk)::value % 4)...};
#pragma unroll
      for (int ks = 0; ks < NKK; ++ks) {
        FR kf[4], qf[4];
#pragma unroll
        for (int b = 0; b < NBK; ++b) {
          kf[br[b]] = tile_frag<E, RK>(sm.Kt, 16 * br[b], ks * KS, lane);
          qf[br[b]] = tile_frag<E, RK>(sm.Qt, 16 * br[b], ks * KS, lane);
          kf[bc[b]] = tile_frag<E, RK>(sm.Kt, 16 * bc[b], ks * KS, lane);
        }
#pragma unroll
        for (int b = 0; b < NBK; ++b) {
          kk[b] = Mma<E>::mma(kf[bc[b]], kf[br[b]], kk[b]);
          qk[b] = Mma<E>::mma(kf[bc[b]], qf[br[b]], qk[b]);
        }
      }
    };
    typedef std::integral_constant<int, 0> B00;
    typedef std::integral_constant<int, 4> B10;
    typedef std::integral_constant<int, 5> B11;
    typedef std::integral_constant<int, 8> B20;
    typedef std::integral_constant<int, 9> B21;
    typedef std::integral_constant<int, 10> B22;
    typedef std::integral_constant<int, 12> B30;
    typedef std::integral_constant<int, 13> B31;
    typedef std::integral_constant<int, 14> B32;
    typedef std::integral_constant<int, 15> B33;
    if (ws == 0) gram(B00(), B10(), B11());
    else if (ws == 1) gram(B20(), B21(), B22());
    else if (ws == 2) gram(B30(), B31());
    else gram(B32(), B33());
    block_sync_lds();                        // gates visible; K and Q no longer read
    issue(nx);                               // lands during the solve
    {
      // A = strictLower(diag(beta) Gam * X K^T), X K^T = K K^T + diag(lambda) Q K^T,
      // and P, the wave's blocks: lane row 16 m + (l & 15), columns 16 n + 4 (l >> 4)..
      // Rows past the chunk's end are zero in both (in A through beta; no
      // output reads those rows of P).  P is stored packed, block (m, n) as
      // one contiguous 16 x 16 block written by the wave's 64 lanes.
      typedef typename Quad<E>::raw QR;
      E* Pg = (E*)p.wP + gi * LBT_ELEMS;
      const int rl = fcol(lane), c4 = frow(lane, 0);
      auto epilogue = [&](int m, int n, const f4& kkb, const f4& qkb) {
        const int r = 16 * m + rl, i0 = 16 * n + c4;
        const float br = sm.b[r], ber = sm.beta[r], lmr = sm.lam[r];
        const f4 bi = *(const f4*)&sm.b[i0];
        f4 a, pv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = i0 + j;
          const float gam = (r >= i && r < x.len) ? __expf(br - bi[j]) : 0.f;
          a[j] = (r > i) ? ber * gam * (kkb[j] + lmr * qkb[j]) : 0.f;
          pv[j] = gam * qkb[j];
        }
        *(f4*)(blkA(m, n) + rl * LB + c4) = a;
        *(QR*)(Pg + (size_t)lbt_block(m, n) * 256 + rl * 16 + c4) = Quad<E>::pack(pv);
      };
      if (ws == 0) {
        epilogue(0, 0, kk[0], qk[0]);
        epilogue(1, 0, kk[1], qk[1]);
        epilogue(1, 1, kk[2], qk[2]);
      } else if (ws == 1) {
        epilogue(2, 0, kk[0], qk[0]);
        epilogue(2, 1, kk[1], qk[1]);
        epilogue(2, 2, kk[2], qk[2]);
      } else if (ws == 2) {
        epilogue(3, 0, kk[0], qk[0]);
        epilogue(3, 1, kk[1], qk[1]);
      } else {
        epilogue(3, 2, kk[0], qk[0]);
        epilogue(3, 3, kk[1], qk[1]);
      }
    }
    block_sync_lds();
    if (lane < 16) {
      // column j of (I + A_ww)^{-1}, written over A_ww; row r of the block is
      // read as four broadcast 16-byte loads one row ahead of its use
      const int j = lane;
      float* blk = blkA(w, w);
      float m[16];
      f4 cu[4], nxt[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) cu[qq] = *(const f4*)(blk + (size_t)1 * LB + 4 * qq);
      m[0] = (j == 0) ? 1.f : 0.f;
#pragma unroll
      for (int r = 1; r < 16; ++r) {
        if (r + 1 < 16) {
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) nxt[qq] = *(const f4*)(blk + (size_t)(r + 1) * LB + 4 * qq);
        }
        float s4[4] = {(r == j) ? 1.f : 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < r; ++i) s4[i & 3] -= cu[i >> 2][i & 3] * m[i];
        m[r] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) cu[qq] = nxt[qq];
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) blk[r * LB + j] = m[r];
    }
    block_sync_lds();
    {
      // A~ blocks: wave 0 (1,0) and (3,1), wave 1 (2,1) and (3,0), wave 2 (3,2), wave 3 (2,0)
      auto tilde = [&](int bm, int bj) { put(blkA(bm, bj), prod(blkA(bm, bj), blkM(bj, bj), zero4()), 1.f); };
      if (w == 0) { tilde(1, 0); tilde(3, 1); }
      else if (w == 1) { tilde(2, 1); tilde(3, 0); }
      else if (w == 2) tilde(3, 2);
      else tilde(2, 0);
    }
    block_sync_lds();
    // level 1: M_10, M_21, M_32 and the diagonal-block parts of M_20, M_31, M_30
    // (M_32 goes over A~_32, which only this product reads)
    f4 part = zero4();
    if (w < 3) {
      const int bb = w + 1;                  // M_b,b-1 = -M_bb A~_b,b-1
      put(blkM(bb, bb - 1), prod(blkM(bb, bb), blkA(bb, bb - 1), zero4()), -1.f);
      if (w == 0) part = prod(blkM(2, 2), blkA(2, 0), zero4());        // M_20
      else if (w == 1) part = prod(blkM(3, 3), blkA(3, 1), zero4());   // M_31
      else part = prod(blkM(3, 3), blkA(3, 0), zero4());               // M_30
    }
    block_sync_lds();
    // level 2: M_20 += M_21 A~_10, M_31 += M_32 A~_21, M_30 += M_32 A~_20
    // (M_20 over A~_30, M_31 over A~_31: both last read in level 1)
    if (w == 0) {
      part = prod(blkM(2, 1), blkA(1, 0), part);
      put(blkM(2, 0), part, -1.f);
    } else if (w == 1) {
      part = prod(blkM(3, 2), blkA(2, 1), part);
      put(blkM(3, 1), part, -1.f);
    } else if (w == 2) {
      part = prod(blkM(3, 2), blkA(2, 0), part);
    }
    block_sync_lds();
    // level 3: M_30 += M_31 A~_10 (over A~_20, last read in level 2)
    if (w == 2) {
      part = prod(blkM(3, 1), blkA(1, 0), part);
      put(blkM(3, 0), part, -1.f);
    }
    block_sync_lds();
    {
      // M (only the backward reads it, so only when the context is kept) and
      // T = M diag(beta), packed like P; a thread takes VEC consecutive
      // columns of one block row.  The stores per matrix are a multiple of
      // 64, so whole waves run a round or skip it.
      E* wM = keep_m ? (E*)p.wM + gi * LBT_ELEMS : nullptr;
      E* wT = (E*)p.wT + gi * LBT_ELEMS;
#pragma unroll
      for (int it = 0; it < MT_ROUNDS; ++it) {
        if (it * NT + ws * 64 >= MT_STORES) break;
        const int idx = tid + it * NT;
        const int k = idx / (16 * BCH), q = idx % (16 * BCH);
        const int rr = q / BCH, cc = (q % BCH) * VEC;   // row and first column inside block k
        const int br = k < 1 ? 0 : k < 3 ? 1 : k < 6 ? 2 : 3, bc = k - br * (br + 1) / 2;
        const float* src = blkM(br, bc) + rr * LB + cc;
        uint4 mr, tr;
        E* me = (E*)&mr;
        E* te = (E*)&tr;
        float mv[VEC], bv[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j += 4) {
          *(f4*)&mv[j] = *(const f4*)(src + j);
          *(f4*)&bv[j] = *(const f4*)&sm.beta[16 * bc + cc + j];
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          me[j] = fromf<E>(mv[j]);
          te[j] = fromf<E>(mv[j] * bv[j]);
        }
        const int at = k * 256 + rr * 16 + cc;
        if (keep_m) *(uint4*)(wM + at) = mr;
        *(uint4*)(wT + at) = tr;
      }
      // the next unit's loads went out before P's and these stores (in-order
      // counter): three or two P blocks per wave, then its rounds of M and T
      const int rounds = (MT_STORES - ws * 64 + NT - 1) / NT;
      wait_vm_n((ws < 2 ? 3 : 2) + (keep_m ? 2 : 1) * rounds);
    }
    cur = nx;
  }
}

// Forward-scan operands of one chunk, filled by direct global->LDS loads as
// swizzled row-major tiles, in sets by the phases that read them:
//   set A (phases 2-4): Q, K (C x Dk) and the gate block (b, beta, lambda);
//   set B (phase 3):    T = (I + A)^{-1} diag(beta) (C x C) and this tile's
//                       columns of V (C x BV);
//   P (phase 4):        the output operator Gam * M_causal * Q K^T (C x C).
// Set A has a ring of NA chunks, P of NP, set B one buffer.  The four
// producer waves split every tile's 1 KB instructions evenly; producers 0-2
// also load one gate vector each.
template <typename E, int DK, int BV>
struct ScanFwdRing {
  static constexpr int RK = DK * (int)sizeof(E), RC = C * (int)sizeof(E), RO = BV * (int)sizeof(E);   // row bytes
  static constexpr int AQ = 0, AK = AQ + C * RK, AG = AK + C * RK, ABYTES = AG + 3 * C * 4;
  static constexpr int BT = 0, BV_ = BT + C * RC, BBYTES = BV_ + C * RO;
  // ring depths: fp32 tiles and 64-column value tiles leave room for two
  // chunks of set A and one P buffer
  static constexpr bool DEEP = sizeof(E) == 2 && BV == 32;
  static constexpr int NA = DEEP ? 3 : 2;
  static constexpr int NP = DEEP ? 2 : 1;                   // P buffers
  static constexpr int LQ = C * RK / 1024 / 4;              // loads per producer: Q
  static constexpr int LK = C * RK / 1024 / 4;              // K (plus one gate vector for producers 0-2)
  static constexpr int LB = (C * RC + C * RO) / 1024 / 4;   // T and V
  static constexpr int LP = C * RC / 1024 / 4;              // P
  static_assert((C * RK / 1024) % 4 == 0 && (C * RC / 1024) % 4 == 0 && (C * RO / 1024) % 4 == 0, "even split");
  static_assert(2 * LB + LQ + LP + 2 * (LK + 1) <= 63, "outstanding-load counter range");
};

template <typename E, int DK, int BV>
struct alignas(16) ScanFwdSmem {
  static constexpr int P = Pad<E>::v;
  typedef ScanFwdRing<E, DK, BV> R;
  alignas(16) char ringA[R::NA][R::ABYTES];
  alignas(16) char ringB[R::BBYTES];
  alignas(16) char Pt[R::NP][C * R::RC];
  E S[BV][DK + P];    // state tile (row v, column k): MFMA operand and saved-state source
  E Y[C][BV + P];     // -diag(g) X S^T (row r, column v)
  E D[C][BV + P];     // D = T V - T diag(g) X S^T
  E Dk[C][BV + P];    // diag(g_C / g) D
  E O[C][BV + P];     // output tile staging
};

// One workgroup per (sequence, head, Dv tile of BV value rows): NCW compute
// waves and four producer waves (one wave alone issues direct loads at only
// about 12 bytes per clock).  bf16 runs eight compute waves, two per SIMD:
// a single wave reads LDS at only about 26 bytes per clock (16 with transpose
// reads), so a chunk's fragment reads take half as long on each of twice as
// many waves.  The state tile S^T (Dk x BV) lives in fp32 MFMA accumulators
// across the whole sequence, split over the compute waves by key blocks (and
// value blocks when there are more waves than key blocks); compute wave w
// owns chunk rows 16 (w & 3).. of every C-row result and a range of its
// value blocks.
//
// The chunk step never forms W = T diag(g) X nor U = T V:
//   D = U - W S^T = T V + T Y,  Y = -diag(g) (K S^T + diag(lambda) Q S^T),
// and Q S^T also serves the output, so a chunk reads Q, K, P, T, V and the
// gates only.  Per chunk the compute waves pass three barriers:
//   B_a  S staged, set A visible    phase 2: saved S; S K^T, S Q^T (as their
//                                   transposes); Y;
//   B_b  Y staged, set B visible    phase 3: output of the previous chunk;
//                                   D = T V + T Y;
//   B_c  D staged, P visible        phase 4: saved D; O = diag(g) Q S^T + P D
//                                   (as O^T = g (S Q^T)^T + D^T P^T); state
//                                   update S^T <- g_C S^T + K^T Dk; S staged.
// Producers: Q of chunk c+NA-1 and P of chunk c+NP-1 in phase 2, K and gates
// of chunk c+NA-1 in phase 3, set B of chunk c+1 in phase 4; they wait for
// set B of chunk c in phase 2, for P of chunk c in phase 3 and for set A of
// chunk c+1 in phase 4.  They issue no other memory operations, so their outstanding-load
// counts are exact.  When p.o is null only the states are produced.
//
// SEG selects the segment-parallel passes over long sequences (each
// sequence split into p.n_seg segments of p.seg_chunks chunks; a chunk is an
// affine map S -> S A + B of the state, Sec. 3.3 compact chunk update, and so
// is a segment):
//   SEG_NONE  one workgroup walks the whole sequence (the single pass);
//   SEG_MAPS  per segment from a zero state, no outputs: the value tiles end
//             at the segment's B, and DK / BV extra tiles whose rows start as
//             rows of the identity and see no values (their V product is
//             skipped) end at the rows of its A; both go to p.wSegOut;
//   SEG_OUT   per segment from its entry state in p.wSegIn, with every
//             output; the last segment writes the final state.
enum { SEG_NONE = 0, SEG_MAPS = 1, SEG_OUT = 2 };

template <typename E, int DK, int DV, int BV, int NCW, int SEG>
__global__ __launch_bounds__(NCW * 64 + 256) void k_scan_fwd(Params p) {
  constexpr int P = Pad<E>::v;
  constexpr int LK = DK + P, LV = BV + P;
  constexpr int NVT = DV / BV;
  constexpr int NB = BV / 16;                 // 16-column blocks per tile
  constexpr int KS = Mma<E>::KS;
  constexpr int NKS = DK / KS;
  constexpr int NCT = NCW * 64;               // compute threads
  // compute wave w: chunk rows 16 cb.. (cb = w & 3) of the C-row results,
  // NBW value blocks from nb0 = (w >> 2) NBW; state tile S^T: KPW key
  // blocks from kb0 and NBS value blocks from ns0
  constexpr int NBW = NB / (NCW / 4);
  constexpr int KB = DK / 16;
  constexpr int KPW = KB >= NCW ? KB / NCW : 1;
  constexpr int SG = KB >= NCW ? 1 : NCW / KB;   // waves that share a key block
  constexpr int NBS = NB / SG;
  static_assert(NCW % 4 == 0 && NBW >= 1 && NBS >= 1 && KPW * (NCW / SG) == KB, "wave mapping");
  constexpr size_t ES = sizeof(E);
  typedef typename Quad<E>::raw QR;
  typedef typename Mma<E>::frag FR;
  typedef ScanFwdRing<E, DK, BV> R;
  constexpr int NA = R::NA;
  // the maps pass produces no output: it loads no P, and its map tiles load
  // no V (their V product is skipped), so their set B is T alone
  constexpr bool MAPS = SEG == SEG_MAPS;
  static_assert(!MAPS || (NA == 2 && R::NP == 1), "the maps pass runs the two-deep ring with one P buffer");
  constexpr int LT = C * R::RC / 1024 / 4;    // loads per producer: T alone
  __shared__ ScanFwdSmem<E, DK, BV> sm;
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id(tid);
  const int prod = w - NCW;                   // 0-3 for the producer waves, negative otherwise
  const bool producer = prod >= 0;
  const int cb = w & 3, nb0 = (w >> 2) * NBW;
  const int kb0 = (w % (NCW / SG)) * KPW, ns0 = (w / (NCW / SG)) * NBS;
  constexpr int G = SEG == SEG_NONE ? 1 : 0;          // 0: the run-time segment count
  const int nseg = G ? G : p.n_seg;
  constexpr int NTILE = NVT + (SEG == SEG_MAPS ? DK / BV : 0);
  int su, vt;
  if (!xcd_unit_tile(blockIdx.x, p.N * p.H * nseg, NTILE, su, vt)) return;
  const int unit = G ? su : su / nseg, g = G ? 0 : su % nseg;
  const bool map_tile = SEG == SEG_MAPS && vt >= NVT;  // rows of the segment's A (no values)
  const int H = p.H, n = unit / H, h = unit % H;
  const int v0 = map_tile ? 0 : vt * BV;               // V columns read (a map tile's are ignored)
  const int r0 = vt * BV;                              // first state row (map rows follow the value rows)
  int s, e;
  if (!seq_range(p, n, s, e)) return;
  const int base = slot_base(p, n, s);
  const int nch_all = max(0, min((e - s + C - 1) / C, p.n_slots - base));
  const int cbeg = G ? 0 : min(g * p.seg_chunks, nch_all);
  const int nch = G ? nch_all : min(cbeg + p.seg_chunks, nch_all);   // end of this workgroup's chunks
  const bool with_o = SEG != SEG_MAPS && p.o != nullptr;
  void* const saved = SEG == SEG_MAPS ? nullptr : p.saved;

  auto chunk_at = [&](int c, size_t& gi, size_t& arow, int& len) {
    const int t0 = s + c * C;
    len = min(C, e - t0);
    gi = (size_t)(base + c) * H + h;
    arow = (size_t)t0 * H + h;
  };
  // producers: Q of chunk c (rows past the chunk re-read its last row: they
  // only meet zero gates)
  auto issueQ = [&](int c) {
    size_t gi, arow;
    int len;
    chunk_at(c, gi, arow, len);
    const char* Qg = (const char*)((const E*)p.q + arow * DK);
    dma_rows<R::RK, C, 4, true>(sm.ringA[c % NA] + R::AQ, Qg, (size_t)H * R::RK, len,
                                Qg + (size_t)(len - 1) * H * R::RK, 0, prod, lane);
  };
  // producers: K and the gate block of chunk c
  auto issueK = [&](int c) {
    size_t gi, arow;
    int len;
    chunk_at(c, gi, arow, len);
    char* r = sm.ringA[c % NA];
    const char* Kg = (const char*)((const E*)p.k + arow * DK);
    dma_rows<R::RK, C, 4, true>(r + R::AK, Kg, (size_t)H * R::RK, len, Kg + (size_t)(len - 1) * H * R::RK, 0,
                                prod, lane);
    if (prod < 3) dma4_asm(p.wb + gi * 3 * C + prod * C + lane, r + R::AG + prod * C * 4);
  };
  // producers: P of chunk c
  auto issueP = [&](int c) {
    if constexpr (MAPS) return;
    size_t gi, arow;
    int len;
    chunk_at(c, gi, arow, len);
    dma_lbt<E, 4>(sm.Pt[c % R::NP], (const char*)((const E*)p.wP + gi * LBT_ELEMS), prod, lane);
  };
  // producers: T and this tile's columns of V of chunk c (rows of V past the
  // chunk re-read its last row: they only meet zero columns of T)
  auto issueB = [&](int c) {
    size_t gi, arow;
    int len;
    chunk_at(c, gi, arow, len);
    const char* Vg = (const char*)((const E*)p.v + arow * DV + v0);
    dma_lbt<E, 4>(sm.ringB + R::BT, (const char*)((const E*)p.wT + gi * LBT_ELEMS), prod, lane);
    if (!map_tile)
      dma_rows<R::RO, C, 4, true>(sm.ringB + R::BV_, Vg, (size_t)H * DV * ES, len,
                                  Vg + (size_t)(len - 1) * H * DV * ES, 0, prod, lane);
  };

  // state: acc[i][j] = S^T rows 16 (kb0 + i).., columns 16 (ns0 + j).. of this tile
  f4 acc[KPW][NBS];
#pragma unroll
  for (int i = 0; i < KPW; ++i)
#pragma unroll
    for (int j = 0; j < NBS; ++j) {
      const int kt = kb0 + i, nb = ns0 + j;
      if constexpr (SEG == SEG_NONE) {
        acc[i][j] = (p.S0 && !producer)
                        ? *(const f4*)(p.S0 + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 +
                                       frow(lane, 0))
                        : zero4();
      } else if constexpr (SEG == SEG_OUT) {
        acc[i][j] = producer ? zero4()
                             : *(const f4*)(p.wSegIn + ((size_t)su * DV + v0 + nb * 16 + fcol(lane)) * DK +
                                            kt * 16 + frow(lane, 0));
      } else {
        // zero for the value rows; map row r starts as row r of the identity
        const int r = r0 - DV + nb * 16 + fcol(lane);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc[i][j][jj] = (map_tile && r == kt * 16 + frow(lane, jj)) ? 1.f : 0.f;
      }
    }
  // S (row v, column k) into LDS for the next chunk
  auto stage_S = [&]() {
#pragma unroll
    for (int i = 0; i < KPW; ++i)
#pragma unroll
      for (int j = 0; j < NBS; ++j)
        *(QR*)&sm.S[(ns0 + j) * 16 + fcol(lane)][(kb0 + i) * 16 + frow(lane, 0)] = Quad<E>::pack(acc[i][j]);
  };
  // output rows of chunk c from the staging tile
  auto store_O = [&](int c) {
    constexpr int VEC = 16 / sizeof(E), PR = BV / VEC;
    const int t0 = s + c * C, len = min(C, e - t0);
    E* obase = (E*)p.o + ((size_t)t0 * H + h) * DV + v0;
    for (int idx = tid; idx < C * PR; idx += NCT) {
      const int r = idx / PR, cc = (idx % PR) * VEC;
      if (r < len) *(uint4*)(obase + (size_t)r * H * DV + cc) = *(const uint4*)&sm.O[r][cc];
    }
  };

  // T and P arrive packed: the chunks above their diagonal blocks are zeroed
  // once here and never loaded (the first barrier of the loop orders these
  // stores before any read)
  zero_upper_chunks<E>(sm.ringB + R::BT, tid, NCT + 256);
  if constexpr (!MAPS) {
#pragma unroll
    for (int i = 0; i < R::NP; ++i) zero_upper_chunks<E>(sm.Pt[i], tid, NCT + 256);
  }
  if (nch > cbeg) {
    if (producer) {
      for (int c = cbeg; c < cbeg + NA - 1 && c < nch; ++c) {
        issueQ(c);
        issueK(c);
      }
      if (R::NP == 2) issueP(cbeg);
      issueB(cbeg);
      wait_vm<0>();
    } else {
      stage_S();
    }
  }
  for (int c = cbeg; c < nch; ++c) {
    const size_t gi = (size_t)(base + c) * H + h;
    const char* ra = sm.ringA[c % NA];
    const float* gb = (const float*)(ra + R::AG);   // b, then beta, then lambda
    const int rr = 16 * cb + fcol(lane);            // chunk row of this lane's result columns
    f4 sq[NBW];                                     // (S Q^T) blocks (v-block nb0 + j, r-block cb), scaled by g_r
    block_sync_lds();                      // B_a: S staged; set A of chunk c visible
    // ---- phase 2
    if (!producer) {
      // (S K^T), (S Q^T): value rows, chunk columns 16w..; the S fragments
      // of one k step at a time are live
      f4 sk[NBW];
#pragma unroll
      for (int j = 0; j < NBW; ++j) sk[j] = sq[j] = zero4();
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const FR kB = tile_frag<E, R::RK>(ra + R::AK, 16 * cb, ks * KS, lane);
        const FR qB = tile_frag<E, R::RK>(ra + R::AQ, 16 * cb, ks * KS, lane);
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
          const FR sa = Frag<E>::load(kmaj(&sm.S[0][0], LK), (nb0 + j) * 16, ks * KS, lane);
          sk[j] = Mma<E>::mma(sa, kB, sk[j]);
          sq[j] = Mma<E>::mma(sa, qB, sq[j]);
        }
      }
      const float gr = __expf(gb[rr]), ngr = -gr, lr = gb[2 * C + rr];
      // Y (row r, column v) = -g_r ((S K^T) + lambda_r (S Q^T))^T
#pragma unroll
      for (int jn = 0; jn < NBW; ++jn) {
        f4 y;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          y[j] = ngr * (sk[jn][j] + lr * sq[jn][j]);
          sq[jn][j] *= gr;
        }
        *(QR*)&sm.Y[rr][(nb0 + jn) * 16 + frow(lane, 0)] = Quad<E>::pack(y);
      }
      // Global stores go out at the end of a phase: at its start they would
      // queue behind the producers' direct loads for that phase and stall
      // the compute wave.
      if (saved) {
        // saved entry state S (row v, column k) of this tile, 16-byte stores
        constexpr int VEC = 16 / sizeof(E), PR = DK / VEC;
        E* dst = (E*)saved + gi * DV * DK + (size_t)v0 * DK;
        for (int idx = tid; idx < BV * PR; idx += NCT) {
          const int r = idx / PR, cc = (idx % PR) * VEC;
          *(uint4*)(dst + (size_t)r * DK + cc) = *(const uint4*)&sm.S[r][cc];
        }
      }
    } else {
      // Q of chunk c+NA-1 (its ring slot was freed at B_a) and P of chunk
      // c+NP-1 (its buffer was last read in the previous phase 4); then set B
      // of chunk c must have landed
      const bool q_next = c + NA - 1 < nch, p_next = c + R::NP - 1 < nch;
      if (q_next) issueQ(c + NA - 1);
      if (p_next) issueP(c + R::NP - 1);
      if constexpr (MAPS) {
        // set B of chunk c was issued before Q of chunk c+1
        if (q_next) wait_vm<R::LQ>();
        else wait_vm<0>();
      } else {
        if (q_next && p_next) wait_vm<R::LQ + R::LP>();
        else if (p_next) wait_vm<R::LP>();
        else wait_vm<0>();
      }
    }
    block_sync_lds();                      // B_b: Y staged; set B of chunk c visible
    // ---- phase 3
    if (!producer) {
      // D^T (value rows, chunk columns 16 cb..) = (V + Y)^T T^T as two
      // products; T is lower triangular (k blocks past this wave's rows are zero)
      const float kbr = __expf(gb[C - 1] - gb[rr]);
#pragma unroll
      for (int jn = 0; jn < NBW; ++jn) {
        const int nb = nb0 + jn;
        f4 d = zero4();
#pragma unroll
        for (int ks = 0; ks < C / KS; ++ks)
          if (keep_kblock<E>(ks * KS <= 16 * cb + 15)) {
            const FR tB = tile_frag<E, R::RC>(sm.ringB + R::BT, 16 * cb, ks * KS, lane);
            if (!map_tile)   // the map rows see no values
              d = Mma<E>::mma(tile_tr_frag<E, R::RO>(sm.ringB + R::BV_, ks * KS, nb * 16, lane), tB, d);
            d = Mma<E>::mma(tr_frag<E>(&sm.Y[0][0], LV, ks * KS, nb * 16, lane), tB, d);
          }
        f4 dk;
#pragma unroll
        for (int j = 0; j < 4; ++j) dk[j] = kbr * d[j];
        *(QR*)&sm.D[rr][nb * 16 + frow(lane, 0)] = Quad<E>::pack(d);
        *(QR*)&sm.Dk[rr][nb * 16 + frow(lane, 0)] = Quad<E>::pack(dk);
      }
      if (with_o && c > cbeg) store_O(c - 1);
    } else {
      // K and gates of chunk c+NA-1; then P of chunk c must have landed
      const bool k_next = c + NA - 1 < nch;
      if (k_next) issueK(c + NA - 1);
      if constexpr (MAPS) {
        // no P to wait for
      } else if constexpr (R::NP == 1) {
        // issued in this chunk's phase 2: only the K loads follow
        if (!k_next) wait_vm<0>();
        else if (prod < 3) wait_vm<R::LK + 1>();
        else wait_vm<R::LK>();
      } else if (c > cbeg) {
        // issued in the previous phase 2; followed by K of chunk c+1, set B
        // of chunk c, Q of chunk c+2, P of chunk c+1 and K of chunk c+2
        if (k_next) {
          if (prod < 3) wait_vm<R::LB + R::LQ + R::LP + 2 * (R::LK + 1)>();
          else wait_vm<R::LB + R::LQ + R::LP + 2 * R::LK>();
        } else if (c + 1 < nch) {
          if (prod < 3) wait_vm<R::LB + R::LP + R::LK + 1>();
          else wait_vm<R::LB + R::LP + R::LK>();
        } else {
          wait_vm<R::LB>();
        }
      }
    }
    block_sync_lds();                      // B_c: D staged; P visible; set B of chunk c free
    // ---- phase 4
    if (!producer) {
      if (with_o) {
        // O^T (value rows, chunk columns 16 cb..) = g_r (S Q^T) + D^T P^T; P
        // is causal (k blocks past this wave's rows are zero)
#pragma unroll
        for (int jn = 0; jn < NBW; ++jn) {
          const int nb = nb0 + jn;
          f4 o = sq[jn];
#pragma unroll
          for (int ks = 0; ks < C / KS; ++ks)
            if (keep_kblock<E>(ks * KS <= 16 * cb + 15))
              o = Mma<E>::mma(tr_frag<E>(&sm.D[0][0], LV, ks * KS, nb * 16, lane),
                              tile_frag<E, R::RC>(sm.Pt[c % R::NP], 16 * cb, ks * KS, lane), o);
          *(QR*)&sm.O[rr][nb * 16 + frow(lane, 0)] = Quad<E>::pack(o);
        }
      }
      // S^T <- g_C S^T + K^T diag(g_C/g) D  (K^T fragments are transpose reads of the K tile)
      const float gC = __expf(gb[C - 1]);
#pragma unroll
      for (int i = 0; i < KPW; ++i)
#pragma unroll
        for (int j = 0; j < NBS; ++j) acc[i][j] = gC * acc[i][j];
#pragma unroll
      for (int ks = 0; ks < C / KS; ++ks) {
        FR ka[KPW];
#pragma unroll
        for (int i = 0; i < KPW; ++i) ka[i] = tile_tr_frag<E, R::RK>(ra + R::AK, ks * KS, 16 * (kb0 + i), lane);
#pragma unroll
        for (int j = 0; j < NBS; ++j) {
          const FR bf = tr_frag<E>(&sm.Dk[0][0], LV, ks * KS, (ns0 + j) * 16, lane);
#pragma unroll
          for (int i = 0; i < KPW; ++i) acc[i][j] = Mma<E>::mma(ka[i], bf, acc[i][j]);
        }
      }
      stage_S();
      if (saved) {
        // D rows of this tile into the saved context (rows past the chunk are
        // zero), whose 32-column tiles are contiguous C x 32 blocks: each
        // workgroup writes whole blocks
        constexpr int VEC = 16 / sizeof(E), PR = BV / VEC, PT = 32 / VEC;
        E* dbase = (E*)p.savedD + gi * C * DV + (size_t)v0 * C;
        for (int idx = tid; idx < C * PR; idx += NCT) {
          const int sub = idx / (C * PT), r = (idx / PT) % C, cc = (idx % PT) * VEC;
          *(uint4*)(dbase + (size_t)sub * C * 32 + (size_t)r * 32 + cc) = *(const uint4*)&sm.D[r][sub * 32 + cc];
        }
      }
    } else if (c + 1 < nch) {
      issueB(c + 1);
      // set A of chunk c+1 complete: what was issued after its last part may
      // still be in flight
      if constexpr (NA == 2) {
        if (MAPS && map_tile) wait_vm<LT>();
        else wait_vm<R::LB>();
      } else {
        if (c == cbeg) {
          // set A of chunk 1 came with the prologue, which waited for it
        } else if (c + 2 < nch) {
          if (prod < 3) wait_vm<2 * R::LB + R::LQ + R::LP + R::LK + 1>();
          else wait_vm<2 * R::LB + R::LQ + R::LP + R::LK>();
        } else {
          wait_vm<2 * R::LB + R::LP>();
        }
      }
    }
  }
  block_sync_lds();                        // output of the last chunk staged
  if (producer) {
    wait_vm<0>();
  } else {
    if (with_o && nch > cbeg) store_O(nch - 1);
    if (SEG == SEG_MAPS) {
      // the segment's B (value rows) and A (map rows): [su][DV + DK][DK]
#pragma unroll
      for (int i = 0; i < KPW; ++i)
#pragma unroll
        for (int j = 0; j < NBS; ++j) {
          const int kt = kb0 + i, nb = ns0 + j;
          *(f4*)(p.wSegOut + ((size_t)su * (DV + DK) + r0 + nb * 16 + fcol(lane)) * DK + kt * 16 +
                 frow(lane, 0)) = acc[i][j];
        }
    } else if (p.Sfin && (SEG == SEG_NONE || g == nseg - 1)) {
#pragma unroll
      for (int i = 0; i < KPW; ++i)
#pragma unroll
        for (int j = 0; j < NBS; ++j) {
          const int kt = kb0 + i, nb = ns0 + j;
          *(f4*)(p.Sfin + ((size_t)unit * DV + v0 + nb * 16 + fcol(lane)) * DK + kt * 16 + frow(lane, 0)) =
              acc[i][j];
        }
    }
  }
}

// ------------------------------------------------------------------ launchers
template <typename E, int DK, int DV>
static hipError_t launch_fwd_t(const Params& p, int in_bwd, int with_scan, hipStream_t st) {
  if (p.n_slots > 0) {
    const int units = p.n_slots * p.H;
    // persistent four-wave workgroups, as many per CU as fit
    dim3 gp(min(units, prep_per_cu<E, DK>() * device_cu_count()));
    const int stage = in_bwd ? ST_PREP_BWD : ST_PREP_FWD;
    prof_mark(stage, 0, st);
    hipLaunchKernelGGL((k_prep<E, DK, DV>), gp, dim3(PREP_THREADS), 0, st, p);
    prof_mark(stage, 1, st);
  }
  if (with_scan) {
    const int units = p.N * p.H;
    const int bv = scan_bv<E, DV>(units);
    const int nb = ((units + 7) / 8) * 8 * (DV / bv);
    if (nb > 0) {
      prof_mark(ST_SCAN_FWD, 0, st);
      // bf16: eight compute waves (two per SIMD, each with half of the LDS
      // reads of a chunk); fp32: four
      constexpr int NCW = sizeof(E) == 2 ? 8 : 4;
      if constexpr (scan_bv_max<E, DV>() == 64) {
        if (bv == 64)
          hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, 64, NCW, SEG_NONE>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
        else
          hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, 32, NCW, SEG_NONE>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
      } else {
        hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, 32, NCW, SEG_NONE>), dim3(nb), dim3(NCW * 64 + 256), 0, st, p);
      }
      prof_mark(ST_SCAN_FWD, 1, st);
    }
  }
  return hipGetLastError();
}

// Entry states of the segments of every (sequence, head): S_0 = the initial
// state (or zero), S_{g+1} = S_g A_g + B_g with segment g's map from the
// SEG_MAPS pass, in fp32.  One workgroup per (sequence, head, 8 value rows)
// walks the segments in order: each step stages A_g in LDS (coalesced
// 16-byte loads, issued one step ahead so that their latency overlaps the
// previous step), then every thread forms one column of its rows from LDS.
constexpr int SEG_COMPOSE_RB = 8;
template <int DK, int DV>
__global__ __launch_bounds__(NTHREADS) void k_seg_compose(Params p) {
  constexpr int RB = SEG_COMPOSE_RB;           // value rows per workgroup
  constexpr int RPT = RB * DK / NTHREADS;      // rows per thread (one column each)
  constexpr int TPR = NTHREADS / DK;           // threads per column
  constexpr int AV = DK * DK / 4 / NTHREADS;   // float4 loads of A per thread
  static_assert(RB * DK % NTHREADS == 0 && NTHREADS % DK == 0 && AV * 4 * NTHREADS == DK * DK,
                "thread mapping");
  __shared__ __align__(16) float Am[DK][DK];
  __shared__ __align__(16) float Srow[RB][DK];
  const int nrb = DV / RB;
  const int unit = blockIdx.x / nrb, rb = blockIdx.x % nrb, tid = threadIdx.x;
  const int G = p.n_seg;
  const int k = tid % DK, rsub = tid / DK;     // column k; rows rsub, rsub + TPR, ...
  float cur[RPT], bn[RPT];
  f4 av[AV];
  // map g's A (registers) and B rows of this thread, loaded one step ahead
  auto fetch = [&](int g) {
    const float* Bm = p.wSegOut + ((size_t)unit * G + g) * (DV + DK) * DK;
    const f4* Ag = (const f4*)(Bm + (size_t)DV * DK);
#pragma unroll
    for (int i = 0; i < AV; ++i) av[i] = Ag[tid + i * NTHREADS];
#pragma unroll
    for (int m = 0; m < RPT; ++m) bn[m] = Bm[(size_t)(rb * RB + rsub + m * TPR) * DK + k];
  };
#pragma unroll
  for (int m = 0; m < RPT; ++m) {
    const int v = rb * RB + rsub + m * TPR;
    cur[m] = p.S0 ? p.S0[((size_t)unit * DV + v) * DK + k] : 0.f;
  }
  if (G > 1) fetch(0);
  for (int g = 0; g < G; ++g) {
    const size_t su = (size_t)unit * G + g;
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
      const int v = rb * RB + rsub + m * TPR;
      p.wSegIn[(su * DV + v) * DK + k] = cur[m];
      Srow[rsub + m * TPR][k] = cur[m];
    }
    if (g + 1 == G) break;
#pragma unroll
    for (int i = 0; i < AV; ++i) ((f4*)&Am[0][0])[tid + i * NTHREADS] = av[i];
#pragma unroll
    for (int m = 0; m < RPT; ++m) cur[m] = bn[m];
    if (g + 2 < G) fetch(g + 1);                 // in flight during this step
    __syncthreads();
    // next entry: rows of S_g A_g + B_g (four state columns per LDS read)
#pragma unroll 4
    for (int r = 0; r < DK; r += 4) {
      const float a0 = Am[r][k], a1 = Am[r + 1][k], a2 = Am[r + 2][k], a3 = Am[r + 3][k];
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const f4 sr = *(const f4*)&Srow[rsub + m * TPR][r];
        cur[m] += sr[0] * a0 + sr[1] * a1 + sr[2] * a2 + sr[3] * a3;
      }
    }
    __syncthreads();                           // Am and Srow are rewritten in the next step
  }
}

// Segment-parallel forward (dense batch): preparation, the maps of every
// segment (from zero), their composition into segment entry states, and the
// outputs pass of every segment from its entry state.  The maps pass takes
// the widest value tiles (it has (DV + DK) / BV of them per segment, and
// wider tiles re-read the operands their segment shares fewer times); the
// outputs pass takes them too once they still give every CU a workgroup.
template <typename E, int DK, int DV>
static hipError_t launch_fwd_seg_t(const Params& p, hipStream_t st) {
  hipError_t e = launch_fwd_t<E, DK, DV>(p, 0, 0, st);    // preparation only
  if (e != hipSuccess) return e;
  const int units = p.N * p.H;
  if (units == 0) return hipSuccess;
  constexpr int NCW = sizeof(E) == 2 ? 8 : 4;
  constexpr int BW = scan_bv_max<E, DV>();     // 64 for bf16, else 32
  const int su8 = ((units * p.n_seg + 7) / 8) * 8;
  const bool out_wide = BW == 64 && (long long)units * p.n_seg * (DV / 64) >= device_cu_count();
  prof_mark(ST_SEG_MAPS, 0, st);
  hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, BW, NCW, SEG_MAPS>), dim3(su8 * (DV + DK) / BW),
                     dim3(NCW * 64 + 256), 0, st, p);
  prof_mark(ST_SEG_MAPS, 1, st);
  prof_mark(ST_SEG_COMPOSE, 0, st);
  hipLaunchKernelGGL((k_seg_compose<DK, DV>), dim3(units * (DV / SEG_COMPOSE_RB)), dim3(NTHREADS), 0, st, p);
  prof_mark(ST_SEG_COMPOSE, 1, st);
  prof_mark(ST_SEG_OUT, 0, st);
  if (out_wide)
    hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, BW, NCW, SEG_OUT>), dim3(su8 * DV / BW), dim3(NCW * 64 + 256), 0,
                       st, p);
  else
    hipLaunchKernelGGL((k_scan_fwd<E, DK, DV, 32, NCW, SEG_OUT>), dim3(su8 * DV / 32), dim3(NCW * 64 + 256), 0,
                       st, p);
  prof_mark(ST_SEG_OUT, 1, st);
  return hipGetLastError();
}

hipError_t launch_fwd_seg(const Params& p, int dtype, int Dk, int Dv, hipStream_t st) {
#define QD_CASE(ET, DKV, DVV) \
  if (Dk == DKV && Dv == DVV) return launch_fwd_seg_t<ET, DKV, DVV>(p, st);
  if (dtype == 1) {
    QD_CASE(__bf16, 64, 64) QD_CASE(__bf16, 64, 128) QD_CASE(__bf16, 64, 256)
    QD_CASE(__bf16, 128, 64) QD_CASE(__bf16, 128, 128) QD_CASE(__bf16, 128, 256)
  } else {
    QD_CASE(float, 64, 64) QD_CASE(float, 64, 128) QD_CASE(float, 64, 256)
  }
#undef QD_CASE
  return hipErrorInvalidValue;
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
