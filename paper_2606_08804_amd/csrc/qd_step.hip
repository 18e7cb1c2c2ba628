// Single-token Q-Delta update for N sequences (decode), Sec. 3.3
// Eq. (qdelta_decay) applied once per (sequence, head):
//
//   x = k + lambda q;  p = S x;  S <- alpha S + beta (v - alpha p) k^T;  o = S q
//
// Each state row S[v, :] is independent, so a row is owned by a group of
// Dk/4 lanes (one float4 each): the state is read once and written once with
// fully coalesced 16-byte accesses, and the two row dot products are reduced
// with DPP lane moves (one shuffle across rows of 16).  The kernel is bound by
// HBM (or MALL) bandwidth.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

// Sum over each aligned group of L = 16 or 32 lanes: DPP within rows of 16
// lanes, then one cross-row exchange for 32.
template <int L>
__device__ inline float row_sum(float x) {
  static_assert(L == 16 || L == 32, "lane group of 16 or 32");
  x = sum16(x);
  if (L == 32) x += __shfl_xor(x, 16, 64);
  return x;
}

// Each lane group owns RPT state rows RPB apart (RPB = rows per workgroup
// pass), so a wave has RPT independent 16-byte loads in flight instead of
// one; the per-row dot products are reduced side by side.
constexpr int STEP_RPT = 4;

template <typename E, int DK>
__global__ __launch_bounds__(NTHREADS) void k_step(int DV, int nrb, const E* __restrict__ q,
                                                  const E* __restrict__ k, const E* __restrict__ v,
                                                  const float* __restrict__ beta,
                                                  const float* __restrict__ lam, float lam_c,
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
  const float lm = lam ? lam[u] : lam_c, bt = beta[u];
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
  for (int i = 0; i < RPT; ++i) px[i] = row_sum<LPR>(px[i]);
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
  for (int i = 0; i < RPT; ++i) oq[i] = row_sum<LPR>(oq[i]);
  if ((tid % LPR) == 0) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int row = row0 + i * RPB;
      if (row < DV) o[u * DV + row] = fromf<E>(oq[i]);
    }
  }
}

hipError_t launch_step(int N, int H, int Dk, int Dv, int dtype, const void* q, const void* k,
                       const void* v, const float* beta, const float* lam, float lam_c, const float* la,
                       float* state, void* o, hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int RPB = NTHREADS / (Dk / 4) * STEP_RPT;   // state rows per workgroup
  const int nrb = (Dv + RPB - 1) / RPB;
  dim3 grid((unsigned)((size_t)N * H * nrb));
#define QD_STEP(ET, DKV)                                                                        \
  hipLaunchKernelGGL((k_step<ET, DKV>), grid, dim3(NTHREADS), 0, st, Dv, nrb, (const ET*)q,     \
                     (const ET*)k, (const ET*)v, beta, lam, lam_c, la, state, (ET*)o)
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

// Fully recurrent forward over whole sequences (Sec. 3.3, Eq. (qdelta_decay)
// token by token; the paper offers this form beside the chunkwise one).
//
// A state row is owned by a group of LPR = 8 lanes, each holding Dk/8
// columns, so both per-token row dot products reduce in three DPP steps;
// the NT/8 lane groups of a workgroup hold RPT rows each in registers for
// the whole sequence: the state is read once (initial state or zero) and
// written once (final state).  Both row dot products use the state before
// the update (o_t = alpha S_{t-1} q + e (k . q)), so they reduce side by
// side, and the decay multiplies a scale instead of every element (the rows
// are held as true state / scale, folded back once per block), so the
// update is one FMA per element.  Tokens are processed in blocks of
// TB: the block's q, k, v slice and gates are staged in LDS (two buffers;
// block b + 1 is loaded into registers while block b is computed, then
// written to the other buffer), so each token reads LDS, not HBM.
// Sequence n of unit u = n * H + h spans tokens [cu[n], cu[n+1]) when cu is
// given (clamped to [0, T_total]), else [n * T, (n + 1) * T); token t of head
// h sits at row t * H + h of the activations and gates.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Sum over each aligned group of 8 lanes, result in every lane of the group,
// with DPP lane moves (no LDS round trip): lanes xor 1 and xor 2 (quad permutations [1,0,3,2] and [2,3,0,1]) give each
// quad its total; the half-row mirror (lane i <-> 7 - i within 8) then adds
// the other quad's total.
__device__ inline float group8_sum(float x) {
  x += dpp_mov<0xB1>(x);
  x += dpp_mov<0x4E>(x);
  x += dpp_mov<0x141>(x);
  return x;
}

template <typename E, int DK, int RPT, int NT>
__global__ __launch_bounds__(NT) void k_rec_fwd(
    int T, int H, int DV, int nrb, const int* __restrict__ cu, int T_total, const E* __restrict__ q,
    const E* __restrict__ k, const E* __restrict__ v, const float* __restrict__ beta,
    const float* __restrict__ lam, float lam_c, const float* __restrict__ la, const float* __restrict__ S0,
    float* __restrict__ Sfin, E* __restrict__ o) {
  constexpr int LPR = 8;                       // lanes per state row (group8_sum)
  constexpr int CPL = DK / LPR;                // columns per lane
  constexpr int NG = NT / LPR;                 // lane groups (rows per pass)
  constexpr int R = NG * RPT;                  // state rows per workgroup
  constexpr int TB = 16;                       // tokens per staged block
  constexpr int EPP = 16 / (int)sizeof(E);     // elements per 16-byte piece
  constexpr int QKP = TB * DK / EPP;           // pieces of one block of q (or k)
  constexpr int VP = TB * R / EPP;             // pieces of one block of v
  constexpr int QKT = (QKP + NT - 1) / NT;
  constexpr int VT = (VP + NT - 1) / NT;
  static_assert(CPL % 4 == 0, "columns per lane");
  __shared__ __align__(16) E qs[2][TB * DK];
  __shared__ __align__(16) E ks[2][TB * DK];
  __shared__ __align__(16) E vs[2][TB * R];
  __shared__ float gs[2][3 * TB];

  const int u = blockIdx.x / nrb;              // (sequence, head) unit
  const int rb = blockIdx.x % nrb;
  const int n = u / H, h = u % H;
  const int tid = threadIdx.x;
  const int grp = tid / LPR;
  const int c0 = (tid % LPR) * CPL;
  int t0, t1;
  if (cu) {
    t0 = min(max(cu[n], 0), T_total);
    t1 = min(max(cu[n + 1], t0), T_total);
  } else {
    t0 = n * T;
    t1 = t0 + T;
  }
  float s[RPT][CPL];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int row = rb * R + grp + i * NG;
#pragma unroll
    for (int j = 0; j < CPL; j += 4) {
      f4 x = zero4();
      if (S0 && row < DV) x = *(const f4*)(S0 + ((size_t)u * DV + row) * DK + c0 + j);
      s[i][j] = x[0]; s[i][j + 1] = x[1]; s[i][j + 2] = x[2]; s[i][j + 3] = x[3];
    }
  }

  // staging registers of one block
  u32x4 rq[QKT], rk[QKT], rv[VT];
  float rg = 0.f;
  auto load_block = [&](int tb) {
#pragma unroll
    for (int j = 0; j < QKT; ++j) {
      const int idx = tid + j * NT;
      rq[j] = u32x4{0, 0, 0, 0};
      rk[j] = u32x4{0, 0, 0, 0};
      const int t = tb + idx / (DK / EPP);
      if (idx < QKP && t < t1) {
        const size_t off = ((size_t)t * H + h) * DK + (size_t)(idx % (DK / EPP)) * EPP;
        rq[j] = *(const u32x4*)(q + off);
        rk[j] = *(const u32x4*)(k + off);
      }
    }
#pragma unroll
    for (int j = 0; j < VT; ++j) {
      const int idx = tid + j * NT;
      rv[j] = u32x4{0, 0, 0, 0};
      const int t = tb + idx / (R / EPP);
      const int row = rb * R + (idx % (R / EPP)) * EPP;   // DV is a multiple of 8: a piece is all in or all out
      if (idx < VP && t < t1 && row < DV) rv[j] = *(const u32x4*)(v + ((size_t)t * H + h) * DV + row);
    }
    rg = 0.f;
    if (tid < 3 * TB) {
      const int which = tid / TB, t = tb + tid % TB;
      const float* src = which == 0 ? beta : which == 1 ? lam : la;
      if (src && t < t1) rg = src[(size_t)t * H + h];
      else if (which == 1 && t < t1) rg = lam_c;           // constant lambda
    }
  };
  auto store_block = [&](int buf) {
#pragma unroll
    for (int j = 0; j < QKT; ++j) {
      const int idx = tid + j * NT;
      if (idx < QKP) {
        *(u32x4*)(&qs[buf][idx * EPP]) = rq[j];
        *(u32x4*)(&ks[buf][idx * EPP]) = rk[j];
      }
    }
#pragma unroll
    for (int j = 0; j < VT; ++j) {
      const int idx = tid + j * NT;
      if (idx < VP) *(u32x4*)(&vs[buf][idx * EPP]) = rv[j];
    }
    if (tid < 3 * TB) gs[buf][tid] = rg;
  };

  float sc = 1.f;                              // true state = sc * s
  const int nblk = (t1 - t0 + TB - 1) / TB;
  if (nblk > 0) {
    load_block(t0);
    store_block(0);
  }
  __syncthreads();
  for (int b = 0; b < nblk; ++b) {
    const int buf = b & 1;
    const int tb = t0 + b * TB;
    const int nt = min(TB, t1 - tb);
    if (b + 1 < nblk) load_block(tb + TB);
    for (int tt = 0; tt < nt; ++tt) {
      float qv[CPL], kv[CPL];
      const float bt = gs[buf][tt], lm = gs[buf][TB + tt];
      const float al = la ? __expf(gs[buf][2 * TB + tt]) : 1.f;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        qv[j] = tof(qs[buf][tt * DK + c0 + j]);
        kv[j] = tof(ks[buf][tt * DK + c0 + j]);
      }
      // S_{t-1} k and S_{t-1} q of the stored rows (true state = sc * stored)
      float pk[RPT], pq[RPT], vr[RPT];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        float a0 = 0.f, a1 = 0.f, b0 = 0.f, b1 = 0.f;
#pragma unroll
        for (int j = 0; j < CPL; j += 2) {
          a0 += s[i][j] * kv[j];
          a1 += s[i][j + 1] * kv[j + 1];
          b0 += s[i][j] * qv[j];
          b1 += s[i][j + 1] * qv[j + 1];
        }
        pk[i] = a0 + a1;
        pq[i] = b0 + b1;
        vr[i] = tof(vs[buf][tt * R + grp + i * NG]);
      }
      float kq = 0.f;
#pragma unroll
      for (int j = 0; j < CPL; ++j) kq += kv[j] * qv[j];
      kq = group8_sum(kq);
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        pk[i] = group8_sum(pk[i]);
        pq[i] = group8_sum(pq[i]);
      }
      // S_t = alpha S_{t-1} + e k^T with e = beta (v - alpha S_{t-1} x), x = k + lambda q,
      // and o_t = S_t q = alpha S_{t-1} q + e (k . q)
      float oq[RPT], ev[RPT];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const float sq = sc * pq[i];
        const float e = bt * (vr[i] - al * (sc * pk[i] + lm * sq));
        oq[i] = al * sq + e * kq;
        ev[i] = e;
      }
      if (al >= 0x1p-6f) {               // decay folded into the scale: one FMA per element
        sc *= al;
        const float rs = 1.f / sc;
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          const float g = ev[i] * rs;
#pragma unroll
          for (int j = 0; j < CPL; ++j) s[i][j] += g * kv[j];
        }
      } else {                           // strong decay: explicit update, scale reset
        const float f = sc * al;
#pragma unroll
        for (int i = 0; i < RPT; ++i)
#pragma unroll
          for (int j = 0; j < CPL; ++j) s[i][j] = f * s[i][j] + ev[i] * kv[j];
        sc = 1.f;
      }
      if ((tid % LPR) == 0) {
        const size_t r = ((size_t)(tb + tt) * H + h) * DV;
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          const int row = rb * R + grp + i * NG;
          if (row < DV) o[r + row] = fromf<E>(oq[i]);
        }
      }
    }
    // fold the scale back in once per block: it stays >= 2^-96 (16 tokens of
    // alpha >= 2^-6), inside the normal fp32 range
#pragma unroll
    for (int i = 0; i < RPT; ++i)
#pragma unroll
      for (int j = 0; j < CPL; ++j) s[i][j] *= sc;
    sc = 1.f;
    if (b + 1 < nblk) store_block(buf ^ 1);   // the buffer read in block b - 1
    __syncthreads();
  }
  if (Sfin) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int row = rb * R + grp + i * NG;
      if (row < DV) {
#pragma unroll
        for (int j = 0; j < CPL; j += 4)
          *(f4*)(Sfin + ((size_t)u * DV + row) * DK + c0 + j) =
              f4{s[i][j], s[i][j + 1], s[i][j + 2], s[i][j + 3]};
      }
    }
  }
}

hipError_t launch_rec_fwd(int N, int T, const int* cu, int T_total, int H, int Dk, int Dv,
                          int dtype, const void* q, const void* k, const void* v,
                          const float* beta, const float* lam, float lam_c, const float* la,
                          const float* S0, float* Sfin, void* o, hipStream_t st) {
  if (N == 0) return hipSuccess;
  if (!((dtype == 1 || dtype == 0) && (Dk == 128 || Dk == 64))) return hipErrorInvalidValue;
  // 128 threads = 16 lane groups; up to eight rows per group, so one
  // workgroup holds up to 128 rows of a unit and a single round of
  // workgroups (two waves per SIMD) covers the whole grid at 64 x 16 units
  constexpr int NT = 128, NG = NT / 8;
  const int rpt = Dv > 4 * NG ? 8 : Dv > 2 * NG ? 4 : Dv > NG ? 2 : 1;
  const int nrb = (Dv + NG * rpt - 1) / (NG * rpt);
  dim3 grid((unsigned)((size_t)N * H * nrb));
#define QD_REC(ET, DKV, RPTV)                                                                   \
  hipLaunchKernelGGL((k_rec_fwd<ET, DKV, RPTV, NT>), grid, dim3(NT), 0, st, T, H, Dv, nrb, cu, \
                     T_total, (const ET*)q, (const ET*)k, (const ET*)v, beta, lam, lam_c, la,  \
                     S0, Sfin, (ET*)o)
#define QD_REC_R(ET, DKV)                                                    \
  if (rpt == 8) QD_REC(ET, DKV, 8); else if (rpt == 4) QD_REC(ET, DKV, 4);   \
  else if (rpt == 2) QD_REC(ET, DKV, 2); else QD_REC(ET, DKV, 1)
  prof_mark(ST_REC_FWD, 0, st);
  if (dtype == 1 && Dk == 128) { QD_REC_R(__bf16, 128); }
  else if (dtype == 1 && Dk == 64) { QD_REC_R(__bf16, 64); }
  else if (dtype == 0 && Dk == 128) { QD_REC_R(float, 128); }
  else { QD_REC_R(float, 64); }
  prof_mark(ST_REC_FWD, 1, st);
#undef QD_REC_R
#undef QD_REC
  return hipGetLastError();
}

}  // namespace qd
