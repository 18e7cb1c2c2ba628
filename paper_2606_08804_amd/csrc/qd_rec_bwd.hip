// Backward of the fully recurrent form (Sec. 3.3, Eq. (qdelta_decay) token
// by token; the paper ships kernels for both the recurrent and the chunkwise
// form).  The paper states no backward; this is the chain rule through
//
//   x_t = k_t + lambda_t q_t,  p_t = S_{t-1} x_t,  e_t = beta_t (v_t - alpha_t p_t),
//   S_t = alpha_t S_{t-1} + e_t k_t^T,  o_t = S_t q_t
//
// for L = <dO, o> + <dS_T, S_T>, with G_t the adjoint of S_t:
//
//   G_t   = G'_t + dO_t q_t^T            (G'_T = dS_T; G'_{t-1} = alpha_t G_t + dp_t x_t^T)
//   s_t   = G_t k_t,  dv_t = beta_t s_t,  dp_t = -alpha_t beta_t s_t
//   dbeta_t = (v_t - alpha_t p_t) . s_t
//   dlog alpha_t = alpha_t (<G_t, S_{t-1}> - beta_t p_t . s_t)
//   dx_t  = S_{t-1}^T dp_t,  dk_t = G_t^T e_t + dx_t,  dlambda_t = q_t . dx_t
//   dq_t  = S_t^T dO_t + lambda_t dx_t = alpha_t S_{t-1}^T dO_t + (dO_t . e_t) k_t + lambda_t dx_t
//   d S_0 = G'_0
//
// The reverse walk needs S_{t-1} only through <G_t, S_{t-1}> and the column
// sums S_{t-1}^T dp_t, S_{t-1}^T dO_t.  Per state row i the scalar
// F_{t,i} = <G_t[i,:], S_t[i,:]> obeys
//   alpha_t <G_t[i,:], S_{t-1}[i,:]> = F_{t,i} - e_{t,i} s_{t,i}
//   F_{t-1,i} = F_{t,i} - e_{t,i} s_{t,i} + dp_{t,i} p_{t,i} + dO_{t-1,i} o_{t-1,i}
// (F_T = <dS_T, S_T> + dO_T . o_T per row), so
//   dlog alpha_t = sum_i (F_{t,i} - e_{t,i} s_{t,i} + dp_{t,i} p_{t,i})
// needs no state at all, and the column sums are formed by a second forward
// sweep once dp is known.  One workgroup per (sequence, head) runs three
// sweeps over its tokens:
//   A (forward)  recompute the states; store p_t and z_t = dO_t * o_t per row, and F_T;
//   B (reverse)  carry G; write dv, dbeta, dlog alpha, dp_t and sum_i e_i G[i,:];
//   C (forward)  recompute the states (p_t read back from sweep A); the
//                column sums S^T dO, S^T dp and dO . e give dq, dk and dlambda.
// Every sweep has the layout of the recurrent forward: a state row is held
// by a group of 8 lanes (Dk / 8 columns each), 32 groups hold Dv / 32 rows
// each.  Row dot products reduce over the 8 lanes with DPP; sums over rows
// reduce in-lane over a group's rows, then over the 8 groups of a wave by a
// butterfly that leaves each lane Dk / 64 finished columns, then over the 4
// waves through LDS once per block of TB tokens, in a fixed order (the
// results are the same on every run).  Tokens are staged in LDS in blocks
// of TB, the next block loaded into registers while the current one is
// computed.
#include "qd_common.h"
#include "qd_launch.h"

namespace qd {

namespace {

typedef unsigned int rb_u32x4 __attribute__((ext_vector_type(4)));

constexpr int RB_NT = 256;        // threads: 4 waves, 32 row groups of 8 lanes
constexpr int RB_NG = RB_NT / 8;  // row groups
constexpr int RB_TB = 8;          // tokens per staged block

// Sum over each aligned group of 8 lanes, in every lane of the group.
__device__ inline float g8sum(float x) {
  x += dpp_mov<0xB1>(x);
  x += dpp_mov<0x4E>(x);
  x += dpp_mov<0x141>(x);
  return x;
}

// Sum over the 8 row groups of a wave (lane bits 3..5) of a value that all
// 8 lanes of each group hold.
__device__ inline float wave_groups_sum(float x) {
  x += __shfl_xor(x, 8, 64);
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

// Butterfly reduce-scatter of a CPL-vector (this lane's columns
// (lane & 7) * CPL ..) over the 8 row groups of a wave: afterwards the lane
// holds CPL / 8 finished columns starting at rs_col(lane).
template <int CPL>
__device__ inline void rs8(const float (&v)[CPL], float (&out)[CPL / 8], int lane) {
  float h1[CPL / 2], h2[CPL / 4];
  const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
#pragma unroll
  for (int e = 0; e < CPL / 2; ++e) {
    const float send = b5 ? v[e] : v[e + CPL / 2];
    const float keep = b5 ? v[e + CPL / 2] : v[e];
    h1[e] = keep + __shfl_xor(send, 32, 64);
  }
#pragma unroll
  for (int e = 0; e < CPL / 4; ++e) {
    const float send = b4 ? h1[e] : h1[e + CPL / 4];
    const float keep = b4 ? h1[e + CPL / 4] : h1[e];
    h2[e] = keep + __shfl_xor(send, 16, 64);
  }
#pragma unroll
  for (int e = 0; e < CPL / 8; ++e) {
    const float send = b3 ? h2[e] : h2[e + CPL / 8];
    const float keep = b3 ? h2[e + CPL / 8] : h2[e];
    out[e] = keep + __shfl_xor(send, 8, 64);
  }
}
template <int CPL>
__device__ inline int rs_col(int lane) {
  return (lane & 7) * CPL + ((lane & 32) ? CPL / 2 : 0) + ((lane & 16) ? CPL / 4 : 0) + ((lane & 8) ? CPL / 8 : 0);
}

// Register staging of one block of TB token rows of W bytes each (row t at
// base + t * stride); rows outside [lo, hi) read as zero.
template <int W>
struct Rows {
  static constexpr int PPR = W / 16;              // 16-byte pieces per row
  static constexpr int PCS = RB_TB * PPR;
  static constexpr int N = (PCS + RB_NT - 1) / RB_NT;
  rb_u32x4 r[N];
  __device__ inline void load(const char* base, size_t stride, int t_first, int lo, int hi, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * RB_NT;
      const int t = t_first + idx / PPR;
      r[i] = rb_u32x4{0, 0, 0, 0};
      if (idx < PCS && t >= lo && t < hi) r[i] = *(const rb_u32x4*)(base + (size_t)t * stride + (idx % PPR) * 16);
    }
  }
  __device__ inline void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * RB_NT;
      if (idx < PCS) *(rb_u32x4*)(lds + idx * 16) = r[i];
    }
  }
};

}  // namespace

template <typename E, int DK, int RPT>
struct alignas(16) RecBwdSmem {
  static constexpr int DVP = RPT * RB_NG;
  alignas(16) E q[2][RB_TB][DK];
  alignas(16) E k[2][RB_TB][DK];
  alignas(16) E v[2][RB_TB][DVP];
  alignas(16) E dO[2][RB_TB][DVP];
  alignas(16) float a[2][RB_TB][DVP];        // B: p_t;  C: dp_t
  alignas(16) float b[2][RB_TB][DVP];        // B: z_{t-1};  C: p_t
  alignas(16) float g[2][3][RB_TB];          // beta, lambda, log alpha
  float pv[RB_TB][4][2][DK];                 // per-wave column sums (B: e G; C: S^T dO, S^T dp)
  float ps[RB_TB][4][2];                     // per-wave row-scalar sums
};

template <typename E, int DK, int RPT>
__global__ __launch_bounds__(RB_NT) void k_rec_bwd(RecBwdArgs a) {
  constexpr int CPL = DK / 8;                // columns per lane
  constexpr int CPT = DK / 32;               // columns per thread in the block epilogue
  constexpr int EB = (int)sizeof(E);
  constexpr int DV = RPT * RB_NG;
  typedef RecBwdSmem<E, DK, RPT> SM;
  __shared__ SM sm;
  const int H = a.H, unit = blockIdx.x, n = unit / H, h = unit % H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, grp = tid >> 3, c = tid & 7, c0 = c * CPL;
  int t0, t1;
  if (a.cu) {
    t0 = min(max(a.cu[n], 0), a.T_total);
    t1 = min(max(a.cu[n + 1], t0), a.T_total);
  } else {
    t0 = n * a.T;
    t1 = t0 + a.T;
  }
  const int nblk = (t1 - t0 + RB_TB - 1) / RB_TB;
  const size_t rowK = (size_t)H * DK * EB, rowV = (size_t)H * DV * EB, rowF = (size_t)H * DV * 4;
  const char* qb = (const char*)a.q + (size_t)h * DK * EB;
  const char* kb = (const char*)a.k + (size_t)h * DK * EB;
  const char* vb = (const char*)a.v + (size_t)h * DV * EB;
  const char* ob = (const char*)a.dO + (size_t)h * DV * EB;
  auto row = [&](int m) { return grp + m * RB_NG; };
  auto fw = [&](float* base, int t, int i) { return base + ((size_t)t * H + h) * DV + i; };

  Rows<DK * EB> rq, rk;
  Rows<DV * EB> rv, ro;
  Rows<DV * 4> ra, rb2;
  float rg = 0.f;
  // stages the block starting at token tb; `sweep` selects the per-row
  // arrays (A: none; B: p_t and z_{t-1}; C: dp_t and p_t)
  auto load = [&](int tb, int sweep) {
    rq.load(qb, rowK, tb, t0, t1, tid);
    rk.load(kb, rowK, tb, t0, t1, tid);
    rv.load(vb, rowV, tb, t0, t1, tid);
    ro.load(ob, rowV, tb, t0, t1, tid);
    if (sweep == 1) {
      ra.load((const char*)a.wP + (size_t)h * DV * 4, rowF, tb, t0, t1, tid);
      rb2.load((const char*)a.wZ + (size_t)h * DV * 4, rowF, tb - 1, t0, t1 - 1, tid);   // z_{t-1}
    } else if (sweep == 2) {
      ra.load((const char*)a.wDP + (size_t)h * DV * 4, rowF, tb, t0, t1, tid);
      rb2.load((const char*)a.wP + (size_t)h * DV * 4, rowF, tb, t0, t1, tid);
    }
    rg = 0.f;
    if (tid < 3 * RB_TB) {
      const int which = tid / RB_TB, t = tb + tid % RB_TB;
      if (t < t1) {
        const float* src = which == 0 ? a.beta : which == 1 ? a.lam : a.la;
        rg = src ? src[(size_t)t * H + h] : (which == 1 ? a.lam_c : 0.f);
      }
    }
  };
  auto store = [&](int buf, int sweep) {
    rq.store((char*)&sm.q[buf][0][0], tid);
    rk.store((char*)&sm.k[buf][0][0], tid);
    rv.store((char*)&sm.v[buf][0][0], tid);
    ro.store((char*)&sm.dO[buf][0][0], tid);
    if (sweep >= 1) ra.store((char*)&sm.a[buf][0][0], tid);
    if (sweep >= 1) rb2.store((char*)&sm.b[buf][0][0], tid);
    if (tid < 3 * RB_TB) sm.g[buf][tid / RB_TB][tid % RB_TB] = rg;
  };
  // per-token operands of this lane: q, k, x = k + lambda q, and the gates
  float qv[CPL], kv[CPL], xv[CPL];
  float bt, lm, al;
  auto token = [&](int buf, int tt) {
    bt = sm.g[buf][0][tt];
    lm = sm.g[buf][1][tt];
    al = a.la ? __expf(sm.g[buf][2][tt]) : 1.f;
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      qv[j] = tof(sm.q[buf][tt][c0 + j]);
      kv[j] = tof(sm.k[buf][tt][c0 + j]);
      xv[j] = kv[j] + lm * qv[j];
    }
  };
  float st[RPT][CPL];          // A, C: the state rows S; B: the adjoint rows G
  auto load_state = [&](const float* src) {
#pragma unroll
    for (int m = 0; m < RPT; ++m)
#pragma unroll
      for (int j = 0; j < CPL; j += 4) {
        f4 x = zero4();
        if (src) x = *(const f4*)(src + ((size_t)unit * DV + row(m)) * DK + c0 + j);
        st[m][j] = x[0]; st[m][j + 1] = x[1]; st[m][j + 2] = x[2]; st[m][j + 3] = x[3];
      }
  };
  auto dot = [&](const float (&r)[CPL], const float (&u)[CPL]) {
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int j = 0; j < CPL; j += 2) {
      s0 += r[j] * u[j];
      s1 += r[j + 1] * u[j + 1];
    }
    return g8sum(s0 + s1);
  };
  // the value of row m held by this lane group's lane m (m < RPT <= 8)
  auto pick = [&](const float (&x)[RPT]) {
    float r = x[0];
#pragma unroll
    for (int m = 1; m < RPT; ++m)
      if (c == m) r = x[m];
    return r;
  };

  // ---------------- sweep A: states forward; p_t, z_t = dO_t o_t per row; F_T
  load_state(a.S0);
  float zl[RPT];
#pragma unroll
  for (int m = 0; m < RPT; ++m) zl[m] = 0.f;
  if (nblk > 0) {
    load(t0, 0);
    store(0, 0);
  }
  __syncthreads();
  for (int bk = 0; bk < nblk; ++bk) {
    const int buf = bk & 1, tb = t0 + bk * RB_TB, nt = min(RB_TB, t1 - tb);
    if (bk + 1 < nblk) load(tb + RB_TB, 0);
    for (int tt = 0; tt < nt; ++tt) {
      token(buf, tt);
      float pm[RPT], zm[RPT];
#pragma unroll
      for (int m = 0; m < RPT; ++m) pm[m] = dot(st[m], xv);
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const float e = bt * (tof(sm.v[buf][tt][row(m)]) - al * pm[m]);
#pragma unroll
        for (int j = 0; j < CPL; ++j) st[m][j] = al * st[m][j] + e * kv[j];
      }
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        zm[m] = tof(sm.dO[buf][tt][row(m)]) * dot(st[m], qv);
        zl[m] = zm[m];
      }
      if (c < RPT) {
        const int t = tb + tt;
        *fw(a.wP, t, row(c)) = pick(pm);
        *fw(a.wZ, t, row(c)) = pick(zm);
      }
    }
    if (bk + 1 < nblk) store(buf ^ 1, 0);
    __syncthreads();
  }
  {
    // F_T = <dS_T, S_T> + dO_T . o_T per row
    float fm[RPT];
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
      float d[CPL];
#pragma unroll
      for (int j = 0; j < CPL; j += 4) {
        f4 x = zero4();
        if (a.dSfin) x = *(const f4*)(a.dSfin + ((size_t)unit * DV + row(m)) * DK + c0 + j);
        d[j] = x[0]; d[j + 1] = x[1]; d[j + 2] = x[2]; d[j + 3] = x[3];
      }
      fm[m] = dot(st[m], d) + zl[m];
    }
    if (c < RPT) a.wF[(size_t)unit * DV + row(c)] = pick(fm);
  }
  __syncthreads();             // p, z and F visible to the whole workgroup

  // ---------------- sweep B: adjoint G in reverse
  load_state(a.dSfin);
  float F[RPT];
#pragma unroll
  for (int m = 0; m < RPT; ++m) F[m] = a.wF[(size_t)unit * DV + row(m)];
  if (nblk > 0) {
    load(t0 + (nblk - 1) * RB_TB, 1);
    store((nblk - 1) & 1, 1);
  }
  __syncthreads();
  for (int bk = nblk - 1; bk >= 0; --bk) {
    const int buf = bk & 1, tb = t0 + bk * RB_TB, nt = min(RB_TB, t1 - tb);
    if (bk > 0) load(tb - RB_TB, 1);
    for (int tt = nt - 1; tt >= 0; --tt) {
      token(buf, tt);
      const int t = tb + tt;
      float sm_[RPT], dpm[RPT], dvm[RPT], r1 = 0.f, r2 = 0.f;
      float wk[CPL];
#pragma unroll
      for (int j = 0; j < CPL; ++j) wk[j] = 0.f;
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const float dOi = tof(sm.dO[buf][tt][row(m)]);
#pragma unroll
        for (int j = 0; j < CPL; ++j) st[m][j] += dOi * qv[j];
        sm_[m] = dot(st[m], kv);
      }
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const float pv = sm.a[buf][tt][row(m)], s = sm_[m];
        const float u = tof(sm.v[buf][tt][row(m)]) - al * pv, e = bt * u, dp = -al * bt * s;
        dpm[m] = dp;
        dvm[m] = bt * s;
        r1 += u * s;
        r2 += F[m] - e * s + dp * pv;
        F[m] = F[m] - e * s + dp * pv + sm.b[buf][tt][row(m)];
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          wk[j] += e * st[m][j];
          st[m][j] = al * st[m][j] + dp * xv[j];
        }
      }
      if (c < RPT) {
        ((E*)a.dv)[((size_t)t * H + h) * DV + row(c)] = fromf<E>(pick(dvm));
        *fw(a.wDP, t, row(c)) = pick(dpm);
      }
      float part[CPL / 8];
      rs8<CPL>(wk, part, lane);
#pragma unroll
      for (int e = 0; e < CPL / 8; ++e) sm.pv[tt][w][0][rs_col<CPL>(lane) + e] = part[e];
      r1 = wave_groups_sum(r1);
      r2 = wave_groups_sum(r2);
      if (lane == 0) {
        sm.ps[tt][w][0] = r1;
        sm.ps[tt][w][1] = r2;
      }
    }
    __syncthreads();
    {
      // block epilogue: dbeta, dlog alpha and sum_i e_i G_i per token
      const int tt = tid >> 5, ci = tid & 31;
      if (tt < nt) {
        const int t = tb + tt;
        float* wk = a.wWK + ((size_t)t * H + h) * DK;
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          const int col = ci * CPT + e;
          wk[col] = ((sm.pv[tt][0][0][col] + sm.pv[tt][1][0][col]) + sm.pv[tt][2][0][col]) + sm.pv[tt][3][0][col];
        }
        if (ci == 0) {
          const size_t gt = (size_t)t * H + h;
          a.dbeta[gt] = ((sm.ps[tt][0][0] + sm.ps[tt][1][0]) + sm.ps[tt][2][0]) + sm.ps[tt][3][0];
          if (a.dla) a.dla[gt] = ((sm.ps[tt][0][1] + sm.ps[tt][1][1]) + sm.ps[tt][2][1]) + sm.ps[tt][3][1];
        }
      }
    }
    if (bk > 0) store(buf ^ 1, 1);
    __syncthreads();
  }
  if (a.dS0) {
#pragma unroll
    for (int m = 0; m < RPT; ++m)
#pragma unroll
      for (int j = 0; j < CPL; j += 4)
        *(f4*)(a.dS0 + ((size_t)unit * DV + row(m)) * DK + c0 + j) =
            f4{st[m][j], st[m][j + 1], st[m][j + 2], st[m][j + 3]};
  }
  __syncthreads();             // dp and the e G sums visible to the whole workgroup

  // ---------------- sweep C: states forward; S^T dO, S^T dp, dO . e
  load_state(a.S0);
  if (nblk > 0) {
    load(t0, 2);
    store(0, 2);
  }
  __syncthreads();
  for (int bk = 0; bk < nblk; ++bk) {
    const int buf = bk & 1, tb = t0 + bk * RB_TB, nt = min(RB_TB, t1 - tb);
    if (bk + 1 < nblk) load(tb + RB_TB, 2);
    for (int tt = 0; tt < nt; ++tt) {
      token(buf, tt);
      float w1[CPL], w2[CPL], cs = 0.f;
#pragma unroll
      for (int j = 0; j < CPL; ++j) w1[j] = w2[j] = 0.f;
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        // p_t = S_{t-1} x_t as sweep A computed it from the same states
        const float dOi = tof(sm.dO[buf][tt][row(m)]), dpi = sm.a[buf][tt][row(m)];
        const float e = bt * (tof(sm.v[buf][tt][row(m)]) - al * sm.b[buf][tt][row(m)]);
        cs += dOi * e;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          w1[j] += dOi * st[m][j];
          w2[j] += dpi * st[m][j];
          st[m][j] = al * st[m][j] + e * kv[j];
        }
      }
      float p1[CPL / 8], p2[CPL / 8];
      rs8<CPL>(w1, p1, lane);
      rs8<CPL>(w2, p2, lane);
#pragma unroll
      for (int e = 0; e < CPL / 8; ++e) {
        sm.pv[tt][w][0][rs_col<CPL>(lane) + e] = p1[e];
        sm.pv[tt][w][1][rs_col<CPL>(lane) + e] = p2[e];
      }
      cs = wave_groups_sum(cs);
      if (lane == 0) sm.ps[tt][w][0] = cs;
    }
    __syncthreads();
    {
      // block epilogue: dq, dk, dlambda per token
      const int tt = tid >> 5, ci = tid & 31;
      if (tt < nt) {
        const int t = tb + tt;
        const size_t gt = (size_t)t * H + h;
        const float lmt = sm.g[buf][1][tt];
        const float alt = a.la ? __expf(sm.g[buf][2][tt]) : 1.f;
        const float cst = ((sm.ps[tt][0][0] + sm.ps[tt][1][0]) + sm.ps[tt][2][0]) + sm.ps[tt][3][0];
        const float* wk = a.wWK + gt * DK;
        float dl = 0.f;
        E oq[CPT], ok[CPT];
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          const int col = ci * CPT + e;
          const float W1 = ((sm.pv[tt][0][0][col] + sm.pv[tt][1][0][col]) + sm.pv[tt][2][0][col]) + sm.pv[tt][3][0][col];
          const float W2 = ((sm.pv[tt][0][1][col] + sm.pv[tt][1][1][col]) + sm.pv[tt][2][1][col]) + sm.pv[tt][3][1][col];
          const float qc = tof(sm.q[buf][tt][col]), kc = tof(sm.k[buf][tt][col]);
          oq[e] = fromf<E>(alt * W1 + cst * kc + lmt * W2);
          ok[e] = fromf<E>(wk[col] + W2);
          dl += qc * W2;
        }
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          ((E*)a.dq)[gt * DK + ci * CPT + e] = oq[e];
          ((E*)a.dk)[gt * DK + ci * CPT + e] = ok[e];
        }
#pragma unroll
        for (int off = 1; off < 32; off <<= 1) dl += __shfl_xor(dl, off, 64);
        if (ci == 0) {
          if (a.dlam) a.dlam[gt] = dl;
          if (a.wDL) a.wDL[gt] = dl;
        }
      }
    }
    if (bk + 1 < nblk) store(buf ^ 1, 2);
    __syncthreads();
  }
}

// Sum of n floats in a fixed order (one workgroup: strided per-thread sums,
// then a tree), written to *out.
__global__ __launch_bounds__(NTHREADS) void k_sum_floats(const float* x, long long n, float* out) {
  __shared__ float part[NTHREADS];
  const int tid = threadIdx.x;
  float acc = 0.f;
  for (long long i = tid; i < n; i += NTHREADS) acc += x[i];
  part[tid] = acc;
  __syncthreads();
#pragma unroll
  for (int off = NTHREADS / 2; off >= 1; off >>= 1) {
    if (tid < off) part[tid] += part[tid + off];
    __syncthreads();
  }
  if (tid == 0) *out = part[0];
}

hipError_t launch_rec_bwd(const RecBwdArgs& a, int units, int dtype, int Dk, float* dlam_sum, long long n_tok_heads,
                          hipStream_t st) {
  if (units > 0) {
    const int rpt = a.DV / RB_NG;
#define QD_RB(ET, DKV, R) \
  hipLaunchKernelGGL((k_rec_bwd<ET, DKV, R>), dim3(units), dim3(RB_NT), 0, st, a)
#define QD_RB_R(ET, DKV)                                            \
  if (rpt == 8) QD_RB(ET, DKV, 8); else if (rpt == 4) QD_RB(ET, DKV, 4); \
  else if (rpt == 2) QD_RB(ET, DKV, 2); else QD_RB(ET, DKV, 1)
    prof_mark(ST_REC_BWD, 0, st);
    if (dtype == 1 && Dk == 128) { QD_RB_R(__bf16, 128); }
    else if (dtype == 1 && Dk == 64) { QD_RB_R(__bf16, 64); }
    else if (dtype == 0 && Dk == 128) { QD_RB_R(float, 128); }
    else { QD_RB_R(float, 64); }
    prof_mark(ST_REC_BWD, 1, st);
#undef QD_RB_R
#undef QD_RB
  }
  if (dlam_sum) hipLaunchKernelGGL(k_sum_floats, dim3(1), dim3(NTHREADS), 0, st, a.wDL, n_tok_heads, dlam_sum);
  return hipGetLastError();
}

}  // namespace qd
