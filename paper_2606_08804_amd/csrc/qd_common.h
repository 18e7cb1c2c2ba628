// Shared device-side building blocks of the Q-Delta HIP kernels (gfx950).
//
//  * MFMA traits: bf16 operands use v_mfma_f32_16x16x32_bf16, fp32 operands
//    v_mfma_f32_16x16x4_f32; both accumulate in fp32.  Lane layouts (wave64):
//      A (16 x K)  lane l holds row l%16, k = KPL*(l/16) .. +KPL-1
//      B (K x 16)  lane l holds col l%16, k = KPL*(l/16) .. +KPL-1
//      C (16 x 16) lane l holds col l%16, rows 4*(l/16) .. +3
//  * Operand views over LDS (or global) matrices, in either storage order.
//  * Chunk/sequence mapping for dense and packed (cu_seqlens) batches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qd {

constexpr int C = 64;          // chunk length (tokens)
constexpr int NTHREADS = 256;  // 4 wave64s per workgroup
constexpr int NWAVES = NTHREADS / 64;

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf4 __attribute__((ext_vector_type(4)));

// ----------------------------------------------------------------- MFMA traits
template <typename E> struct Mma;

template <> struct Mma<__bf16> {
  static constexpr int KS = 32;   // k per instruction
  static constexpr int KPL = 8;   // k values per lane
  typedef bf8 frag;
  __device__ static inline f4 mma(frag a, frag b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  static constexpr int KS = 4;
  static constexpr int KPL = 1;
  typedef float frag;
  __device__ static inline f4 mma(frag a, frag b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

__device__ inline float tof(float x) { return x; }
__device__ inline float tof(__bf16 x) { return (float)x; }
template <typename E> __device__ inline E fromf(float x);
template <> __device__ inline float fromf<float>(float x) { return x; }
template <> __device__ inline __bf16 fromf<__bf16>(float x) { return (__bf16)x; }

// Row padding (elements) that keeps 16-byte alignment and spreads rows over
// LDS banks: rows of 16*(D/8)+16 bytes (bf16) or 4*D+16 bytes (fp32).
template <typename E> struct Pad { static constexpr int v = 16 / sizeof(E); };

// ----------------------------------------------------------------- operand views
// KMaj: element (i, k) at p[i*ld + k]   (k contiguous)
// IMaj: element (i, k) at p[k*ld + i]   (i contiguous)
// "i" is the row of an A operand or the column of a B operand.
template <typename S> struct KMaj { const S* p; int ld; };
template <typename S> struct IMaj { const S* p; int ld; };

template <typename S> __device__ inline KMaj<S> kmaj(const S* p, int ld) { return KMaj<S>{p, ld}; }
template <typename S> __device__ inline IMaj<S> imaj(const S* p, int ld) { return IMaj<S>{p, ld}; }

template <typename E> struct Frag;

template <> struct Frag<__bf16> {
  __device__ static inline bf8 load(KMaj<__bf16> v, int i0, int k0, int lane) {
    return *(const bf8*)(v.p + (size_t)(i0 + (lane & 15)) * v.ld + k0 + (lane >> 4) * 8);
  }
  __device__ static inline bf8 load(KMaj<float> v, int i0, int k0, int lane) {
    const float* s = v.p + (size_t)(i0 + (lane & 15)) * v.ld + k0 + (lane >> 4) * 8;
    f4 a = *(const f4*)s, b = *(const f4*)(s + 4);
    bf8 r;
    r[0] = (__bf16)a[0]; r[1] = (__bf16)a[1]; r[2] = (__bf16)a[2]; r[3] = (__bf16)a[3];
    r[4] = (__bf16)b[0]; r[5] = (__bf16)b[1]; r[6] = (__bf16)b[2]; r[7] = (__bf16)b[3];
    return r;
  }
  template <typename S>
  __device__ static inline bf8 load(IMaj<S> v, int i0, int k0, int lane) {
    const S* s = v.p + (size_t)(k0 + (lane >> 4) * 8) * v.ld + i0 + (lane & 15);
    bf8 r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = (__bf16)tof(s[(size_t)j * v.ld]);
    return r;
  }
};

template <> struct Frag<float> {
  template <typename S>
  __device__ static inline float load(KMaj<S> v, int i0, int k0, int lane) {
    return tof(v.p[(size_t)(i0 + (lane & 15)) * v.ld + k0 + (lane >> 4)]);
  }
  template <typename S>
  __device__ static inline float load(IMaj<S> v, int i0, int k0, int lane) {
    return tof(v.p[(size_t)(k0 + (lane >> 4)) * v.ld + i0 + (lane & 15)]);
  }
};

// acc += A[m0:m0+16, 0:K] * B[0:K, n0:n0+16]
template <typename E, int K, typename AV, typename BV>
__device__ inline f4 mma_k(AV a, BV b, int m0, int n0, f4 acc, int lane) {
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += Mma<E>::KS)
    acc = Mma<E>::mma(Frag<E>::load(a, m0, k0, lane), Frag<E>::load(b, n0, k0, lane), acc);
  return acc;
}

// Same with a run-time contraction length (multiple of KS).
template <typename E, typename AV, typename BV>
__device__ inline f4 mma_kn(AV a, BV b, int m0, int n0, int K, f4 acc, int lane) {
  for (int k0 = 0; k0 < K; k0 += Mma<E>::KS)
    acc = Mma<E>::mma(Frag<E>::load(a, m0, k0, lane), Frag<E>::load(b, n0, k0, lane), acc);
  return acc;
}

__device__ inline f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }

// Row of C-fragment element j for this lane, relative to the tile origin.
__device__ inline int frow(int lane, int j) { return ((lane >> 4) << 2) + j; }
__device__ inline int fcol(int lane) { return lane & 15; }

// ----------------------------------------------------------------- tile loads
// Load rows [0, C) of a [*, ld_g] global matrix block (row stride `gs`
// elements, D columns) into LDS dst[r*ld + c], zero-filling rows >= len.
template <typename E, int D, int NT = NTHREADS>
__device__ inline void load_rows(E* dst, int ld, const E* src, size_t gs, int len, int tid) {
  constexpr int VEC = 16 / sizeof(E);
  constexpr int PR = D / VEC;
  for (int idx = tid; idx < C * PR; idx += NT) {
    const int r = idx / PR, c = (idx % PR) * VEC;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r < len) val = *(const uint4*)(src + (size_t)r * gs + c);
    *(uint4*)(dst + (size_t)r * ld + c) = val;
  }
}

// Same, storing the transpose: dst[c*ld + r] = scale(r) * src[r][c].
template <typename E, int D, typename Scale, int NT = NTHREADS>
__device__ inline void load_rows_t(E* dst, int ld, const E* src, size_t gs, int len, int tid,
                                   Scale scale) {
  constexpr int VEC = 16 / sizeof(E);
  constexpr int PR = D / VEC;
  for (int idx = tid; idx < C * PR; idx += NT) {
    const int r = idx % C, c = (idx / C) * VEC;   // consecutive threads -> consecutive rows
    E vals[VEC];
    if (r < len) {
      uint4 raw = *(const uint4*)(src + (size_t)r * gs + c);
      const E* pv = (const E*)&raw;
      const float s = scale(r);
#pragma unroll
      for (int j = 0; j < VEC; ++j) vals[j] = fromf<E>(tof(pv[j]) * s);
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) vals[j] = fromf<E>(0.f);
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) dst[(size_t)(c + j) * ld + r] = vals[j];
  }
}

struct One { __device__ float operator()(int) const { return 1.f; } };

// Four consecutive activation-dtype values of one lane's C fragment.
template <typename E> struct Quad;
template <> struct Quad<__bf16> {
  typedef uint2 raw;
  __device__ static inline float get(raw r, int j) {
    const __bf16* e = (const __bf16*)&r;
    return (float)e[j];
  }
  __device__ static inline raw pack(f4 x) {
    raw r;
    __bf16* e = (__bf16*)&r;
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] = (__bf16)x[j];
    return r;
  }
};
template <> struct Quad<float> {
  typedef uint4 raw;
  __device__ static inline float get(raw r, int j) { return ((const float*)&r)[j]; }
  __device__ static inline raw pack(f4 x) {
    raw r;
    float* e = (float*)&r;
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] = x[j];
    return r;
  }
};

// Register staging of an R x COLS tile (row stride `rs` elements in global,
// rows >= valid read as zero) for software prefetch: load() issues the global
// reads, store() writes the tile to LDS with 16-byte stores.
template <typename E, int R, int COLS, int NT = NTHREADS>
struct TileRegs {
  static constexpr int VEC = 16 / sizeof(E);
  static constexpr int PR = COLS / VEC;
  static constexpr int TOTAL = R * PR;
  static constexpr int N = (TOTAL + NT - 1) / NT;
  static_assert(TOTAL % NT == 0 || TOTAL < NT, "tile must split evenly over the workgroup");
  uint4 v[N];
  __device__ static inline bool owns(int i, int tid) { return TOTAL >= NT || tid + i * NT < TOTAL; }
  __device__ inline void load(const E* src, size_t rs, int valid, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx / PR, c = (idx % PR) * VEC;
      v[i] = (owns(i, tid) && r < valid) ? *(const uint4*)(src + (size_t)r * rs + c) : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ inline void store(E* dst, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx / PR, c = (idx % PR) * VEC;
      if (owns(i, tid)) *(uint4*)(dst + (size_t)r * ld + c) = v[i];
    }
  }
};

// As TileRegs, but consecutive threads take consecutive rows, so that the
// transposed LDS store storeT() (dst[c*ld + r]) is free of bank conflicts.
template <typename E, int R, int COLS, int NT = NTHREADS>
struct TileRegsT {
  static constexpr int VEC = 16 / sizeof(E);
  static constexpr int PR = COLS / VEC;
  static constexpr int N = R * PR / NT;
  static_assert(N >= 1 && N * NT == R * PR && NT % R == 0, "tile split");
  uint4 v[N];
  __device__ inline void load(const E* src, size_t rs, int valid, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx % R, c = (idx / R) * VEC;
      v[i] = r < valid ? *(const uint4*)(src + (size_t)r * rs + c) : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ inline void storeT(E* dst, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx % R, c = (idx / R) * VEC;
      const E* e = (const E*)&v[i];
#pragma unroll
      for (int j = 0; j < VEC; ++j) dst[(size_t)(c + j) * ld + r] = e[j];
    }
  }
};

// fp32 tile staged in registers and written to LDS converted to E.
template <typename E, int R, int COLS, int NT = NTHREADS>
struct TileRegsF {
  static constexpr int PR = COLS / 4;
  static constexpr int TOTAL = R * PR;
  static constexpr int N = TOTAL / NT;
  static_assert(N >= 1 && N * NT == TOTAL, "tile split");
  f4 v[N];
  __device__ inline void load(const float* src, size_t rs, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx / PR, c = (idx % PR) * 4;
      v[i] = *(const f4*)(src + (size_t)r * rs + c);
    }
  }
  __device__ inline void store(E* dst, int ld, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int idx = tid + i * NT, r = idx / PR, c = (idx % PR) * 4;
      *(typename Quad<E>::raw*)(dst + (size_t)r * ld + c) = Quad<E>::pack(v[i]);
    }
  }
};

struct NoRegs {};

// Number of compute units of the current device (host side, cached).
int device_cu_count();

template <typename F> __device__ inline F zero_frag();
template <> __device__ inline bf8 zero_frag<bf8>() { return __builtin_bit_cast(bf8, make_uint4(0, 0, 0, 0)); }
template <> __device__ inline float zero_frag<float>() { return 0.f; }

// MFMA A-operand fragments of one 16-row block, loaded straight from global
// memory into registers (row-major source, k contiguous, row stride `ld`).
// Rows at or beyond `valid` (relative to the block's first row) read as zero.
template <typename E, int K>
struct AFrag {
  typedef typename Mma<E>::frag frag;
  static constexpr int NK = K / Mma<E>::KS;
  frag f[NK];
  __device__ inline void load(const E* row0, size_t ld, int valid, int lane) {
    const int r = lane & 15;
    const E* src = row0 + (size_t)r * ld + (lane >> 4) * Mma<E>::KPL;
#pragma unroll
    for (int ks = 0; ks < NK; ++ks)
      f[ks] = r < valid ? *(const frag*)(src + ks * Mma<E>::KS) : zero_frag<frag>();
  }
};

// Workgroup barrier that orders LDS traffic only: outstanding global loads
// (software prefetch) stay in flight across it.
__device__ inline void block_sync_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}



// ----------------------------------------------------------------- parameters
struct Params {
  // sizes
  int T;          // dense: tokens per sequence; varlen: total tokens
  int N;          // sequences
  int H;
  int NT;         // dense: ceil(T / C)
  int n_slots;    // saved-state / workspace slots
  const int* cu;  // varlen cu_seqlens (device) or nullptr
  // forward inputs
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  const float* lam;
  const float* la;       // log alpha or nullptr
  const float* S0;       // initial state or nullptr
  // forward outputs
  void* o;
  float* Sfin;
  float* saved;          // saved context: entry states S^T [slot][H][Dk][Dv] (fp32)
  void* savedD;          // saved context: D [slot][H][C][Dv] (dtype)
  // workspace (per slot and head)
  float* wb;             // [slot][H][C] chunk-local prefix sums of log alpha
  void* wU;              // [slot][H] C x Dv, C-fragment tiled
  void* wW;              // [slot][H][C][Dk]
  void* wP;              // [slot][H][C][C]   P = Gam * M * Q K^T
  void* wKt;             // [slot][H][Dk][C]  K^T
  void* wT;              // [slot][H][2][C][C] T^T and P^T (backward only)
  void* wWt;             // [slot][H][Dk][C]  W^T (backward only)
  void* wQgt;            // [slot][H][Dk][C]  (diag(g) Q)^T (backward only)
  void* wQt;             // [slot][H][Dk][C]  Q^T (backward only)
  void* wM;              // [slot][H][C][C]   (I + A)^{-1} (backward only)
  void* wdOt;            // [slot][H][Dv][C]  dO^T (backward only)
  // backward
  const void* dO;
  const float* dSfin;
  void* dq;
  void* dk;
  void* dv;
  float* dbeta;
  float* dlam;
  float* dla;
  float* dS0;
  float* w_dSo;          // [slot][H][Dk][Dv] gradient w.r.t. each chunk's exit state, transposed
  void* w_dDb;           // [slot][H][C][Dv] dD (dtype)
};

// Token range of sequence n; false when cu_seqlens is malformed for n.
__device__ inline bool seq_range(const Params& p, int n, int& s, int& e) {
  if (!p.cu) {
    s = n * p.T;
    e = s + p.T;
    return true;
  }
  s = p.cu[n];
  e = p.cu[n + 1];
  return s >= 0 && s <= e && e <= p.T;
}

__device__ inline int slot_base(const Params& p, int n, int s) {
  return p.cu ? s / C + n : n * p.NT;
}

// Map slot g to (sequence n, first token t0, valid rows len).  False for
// slots no chunk maps to.
__device__ inline bool locate(const Params& p, int g, int& n, int& t0, int& len) {
  if (!p.cu) {
    n = g / p.NT;
    const int c = g - n * p.NT;
    if (n >= p.N) return false;
    t0 = n * p.T + c * C;
    len = min(C, p.T - c * C);
    return len > 0;
  }
  int lo = 0, hi = p.N - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    const int cm = p.cu[mid];
    const int bm = (cm >= 0 ? cm / C : 0) + mid;
    if (bm <= g) lo = mid; else hi = mid - 1;
  }
  n = lo;
  int s, e;
  if (!seq_range(p, n, s, e)) return false;
  const int c = g - (s / C + n);
  if (c < 0) return false;
  t0 = s + c * C;
  if (t0 >= e) return false;
  len = min(C, e - t0);
  return true;
}

// ----------------------------------------------------------------- reductions
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// Sum over the 16 lanes that share (lane >> 4).
__device__ inline float sum16(float x) {
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// ----------------------------------------------------------------- UT solve
// In-place-free inverse of the unit lower-triangular C x C matrix I + A,
// A strictly lower, fp32, A at sA[r*lda + i].  Writes Minv = (I + A)^{-1} to
// sM[r*ldm + i] (upper part zero).  `tmp` is scratch of >= 4*16*17 floats.
// Diagonal 16x16 blocks by forward substitution (one lane per column), then
// the off-diagonal blocks by increasing block distance,
//   Minv_ij = - Minv_ii * sum_{m=j}^{i-1} A_im Minv_mj,
// with fp32 MFMA products.  Must be called by all threads of the block.
template <int NT = NTHREADS>
__device__ inline void unit_lower_inverse(const float* sA, int lda, float* sM, int ldm,
                                          float* tmp, int tid) {
  static_assert(NT >= 256, "needs at least four waves");
  const int lane = tid & 63, w = tid >> 6;
  // zero the strictly-upper blocks
  for (int idx = tid; idx < C * C; idx += NT) {
    const int r = idx / C, i = idx % C;
    if ((i >> 4) > (r >> 4)) sM[r * ldm + i] = 0.f;
  }
  if (lane < 16 && w < 4) {
    // forward substitution for column j of the inverse of diagonal block w;
    // row r of the block is read as four broadcast 16-byte loads, one row
    // ahead of its use, so the dependent FMA chain runs from registers
    const int base = w * 16, j = lane;
    const float* blk = sA + (size_t)base * lda + base;
    float m[16];
    f4 cur[4], nxt[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) cur[q] = *(const f4*)(blk + (size_t)1 * lda + 4 * q);
    m[0] = (j == 0) ? 1.f : 0.f;
#pragma unroll
    for (int r = 1; r < 16; ++r) {
      if (r + 1 < 16) {
#pragma unroll
        for (int q = 0; q < 4; ++q) nxt[q] = *(const f4*)(blk + (size_t)(r + 1) * lda + 4 * q);
      }
      float s = (r == j) ? 1.f : 0.f;
#pragma unroll
      for (int i = 0; i < r; ++i) s -= cur[i >> 2][i & 3] * m[i];
      m[r] = s;
#pragma unroll
      for (int q = 0; q < 4; ++q) cur[q] = nxt[q];
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) sM[(base + r) * ldm + base + j] = m[r];
  }
  __syncthreads();
  float* X = tmp + w * (16 * 17);
  for (int d = 1; d < 4; ++d) {
    const int nb = 4 - d;            // blocks at this distance
    if (w < nb) {
      const int bj = w, bi = w + d;
      f4 acc = zero4();
      for (int m = bj; m < bi; ++m)
        acc = mma_k<float, 16>(kmaj(sA + bi * 16 * lda + m * 16, lda),
                               imaj(sM + m * 16 * ldm + bj * 16, ldm), 0, 0, acc, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) X[frow(lane, j) * 17 + fcol(lane)] = acc[j];
      // same wave wrote X; wave-level barrier is enough but keep block-uniform flow
    }
    __syncthreads();
    if (w < nb) {
      const int bj = w, bi = w + d;
      f4 acc = zero4();
      acc = mma_k<float, 16>(kmaj(sM + bi * 16 * ldm + bi * 16, ldm), imaj(X, 17), 0, 0, acc, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) sM[(bi * 16 + frow(lane, j)) * ldm + bj * 16 + fcol(lane)] = -acc[j];
    }
    __syncthreads();
  }
}

// Inclusive prefix sum of 64 values held one per lane of wave 0 (lane < 64).
__device__ inline float wave_incl_scan(float x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  return x;
}

// XCD-aware mapping of a flat block id onto (unit, tile) pairs so that all
// tiles of one unit are dispatched to the same XCD (blocks are handed to the
// 8 XCDs round-robin).  Returns false for padding blocks.
__device__ inline bool xcd_unit_tile(int bid, int n_units, int n_tiles, int& unit, int& tile) {
  const int xcd = bid & 7, slot = bid >> 3;
  tile = slot % n_tiles;
  unit = (slot / n_tiles) * 8 + xcd;
  return unit < n_units;
}

}  // namespace qd
