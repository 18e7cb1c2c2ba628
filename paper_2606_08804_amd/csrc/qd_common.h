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
#include <cstdint>
#include <stdint.h>

namespace qd {

constexpr int C = 64;          // chunk length (tokens)
constexpr int NTHREADS = 256;  // 4 wave64s per workgroup
constexpr int NWAVES = NTHREADS / 64;

typedef float f4 __attribute__((ext_vector_type(4)));

// Lower-triangular chunk operands (T, M, P) are stored with exact zeros above
// the 16 x 16 block diagonal, so products with them may skip those k blocks
// or not: the fp32 forms (16 k steps per chunk) skip them; the bf16 forms
// (two k steps) run every block, which keeps the waves' work equal and each
// phase one basic block whose LDS reads can all be issued ahead of the MFMAs.
template <typename E>
__device__ constexpr bool keep_kblock(bool needed) { return sizeof(E) == 2 || needed; }

// Wave index within the workgroup, in a scalar register: branches on it are
// uniform, so they compile to scalar branches instead of exec-mask regions.
__device__ inline int wave_id(int tid) { return __builtin_amdgcn_readfirstlane(tid >> 6); }
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

__device__ inline f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }

// Row of C-fragment element j for this lane, relative to the tile origin.
__device__ inline int frow(int lane, int j) { return ((lane >> 4) << 2) + j; }
__device__ inline int fcol(int lane) { return lane & 15; }

// Four consecutive activation-dtype values of one lane's C fragment.
template <typename E> struct Quad;
template <> struct Quad<__bf16> {
  typedef uint2 raw;
  __device__ static inline float get(raw r, int j) {
    const __bf16* e = (const __bf16*)&r;
    return (float)e[j];
  }
  // one vector conversion, so that each pair of values takes a single
  // two-source v_cvt_pk_bf16_f32 (element-wise conversions are rejoined with
  // shifts and ors)
  __device__ static inline raw pack(f4 x) { return __builtin_bit_cast(raw, __builtin_convertvector(x, bf4)); }
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

// Number of compute units of the current device (host side, cached).
int device_cu_count();

// Workgroup barrier that orders LDS traffic only: outstanding global loads
// (software prefetch) stay in flight across it.
__device__ inline void block_sync_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (they complete in issue order).  Needed for direct global->LDS loads, whose
// LDS writes the compiler does not track.
template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// wait_vm with a count known only at run time (uniform across the wave, 0-15).
__device__ inline void wait_vm_n(int n) {
  switch (n) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<1>(); break;
    case 2: wait_vm<2>(); break;
    case 3: wait_vm<3>(); break;
    case 4: wait_vm<4>(); break;
    case 5: wait_vm<5>(); break;
    case 6: wait_vm<6>(); break;
    case 7: wait_vm<7>(); break;
    case 8: wait_vm<8>(); break;
    case 9: wait_vm<9>(); break;
    case 10: wait_vm<10>(); break;
    case 11: wait_vm<11>(); break;
    case 12: wait_vm<12>(); break;
    case 13: wait_vm<13>(); break;
    case 14: wait_vm<14>(); break;
    case 15: wait_vm<15>(); break;
    default: wait_vm<0>(); break;
  }
}

// LDS tiles written by direct loads are rows of RB bytes (64, 128 or 256) made of
// 16-byte chunks; chunk c of row r sits at slot c ^ swz(r).  swz is a linear
// (XOR) map of the low four row bits, chosen by measuring on gfx950 every such
// map of full rank for three read patterns: MFMA fragments (16 consecutive
// rows at one chunk per 16 lanes, 16-byte reads), transpose reads (4
// consecutive rows times two adjacent chunks per 16 lanes, 8-byte reads) and
// fp32 rows read as bf16 fragments (two adjacent 16-byte chunks per lane).
// The maps below run all three at the rate of conflict-free contiguous reads.
template <int RB>
__device__ inline int tile_swz(int row) {
  static_assert(RB == 64 || RB == 128 || RB == 256, "row size");
  const int b0 = row & 1, b1 = (row >> 1) & 1, b2 = (row >> 2) & 1, b3 = (row >> 3) & 1;
  if constexpr (RB == 64) return b3 | ((b0 ^ b3) << 1);
  if constexpr (RB == 128) return (b0 ^ b1) | (b1 << 1) | (b3 << 2);
  return b3 | ((b2 ^ b3) << 1) | (b1 << 2) | (b0 << 3);
}
template <int RB>
__device__ inline int tile_off(int row, int byte) {
  return row * RB + (((byte >> 4) ^ tile_swz<RB>(row)) << 4) + (byte & 15);
}

// One 16-byte (or 4-byte) direct global->LDS load per lane through inline
// assembly: lane i's bytes land at LDS byte `lds` + 16i (4i).  The compiler
// does not see these as LDS writes, so it adds no waits of its own for them
// (it would otherwise wait on every wave's stores before LDS accesses that it
// cannot prove disjoint); every consumer must be ordered by an explicit
// vmcnt wait in the issuing wave plus a barrier.  m0 holds the LDS base;
// kernels using this form issue no compiler-generated direct loads, the only
// other user of m0 here.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ inline void dma16_asm(const void* g, char* lds) {
  // a generic pointer into LDS holds the LDS byte address in its low 32 bits;
  // the address is uniform across the wave (callers pass per-wave bases)
  const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(base), "v"(g) : "memory", "m0");
}
__device__ inline void dma4_asm(const void* g, char* lds) {
  const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(base), "v"(g) : "memory", "m0");
}
#pragma clang diagnostic pop

// Direct global->LDS copy of a ROWS x RB-byte block (row stride `stride`
// bytes) into the swizzled layout at `dst`.  Each instruction moves 1 KB
// (lane i writes LDS bytes 16i..16i+15 of it); wave w of NW issues
// instructions w, w + NW, ...  Rows at or past `valid` are read from `zsrc` (stride
// `zstride`) instead, which the caller points at rows known to be zero.
template <int RB, int ROWS, int NW = NWAVES, bool ASM = false>
__device__ inline void dma_rows(char* dst, const char* src, size_t stride, int valid, const char* zsrc,
                                size_t zstride, int w, int lane) {
  constexpr int NCH = RB / 16, RPI = 1024 / RB, NI = ROWS / RPI;
  static_assert(NI % NW == 0, "instructions split evenly over the waves");
#pragma unroll
  for (int j = 0; j < NI / NW; ++j) {
    const int i = j * NW + w;
    const int row = i * RPI + lane / NCH;
    const int c = (lane % NCH) ^ tile_swz<RB>(row);
    const char* g = row < valid ? src + (size_t)row * stride + c * 16 : zsrc + (size_t)row * zstride + c * 16;
    if constexpr (ASM)
      dma16_asm(g, dst + i * 1024);
    else
      __builtin_amdgcn_global_load_lds((const void*)g, (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                       16, 0, 0);
  }
}

// C x C operators whose 16 x 16 blocks above the diagonal are zero (P, M, T)
// are stored packed: the ten blocks on and below the diagonal, block (r, c)
// (c <= r) at index r (r + 1) / 2 + c, each row-major.  Stores then cover
// whole blocks (whole cache lines) and 37.5% fewer bytes move.
constexpr int LBT_ELEMS = 10 * 256;
__device__ inline int lbt_block(int br, int bc) { return br * (br + 1) / 2 + bc; }

// Direct load of a packed C x C operand into the swizzled row-major LDS tile
// at `dst` (rows of C elements): the same instructions as a full tile, with
// the lanes of chunks above the diagonal masked off, so those LDS bytes keep
// what zero_upper_chunks wrote there once.  Every instruction covers whole
// rows, whose first block is on or below the diagonal, so each has active
// lanes and the outstanding-load count is that of a full tile.
template <typename E, int NW>
__device__ inline void dma_lbt(char* dst, const char* src, int w, int lane) {
  constexpr int RB = C * (int)sizeof(E), NCH = RB / 16, RPI = 1024 / RB, NI = C / RPI;
  constexpr int BCH = 16 * (int)sizeof(E) / 16;   // 16-byte chunks per block row
  static_assert(NI % NW == 0, "instructions split evenly over the waves");
#pragma unroll
  for (int j = 0; j < NI / NW; ++j) {
    int l = lane;                     // formed again per instruction: no address kept live across them
    asm volatile("" : "+v"(l));
    const int i = j * NW + w;
    const int row = i * RPI + l / NCH;
    const int c = (l % NCH) ^ tile_swz<RB>(row);
    const int br = row >> 4, bc = c / BCH;
    if (bc <= br)
      dma16_asm(src + ((size_t)lbt_block(br, bc) * 256 + (row & 15) * 16) * sizeof(E) + (c % BCH) * 16,
                dst + i * 1024);
  }
}

// Zeroes the chunks above the diagonal blocks of a swizzled C x C LDS tile
// (the ones dma_lbt never writes), nthreads threads from thread t.
template <typename E>
__device__ inline void zero_upper_chunks(char* dst, int t, int nthreads) {
  constexpr int RB = C * (int)sizeof(E), NCH = RB / 16, BCH = 16 * (int)sizeof(E) / 16;
  for (int idx = t; idx < C * NCH; idx += nthreads) {
    const int row = idx / NCH, c = idx % NCH;
    if (c / BCH > (row >> 4)) *(uint4*)(dst + row * RB + ((c ^ tile_swz<RB>(row)) << 4)) = make_uint4(0, 0, 0, 0);
  }
}

// MFMA fragment (A or B operand; both map lane l to row l & 15 and to the
// KPL consecutive k from (l >> 4) * KPL) read from a swizzled LDS tile of
// element type E.
//
// 16-bit fragments start at a row that is a multiple of 16, so the swizzle of
// each lane's row depends on the lane alone, and at a k offset that is a
// multiple of 32 elements (whole groups of four 16-byte chunks), which enters
// the chunk index as an XOR: the address is row0 RB + (frag_x(l) ^ 2 k0), one
// lane constant per row size, and the rest folds into the instruction offset.
template <int RB>
__device__ inline int frag_x(int lane) {
  return (lane & 15) * RB + (((lane >> 4) ^ tile_swz<RB>(lane & 15)) << 4);
}
template <typename E, int RB>
__device__ inline typename Mma<E>::frag tile_frag(const char* t, int row0, int k0, int lane) {
  if constexpr (sizeof(E) == 2) {
    return *(const typename Mma<E>::frag*)(t + row0 * RB + (frag_x<RB>(lane) ^ (2 * k0)));
  } else {
    const int row = row0 + (lane & 15), k = k0 + (lane >> 4) * Mma<E>::KPL;
    return *(const typename Mma<E>::frag*)(t + tile_off<RB>(row, k * (int)sizeof(E)));
  }
}
// Fragment of the TRANSPOSE of a swizzled LDS tile (rows of RB bytes): for
// lane l the values at tile rows k0 + (l >> 4) * KPL + e, e < KPL, and column
// j0 + (l & 15) (j0 a multiple of 16), i.e. the operand whose "row" index is
// the tile column.  16-bit tiles use the LDS transpose read (see tr_frag
// below): each 8-byte piece lies inside one 16-byte chunk, so the swizzle
// applies per piece.
//
// With k0 a multiple of 16 and j0 a multiple of 16, the two 8-byte pieces of
// lane l sit at k0 RB + (tr_y(l, 0) ^ 2 j0) and k0 RB + (tr_y(l, 4) ^ 2 j0)
// (same reasoning as frag_x: the row swizzle depends on the lane alone and
// the column offset is an XOR of whole chunk pairs).
template <int RB>
__device__ inline int tr_y(int lane, int dr) {
  const int L = lane & 15, r = (lane >> 4) * 8 + (L >> 2) + dr;
  return r * RB + ((((L & 3) >> 1) ^ tile_swz<RB>(r & 15)) << 4) + 8 * (L & 1);
}
template <typename E, int RB>
__device__ inline typename Mma<E>::frag tile_tr_frag(const char* t, int k0, int j0, int lane) {
  if constexpr (sizeof(E) == 2) {
    typedef __bf16 v4b __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4b* lp;
    const char* b = t + k0 * RB;
    const v4b lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lp)(uintptr_t)(uint32_t)(uintptr_t)(b + (tr_y<RB>(lane, 0) ^ (2 * j0))));
    const v4b hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lp)(uintptr_t)(uint32_t)(uintptr_t)(b + (tr_y<RB>(lane, 4) ^ (2 * j0))));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  } else {
    return *(const float*)(t + tile_off<RB>(k0 + (lane >> 4), 4 * (j0 + (lane & 15))));
  }
}
// MFMA fragment of the TRANSPOSE of a row-major 16-bit LDS matrix: with
// element (i, j) at base + i * ld + j (ld in elements), returns for lane l the
// fragment values (i = k0 + (l >> 4) * KPL + e, j = j0 + (l & 15)), e < KPL,
// i.e. the operand whose "row" index is j and whose k index is i.  Uses the
// LDS transpose read: in each 16-lane group, lane L names the 8 bytes at row
// (L >> 2) and columns 4 (L & 3) .. +3 of a 4 x 16 block and receives column
// L of that block.  The fp32 form is a plain strided read.
template <typename E>
__device__ inline typename Mma<E>::frag tr_frag(const E* base, int ld, int k0, int j0, int lane);
template <>
__device__ inline bf8 tr_frag<__bf16>(const __bf16* base, int ld, int k0, int j0, int lane) {
  typedef __bf16 v4b __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4b* lp;
  const int L = lane & 15, i0 = k0 + (lane >> 4) * 8 + (L >> 2), j = j0 + 4 * (L & 3);
  const __bf16* a = base + (size_t)i0 * ld + j;
  const v4b lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lp)(uintptr_t)(uint32_t)(uintptr_t)a);
  const v4b hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lp)(uintptr_t)(uint32_t)(uintptr_t)(a + (size_t)4 * ld));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}
template <>
__device__ inline float tr_frag<float>(const float* base, int ld, int k0, int j0, int lane) {
  return base[(size_t)(k0 + (lane >> 4)) * ld + j0 + (lane & 15)];
}


// ----------------------------------------------------------------- parameters
struct Params {
  // sizes
  int T;          // dense: tokens per sequence; varlen: total tokens
  int N;          // sequences
  int H;
  int NT;         // dense: ceil(T / C)
  int n_slots;    // saved-state / workspace slots
  int lead;         // intra-chunk backward: leading workgroups that only wait
  int lead_cycles;  // ... and for how many clock cycles
  const int* cu;  // varlen cu_seqlens (device) or nullptr
  // forward inputs
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  const float* lam;      // per token and head, or nullptr: lambda == lam_c everywhere
  float lam_c;
  const float* la;       // log alpha or nullptr
  const float* S0;       // initial state or nullptr
  // forward outputs
  void* o;
  float* Sfin;
  void* saved;           // saved context: entry states S [slot][H][Dv][Dk] (dtype)
  void* savedD;          // saved context: D [slot][H][Dv/32][C][32] (dtype), 32-column tiles
  // chunk factors from the preparation, per slot and head (in the saved
  // context when one is kept, else in the workspace)
  float* wb;             // [slot][H][3][C] gate block: chunk-local prefix sums b of
                         // log alpha, beta, lambda (beta, lambda zero past the chunk)
  void* wP;              // [slot][H][LBT_ELEMS] P = Gam * M_causal * Q K^T (packed lower blocks)
  void* wM;              // [slot][H][LBT_ELEMS] M = (I + A)^{-1}           (packed lower blocks)
  void* wT;              // [slot][H][LBT_ELEMS] T = M diag(beta) (workspace only; packed)
  void* wZ;              // 1 KB of zeros, written by the preparation kernel: zero rows for direct loads
  // backward
  const void* dO;
  const float* dSfin;
  void* dq;
  void* dk;
  void* dv;
  float* dbeta;
  float* dlam;           // per token and head (lam given), else nullptr
  float* dlam_sum;       // one float: gradient of the constant lambda (lam == nullptr), or nullptr
  float* w_dlam;         // [slot][H] per-unit partial sums of the constant-lambda gradient
  float* dla;
  float* dS0;
  void* w_dSo;           // [slot][H][Dv][Dk] gradient w.r.t. each chunk's exit state (dtype)
  // segment-parallel forward (dense batches): each sequence in n_seg
  // segments of seg_chunks chunks
  int n_seg;
  int seg_chunks;
  float* wSegOut;        // [N*H][n_seg][Dv + Dk][Dk] fp32: each segment's B (value rows) and A (map rows)
  float* wSegIn;         // [N*H][n_seg][Dv][Dk] fp32: each segment's entry state
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
// Lane exchanges (ds_bpermute) addressed from a lane index the caller
// supplies: a kernel near its register limit passes an index laundered per
// phase, so that the exchange addresses of one phase are not kept alive
// through the next.  Same values and order as the __shfl forms.
__device__ inline float lane_from(float x, int src) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src << 2, __builtin_bit_cast(int, x)));
}
__device__ inline float lane_xor(float x, int off, int lane) { return lane_from(x, lane ^ off); }
__device__ inline float wave_sum_l(float x, int lane) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += lane_xor(x, off, lane);
  return x;
}

// Sum over each row of 16 lanes with DPP lane moves (no LDS crossbar):
// swaps within pairs and quads, then rotations by 4 and 8 within the row.
template <int CTRL>
__device__ inline float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ inline float sum16(float x) {
  x += dpp_mov<0xB1>(x);    // quad_perm [1,0,3,2]
  x += dpp_mov<0x4E>(x);    // quad_perm [2,3,0,1]
  x += dpp_mov<0x124>(x);   // row_ror:4
  x += dpp_mov<0x128>(x);   // row_ror:8
  return x;
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP lane moves (no
// LDS crossbar): shifts by 1, 2, 4 and 8 within each row of 16 (lanes
// shifted in from outside the row read 0), then row 0's total added to row 1
// and row 2's to row 3 (row broadcast of lane 15), then rows 0-1's total to
// rows 2-3 (row broadcast of lane 31).
template <int CTRL, int ROWS, bool BOUND>
__device__ inline float dpp_src(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROWS, 0xF, BOUND));
}
__device__ inline float wave_incl_scan_dpp(float x) {
  x += dpp_src<0x111, 0xF, true>(x);    // row_shr:1
  x += dpp_src<0x112, 0xF, true>(x);    // row_shr:2
  x += dpp_src<0x114, 0xF, true>(x);    // row_shr:4
  x += dpp_src<0x118, 0xF, true>(x);    // row_shr:8
  x += dpp_src<0x142, 0xA, false>(x);   // row_bcast:15 into rows 1 and 3
  x += dpp_src<0x143, 0xC, false>(x);   // row_bcast:31 into rows 2 and 3
  return x;
}


// Value rows per scan workgroup.  Every value tile of a (sequence, head)
// re-reads the chunk operands shared by all its tiles (Q, K, T, P, gates), so
// wider tiles move fewer bytes per unit of work; 64-row tiles (bf16 only, for
// LDS room) are used once they still give every CU at least two workgroups.
template <typename E, int DV>
constexpr int scan_bv_max() {
  return (sizeof(E) == 2 && DV >= 64) ? 64 : 32;
}
template <typename E, int DV>
inline int scan_bv(int units) {
  if (scan_bv_max<E, DV>() == 64 && (long long)units * (DV / 64) >= 2LL * device_cu_count()) return 64;
  return 32;
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
