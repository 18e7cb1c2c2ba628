/*
 * qdelta.h -- C ABI of libqdelta.so: the Q-Delta layer on AMD Instinct MI355X
 * (gfx950), as hand-written HIP kernels.
 *
 * The operation (Sec. 3.3, Eq. (qdelta_decay), with the mixed input of
 * Eq. (qdelta_gated_form)).  For every sequence n and head h independently,
 * with a state S in R^{Dv x Dk} (row = value component):
 *
 *     x_t = k_t + lam_t q_t
 *     S_t = alpha_t S_{t-1} (I - beta_t x_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t q_t                           (read-out from the updated state)
 *
 * The chunk entry points evaluate this with the chunkwise-parallel form of
 * Sec. 3.3 ("Chunkwise parallel form"; App. D.1 WY representation, App. D.2 UT
 * transform): chunks of `chunk` consecutive tokens, a UT-transform triangular
 * solve inside each chunk, and a sequential fp32 scan of the state across
 * chunks.  The result equals the recurrence up to floating-point rounding.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller.  Inputs are
 *    never written.  Every output is fully overwritten (never accumulated).
 *  - Tensors are dense, row-major, contiguous, 16-byte aligned.
 *  - Activations q, k, v, o (and dO, dq, dk, dv) use `dtype`: QDELTA_BF16 or
 *    QDELTA_F32.  Gates, states and gate gradients are always float32.
 *  - Decay is passed as log(alpha) (float32, <= 0 expected); log_alpha == NULL
 *    means alpha == 1 everywhere.  Gate values are not clamped.
 *  - The query-feedback gate lambda is either per token and head (`lam`, a
 *    [.., H] float32 tensor) or one constant for every token and head
 *    (`lam` == NULL, value `lam_scalar`): the paper's ablations fix it to a
 *    scalar (Sec. 4.2, table "Ablation on the query-feedback coefficient
 *    lambda": 0.2, 0.5, 0.8, and 1 for no gating), and lam_scalar == 0 is the
 *    gated delta rule of Sec. 2 (x_t = k_t).  The constant form reads no
 *    lambda stream.
 *  - Calls are asynchronous on `stream` (0 = the null stream): no host
 *    synchronisation and no device allocation.  Scratch memory is a caller
 *    workspace of at least the size reported by qdelta_chunk_workspace_bytes.
 *  - Validation of every host-visible argument happens before the first
 *    launch; on any error nothing is launched and nothing is written.
 *  - Apart from the opt-in measurement facility at the end of this file and
 *    the scratch array of qdelta_chunk_fwd_noalloc, there is no global mutable
 *    state; calls on different streams may overlap provided their workspaces
 *    and outputs do not.
  *  - Supported: Dk in {64, 128}; Dv in {64, 128, 256}; chunk == 64; T >= 0 need
 *    not be a multiple of chunk.  The chunk entry points additionally require
 *    Dk == 64 for QDELTA_F32 (their fp32 operand tiles at Dk == 128 exceed the
 *    160 KB of LDS of a compute unit).  Anything else returns
 *    QDELTA_EUNSUPPORTED.
 *
 * Sequence layouts
 * ----------------
 *  dense   q,k [B,T,H,Dk]  v,o [B,T,H,Dv]  gates [B,T,H]  states [B,H,Dv,Dk]
 *  varlen  the same with B == 1 and T = total tokens, split into N sequences by
 *          cu_seqlens (device int32[N+1], cu[0] = 0, non-decreasing,
 *          cu[N] = T); states are [N,H,Dv,Dk].  Chunks restart at every
 *          sequence start, so results do not depend on how sequences are packed.
 *          A malformed cu_seqlens cannot be checked without a host copy: the
 *          kernels then skip the offending sequences (their outputs are left
 *          unspecified) but never access memory out of bounds.
 *
 * Saved context (written by the forward, read by the backward)
 * --------------------------------------------------------------
 *  A caller-owned device buffer of qdelta_saved_bytes() bytes (16-byte
 *  aligned) with six regions, one after the other, all but the fourth
 *  indexed by unit u = slot * H + h (U = n_slots * H units):
 *    states  dtype [U, Dv, Dk]: the entry state S of the chunk, rounded to
 *            the activation dtype (the backward's products take it as an MFMA
 *            operand of that type);
 *    D       dtype [U, Dv/32, C, 32]: the chunk's "new values" D = U - W S^T
 *            (App. D, WY form) in tiles of 32 value columns, each tile a
 *            contiguous C x 32 row-major block; rows >= the chunk's length
 *            zero;
 *    gates   float32 [U, 3, C]: chunk-local prefix sums b of log alpha, then
 *            beta and lambda (zero past the chunk's length);
 *    zero    1024 bytes of zeros (rows of zeros for the backward's loads);
 *    P       dtype [U, 10, 16, 16]: the intra-chunk output operator
 *            Gam * M * (Q K^T) (Sec. 3.3 chunkwise form), lower triangular
 *            in 16 x 16 blocks and stored as those ten blocks: block (r, c),
 *            c <= r, at index r (r + 1) / 2 + c, each row-major; rows >= the
 *            chunk's length zero;
 *    M       dtype [U, 10, 16, 16]: (I + A)^{-1} of the UT transform
 *            (App. D.2), its ten blocks on and below the diagonal, as P.
 *  The backward reads all of it and so needs no preparation pass of its own.
 *  n_slots from qdelta_saved_state_slots.  Chunk c (0-based) of sequence n
 *  occupies slot  n*ceil(T/chunk) + c  (dense) or  floor(cu[n]/chunk) + n + c
 *  (varlen); slots no chunk maps to are untouched.
 */
#ifndef QDELTA_H
#define QDELTA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QDELTA_OK = 0,
  QDELTA_EINVAL = 1,        /* NULL where a pointer is required, negative or inconsistent size, misalignment */
  QDELTA_EUNSUPPORTED = 2,  /* valid but not implemented: head dims, chunk, dtype combination */
  QDELTA_ENOWORKSPACE = 3,  /* workspace smaller than qdelta_chunk_workspace_bytes() */
  QDELTA_EHIP = 4           /* a kernel launch reported an error */
} qdelta_status;

typedef enum { QDELTA_F32 = 0, QDELTA_BF16 = 1 } qdelta_dtype;

/* Static text for a status code (never NULL). */
const char* qdelta_status_string(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int qdelta_version(void);

/* Number of saved-context slots (chunks, counting the varlen holes).
 * n_seqs == 0: dense batch of B sequences of T tokens -> B*ceil(T/chunk).
 * n_seqs  > 0: varlen batch of T total tokens in n_seqs sequences ->
 *              floor(T/chunk) + n_seqs (an upper bound that needs no host copy
 *              of cu_seqlens).  Returns 0 for invalid sizes. */
size_t qdelta_saved_state_slots(int32_t B, int32_t T, int32_t chunk, int32_t n_seqs);

/* Bytes of the saved context for these sizes (0 for unsupported sizes). */
size_t qdelta_saved_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                          int32_t dtype, int32_t n_seqs);

/* Workspace bytes needed by qdelta_chunk_fwd[_varlen] (is_bwd == 0) or
 * qdelta_chunk_bwd[_varlen] (is_bwd != 0) for these sizes (same meaning of
 * n_seqs as above).  Returns 0 for unsupported or invalid sizes. */
size_t qdelta_chunk_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                    int32_t chunk, int32_t dtype, int32_t n_seqs, int32_t is_bwd);

/* Chunkwise forward (Sec. 3.3 chunkwise form; App. D).
 *   q, k [B,T,H,Dk], v [B,T,H,Dv]           activations (dtype)
 *   beta [B,T,H]                             write strength (fp32)
 *   lam [B,T,H] or NULL                      query-feedback gate (fp32); NULL: lambda == lam_scalar
 *   lam_scalar                               the constant lambda when lam is NULL (0: the gated
 *                                            delta rule of Sec. 2, x_t = k_t)
 *   log_alpha [B,T,H] or NULL                log of the forget gate (fp32)
 *   initial_state [B,H,Dv,Dk] or NULL        entry state (NULL = zero)
 *   o [B,T,H,Dv]                             output o_t = S_t q_t (dtype)
 *   final_state [B,H,Dv,Dk] or NULL          state after the last token
 *   saved or NULL                            saved context for the backward (see above)
 *   ws, ws_bytes                             device workspace */
int qdelta_chunk_fwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                     int32_t dtype, const void* q, const void* k, const void* v,
                     const float* beta, const float* lam, float lam_scalar, const float* log_alpha,
                     const float* initial_state, void* o, float* final_state,
                     void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/* Segment-parallel forward (dense batch) for long sequences over few
 * (sequence, head) pairs, where the single pass's one workgroup per
 * (sequence, head, value tile) would leave most compute units idle.  Each
 * chunk acts on the state as an affine map S -> S A_c + B_c (Sec. 3.3, the
 * compact chunk update S' = S (g_C I - W^T Kbar) + U^T Kbar), so a run of
 * chunks is one too.  Each sequence is cut into segments of
 * ceil(ceil(T/chunk) / n_segments) chunks; every segment's map (A: Dk x Dk,
 * B: Dv x Dk) is formed in parallel from a zero state, the segments' entry
 * states follow in order (S_{g+1} = S_g A_g + B_g, fp32), and every segment
 * is then run again from its entry state, writing its outputs.  About three
 * times the scan work of the single pass (A has Dk rows) for up to
 * n_segments times its parallelism.
 *   Arguments as qdelta_chunk_fwd, plus n_segments >= 1 (1: the single
 *   pass); ws_bytes >= qdelta_segmented_workspace_bytes(..., n_segments).
 *   Results equal qdelta_chunk_fwd's up to rounding (not bit for bit: the
 *   entry states come from composed maps). */
int qdelta_chunk_fwd_segmented(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                               int32_t dtype, const void* q, const void* k, const void* v,
                               const float* beta, const float* lam, float lam_scalar,
                               const float* log_alpha, const float* initial_state, void* o,
                               float* final_state, void* saved, int32_t n_segments, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/* Workspace bytes of qdelta_chunk_fwd_segmented (0 for invalid sizes). */
size_t qdelta_segmented_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                        int32_t chunk, int32_t dtype, int32_t n_segments);

/* Segment count that qdelta_chunk_fwd_segmented is expected to run fastest
 * with on the current device (1: use the single pass).  Host-side only. */
int32_t qdelta_suggest_segments(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype);

/* Allocation-free forward, for callers that cannot allocate device memory
 * or hand over a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Same arguments and results as
 * qdelta_chunk_fwd (dense layout, no saved context); its workspace is a
 * library-owned scratch array of QDELTA_NOALLOC_SCRATCH_BYTES per device,
 * held from the first call on that device until the process ends.
 *  - Sizes whose forward workspace (qdelta_chunk_workspace_bytes with
 *    is_bwd == 0) exceeds QDELTA_NOALLOC_SCRATCH_BYTES return
 *    QDELTA_ENOWORKSPACE before any device call (about 6100 chunk-head units
 *    at bf16, e.g. B=4 T=4096 H=16 fits; about 3100 at fp32).
 *  - Calls no allocating routine.  The first call on a device looks up the
 *    scratch array's device address (QDELTA_EHIP if that fails).
 *  - Every call on a device shares that device's scratch array: calls that
 *    overlap in time on one device (different streams or host threads) race
 *    and must be serialised by the caller.  The array keeps the last call's
 *    contents; no call relies on its initial contents. */
#define QDELTA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int qdelta_chunk_fwd_noalloc(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                             int32_t dtype, const void* q, const void* k, const void* v,
                             const float* beta, const float* lam, float lam_scalar,
                             const float* log_alpha, const float* initial_state, void* o,
                             float* final_state, hipStream_t stream);

/* Varlen forward: as qdelta_chunk_fwd with B == 1, T total tokens, N sequences
 * delimited by the device array cu_seqlens[N+1]; states are [N,H,Dv,Dk]. */
int qdelta_chunk_fwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                            int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype,
                            const void* q, const void* k, const void* v, const float* beta,
                            const float* lam, float lam_scalar, const float* log_alpha,
                            const float* initial_state, void* o, float* final_state,
                            void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/* Chunkwise backward: exact gradients (up to rounding) of
 *     L = <d_o, o> + <d_final_state, final_state>
 * with respect to q, k, v, beta, lam, log_alpha and initial_state.  The paper
 * states no backward pass; this is the derivative of the forward above.
 *   saved           the saved context from qdelta_chunk_fwd on the same inputs,
 *                   or NULL to recompute the state scan inside this call
 *   d_o [B,T,H,Dv]  (dtype);  d_final_state [B,H,Dv,Dk] or NULL (= zero)
 *   dq, dk [B,T,H,Dk], dv [B,T,H,Dv] (dtype); dbeta [B,T,H] (fp32)
 *   dlam: lam != NULL: [B,T,H] fp32, required;
 *         lam == NULL: NULL (no lambda gradient) or ONE fp32 that receives the
 *         gradient with respect to the constant lambda (summed over every token
 *         and head, in a fixed order: the same value on every run)
 *   dlog_alpha [B,T,H] fp32: required iff log_alpha != NULL, else must be NULL
 *   d_initial_state [B,H,Dv,Dk] or NULL */
int qdelta_chunk_bwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                     int32_t dtype, const void* q, const void* k, const void* v,
                     const float* beta, const float* lam, float lam_scalar, const float* log_alpha,
                     const float* initial_state, const void* saved, const void* d_o,
                     const float* d_final_state, void* dq, void* dk, void* dv, float* dbeta,
                     float* dlam, float* dlog_alpha, float* d_initial_state, void* ws,
                     size_t ws_bytes, hipStream_t stream);

/* Varlen backward: as qdelta_chunk_bwd with the varlen layout. */
int qdelta_chunk_bwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                            int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype,
                            const void* q, const void* k, const void* v, const float* beta,
                            const float* lam, float lam_scalar, const float* log_alpha,
                            const float* initial_state, const void* saved,
                            const void* d_o, const float* d_final_state, void* dq, void* dk,
                            void* dv, float* dbeta, float* dlam, float* dlog_alpha,
                            float* d_initial_state, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* One token of the recurrence for N sequences (decode), Sec. 3.3
 * Eq. (qdelta_decay) applied once:
 *   q, k [N,H,Dk], v [N,H,Dv] (dtype); beta, lam, log_alpha [N,H] (fp32,
 *   lam (NULL: lambda == lam_scalar) and log_alpha (NULL: alpha == 1) may be
 *   NULL);  state [N,H,Dv,Dk] fp32, updated in place;
 *   o [N,H,Dv] (dtype) = updated state times q.
 * Supported: Dk in {64, 128}, Dv a positive multiple of 8 up to 256, any dtype. */
int qdelta_recurrent_step(int32_t N, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                          const void* q, const void* k, const void* v, const float* beta,
                          const float* lam, float lam_scalar, const float* log_alpha, float* state,
                          void* o, hipStream_t stream);

/* Fully recurrent forward over whole sequences: Sec. 3.3 Eq. (qdelta_decay)
 * applied token by token (the paper provides this form beside the chunkwise
 * one).  Same results as qdelta_chunk_fwd up to rounding, one launch, no
 * workspace and no saved context (inference and short sequences).
 *   q, k [B,T,H,Dk], v [B,T,H,Dv] (dtype); beta [B,T,H] fp32;
 *   lam [B,T,H] or NULL (lambda == lam_scalar); log_alpha [B,T,H] or NULL (alpha == 1);
 *   initial_state [B,H,Dv,Dk] fp32 or NULL (zero);
 *   o [B,T,H,Dv] (dtype); final_state [B,H,Dv,Dk] fp32 or NULL.
 * Supported: Dk in {64, 128}, Dv a positive multiple of 8 up to 256, any dtype. */
int qdelta_recurrent_fwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                         const void* q, const void* k, const void* v, const float* beta,
                         const float* lam, float lam_scalar, const float* log_alpha,
                         const float* initial_state, void* o, float* final_state, hipStream_t stream);

/* Varlen recurrent forward: B == 1, T total tokens, N sequences delimited by
 * the device array cu_seqlens[N+1] (entries are clamped to [0, T]); states
 * are [N,H,Dv,Dk]. */
int qdelta_recurrent_fwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                                int32_t Dk, int32_t Dv, int32_t dtype, const void* q,
                                const void* k, const void* v, const float* beta,
                                const float* lam, float lam_scalar, const float* log_alpha,
                                const float* initial_state, void* o, float* final_state,
                                hipStream_t stream);

/* Workspace bytes of qdelta_recurrent_bwd[_varlen] for these sizes
 * (n_seqs == 0: dense B x T; n_seqs > 0: varlen, T total tokens): per
 * token-head 3 Dv + Dk + 1 fp32, per (sequence, head) Dv fp32.  0 for
 * unsupported sizes. */
size_t qdelta_recurrent_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                        int32_t n_seqs);

/* Backward of the fully recurrent form (the paper ships kernels for both the
 * fully recurrent and the chunkwise form, Sec. 3.3): exact gradients (up to
 * rounding) of L = <d_o, o> + <d_final_state, final_state> through
 * Eq. (qdelta_decay) token by token, one launch, no saved context (the
 * states are recomputed).  Arguments and gradient conventions as
 * qdelta_chunk_bwd (dense layout; dlam per token for a lam tensor, one float
 * or NULL for a constant lambda), plus a workspace of
 * qdelta_recurrent_workspace_bytes.  Same results as qdelta_chunk_bwd up to
 * rounding; meant for short sequences, where the chunk form's per-chunk
 * work does not pay off.
 * Supported: Dk in {64, 128}, Dv in {32, 64, 128, 256}, any dtype. */
int qdelta_recurrent_bwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                         const void* q, const void* k, const void* v, const float* beta,
                         const float* lam, float lam_scalar, const float* log_alpha,
                         const float* initial_state, const void* d_o, const float* d_final_state,
                         void* dq, void* dk, void* dv, float* dbeta, float* dlam, float* dlog_alpha,
                         float* d_initial_state, void* ws, size_t ws_bytes, hipStream_t stream);

/* Varlen recurrent backward: B == 1, T total tokens, N sequences delimited
 * by the device array cu_seqlens[N+1] (entries clamped to [0, T]); states
 * are [N,H,Dv,Dk]. */
int qdelta_recurrent_bwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H, int32_t Dk,
                                int32_t Dv, int32_t dtype, const void* q, const void* k, const void* v,
                                const float* beta, const float* lam, float lam_scalar,
                                const float* log_alpha, const float* initial_state, const void* d_o,
                                const float* d_final_state, void* dq, void* dk, void* dv, float* dbeta,
                                float* dlam, float* dlog_alpha, float* d_initial_state, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/* Row L2 normalisation for the layer's q and k (unit-norm keys are the
 * condition of Sec. 3.4 Lemma 1): y = x / max(|x|, 1e-12) per row of D.
 *   x        rows of D elements (dtype), row r at x + r * ld_x (ld_x >= D,
 *            ld_x * element size a multiple of 16 bytes): strided views allowed
 *   y        [rows, D] (dtype), contiguous
 *   rnorm    [rows] fp32: 1 / max(|x|, 1e-12), negated for rows whose norm was
 *            clamped; pass it to the backward unchanged
 * Supported: D in {64, 128}, any dtype. */
int qdelta_l2norm_fwd(int64_t rows, int32_t D, int64_t ld_x, int32_t dtype, const void* x, void* y,
                      float* rnorm, hipStream_t stream);

/* Backward of qdelta_l2norm_fwd: dx = r (dy - y (y . dy)) per row, r = |rnorm|
 * (dx = r dy for a clamped row).  y, dy, dx [rows, D] contiguous (dtype). */
int qdelta_l2norm_bwd(int64_t rows, int32_t D, int32_t dtype, const void* y, const float* rnorm,
                      const void* dy, void* dx, hipStream_t stream);

/* Measurement facility (benchmarks and profiling only; not thread-safe).
 * qdelta_profile_begin() starts recording a pair of HIP events around every
 * kernel launch of the library, on the launch stream, tagged by stage:
 *   0 chunk preparation (forward)       1 forward state scan + chunk output
 *   2 chunk preparation (backward)      3 backward state scan (+ dv)
 *   4 intra-chunk backward              5 recurrent step
 *   6 recurrent forward                 7 segment maps (segmented forward)
 *   8 segment entry states              9 segment outputs
 *  10 recurrent backward
 * qdelta_profile_end() waits for the recorded events, writes the summed kernel
 * time (milliseconds) and the number of launches of each stage into the
 * caller's arrays of QDELTA_N_STAGES entries (either may be NULL) and stops
 * recording.  Returns QDELTA_EHIP if an event call failed. */
#define QDELTA_N_STAGES 11
int qdelta_profile_begin(void);
int qdelta_profile_end(float* ms, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* QDELTA_H */
