// C ABI of libqdelta.so (declared in include/qdelta.h): argument validation,
// workspace carving and kernel launches on the caller's stream.  No host
// synchronisation and no device allocation happen here.
#include <stddef.h>
#include <stdint.h>

#include <mutex>
#include <vector>

#include "qd_launch.h"
#include "qdelta.h"

namespace {

using qd::C;

constexpr int kVersion = 10000;  // 1.0.0

struct Layout {
  size_t wb = 0, wT = 0, wP = 0, wZ = 0;   // forward: chunk factors (T always; gates, P and the zero block when no saved context is kept)
  size_t dSo = 0, ctx = 0;                 // backward: scan output dS', room to recompute the context
  size_t dlam = 0;                         // backward: per-unit partials of a constant lambda's gradient
  size_t total = 0;
};

// Saved context, region after region: per unit (slot, head) S [Dv][Dk] and
// D [Dv/32][C][32]; per unit the gate block fp32 [3][C] (b, beta, lambda);
// one 1 KB zero block; per unit P and M, each as the ten 16 x 16 blocks on
// and below the diagonal (all but the gates in the activation dtype).
struct Ctx {
  size_t states, D, b, Z, P, M, total;
};
Ctx ctx_layout(size_t units, int Dk, int Dv, int esz) {
  Ctx c;
  c.states = 0;
  c.D = c.states + units * (size_t)Dk * Dv * esz;
  c.b = c.D + units * (size_t)C * Dv * esz;
  c.Z = c.b + units * (size_t)3 * C * 4;
  c.P = c.Z + (units > 0 ? 1024 : 0);
  c.M = c.P + units * (size_t)qd::LBT_ELEMS * esz;
  c.total = c.M + units * (size_t)qd::LBT_ELEMS * esz;
  return c;
}

Layout make_layout(size_t units, int Dk, int Dv, int esz, bool bwd) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) & ~size_t(255);
    return at;
  };
  L.wT = take(units * qd::LBT_ELEMS * esz);
  if (bwd) {
    L.dSo = take(units * (size_t)Dv * Dk * esz);
    L.ctx = take(ctx_layout(units, Dk, Dv, esz).total);
    L.dlam = take(units * sizeof(float));
  } else {
    L.wb = take(units * 3 * C * 4);
    L.wZ = take(units > 0 ? 1024 : 0);
    L.wP = take(units * qd::LBT_ELEMS * esz);
  }
  L.total = off;
  return L;
}

// Segment-parallel forward: the forward layout, then each segment's map
// (B and A rows, fp32) and each segment's entry state (fp32).
struct SegLayout {
  Layout fwd;
  size_t out = 0, in = 0, total = 0;
};
SegLayout make_seg_layout(size_t units, size_t seq_heads, int G, int Dk, int Dv, int esz) {
  SegLayout S;
  S.fwd = make_layout(units, Dk, Dv, esz, false);
  size_t off = S.fwd.total;
  S.out = off;
  off += (seq_heads * G * (size_t)(Dv + Dk) * Dk * 4 + 255) & ~size_t(255);
  S.in = off;
  off += (seq_heads * G * (size_t)Dv * Dk * 4 + 255) & ~size_t(255);
  S.total = off;
  return S;
}

// Chunks per segment and the number of non-empty segments for n_segments
// requested over NT chunks.
void seg_split(int NT, int n_segments, int& L, int& G) {
  L = NT > 0 ? (NT + n_segments - 1) / n_segments : 1;
  G = NT > 0 ? (NT + L - 1) / L : 1;
}

// Points the context fields of p (states, D, gates, P, M) into a context buffer.
void bind_ctx(qd::Params& p, char* base, size_t units, int Dk, int Dv, int esz) {
  const Ctx c = ctx_layout(units, Dk, Dv, esz);
  p.saved = base + c.states;
  p.savedD = base + c.D;
  p.wb = reinterpret_cast<float*>(base + c.b);
  p.wZ = base + c.Z;
  p.wP = base + c.P;
  p.wM = base + c.M;
}

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool ok_ptr(const void* p) { return p != nullptr && aligned(p); }
bool ok_opt(const void* p) { return p == nullptr || aligned(p); }

int check_dims(int64_t tokens, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype) {
  if (tokens < 0 || H <= 0 || chunk <= 0 || Dk <= 0 || Dv <= 0) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if (chunk != C) return QDELTA_EUNSUPPORTED;
  if (Dk != 64 && Dk != 128) return QDELTA_EUNSUPPORTED;
  if (Dv != 64 && Dv != 128 && Dv != 256) return QDELTA_EUNSUPPORTED;
  if (dtype == QDELTA_F32 && Dk != 64) return QDELTA_EUNSUPPORTED;
  // element offsets of the largest tensors stay below 2^31 tokens * heads
  if (tokens * (int64_t)H >= (int64_t(1) << 31)) return QDELTA_EUNSUPPORTED;
  return QDELTA_OK;
}

size_t slots_for(int32_t B, int32_t T, int32_t n_seqs) {
  if (n_seqs > 0) return (size_t)(T / C) + (size_t)n_seqs;
  return (size_t)B * (size_t)((T + C - 1) / C);
}

struct Sizes {
  int32_t T;        // dense: per-sequence tokens; varlen: total tokens
  int32_t N;        // sequences
  const int32_t* cu;
  size_t slots;
  int64_t tokens;   // total tokens
};

int make_sizes(bool varlen, int32_t B, int32_t T, int32_t N, const int32_t* cu, Sizes& s) {
  if (T < 0) return QDELTA_EINVAL;
  if (varlen) {
    if (N < 0 || cu == nullptr) return QDELTA_EINVAL;
    s.T = T;
    s.N = N;
    s.cu = cu;
    s.slots = slots_for(1, T, N > 0 ? N : 0);
    if (N == 0) s.slots = 0;
    s.tokens = T;
  } else {
    if (B < 0) return QDELTA_EINVAL;
    s.T = T;
    s.N = B;
    s.cu = nullptr;
    s.slots = slots_for(B, T, 0);
    s.tokens = (int64_t)B * T;
  }
  return QDELTA_OK;
}

// dry == true: validation only (ws is not dereferenced); returns what the
// call would return up to its first launch.
int fwd_impl(bool varlen, int32_t B, int32_t T, int32_t N, const int32_t* cu, int32_t H,
             int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype, const void* q, const void* k,
             const void* v, const float* beta, const float* lam, float lam_c, const float* log_alpha,
             const float* initial_state, void* o, float* final_state, void* saved,
             void* ws, size_t ws_bytes, hipStream_t stream, bool dry = false) {
  Sizes s;
  int rc = make_sizes(varlen, B, T, N, cu, s);
  if (rc) return rc;
  rc = check_dims(s.tokens, H, Dk, Dv, chunk, dtype);
  if (rc) return rc;
  const bool has_tokens = s.tokens > 0;
  if (has_tokens && !(ok_ptr(q) && ok_ptr(k) && ok_ptr(v) && ok_ptr(beta) && ok_ptr(o)))
    return QDELTA_EINVAL;
  if (!ok_opt(lam) || !ok_opt(log_alpha) || !ok_opt(initial_state) || !ok_opt(final_state) ||
      !ok_opt(saved))
    return QDELTA_EINVAL;
  const int esz = dtype == QDELTA_BF16 ? 2 : 4;
  const Layout L = make_layout(s.slots * (size_t)H, Dk, Dv, esz, false);
  if (L.total > 0 && (ws == nullptr || !aligned(ws))) return QDELTA_EINVAL;
  if (ws_bytes < L.total) return QDELTA_ENOWORKSPACE;
  if (s.N == 0 || dry) return QDELTA_OK;

  char* w = static_cast<char*>(ws);
  qd::Params p{};
  p.T = s.T;
  p.N = s.N;
  p.H = H;
  p.NT = varlen ? 0 : (s.T + C - 1) / C;
  p.n_slots = (int)s.slots;
  p.cu = s.cu;
  p.q = q; p.k = k; p.v = v;
  p.beta = beta; p.lam = lam; p.lam_c = lam_c; p.la = log_alpha; p.S0 = initial_state;
  p.o = has_tokens ? o : nullptr;
  p.Sfin = final_state;
  const size_t units = s.slots * (size_t)H;
  p.wT = w + L.wT;
  if (saved) {
    bind_ctx(p, static_cast<char*>(saved), units, Dk, Dv, esz);
  } else {
    p.wb = reinterpret_cast<float*>(w + L.wb);
    p.wZ = w + L.wZ;
    p.wP = w + L.wP;
    p.wM = nullptr;    // M feeds only the backward
  }
  hipError_t e = qd::launch_fwd(p, dtype, Dk, Dv, 0, 1, stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int bwd_impl(bool varlen, int32_t B, int32_t T, int32_t N, const int32_t* cu, int32_t H,
             int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype, const void* q, const void* k,
             const void* v, const float* beta, const float* lam, float lam_c, const float* log_alpha,
             const float* initial_state, const void* saved, const void* d_o,
             const float* d_final_state, void* dq, void* dk, void* dv, float* dbeta, float* dlam,
             float* dlog_alpha, float* d_initial_state, void* ws, size_t ws_bytes,
             hipStream_t stream) {
  Sizes s;
  int rc = make_sizes(varlen, B, T, N, cu, s);
  if (rc) return rc;
  rc = check_dims(s.tokens, H, Dk, Dv, chunk, dtype);
  if (rc) return rc;
  const bool has_tokens = s.tokens > 0;
  if (has_tokens &&
      !(ok_ptr(q) && ok_ptr(k) && ok_ptr(v) && ok_ptr(beta) && ok_ptr(d_o) &&
        ok_ptr(dq) && ok_ptr(dk) && ok_ptr(dv) && ok_ptr(dbeta)))
    return QDELTA_EINVAL;
  if ((log_alpha == nullptr) != (dlog_alpha == nullptr) && has_tokens) return QDELTA_EINVAL;
  // per-token lambda: its gradient is required; constant lambda: dlam is
  // optional and then receives one float
  if (lam != nullptr && dlam == nullptr && has_tokens) return QDELTA_EINVAL;
  if (lam == nullptr && dlam != nullptr && (reinterpret_cast<uintptr_t>(dlam) & 3u)) return QDELTA_EINVAL;
  if (!ok_opt(lam) || (lam != nullptr && !ok_opt(dlam)) || !ok_opt(log_alpha) || !ok_opt(dlog_alpha) ||
      !ok_opt(initial_state) ||
      !ok_opt(saved) || !ok_opt(d_final_state) || !ok_opt(d_initial_state))
    return QDELTA_EINVAL;
  const int esz = dtype == QDELTA_BF16 ? 2 : 4;
  const Layout L = make_layout(s.slots * (size_t)H, Dk, Dv, esz, true);
  if (L.total > 0 && (ws == nullptr || !aligned(ws))) return QDELTA_EINVAL;
  if (ws_bytes < L.total) return QDELTA_ENOWORKSPACE;
  const bool dlam_const = lam == nullptr && dlam != nullptr;
  if (s.N == 0) {
    // nothing to differentiate: a requested constant-lambda gradient is zero
    if (dlam_const) return qd::launch_zero(dlam, stream) == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
    return QDELTA_OK;
  }

  char* w = static_cast<char*>(ws);
  qd::Params p{};
  p.T = s.T;
  p.N = s.N;
  p.H = H;
  p.NT = varlen ? 0 : (s.T + C - 1) / C;
  p.n_slots = (int)s.slots;
  p.cu = s.cu;
  p.q = q; p.k = k; p.v = v;
  p.beta = beta; p.lam = lam; p.lam_c = lam_c; p.la = log_alpha; p.S0 = initial_state;
  p.dO = d_o;
  p.dSfin = d_final_state;
  p.dq = dq; p.dk = dk; p.dv = dv;
  p.dbeta = dbeta; p.dla = dlog_alpha; p.dS0 = d_initial_state;
  p.dlam = dlam_const ? nullptr : dlam;
  p.dlam_sum = dlam_const ? dlam : nullptr;
  p.w_dlam = dlam_const ? reinterpret_cast<float*>(w + L.dlam) : nullptr;
  p.w_dSo = w + L.dSo;
  const size_t units = s.slots * (size_t)H;
  hipError_t e = hipSuccess;
  if (saved) {
    bind_ctx(p, const_cast<char*>(static_cast<const char*>(saved)), units, Dk, Dv, esz);
  } else {
    // recompute the saved context (no outputs) into the workspace
    bind_ctx(p, w + L.ctx, units, Dk, Dv, esz);
    p.wT = w + L.wT;
    e = qd::launch_fwd(p, dtype, Dk, Dv, 1, 1, stream);
    if (e != hipSuccess) return QDELTA_EHIP;
  }
  e = qd::launch_bwd(p, dtype, Dk, Dv, stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

// Scratch of the allocation-free forward: one copy per device, held until
// the process ends.  In host code `scratch` is only a stand-in for the
// symbol; its device address (per device) comes from hipGetSymbolAddress and
// is the only form passed to kernels.
__device__ __align__(256) char scratch[QDELTA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and cached.
int scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return QDELTA_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return QDELTA_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return QDELTA_OK;
}

// Measurement facility state (process-wide; benchmarks only).
struct Prof {
  bool on = false;
  bool failed = false;
  std::vector<hipEvent_t> start[qd::ST_COUNT], stop[qd::ST_COUNT];
  int used[qd::ST_COUNT] = {};
};
Prof g_prof;

}  // namespace

int qd::device_cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

void qd::prof_mark(int stage, int after, hipStream_t st) {
  Prof& P = g_prof;
  if (!P.on || stage < 0 || stage >= ST_COUNT) return;
  const int i = P.used[stage];
  if (!after) {
    if (i == (int)P.start[stage].size()) {
      hipEvent_t a = nullptr, b = nullptr;
      // no system-scope fence: the events only time kernels on this device,
      // and the fence made each record cost microseconds between launches
      if (hipEventCreateWithFlags(&a, hipEventDisableSystemFence) != hipSuccess ||
          hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess) {
        P.failed = true;
        return;
      }
      P.start[stage].push_back(a);
      P.stop[stage].push_back(b);
    }
    if (hipEventRecord(P.start[stage][i], st) != hipSuccess) P.failed = true;
  } else {
    if (i >= (int)P.stop[stage].size()) return;
    if (hipEventRecord(P.stop[stage][i], st) != hipSuccess) P.failed = true;
    P.used[stage] = i + 1;
  }
}

extern "C" {

int qdelta_profile_begin(void) {
  g_prof.on = true;
  g_prof.failed = false;
  for (int s = 0; s < qd::ST_COUNT; ++s) g_prof.used[s] = 0;
  return QDELTA_OK;
}

int qdelta_profile_end(float* ms, int32_t* launches) {
  Prof& P = g_prof;
  bool failed = P.failed;
  for (int s = 0; s < qd::ST_COUNT; ++s) {
    float tot = 0.f;
    for (int i = 0; i < P.used[s]; ++i) {
      float t = 0.f;
      if (hipEventSynchronize(P.stop[s][i]) != hipSuccess ||
          hipEventElapsedTime(&t, P.start[s][i], P.stop[s][i]) != hipSuccess) {
        failed = true;
        continue;
      }
      tot += t;
    }
    if (ms) ms[s] = tot;
    if (launches) launches[s] = P.used[s];
    P.used[s] = 0;
  }
  P.on = false;
  return failed ? QDELTA_EHIP : QDELTA_OK;
}

const char* qdelta_status_string(int status) {
  switch (status) {
    case QDELTA_OK: return "ok";
    case QDELTA_EINVAL: return "invalid argument (null or misaligned pointer, bad size)";
    case QDELTA_EUNSUPPORTED: return "unsupported configuration (head dims, chunk or dtype)";
    case QDELTA_ENOWORKSPACE: return "workspace too small";
    case QDELTA_EHIP: return "HIP launch error";
    default: return "unknown status";
  }
}

int qdelta_version(void) { return kVersion; }

size_t qdelta_saved_state_slots(int32_t B, int32_t T, int32_t chunk, int32_t n_seqs) {
  if (B < 0 || T < 0 || n_seqs < 0 || chunk != C) return 0;
  return slots_for(B, T, n_seqs);
}

size_t qdelta_saved_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                          int32_t dtype, int32_t n_seqs) {
  if (B < 0 || T < 0 || n_seqs < 0) return 0;
  const int64_t tokens = n_seqs > 0 ? (int64_t)T : (int64_t)B * T;
  if (check_dims(tokens, H, Dk, Dv, chunk, dtype) != QDELTA_OK) return 0;
  return ctx_layout(slots_for(B, T, n_seqs) * (size_t)H, Dk, Dv, dtype == QDELTA_BF16 ? 2 : 4).total;
}

size_t qdelta_chunk_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                    int32_t chunk, int32_t dtype, int32_t n_seqs, int32_t is_bwd) {
  if (B < 0 || T < 0 || n_seqs < 0) return 0;
  const int64_t tokens = n_seqs > 0 ? (int64_t)T : (int64_t)B * T;
  if (check_dims(tokens, H, Dk, Dv, chunk, dtype) != QDELTA_OK) return 0;
  const size_t slots = slots_for(B, T, n_seqs);
  return make_layout(slots * (size_t)H, Dk, Dv, dtype == QDELTA_BF16 ? 2 : 4, is_bwd != 0).total;
}

int qdelta_chunk_fwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                     int32_t dtype, const void* q, const void* k, const void* v,
                     const float* beta, const float* lam, float lam_scalar, const float* log_alpha,
                     const float* initial_state, void* o, float* final_state,
                     void* saved, void* ws, size_t ws_bytes, hipStream_t stream) {
  return fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                  log_alpha, initial_state, o, final_state, saved, ws, ws_bytes, stream);
}

int qdelta_chunk_fwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                            int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype,
                            const void* q, const void* k, const void* v, const float* beta,
                            const float* lam, float lam_scalar, const float* log_alpha,
                            const float* initial_state, void* o, float* final_state,
                            void* saved, void* ws, size_t ws_bytes, hipStream_t stream) {
  return fwd_impl(true, 1, T, N, cu_seqlens, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                  log_alpha, initial_state, o, final_state, saved, ws, ws_bytes, stream);
}

size_t qdelta_segmented_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                        int32_t chunk, int32_t dtype, int32_t n_segments) {
  if (B < 0 || T < 0 || n_segments < 1) return 0;
  if (check_dims((int64_t)B * T, H, Dk, Dv, chunk, dtype) != QDELTA_OK) return 0;
  int L, G;
  seg_split((T + C - 1) / C, n_segments, L, G);
  return make_seg_layout(slots_for(B, T, 0) * (size_t)H, (size_t)B * H, G, Dk, Dv,
                         dtype == QDELTA_BF16 ? 2 : 4).total;
}

int32_t qdelta_suggest_segments(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype) {
  if (B <= 0 || T <= 0 || H <= 0 || Dk <= 0 || Dv <= 0) return 1;
  const long long cus = qd::device_cu_count();
  const long long seq_heads = (long long)B * H;
  const int NT = (T + C - 1) / C;
  // the single pass runs one workgroup per (sequence, head, 32 value rows);
  // with half as many of them as CUs or more it is the faster form
  // (measured at B1 T65536 d128 bf16: 16 heads, 64 workgroups, take 1.64 ms
  // in one pass and about 1.0 ms in eight segments)
  if (seq_heads * (Dv / 32) * 2 >= cus) return 1;
  // the maps pass runs (Dv + Dk) / w workgroups per segment (w = 64 value
  // rows for bf16, 32 for fp32): up to two per CU, with segments of at least
  // 16 chunks
  const int w = dtype == QDELTA_BF16 ? 64 : 32;
  int G = 1;
  while (G < 16 && seq_heads * (2 * G) * ((Dv + Dk) / w) <= 2 * cus && NT / (2 * G) >= 16) G *= 2;
  return G;
}

int qdelta_chunk_fwd_segmented(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                               int32_t dtype, const void* q, const void* k, const void* v,
                               const float* beta, const float* lam, float lam_scalar,
                               const float* log_alpha, const float* initial_state, void* o,
                               float* final_state, void* saved, int32_t n_segments, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  if (n_segments < 1) return QDELTA_EINVAL;
  if (n_segments == 1)
    return fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                    log_alpha, initial_state, o, final_state, saved, ws, ws_bytes, stream);
  const size_t need = qdelta_segmented_workspace_bytes(B, T, H, Dk, Dv, chunk, dtype, n_segments);
  // validation of everything else (no device call), with the forward's own workspace
  int rc = fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                    log_alpha, initial_state, o, final_state, saved, ws, ws_bytes, stream, true);
  if (rc != QDELTA_OK) return rc;
  if (ws_bytes < need) return QDELTA_ENOWORKSPACE;
  if (B == 0) return QDELTA_OK;
  const int esz = dtype == QDELTA_BF16 ? 2 : 4;
  const int NT = (T + C - 1) / C;
  int L, G;
  seg_split(NT, n_segments, L, G);
  if (G == 1)    // one segment is the single pass
    return fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                    log_alpha, initial_state, o, final_state, saved, ws, ws_bytes, stream);
  const size_t slots = slots_for(B, T, 0), units = slots * (size_t)H;
  const SegLayout S = make_seg_layout(units, (size_t)B * H, G, Dk, Dv, esz);
  char* w = static_cast<char*>(ws);
  qd::Params p{};
  p.T = T;
  p.N = B;
  p.H = H;
  p.NT = NT;
  p.n_slots = (int)slots;
  p.cu = nullptr;
  p.q = q; p.k = k; p.v = v;
  p.beta = beta; p.lam = lam; p.lam_c = lam_scalar; p.la = log_alpha; p.S0 = initial_state;
  p.o = T > 0 ? o : nullptr;
  p.Sfin = final_state;
  p.wT = w + S.fwd.wT;
  if (saved) {
    bind_ctx(p, static_cast<char*>(saved), units, Dk, Dv, esz);
  } else {
    p.wb = reinterpret_cast<float*>(w + S.fwd.wb);
    p.wZ = w + S.fwd.wZ;
    p.wP = w + S.fwd.wP;
    p.wM = nullptr;
  }
  p.n_seg = G;
  p.seg_chunks = L;
  p.wSegOut = reinterpret_cast<float*>(w + S.out);
  p.wSegIn = reinterpret_cast<float*>(w + S.in);
  hipError_t e = qd::launch_fwd_seg(p, dtype, Dk, Dv, stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int qdelta_chunk_fwd_noalloc(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                             int32_t dtype, const void* q, const void* k, const void* v,
                             const float* beta, const float* lam, float lam_scalar,
                             const float* log_alpha, const float* initial_state, void* o,
                             float* final_state, hipStream_t stream) {
  // validate first (no device call): sizes past the scratch array return
  // QDELTA_ENOWORKSPACE; the workspace pointer is not dereferenced here
  void* const probe = reinterpret_cast<void*>(uintptr_t(256));
  int rc = fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                    log_alpha, initial_state, o, final_state, nullptr, probe, QDELTA_NOALLOC_SCRATCH_BYTES,
                    stream, true);
  if (rc != QDELTA_OK || B == 0) return rc;
  void* ws = nullptr;
  rc = scratch_ptr(&ws);
  if (rc != QDELTA_OK) return rc;
  // every workspace byte the kernels read is written earlier in the same
  // call (preparation before scan), so nothing needs clearing
  return fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                  log_alpha, initial_state, o, final_state, nullptr, ws, QDELTA_NOALLOC_SCRATCH_BYTES, stream);
}

int qdelta_chunk_bwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t chunk,
                     int32_t dtype, const void* q, const void* k, const void* v,
                     const float* beta, const float* lam, float lam_scalar, const float* log_alpha,
                     const float* initial_state, const void* saved, const void* d_o,
                     const float* d_final_state, void* dq, void* dk, void* dv, float* dbeta,
                     float* dlam, float* dlog_alpha, float* d_initial_state, void* ws,
                     size_t ws_bytes, hipStream_t stream) {
  return bwd_impl(false, B, T, B, nullptr, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                  log_alpha, initial_state, saved, d_o, d_final_state, dq, dk, dv, dbeta,
                  dlam, dlog_alpha, d_initial_state, ws, ws_bytes, stream);
}

int qdelta_chunk_bwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                            int32_t Dk, int32_t Dv, int32_t chunk, int32_t dtype,
                            const void* q, const void* k, const void* v, const float* beta,
                            const float* lam, float lam_scalar, const float* log_alpha,
                            const float* initial_state, const void* saved,
                            const void* d_o, const float* d_final_state, void* dq, void* dk,
                            void* dv, float* dbeta, float* dlam, float* dlog_alpha,
                            float* d_initial_state, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  return bwd_impl(true, 1, T, N, cu_seqlens, H, Dk, Dv, chunk, dtype, q, k, v, beta, lam, lam_scalar,
                  log_alpha, initial_state, saved, d_o, d_final_state, dq, dk, dv, dbeta,
                  dlam, dlog_alpha, d_initial_state, ws, ws_bytes, stream);
}

static int rec_fwd_impl(bool varlen, int32_t B, int32_t T, int32_t N, const int32_t* cu, int32_t H,
                 int32_t Dk, int32_t Dv, int32_t dtype, const void* q, const void* k,
                 const void* v, const float* beta, const float* lam, float lam_c, const float* log_alpha,
                 const float* initial_state, void* o, float* final_state, hipStream_t stream) {
  if (T < 0 || H <= 0) return QDELTA_EINVAL;
  if (varlen ? (N < 0 || cu == nullptr) : B < 0) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if ((Dk != 64 && Dk != 128) || Dv <= 0 || Dv > 256 || (Dv % 8) != 0) return QDELTA_EUNSUPPORTED;
  const int64_t tokens = varlen ? T : (int64_t)B * T;
  const int32_t n_seqs = varlen ? N : B;
  // token offsets (t * H + h) and unit indices stay below 2^31
  if (tokens * H >= (int64_t(1) << 31) || (int64_t)n_seqs * H >= (int64_t(1) << 31))
    return QDELTA_EUNSUPPORTED;
  if (tokens > 0 && !(ok_ptr(q) && ok_ptr(k) && ok_ptr(v) && ok_ptr(beta) && ok_ptr(o)))
    return QDELTA_EINVAL;
  if (!ok_opt(lam) || !ok_opt(log_alpha) || !ok_opt(initial_state) || !ok_opt(final_state))
    return QDELTA_EINVAL;
  if (n_seqs == 0) return QDELTA_OK;
  hipError_t e = qd::launch_rec_fwd(n_seqs, varlen ? 0 : T, varlen ? cu : nullptr, (int)tokens, H,
                                    Dk, Dv, dtype, q, k, v, beta, lam, lam_c, log_alpha, initial_state,
                                    final_state, o, stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int qdelta_recurrent_fwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                         const void* q, const void* k, const void* v, const float* beta,
                         const float* lam, float lam_scalar, const float* log_alpha,
                         const float* initial_state, void* o, float* final_state, hipStream_t stream) {
  return rec_fwd_impl(false, B, T, B, nullptr, H, Dk, Dv, dtype, q, k, v, beta, lam, lam_scalar, log_alpha,
                      initial_state, o, final_state, stream);
}

int qdelta_recurrent_fwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H,
                                int32_t Dk, int32_t Dv, int32_t dtype, const void* q,
                                const void* k, const void* v, const float* beta,
                                const float* lam, float lam_scalar, const float* log_alpha,
                                const float* initial_state, void* o, float* final_state,
                                hipStream_t stream) {
  return rec_fwd_impl(true, 1, T, N, cu_seqlens, H, Dk, Dv, dtype, q, k, v, beta, lam, lam_scalar,
                      log_alpha, initial_state, o, final_state, stream);
}

size_t qdelta_recurrent_workspace_bytes(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv,
                                        int32_t n_seqs) {
  if (B < 0 || T < 0 || H <= 0 || n_seqs < 0) return 0;
  if ((Dk != 64 && Dk != 128) || (Dv != 32 && Dv != 64 && Dv != 128 && Dv != 256)) return 0;
  const size_t tok = n_seqs > 0 ? (size_t)T : (size_t)B * T;
  const size_t units = (size_t)(n_seqs > 0 ? n_seqs : B) * H;
  auto r = [](size_t b) { return (b + 255) & ~size_t(255); };
  return 3 * r(tok * H * Dv * 4) + r(tok * H * Dk * 4) + r(units * Dv * 4) + r(tok * H * 4);
}

static int rec_bwd_impl(bool varlen, int32_t B, int32_t T, int32_t N, const int32_t* cu, int32_t H,
                        int32_t Dk, int32_t Dv, int32_t dtype, const void* q, const void* k, const void* v,
                        const float* beta, const float* lam, float lam_c, const float* log_alpha,
                        const float* initial_state, const void* d_o, const float* d_final_state, void* dq,
                        void* dk, void* dv, float* dbeta, float* dlam, float* dlog_alpha,
                        float* d_initial_state, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (T < 0 || H <= 0) return QDELTA_EINVAL;
  if (varlen ? (N < 0 || cu == nullptr) : B < 0) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if ((Dk != 64 && Dk != 128) || (Dv != 32 && Dv != 64 && Dv != 128 && Dv != 256)) return QDELTA_EUNSUPPORTED;
  const int64_t tokens = varlen ? T : (int64_t)B * T;
  const int32_t n_seqs = varlen ? N : B;
  if (tokens * H * (int64_t)(Dv > Dk ? Dv : Dk) >= (int64_t(1) << 31) || (int64_t)n_seqs * H >= (int64_t(1) << 31))
    return QDELTA_EUNSUPPORTED;
  const bool has_tokens = tokens > 0;
  if (has_tokens && !(ok_ptr(q) && ok_ptr(k) && ok_ptr(v) && ok_ptr(beta) && ok_ptr(d_o) && ok_ptr(dq) &&
                      ok_ptr(dk) && ok_ptr(dv) && ok_ptr(dbeta)))
    return QDELTA_EINVAL;
  if ((log_alpha == nullptr) != (dlog_alpha == nullptr) && has_tokens) return QDELTA_EINVAL;
  if (lam != nullptr && dlam == nullptr && has_tokens) return QDELTA_EINVAL;
  if (lam == nullptr && dlam != nullptr && (reinterpret_cast<uintptr_t>(dlam) & 3u)) return QDELTA_EINVAL;
  if (!ok_opt(lam) || (lam != nullptr && !ok_opt(dlam)) || !ok_opt(log_alpha) || !ok_opt(dlog_alpha) ||
      !ok_opt(initial_state) || !ok_opt(d_final_state) || !ok_opt(d_initial_state))
    return QDELTA_EINVAL;
  const size_t need = qdelta_recurrent_workspace_bytes(B, T, H, Dk, Dv, varlen ? (N > 0 ? N : 1) : 0);
  if (need > 0 && (ws == nullptr || !aligned(ws))) return QDELTA_EINVAL;
  if (ws_bytes < need) return QDELTA_ENOWORKSPACE;
  const bool dlam_const = lam == nullptr && dlam != nullptr;
  if (n_seqs == 0) {
    if (dlam_const) return qd::launch_zero(dlam, stream) == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
    return QDELTA_OK;
  }
  const size_t tok = (size_t)tokens;
  auto r = [](size_t b) { return (b + 255) & ~size_t(255); };
  char* w = static_cast<char*>(ws);
  qd::RecBwdArgs a{};
  a.T = varlen ? 0 : T;
  a.cu = varlen ? cu : nullptr;
  a.T_total = (int)tokens;
  a.H = H;
  a.DV = Dv;
  a.q = q; a.k = k; a.v = v; a.dO = d_o;
  a.beta = beta; a.lam = lam; a.lam_c = lam_c; a.la = log_alpha; a.S0 = initial_state; a.dSfin = d_final_state;
  a.dq = dq; a.dk = dk; a.dv = dv;
  a.dbeta = dbeta; a.dla = dlog_alpha; a.dS0 = d_initial_state;
  a.dlam = dlam_const ? nullptr : dlam;
  size_t off = 0;
  a.wP = reinterpret_cast<float*>(w + off); off += r(tok * H * Dv * 4);
  a.wZ = reinterpret_cast<float*>(w + off); off += r(tok * H * Dv * 4);
  a.wDP = reinterpret_cast<float*>(w + off); off += r(tok * H * Dv * 4);
  a.wWK = reinterpret_cast<float*>(w + off); off += r(tok * H * Dk * 4);
  a.wF = reinterpret_cast<float*>(w + off); off += r((size_t)n_seqs * H * Dv * 4);
  a.wDL = dlam_const ? reinterpret_cast<float*>(w + off) : nullptr;
  hipError_t e = qd::launch_rec_bwd(a, n_seqs * H, dtype, Dk, dlam_const ? dlam : nullptr, (long long)tok * H,
                                    stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int qdelta_recurrent_bwd(int32_t B, int32_t T, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                         const void* q, const void* k, const void* v, const float* beta,
                         const float* lam, float lam_scalar, const float* log_alpha,
                         const float* initial_state, const void* d_o, const float* d_final_state,
                         void* dq, void* dk, void* dv, float* dbeta, float* dlam, float* dlog_alpha,
                         float* d_initial_state, void* ws, size_t ws_bytes, hipStream_t stream) {
  return rec_bwd_impl(false, B, T, B, nullptr, H, Dk, Dv, dtype, q, k, v, beta, lam, lam_scalar, log_alpha,
                      initial_state, d_o, d_final_state, dq, dk, dv, dbeta, dlam, dlog_alpha, d_initial_state, ws,
                      ws_bytes, stream);
}

int qdelta_recurrent_bwd_varlen(int32_t T, int32_t N, const int32_t* cu_seqlens, int32_t H, int32_t Dk,
                                int32_t Dv, int32_t dtype, const void* q, const void* k, const void* v,
                                const float* beta, const float* lam, float lam_scalar,
                                const float* log_alpha, const float* initial_state, const void* d_o,
                                const float* d_final_state, void* dq, void* dk, void* dv, float* dbeta,
                                float* dlam, float* dlog_alpha, float* d_initial_state, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
  return rec_bwd_impl(true, 1, T, N, cu_seqlens, H, Dk, Dv, dtype, q, k, v, beta, lam, lam_scalar, log_alpha,
                      initial_state, d_o, d_final_state, dq, dk, dv, dbeta, dlam, dlog_alpha, d_initial_state, ws,
                      ws_bytes, stream);
}

int qdelta_l2norm_fwd(int64_t rows, int32_t D, int64_t ld_x, int32_t dtype, const void* x, void* y,
                      float* rnorm, hipStream_t stream) {
  if (rows < 0 || ld_x < D) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if (D != 64 && D != 128) return QDELTA_EUNSUPPORTED;
  const int esz = dtype == QDELTA_BF16 ? 2 : 4;
  if ((ld_x * esz) % 16 != 0) return QDELTA_EINVAL;
  if (rows >= (int64_t(1) << 31)) return QDELTA_EUNSUPPORTED;
  if (rows == 0) return QDELTA_OK;
  if (!(ok_ptr(x) && ok_ptr(y) && ok_ptr(rnorm))) return QDELTA_EINVAL;
  hipError_t e = qd::launch_l2norm(0, rows, D, ld_x, dtype, x, nullptr, nullptr, rnorm, nullptr, y,
                                   stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int qdelta_l2norm_bwd(int64_t rows, int32_t D, int32_t dtype, const void* y, const float* rnorm,
                      const void* dy, void* dx, hipStream_t stream) {
  if (rows < 0) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if (D != 64 && D != 128) return QDELTA_EUNSUPPORTED;
  if (rows >= (int64_t(1) << 31)) return QDELTA_EUNSUPPORTED;
  if (rows == 0) return QDELTA_OK;
  if (!(ok_ptr(y) && ok_ptr(rnorm) && ok_ptr(dy) && ok_ptr(dx))) return QDELTA_EINVAL;
  hipError_t e = qd::launch_l2norm(1, rows, D, D, dtype, nullptr, y, rnorm, nullptr, dy, dx, stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

int qdelta_recurrent_step(int32_t N, int32_t H, int32_t Dk, int32_t Dv, int32_t dtype,
                          const void* q, const void* k, const void* v, const float* beta,
                          const float* lam, float lam_scalar, const float* log_alpha, float* state,
                          void* o, hipStream_t stream) {
  if (N < 0 || H <= 0) return QDELTA_EINVAL;
  if (dtype != QDELTA_F32 && dtype != QDELTA_BF16) return QDELTA_EINVAL;
  if ((Dk != 64 && Dk != 128) || Dv <= 0 || Dv > 256 || (Dv % 8) != 0) return QDELTA_EUNSUPPORTED;
  if ((int64_t)N * H * 32 >= (int64_t(1) << 31)) return QDELTA_EUNSUPPORTED;
  if (N == 0) return QDELTA_OK;
  if (!(ok_ptr(q) && ok_ptr(k) && ok_ptr(v) && ok_ptr(beta) && ok_ptr(state) && ok_ptr(o) &&
        ok_opt(lam) && ok_opt(log_alpha)))
    return QDELTA_EINVAL;
  hipError_t e = qd::launch_step(N, H, Dk, Dv, dtype, q, k, v, beta, lam, lam_scalar, log_alpha, state, o,
                                 stream);
  return e == hipSuccess ? QDELTA_OK : QDELTA_EHIP;
}

}  // extern "C"
