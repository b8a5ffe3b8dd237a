// Host side of the C ABI: argument validation (before anything is enqueued),
// workspace layout, and the launch sequence of one exit's forward and
// backward passes.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ee_tuning.h"
#include "launch.h"

// The workspace of ee_exit_decide_static: a fixed array in the library's own
// device memory, one per GPU (it comes with the code object when the library
// is loaded on a device and stays until the process ends).  In host code
// `scratch` names a host-side shadow, not device memory: kernels receive the
// device address that hipGetSymbolAddress gives for the current device.
static __device__ __align__(256) char scratch[EE_STATIC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

ee_status fail(ee_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

constexpr int64_t kMaxTokens = 1 << 20;
constexpr int64_t kMaxHidden = 32768;
constexpr int64_t kMaxVocab = 1 << 20;
constexpr int64_t kMaxInter = 65536;
constexpr int64_t kMaxMlpHidden = 8192;  // the exit-norm backward keeps a row in registers
constexpr size_t kAlign = 256;

int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Workspace regions of one exit.  The first 256 bytes are a header shared
// by every exit: the device error flag and a scratch loss slot.
struct Layout {
  int64_t ldn = 0, vtiles = 0, itiles = 0;
  int vtile = 0, itile = 0;
  size_t z = 0, zht = 0, r = 0, P = 0, pm = 0, pl = 0, tgt = 0, lse = 0, sn = 0, bsum = 0, dgp = 0;
  size_t u = 0, uhat = 0, rx = 0, hg = 0, act = 0, y = 0, dz = 0, dy = 0, dhg = 0, dhu = 0,
         dgpg = 0, dgpu = 0;
  size_t mu = 0, gsp = 0, gsum = 0, dbp = 0;  // LayerNorm mean; bias: G row sums, bias partials
  size_t coef = 0, fb = 0;                    // unshifted form: s_n exp(-LSE_n), range-check flag
  ee::SplitTail zs{0, 0, 1};                  // split-K tail of the dZ product
  ee::SplitTail ys{0, 0, 1};                  // split-K tail of the down projection
  int64_t gchunks = 0;
  size_t total = 0;
};
constexpr size_t kFlagOff = 0;
constexpr size_t kLossSlotOff = 16;
constexpr size_t kHeader = 256;

Layout layout(const ee_exit &e, int64_t n) {
  Layout L;
  const size_t es = e.dtype == EE_BF16 ? 2 : 4;
  const size_t h = static_cast<size_t>(e.hidden), V = static_cast<size_t>(e.vocab);
  const size_t I = static_cast<size_t>(e.intermediate), N = static_cast<size_t>(n);
  L.ldn = cdiv64(n, ee::kTokenPad) * ee::kTokenPad;
  const bool f32 = e.dtype == EE_F32;
  L.vtile = ee::gemm_part_cols(f32);  // partial slices of the logits and dW_out GEMMs
  L.itile = ee::gemm_part_cols(f32);  // and of the dW_gate / dW_up GEMMs
  L.vtiles = cdiv64(e.vocab, L.vtile);
  L.itiles = cdiv64(e.intermediate, L.itile);
  const size_t ldn = static_cast<size_t>(L.ldn);
  size_t cur = kHeader;
  auto take = [&](size_t bytes) {
    const size_t o = align_up(cur);
    cur = o + bytes;
    return o;
  };
  const bool normed = e.kind == EE_EXIT_NORM || e.kind == EE_EXIT_MLP;
  if (normed) L.z = take(N * h * es);
  L.zht = take(h * ldn * es);
  L.r = take(ldn * 4);
  L.P = take(V * ldn * es);
  L.pm = take(static_cast<size_t>(L.vtiles) * ldn * 4);
  L.pl = take(static_cast<size_t>(L.vtiles) * ldn * 4);
  L.tgt = take(ldn * 4);
  L.lse = take(ldn * 4);
  L.sn = take(ldn * 4);
  L.bsum = take(static_cast<size_t>(cdiv64(n, 32)) * 4);
  L.coef = take(ldn * 4);
  L.fb = take(4);
  if (normed) L.dgp = take(static_cast<size_t>(L.vtiles) * h * 4);
  if (e.norm == EE_NORM_LAYER) L.mu = take(ldn * 4);
  if (e.beta != nullptr) {
    L.gchunks = ee::seed_chunks(static_cast<int>(L.ldn));
    L.gsp = take(static_cast<size_t>(L.gchunks) * V * 4);
    L.gsum = take(V * 4);
    L.dbp = take(static_cast<size_t>(L.vtiles) * h * 4);
  }
  if (e.kind == EE_EXIT_MLP) {
    L.u = take(N * h * es);
    L.uhat = take(h * ldn * es);  // U_hat^T, token-contiguous
    L.rx = take(ldn * 4);
    L.hg = take(2 * N * I * es);  // (H_g, H_u) side by side per element
    L.act = take(N * I * es);
    L.ys = ee::split_tail(f32, static_cast<int>(n), static_cast<int>(h), static_cast<int>(I));
    L.y = take(static_cast<size_t>(L.ys.splits) * N * h * 4);
    L.zs = ee::split_tail(f32, static_cast<int>(n), static_cast<int>(h), static_cast<int>(V));
    L.dz = take(static_cast<size_t>(L.zs.splits) * N * h * 4);
    L.dy = take(N * h * es);
    L.dhg = take(I * ldn * es);  // dH_g^T, token-contiguous
    L.dhu = take(I * ldn * es);
    L.dgpg = take(static_cast<size_t>(L.itiles) * h * 4);
    L.dgpu = take(static_cast<size_t>(L.itiles) * h * 4);
  }
  L.total = align_up(cur);
  return L;
}

bool misaligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

ee_status check_ptr(const void *p, const char *what) {
  if (p == nullptr) return fail(EE_ERR_NULL, "%s is NULL", what);
  if (misaligned(p)) return fail(EE_ERR_ALIGN, "%s is not 16-byte aligned", what);
  return EE_OK;
}

ee_status check_opt_ptr(const void *p, const char *what) {
  if (p != nullptr && misaligned(p)) return fail(EE_ERR_ALIGN, "%s is not 16-byte aligned", what);
  return EE_OK;
}

#define EE_TRY(expr)                 \
  do {                               \
    const ee_status _s = (expr);     \
    if (_s != EE_OK) return _s;      \
  } while (0)

ee_status validate_exit(const ee_exit *e, int idx) {
  if (e == nullptr) return fail(EE_ERR_NULL, "exit %d descriptor is NULL", idx);
  if (e->kind == EE_EXIT_LAYER)
    return fail(EE_ERR_UNSUPPORTED, "exit %d: the Layer exit (a full Transformer layer) is not implemented", idx);
  if (e->kind < EE_EXIT_EMBEDDING || e->kind > EE_EXIT_MLP)
    return fail(EE_ERR_UNSUPPORTED, "exit %d: unknown exit kind %d", idx, e->kind);
  if (e->dtype != EE_F32 && e->dtype != EE_BF16) return fail(EE_ERR_DTYPE, "exit %d: unknown dtype %d", idx, e->dtype);
  if (e->hidden < 64 || e->hidden > kMaxHidden || e->hidden % 64 != 0)
    return fail(EE_ERR_SHAPE, "exit %d: hidden=%lld must be a multiple of 64 in [64, %lld]", idx,
                static_cast<long long>(e->hidden), static_cast<long long>(kMaxHidden));
  if (e->vocab < 1 || e->vocab > kMaxVocab)
    return fail(EE_ERR_SHAPE, "exit %d: vocab=%lld must be in [1, %lld]", idx, static_cast<long long>(e->vocab),
                static_cast<long long>(kMaxVocab));
  if (e->kind == EE_EXIT_MLP) {
    if (e->hidden > kMaxMlpHidden)
      return fail(EE_ERR_SHAPE, "exit %d: an MLP exit needs hidden <= %lld", idx, static_cast<long long>(kMaxMlpHidden));
    if (e->intermediate < 64 || e->intermediate > kMaxInter || e->intermediate % 64 != 0)
      return fail(EE_ERR_SHAPE, "exit %d: intermediate=%lld must be a multiple of 64 in [64, %lld]", idx,
                  static_cast<long long>(e->intermediate), static_cast<long long>(kMaxInter));
  } else if (e->intermediate != 0) {
    return fail(EE_ERR_SHAPE, "exit %d: intermediate must be 0 for a non-MLP exit", idx);
  }
  if (!(e->rms_eps >= 0.0f) || !std::isfinite(e->rms_eps))
    return fail(EE_ERR_SHAPE, "exit %d: rms_eps must be finite and >= 0", idx);
  if (e->norm != EE_NORM_RMS && e->norm != EE_NORM_LAYER)
    return fail(EE_ERR_UNSUPPORTED, "exit %d: unknown norm %d", idx, e->norm);
  if (e->norm == EE_NORM_LAYER && e->kind != EE_EXIT_NORM)
    return fail(EE_ERR_UNSUPPORTED, "exit %d: LayerNorm is available for Norm exits only", idx);
  if (e->beta != nullptr && e->norm != EE_NORM_LAYER)
    return fail(EE_ERR_SHAPE, "exit %d: beta is the bias of a LayerNorm exit", idx);
  EE_TRY(check_opt_ptr(e->beta, "beta"));
  EE_TRY(check_ptr(e->w_out, "w_out"));
  if (e->kind != EE_EXIT_EMBEDDING) EE_TRY(check_ptr(e->gamma, "gamma"));
  if (e->kind == EE_EXIT_MLP) {
    EE_TRY(check_ptr(e->gamma_mlp, "gamma_mlp"));
    EE_TRY(check_ptr(e->w_gate, "w_gate"));
    EE_TRY(check_ptr(e->w_up, "w_up"));
    EE_TRY(check_ptr(e->w_down, "w_down"));
  }
  return EE_OK;
}

ee_status validate_tokens(int64_t n) {
  if (n < 1 || n > kMaxTokens)
    return fail(EE_ERR_SHAPE, "n_tokens=%lld must be in [1, %lld] (the loss is a mean over tokens)",
                static_cast<long long>(n), static_cast<long long>(kMaxTokens));
  return EE_OK;
}

struct Range {
  uintptr_t lo, hi;
  const char *what;
};

bool overlap(const Range &a, const Range &b) { return a.lo < b.hi && b.lo < a.hi; }

Range make_range(const void *p, size_t bytes, const char *what) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Range{lo, lo + bytes, what};
}

// Gradient buffers of one exit, with their sizes.
int grad_ranges(const ee_exit &e, const ee_exit_grads &g, Range *out) {
  const size_t h = e.hidden, V = e.vocab, I = e.intermediate;
  int k = 0;
  out[k++] = make_range(g.d_w_out, V * h * 4, "d_w_out");
  if (e.kind != EE_EXIT_EMBEDDING) out[k++] = make_range(g.d_gamma, h * 4, "d_gamma");
  if (e.beta != nullptr) out[k++] = make_range(g.d_beta, h * 4, "d_beta");
  if (e.kind == EE_EXIT_MLP) {
    out[k++] = make_range(g.d_gamma_mlp, h * 4, "d_gamma_mlp");
    out[k++] = make_range(g.d_w_gate, I * h * 4, "d_w_gate");
    out[k++] = make_range(g.d_w_up, I * h * 4, "d_w_up");
    out[k++] = make_range(g.d_w_down, h * I * 4, "d_w_down");
  }
  return k;
}

int param_ranges(const ee_exit &e, Range *out) {
  const size_t es = e.dtype == EE_BF16 ? 2 : 4;
  const size_t h = e.hidden, V = e.vocab, I = e.intermediate;
  int k = 0;
  out[k++] = make_range(e.w_out, V * h * es, "w_out");
  if (e.kind != EE_EXIT_EMBEDDING) out[k++] = make_range(e.gamma, h * es, "gamma");
  if (e.beta != nullptr) out[k++] = make_range(e.beta, h * es, "beta");
  if (e.kind == EE_EXIT_MLP) {
    out[k++] = make_range(e.gamma_mlp, h * es, "gamma_mlp");
    out[k++] = make_range(e.w_gate, I * h * es, "w_gate");
    out[k++] = make_range(e.w_up, I * h * es, "w_up");
    out[k++] = make_range(e.w_down, h * I * es, "w_down");
  }
  return k;
}

ee_status validate_grads(const ee_exit &e, const ee_exit_grads *g, int idx) {
  if (g == nullptr) return fail(EE_ERR_NULL, "gradient set of exit %d is NULL", idx);
  EE_TRY(check_ptr(g->d_w_out, "d_w_out"));
  if (e.kind != EE_EXIT_EMBEDDING) EE_TRY(check_ptr(g->d_gamma, "d_gamma"));
  if (e.beta != nullptr) EE_TRY(check_ptr(g->d_beta, "d_beta"));
  if (e.kind == EE_EXIT_MLP) {
    EE_TRY(check_ptr(g->d_gamma_mlp, "d_gamma_mlp"));
    EE_TRY(check_ptr(g->d_w_gate, "d_w_gate"));
    EE_TRY(check_ptr(g->d_w_up, "d_w_up"));
    EE_TRY(check_ptr(g->d_w_down, "d_w_down"));
  }
  return EE_OK;
}

ee_status hip_fail(hipError_t err, const char *where) {
  return fail(EE_ERR_HIP, "%s: %s", where, hipGetErrorString(err));
}

#define EE_HIP(call, where)                           \
  do {                                                \
    const hipError_t _e = (call);                     \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

// ------------------------------------------------------- kernel timing
// Diagnostics only: while enabled, every launch of the step is bracketed by
// a pair of HIP events recorded on the launch stream.
struct ProfRecord {
  const char *name;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
thread_local bool g_prof_suspended = false;  // set while a call must not create events
std::vector<ProfRecord> g_prof_records;
std::vector<hipEvent_t> g_prof_pool;
size_t g_prof_used = 0;

hipEvent_t prof_event() {
  if (g_prof_used == g_prof_pool.size()) {
    hipEvent_t ev = nullptr;
    if (hipEventCreate(&ev) != hipSuccess) return nullptr;
    g_prof_pool.push_back(ev);
  }
  return g_prof_pool[g_prof_used++];
}

// Launch `call` (a hipError_t expression) as kernel `name` on stream s.
#define EE_LAUNCH(name, s, call)                                         \
  do {                                                                   \
    hipEvent_t _a = nullptr, _b = nullptr;                               \
    if (g_prof_on && !g_prof_suspended) {                                \
      std::lock_guard<std::mutex> _g(g_prof_mu);                         \
      _a = prof_event();                                                 \
      _b = prof_event();                                                 \
      if (_a != nullptr) (void)hipEventRecord(_a, s);                    \
    }                                                                    \
    EE_HIP(call, name);                                                  \
    if (_a != nullptr && _b != nullptr) {                                \
      std::lock_guard<std::mutex> _g(g_prof_mu);                         \
      (void)hipEventRecord(_b, s);                                       \
      g_prof_records.push_back(ProfRecord{name, _a, _b});                \
    }                                                                    \
  } while (0)

char *at(void *ws, size_t off) { return static_cast<char *>(ws) + off; }
float *atf(void *ws, size_t off) { return reinterpret_cast<float *>(at(ws, off)); }

bool unshifted_form(const ee_exit &e) { return e.vocab >= 64; }

// Forward of one exit; see ee_head_forward_loss.
ee_status run_forward(const ee_exit &e, const void *x, const int32_t *targets, const float *token_w, int64_t n64,
                      float w_e, uint32_t flags, void *ws, float *loss, float *row_loss, float *total, int first,
                      hipStream_t s) {
  const Layout L = layout(e, n64);
  const bool f32 = e.dtype == EE_F32;
  const int n = static_cast<int>(n64), h = static_cast<int>(e.hidden), V = static_cast<int>(e.vocab);
  const int I = static_cast<int>(e.intermediate), ldn = static_cast<int>(L.ldn);
  const void *zsrc = x;
  // The first exit of a call clears the device error record in its first
  // kernel; every exit's first kernel clears its range-check flag.
  int *clear = first ? reinterpret_cast<int *>(at(ws, kFlagOff)) : nullptr;
  // Exits take the unshifted form of the logits (P = exp(S)), with a bias
  // too (G's row sums for its gradient then come from one read of P'),
  // except for a vocabulary of less than one 64-id slice (where the seed
  // costs nothing, and a single id keeps its loss exactly 0: exp(S - m) = 1).
  const bool unshifted = unshifted_form(e);
  int *fb = reinterpret_cast<int *>(at(ws, L.fb));
  if (e.kind == EE_EXIT_MLP) {
    if (ee::norm_rows(h, f32)) {
      EE_LAUNCH("mlp pre-norm", s, ee::launch_norm_rows(f32, x, h, n, ldn, h, e.rms_eps, e.gamma_mlp, nullptr, atf(ws, L.rx),
                                                        nullptr, at(ws, L.u), at(ws, L.uhat), s, clear, fb));
    } else {
      EE_LAUNCH("mlp pre-norm rms", s, ee::launch_row_rms(f32, x, h, n, h, e.rms_eps, atf(ws, L.rx), s, nullptr, clear, fb));
      EE_LAUNCH("mlp pre-norm apply", s, ee::launch_norm_apply(f32, f32, x, h, atf(ws, L.rx), e.gamma_mlp, n, ldn, h,
                                                               at(ws, L.u), nullptr, at(ws, L.uhat), s));
    }
    EE_LAUNCH("gate and up projections + swiglu", s, ee::gemm_gate_up_swiglu(f32, at(ws, L.u), e.w_gate, e.w_up, n, I, h, at(ws, L.hg),
                                                                             at(ws, L.act), s));
    EE_LAUNCH("down projection + residual", s, ee::gemm_down_residual(f32, at(ws, L.act), e.w_down, x, n, h, I, atf(ws, L.y), s, L.ys));
    EE_LAUNCH("exit norm rms", s, ee::launch_row_rms_split(atf(ws, L.y), n, h, e.rms_eps, atf(ws, L.r), L.ys, s));
    EE_LAUNCH("exit norm apply", s, ee::launch_norm_apply(true, f32, atf(ws, L.y), h, atf(ws, L.r), e.gamma, n, ldn, h, at(ws, L.z),
                                 nullptr, at(ws, L.zht), s));
    zsrc = at(ws, L.z);
  } else if (e.kind == EE_EXIT_NORM) {
    float *mu = e.norm == EE_NORM_LAYER ? atf(ws, L.mu) : nullptr;
    if (ee::norm_rows(h, f32)) {
      EE_LAUNCH("exit norm", s, ee::launch_norm_rows(f32, x, h, n, ldn, h, e.rms_eps, e.gamma, e.beta, atf(ws, L.r), mu,
                                                     at(ws, L.z), at(ws, L.zht), s, clear, fb));
    } else {
      EE_LAUNCH("exit norm rms", s, ee::launch_row_rms(f32, x, h, n, h, e.rms_eps, atf(ws, L.r), s, mu, clear, fb));
      EE_LAUNCH("exit norm apply", s, ee::launch_norm_apply(f32, f32, x, h, atf(ws, L.r), e.gamma, n, ldn, h, at(ws, L.z),
                                                            nullptr, at(ws, L.zht), s, mu, e.beta));
    }
    zsrc = at(ws, L.z);
  } else {
    EE_LAUNCH("hidden-state transpose", s, ee::launch_norm_apply(f32, f32, x, h, nullptr, nullptr, n, ldn, h, nullptr, nullptr, at(ws, L.zht), s,
                                                                 nullptr, nullptr, clear, fb));
  }
  EE_LAUNCH("logits + softmax partials", s, ee::gemm_logits(f32, e.w_out, zsrc, V, n, h, at(ws, L.P), ldn, atf(ws, L.pm), atf(ws, L.pl),
                         atf(ws, L.tgt), targets, s,
                         unshifted ? ((flags & EE_FLAG_DYNAMIC_TOKEN_WEIGHTS) ? 1 : 2) : 0));
  ee::CeReduceArgs a{};
  a.part_m = atf(ws, L.pm);
  a.part_l = atf(ws, L.pl);
  a.tgt = atf(ws, L.tgt);
  a.targets = targets;
  a.token_w = token_w;
  a.lse = atf(ws, L.lse);
  a.sn = atf(ws, L.sn);
  a.row_loss = row_loss;
  a.block_sums = atf(ws, L.bsum);
  a.flag = reinterpret_cast<int *>(at(ws, kFlagOff));
  a.n = n;
  a.ldn = ldn;
  a.vocab = V;
  a.tiles = static_cast<int>(L.vtiles);
  a.exit_weight = w_e;
  a.dynamic_weights = (flags & EE_FLAG_DYNAMIC_TOKEN_WEIGHTS) ? 1 : 0;
  a.shift0 = unshifted ? 1 : 0;
  a.fallback = fb;
  a.coef = atf(ws, L.coef);
  EE_LAUNCH("cross-entropy reduce", s, ee::launch_ce_reduce(a, s));
  const bool bias = e.beta != nullptr;
  if (unshifted) {
    // G = diag(coef) P' (see launch_seed_or_scale), unless a row was out of
    // the unshifted range: then the launches gated on its flag redo the
    // logits, the reduce and the seed in the shifted form.
    EE_LAUNCH("logits, shifted (if out of range)", s, ee::gemm_logits(f32, e.w_out, zsrc, V, n, h, at(ws, L.P), ldn, atf(ws, L.pm),
                                                                      atf(ws, L.pl), atf(ws, L.tgt), targets, s, 0, fb));
    a.shift0 = 0;
    a.run_if = fb;
    EE_LAUNCH("cross-entropy reduce, shifted (if out of range)", s, ee::launch_ce_reduce(a, s));
    EE_LAUNCH("operand scale (or seed, if out of range) and loss", s,
              ee::launch_seed_or_scale(f32, at(ws, L.P), at(ws, L.zht), atf(ws, L.pm), atf(ws, L.lse), atf(ws, L.sn), atf(ws, L.coef),
                                       targets, n, ldn, h, V, L.vtile, fb, atf(ws, L.bsum), static_cast<int>(cdiv64(n, 32)), loss,
                                       total, w_e, first, s, bias ? atf(ws, L.gsp) : nullptr));
    if (bias)
      EE_LAUNCH("logit-gradient row sums (unshifted form)", s,
                ee::launch_gsum_unshifted(f32, at(ws, L.P), atf(ws, L.coef), n, ldn, V, fb, atf(ws, L.gsp), s));
  } else {
    EE_LAUNCH("logit seed", s, ee::launch_seed(f32, at(ws, L.P), atf(ws, L.pm), atf(ws, L.lse), atf(ws, L.sn), targets, n, ldn, V, L.vtile,
                                               s, bias ? atf(ws, L.gsp) : nullptr));
  }
  if (bias)
    EE_LAUNCH("logit-gradient row sums", s, ee::launch_gain_reduce(atf(ws, L.gsp), static_cast<int>(L.gchunks), nullptr, 0, V,
                                                                   atf(ws, L.gsum), 0, s));
  if (!unshifted)
    EE_LAUNCH("loss reduce", s, ee::launch_final_loss(atf(ws, L.bsum), static_cast<int>(cdiv64(n, 32)), n, loss, total, w_e, first, s));
  return EE_OK;
}

// Backward of one exit; see ee_head_backward.
ee_status run_backward(const ee_exit &e, int64_t n64, void *ws, const ee_exit_grads &g, int acc, hipStream_t s) {
  const Layout L = layout(e, n64);
  const bool f32 = e.dtype == EE_F32;
  const int n = static_cast<int>(n64), h = static_cast<int>(e.hidden), V = static_cast<int>(e.vocab);
  const int I = static_cast<int>(e.intermediate), ldn = static_cast<int>(L.ldn);
  const bool normed = e.kind != EE_EXIT_EMBEDDING;
  const bool bias = e.beta != nullptr;
  EE_LAUNCH("output-matrix gradient", s, ee::gemm_weight_grad_kk(f32, at(ws, L.P), at(ws, L.zht), V, h, ldn, normed ? e.gamma : nullptr,
                                 normed ? e.w_out : nullptr, g.d_w_out, normed ? atf(ws, L.dgp) : nullptr, acc, s,
                                 bias ? atf(ws, L.gsum) : nullptr, e.beta, bias ? atf(ws, L.dbp) : nullptr));
  if (normed)
    EE_LAUNCH("exit gain gradient", s, ee::launch_gain_reduce(atf(ws, L.dgp), static_cast<int>(L.vtiles), nullptr, 0, h, g.d_gamma, acc, s));
  if (bias)
    EE_LAUNCH("exit bias gradient", s, ee::launch_gain_reduce(atf(ws, L.dbp), static_cast<int>(L.vtiles), nullptr, 0, h, g.d_beta, acc, s));
  if (e.kind != EE_EXIT_MLP) return EE_OK;
  const bool unshifted = unshifted_form(e);  // as in run_forward: G = diag(coef) P' unless the flag is set
  EE_LAUNCH("dZ", s, ee::gemm_dz(f32, at(ws, L.P), e.w_out, n, ldn, h, V, atf(ws, L.dz), s, L.zs));
  EE_LAUNCH("exit norm backward", s, ee::launch_norm_bwd(f32, atf(ws, L.dz), atf(ws, L.y), atf(ws, L.r), e.gamma, n, h, at(ws, L.dy), s,
                                                         L.zs, unshifted ? atf(ws, L.coef) : nullptr,
                                                         reinterpret_cast<const int *>(at(ws, L.fb))));
  EE_LAUNCH("dA + swiglu backward, down gradient", s,
            ee::gemm_da_swiglu_dw_down(f32, at(ws, L.dy), e.w_down, n, I, h, at(ws, L.hg), at(ws, L.dhg), at(ws, L.dhu),
                                       ldn, at(ws, L.act), g.d_w_down, acc, s));
  EE_LAUNCH("gate and up gradients", s,
            ee::gemm_weight_grad_kk_pair(f32, at(ws, L.dhg), at(ws, L.dhu), at(ws, L.uhat), I, h, ldn, e.gamma_mlp, e.w_gate,
                                         e.w_up, g.d_w_gate, g.d_w_up, atf(ws, L.dgpg), atf(ws, L.dgpu), acc, s));
  EE_LAUNCH("mlp gain gradient", s, ee::launch_gain_reduce(atf(ws, L.dgpg), static_cast<int>(L.itiles), atf(ws, L.dgpu),
                                static_cast<int>(L.itiles), h, g.d_gamma_mlp, acc, s));
  return EE_OK;
}

ee_status check_workspace(void *ws, size_t ws_bytes, size_t need) {
  EE_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < need)
    return fail(EE_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  return EE_OK;
}

// Outputs (gradients, losses) must not overlap each other or any input.
ee_status check_aliasing(int n_exits, const ee_exit *exits, const void *const *hidden, const int32_t *targets,
                         const float *token_w, int64_t n, const ee_exit_grads *grads, const float *loss_a,
                         size_t loss_a_bytes, const float *loss_b, size_t loss_b_bytes, void *ws, size_t ws_bytes) {
  constexpr int kMaxRanges = 8;
  std::vector<Range> outs, ins;
  for (int i = 0; i < n_exits; ++i) {
    Range r[kMaxRanges];
    if (grads != nullptr) {
      const int k = grad_ranges(exits[i], grads[i], r);
      outs.insert(outs.end(), r, r + k);
    }
    const int k = param_ranges(exits[i], r);
    ins.insert(ins.end(), r, r + k);
    const size_t es = exits[i].dtype == EE_BF16 ? 2 : 4;
    if (hidden != nullptr) ins.push_back(make_range(hidden[i], static_cast<size_t>(n) * exits[i].hidden * es, "hidden"));
  }
  if (loss_a != nullptr) outs.push_back(make_range(loss_a, loss_a_bytes, "loss"));
  if (loss_b != nullptr) outs.push_back(make_range(loss_b, loss_b_bytes, "loss"));
  if (targets != nullptr) ins.push_back(make_range(targets, static_cast<size_t>(n) * 4, "targets"));
  if (token_w != nullptr) ins.push_back(make_range(token_w, static_cast<size_t>(n) * 4, "token_w"));
  ins.push_back(make_range(ws, ws_bytes, "workspace"));
  for (size_t i = 0; i < outs.size(); ++i) {
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlap(outs[i], outs[j]))
        return fail(EE_ERR_ALIAS, "output %s overlaps output %s", outs[i].what, outs[j].what);
    for (const Range &r : ins)
      if (overlap(outs[i], r)) return fail(EE_ERR_ALIAS, "output %s overlaps input %s", outs[i].what, r.what);
  }
  return EE_OK;
}

// ------------------------------------------------------------ decode
// Workspace regions of the decode-time decision for n rows.
struct DecLayout {
  size_t z = 0, u = 0, hg = 0, act = 0, y = 0, pm = 0, pl = 0, pa = 0, total = 0;
  int tiles = 0;
};

DecLayout dec_layout(const ee_exit &e, int64_t n) {
  DecLayout L;
  const size_t es = e.dtype == EE_BF16 ? 2 : 4;
  const size_t h = static_cast<size_t>(e.hidden), I = static_cast<size_t>(e.intermediate);
  const size_t N = static_cast<size_t>(n);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.z = take(N * h * es);
  if (e.kind == EE_EXIT_MLP) {
    L.u = take(N * h * es);
    L.hg = take(N * I * es);
    L.act = take(N * I * es);
    L.y = take(N * h * 4);
  }
  L.tiles = ee::decode_tiles(static_cast<int>(e.vocab));
  L.pm = take(static_cast<size_t>(L.tiles) * N * 4);
  L.pl = take(static_cast<size_t>(L.tiles) * N * 4);
  L.pa = take(static_cast<size_t>(L.tiles) * N * 4);
  L.total = off;
  return L;
}

ee_status validate_rows(int64_t n) {
  if (n < 1 || n > kMaxTokens)
    return fail(EE_ERR_SHAPE, "n_rows=%lld must be in [1, %lld]", static_cast<long long>(n),
                static_cast<long long>(kMaxTokens));
  return EE_OK;
}

ee_status validate_decide(const ee_exit *e, const void *hidden, int64_t n_rows, float threshold, int32_t *token,
                          float *confidence, int32_t *exit_flag) {
  EE_TRY(validate_exit(e, 0));
  EE_TRY(validate_rows(n_rows));
  if (std::isnan(threshold)) return fail(EE_ERR_SHAPE, "threshold is NaN");
  EE_TRY(check_ptr(hidden, "hidden"));
  EE_TRY(check_ptr(token, "token"));
  EE_TRY(check_ptr(confidence, "confidence"));
  EE_TRY(check_ptr(exit_flag, "exit_flag"));
  return EE_OK;
}

// Outputs must not overlap each other, the inputs or the workspace (ws may be
// NULL: the fixed array of ee_exit_decide_static is no caller buffer).
ee_status check_decide_aliasing(const ee_exit &e, const void *hidden, int64_t n_rows, int32_t *token,
                                float *confidence, int32_t *exit_flag, void *ws, size_t ws_bytes) {
  const size_t n = static_cast<size_t>(n_rows);
  const size_t es = e.dtype == EE_BF16 ? 2 : 4;
  Range outs[4] = {make_range(token, n * 4, "token"), make_range(confidence, n * 4, "confidence"),
                   make_range(exit_flag, n * 4, "exit_flag"), make_range(ws, ws_bytes, "workspace")};
  const int n_outs = ws != nullptr ? 4 : 3;
  Range ins[8];
  int k = param_ranges(e, ins);
  ins[k++] = make_range(hidden, n * static_cast<size_t>(e.hidden) * es, "hidden");
  for (int a = 0; a < n_outs; ++a) {
    for (int b = a + 1; b < n_outs; ++b)
      if (overlap(outs[a], outs[b])) return fail(EE_ERR_ALIAS, "%s overlaps %s", outs[a].what, outs[b].what);
    for (int b = 0; b < k; ++b)
      if (overlap(outs[a], ins[b])) return fail(EE_ERR_ALIAS, "%s overlaps %s", outs[a].what, ins[b].what);
  }
  return EE_OK;
}

// ------------------------------------------- decode without allocation
constexpr size_t kStaticScratchBytes = EE_STATIC_SCRATCH_BYTES;

std::mutex g_scratch_mu;
std::vector<void *> g_scratch_ptr;  // per device, looked up on the first call there

ee_status static_scratch(void **out) {
  int dev = 0;
  EE_HIP(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_ptr.empty()) {
    int count = 0;
    EE_HIP(hipGetDeviceCount(&count), "hipGetDeviceCount");
    g_scratch_ptr.assign(static_cast<size_t>(count > 0 ? count : 0), nullptr);
  }
  if (dev < 0 || static_cast<size_t>(dev) >= g_scratch_ptr.size())
    return fail(EE_ERR_HIP, "current device %d is not one of the %zu devices", dev, g_scratch_ptr.size());
  if (g_scratch_ptr[dev] == nullptr) {
    void *p = nullptr;
    EE_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (p == nullptr) return fail(EE_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL on device %d", dev);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return EE_OK;
}

ee_status run_decide(const ee_exit &e, const void *x, int64_t n64, float threshold, int32_t *token,
                     float *confidence, int32_t *exit_flag, void *ws, hipStream_t s) {
  const DecLayout L = dec_layout(e, n64);
  const bool f32 = e.dtype == EE_F32;
  const int n = static_cast<int>(n64), h = static_cast<int>(e.hidden), V = static_cast<int>(e.vocab);
  const int I = static_cast<int>(e.intermediate);
  const void *z = x;
  if (e.kind == EE_EXIT_MLP) {
    EE_LAUNCH("decode mlp pre-norm", s,
              ee::launch_row_norm(f32, f32, x, n, h, e.rms_eps, e.gamma_mlp, nullptr, false, at(ws, L.u), s));
    EE_LAUNCH("decode gate projection", s, ee::decode_store(f32, e.w_gate, I, at(ws, L.u), n, h, at(ws, L.hg), s));
    EE_LAUNCH("decode up projection + swiglu", s,
              ee::decode_swiglu(f32, e.w_up, I, at(ws, L.u), n, h, at(ws, L.hg), at(ws, L.act), s));
    EE_LAUNCH("decode down projection + residual", s,
              ee::decode_residual(f32, e.w_down, h, at(ws, L.act), n, I, x, atf(ws, L.y), s));
    EE_LAUNCH("decode exit norm", s,
              ee::launch_row_norm(true, f32, atf(ws, L.y), n, h, e.rms_eps, e.gamma, nullptr, false, at(ws, L.z), s));
    z = at(ws, L.z);
  } else if (e.kind == EE_EXIT_NORM) {
    EE_LAUNCH("decode exit norm", s,
              ee::launch_row_norm(f32, f32, x, n, h, e.rms_eps, e.gamma, e.beta, e.norm == EE_NORM_LAYER, at(ws, L.z),
                                  s));
    z = at(ws, L.z);
  }
  int32_t *pa = reinterpret_cast<int32_t *>(at(ws, L.pa));
  EE_LAUNCH("decode logits partials", s,
            ee::decode_logits(f32, e.w_out, V, z, n, h, atf(ws, L.pm), atf(ws, L.pl), pa, s));
  EE_LAUNCH("decode decision", s,
            ee::decode_decide(atf(ws, L.pm), atf(ws, L.pl), pa, L.tiles, n, threshold, token, confidence, exit_flag,
                              s));
  return EE_OK;
}

}  // namespace

extern "C" {

int ee_abi_version(void) { return EE_ABI_VERSION; }

const char *ee_last_error(void) { return g_last_error.c_str(); }

const char *ee_status_string(ee_status s) {
  switch (s) {
    case EE_OK: return "ok";
    case EE_ERR_NULL: return "a required pointer is NULL";
    case EE_ERR_SHAPE: return "a size is out of range";
    case EE_ERR_DTYPE: return "unknown or mismatched dtype";
    case EE_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case EE_ERR_WORKSPACE: return "workspace too small";
    case EE_ERR_ALIAS: return "an output overlaps another buffer";
    case EE_ERR_UNSUPPORTED: return "unsupported exit kind or flag";
    case EE_ERR_TARGET: return "a target token id is outside [0, V)";
    case EE_ERR_HIP: return "HIP runtime error";
    default: break;
  }
  return "unknown status";
}

size_t ee_workspace_bytes(int n_exits, const ee_exit *exits, int64_t n_tokens) {
  if (n_exits < 1) {
    fail(EE_ERR_SHAPE, "n_exits must be >= 1");
    return 0;
  }
  if (exits == nullptr) {
    fail(EE_ERR_NULL, "exits is NULL");
    return 0;
  }
  if (validate_tokens(n_tokens) != EE_OK) return 0;
  size_t need = 0;
  for (int i = 0; i < n_exits; ++i) {
    if (validate_exit(&exits[i], i) != EE_OK) return 0;
    const size_t t = layout(exits[i], n_tokens).total;
    need = t > need ? t : need;
  }
  return need;
}

ee_status ee_head_forward_loss(const ee_exit *e, const void *hidden, const int32_t *targets, const float *token_w,
                               int64_t n_tokens, float exit_weight, uint32_t flags, void *ws, size_t ws_bytes,
                               float *loss, float *row_loss, void *stream) {
  g_last_error.clear();
  EE_TRY(validate_exit(e, 0));
  EE_TRY(validate_tokens(n_tokens));
  if ((flags & ~EE_FLAG_DYNAMIC_TOKEN_WEIGHTS) != 0) return fail(EE_ERR_UNSUPPORTED, "unknown flags 0x%x", flags);
  if (!std::isfinite(exit_weight)) return fail(EE_ERR_SHAPE, "exit_weight must be finite");
  EE_TRY(check_ptr(hidden, "hidden"));
  EE_TRY(check_ptr(targets, "targets"));
  EE_TRY(check_opt_ptr(token_w, "token_w"));
  EE_TRY(check_ptr(loss, "loss"));
  EE_TRY(check_opt_ptr(row_loss, "row_loss"));
  EE_TRY(check_workspace(ws, ws_bytes, layout(*e, n_tokens).total));
  const void *hs[1] = {hidden};
  EE_TRY(check_aliasing(1, e, hs, targets, token_w, n_tokens, nullptr, loss, 4, row_loss,
                        static_cast<size_t>(n_tokens) * 4, ws, ws_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  return run_forward(*e, hidden, targets, token_w, n_tokens, exit_weight, flags, ws, loss, row_loss, nullptr, 1, s);
}

ee_status ee_head_backward(const ee_exit *e, int64_t n_tokens, void *ws, size_t ws_bytes, const ee_exit_grads *g,
                           int accumulate, void *stream) {
  g_last_error.clear();
  EE_TRY(validate_exit(e, 0));
  EE_TRY(validate_tokens(n_tokens));
  EE_TRY(validate_grads(*e, g, 0));
  if (accumulate != 0 && accumulate != 1) return fail(EE_ERR_SHAPE, "accumulate must be 0 or 1");
  EE_TRY(check_workspace(ws, ws_bytes, layout(*e, n_tokens).total));
  EE_TRY(check_aliasing(1, e, nullptr, nullptr, nullptr, n_tokens, g, nullptr, 0, nullptr, 0, ws, ws_bytes));
  return run_backward(*e, n_tokens, ws, *g, accumulate, static_cast<hipStream_t>(stream));
}

ee_status ee_multi_exit_step(int n_exits, const ee_exit *exits, const void *const *hidden, const int32_t *targets,
                             const float *token_w, int64_t n_tokens, const float *exit_weights, uint32_t flags,
                             const ee_exit_grads *grads, int accumulate, void *ws, size_t ws_bytes,
                             float *loss_total, float *loss_per_exit, void *stream) {
  g_last_error.clear();
  if (n_exits < 1 || n_exits > 64) return fail(EE_ERR_SHAPE, "n_exits=%d must be in [1, 64]", n_exits);
  if (exits == nullptr) return fail(EE_ERR_NULL, "exits is NULL");
  if (hidden == nullptr) return fail(EE_ERR_NULL, "hidden is NULL");
  if (exit_weights == nullptr) return fail(EE_ERR_NULL, "exit_weights is NULL");
  if (grads == nullptr) return fail(EE_ERR_NULL, "grads is NULL");
  EE_TRY(validate_tokens(n_tokens));
  if ((flags & ~EE_FLAG_DYNAMIC_TOKEN_WEIGHTS) != 0) return fail(EE_ERR_UNSUPPORTED, "unknown flags 0x%x", flags);
  if (accumulate != 0 && accumulate != 1) return fail(EE_ERR_SHAPE, "accumulate must be 0 or 1");
  size_t need = 0;
  for (int i = 0; i < n_exits; ++i) {
    EE_TRY(validate_exit(&exits[i], i));
    if (exits[i].vocab != exits[0].vocab) return fail(EE_ERR_SHAPE, "all exits must share the vocabulary size");
    if (exits[i].dtype != exits[0].dtype) return fail(EE_ERR_DTYPE, "all exits must share one dtype");
    EE_TRY(validate_grads(exits[i], &grads[i], i));
    EE_TRY(check_ptr(hidden[i], "hidden[e]"));
    if (!std::isfinite(exit_weights[i])) return fail(EE_ERR_SHAPE, "exit_weights[%d] must be finite", i);
    const size_t t = layout(exits[i], n_tokens).total;
    need = t > need ? t : need;
  }
  EE_TRY(check_ptr(targets, "targets"));
  EE_TRY(check_opt_ptr(token_w, "token_w"));
  EE_TRY(check_ptr(loss_total, "loss_total"));
  EE_TRY(check_opt_ptr(loss_per_exit, "loss_per_exit"));
  EE_TRY(check_workspace(ws, ws_bytes, need));
  EE_TRY(check_aliasing(n_exits, exits, hidden, targets, token_w, n_tokens, grads, loss_total, 4, loss_per_exit,
                        static_cast<size_t>(n_exits) * 4, ws, ws_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int i = 0; i < n_exits; ++i) {
    float *loss = loss_per_exit != nullptr ? loss_per_exit + i : atf(ws, kLossSlotOff);
    EE_TRY(run_forward(exits[i], hidden[i], targets, token_w, n_tokens, exit_weights[i], flags, ws, loss, nullptr,
                       loss_total, i == 0, s));
    EE_TRY(run_backward(exits[i], n_tokens, ws, grads[i], accumulate, s));
  }
  return EE_OK;
}

ee_status ee_adam_update(int n_tensors, const ee_adam_tensor *tensors, float lr, float beta1, float beta2,
                         float eps, int64_t step, void *stream) {
  if (n_tensors < 0) return fail(EE_ERR_SHAPE, "n_tensors = %d is negative", n_tensors);
  if (n_tensors == 0) return EE_OK;
  if (tensors == nullptr) return fail(EE_ERR_NULL, "tensors is NULL");
  if (!std::isfinite(lr)) return fail(EE_ERR_SHAPE, "lr is not finite");
  if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
    return fail(EE_ERR_SHAPE, "beta1 = %g and beta2 = %g must lie in [0, 1)", beta1, beta2);
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(EE_ERR_SHAPE, "eps = %g must be finite and >= 0", eps);
  if (step < 1) return fail(EE_ERR_SHAPE, "step = %lld must be >= 1", static_cast<long long>(step));
  std::vector<Range> written, read;
  for (int i = 0; i < n_tensors; ++i) {
    const ee_adam_tensor &t = tensors[i];
    if (t.reserved != 0) return fail(EE_ERR_SHAPE, "tensor %d: reserved field must be 0", i);
    if (t.numel < 0) return fail(EE_ERR_SHAPE, "tensor %d: numel is negative", i);
    if (t.dtype != EE_F32 && t.dtype != EE_BF16) return fail(EE_ERR_DTYPE, "tensor %d: unknown dtype %d", i, t.dtype);
    if (t.numel == 0) continue;
    if (t.numel > (int64_t{1} << 40)) return fail(EE_ERR_SHAPE, "tensor %d: numel above 2^40", i);
    char what[64];
    snprintf(what, sizeof(what), "tensor %d param", i);
    EE_TRY(check_ptr(t.param, what));
    snprintf(what, sizeof(what), "tensor %d grad", i);
    EE_TRY(check_ptr(t.grad, what));
    snprintf(what, sizeof(what), "tensor %d exp_avg", i);
    EE_TRY(check_ptr(t.exp_avg, what));
    snprintf(what, sizeof(what), "tensor %d exp_avg_sq", i);
    EE_TRY(check_ptr(t.exp_avg_sq, what));
    snprintf(what, sizeof(what), "tensor %d master", i);
    EE_TRY(check_opt_ptr(t.master, what));
    const size_t n = static_cast<size_t>(t.numel);
    written.push_back(make_range(t.param, n * (t.dtype == EE_BF16 ? 2 : 4), "a param"));
    written.push_back(make_range(t.exp_avg, n * 4, "an exp_avg"));
    written.push_back(make_range(t.exp_avg_sq, n * 4, "an exp_avg_sq"));
    if (t.master != nullptr) written.push_back(make_range(t.master, n * 4, "a master"));
    read.push_back(make_range(t.grad, n * 4, "a grad"));
  }
  for (size_t a = 0; a < written.size(); ++a) {
    for (size_t b = a + 1; b < written.size(); ++b)
      if (overlap(written[a], written[b]))
        return fail(EE_ERR_ALIAS, "%s buffer overlaps %s buffer", written[a].what, written[b].what);
    for (const Range &r : read)
      if (overlap(written[a], r)) return fail(EE_ERR_ALIAS, "%s buffer overlaps %s buffer", written[a].what, r.what);
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  ee::AdamBatchArgs b{};
  b.beta1 = beta1;
  b.beta2 = beta2;
  b.eps = eps;
  const double t = static_cast<double>(step);
  b.lr_bc1 = static_cast<float>(static_cast<double>(lr) / (1.0 - std::pow(static_cast<double>(beta1), t)));
  b.inv_bc2 = static_cast<float>(1.0 / (1.0 - std::pow(static_cast<double>(beta2), t)));
  int64_t blocks = 0;
  for (int i = 0; i < n_tensors; ++i) {
    const ee_adam_tensor &t = tensors[i];
    if (t.numel == 0) continue;
    const int64_t nb = ee::adam_blocks(t.numel);
    if (b.count == ee::kAdamMaxTensors || blocks + nb > 0x7FFFFFFF) {
      EE_LAUNCH("adam update", s, ee::launch_adam(b, s));
      b.count = 0;
      blocks = 0;
    }
    ee::AdamTensorArgs &a = b.t[b.count++];
    a = ee::AdamTensorArgs{};
    a.param = t.param;
    a.master = t.master;
    a.grad = t.grad;
    a.exp_avg = t.exp_avg;
    a.exp_avg_sq = t.exp_avg_sq;
    a.numel = t.numel;
    a.bf16 = t.dtype == EE_BF16;
    blocks += nb;
  }
  if (b.count > 0) EE_LAUNCH("adam update", s, ee::launch_adam(b, s));
  return EE_OK;
}

double ee_lr_schedule(int64_t step, int64_t total_steps, double warmup_fraction, double lr_max, double lr_min) {
  if (step < 1 || total_steps < 1 || !(warmup_fraction >= 0.0 && warmup_fraction < 1.0)) {
    fail(EE_ERR_SHAPE, "ee_lr_schedule: need step >= 1, total_steps >= 1, 0 <= warmup_fraction < 1");
    return std::nan("");
  }
  const int64_t warmup = static_cast<int64_t>(std::floor(warmup_fraction * static_cast<double>(total_steps)));
  if (step <= warmup) return lr_max * static_cast<double>(step) / static_cast<double>(warmup);
  if (step <= total_steps)
    return lr_min + (lr_max - lr_min) * static_cast<double>(total_steps - step) /
                        static_cast<double>(total_steps - warmup);
  return lr_min;
}

size_t ee_decode_workspace_bytes(const ee_exit *e, int64_t n_rows) {
  g_last_error.clear();
  if (validate_exit(e, 0) != EE_OK || validate_rows(n_rows) != EE_OK) return 0;
  return dec_layout(*e, n_rows).total;
}

ee_status ee_exit_decide(const ee_exit *e, const void *hidden, int64_t n_rows, float threshold, int32_t *token,
                         float *confidence, int32_t *exit_flag, void *ws, size_t ws_bytes, void *stream) {
  g_last_error.clear();
  EE_TRY(validate_decide(e, hidden, n_rows, threshold, token, confidence, exit_flag));
  EE_TRY(check_workspace(ws, ws_bytes, dec_layout(*e, n_rows).total));
  EE_TRY(check_decide_aliasing(*e, hidden, n_rows, token, confidence, exit_flag, ws, ws_bytes));
  return run_decide(*e, hidden, n_rows, threshold, token, confidence, exit_flag, ws,
                    static_cast<hipStream_t>(stream));
}

ee_status ee_exit_decide_static(const ee_exit *e, const void *hidden, int64_t n_rows, float threshold,
                                int32_t *token, float *confidence, int32_t *exit_flag, void *stream) {
  g_last_error.clear();
  EE_TRY(validate_decide(e, hidden, n_rows, threshold, token, confidence, exit_flag));
  const size_t need = dec_layout(*e, n_rows).total;
  if (need > kStaticScratchBytes)
    return fail(EE_ERR_WORKSPACE, "ee_exit_decide_static: %lld rows of this exit need %zu bytes of workspace, "
                "above the fixed %zu-byte array (use ee_exit_decide with a workspace)",
                static_cast<long long>(n_rows), need, kStaticScratchBytes);
  EE_TRY(check_decide_aliasing(*e, hidden, n_rows, token, confidence, exit_flag, nullptr, 0));
  void *ws = nullptr;
  EE_TRY(static_scratch(&ws));
  // no profiling events: creating them would allocate
  const bool was = g_prof_suspended;
  g_prof_suspended = true;
  const ee_status st = run_decide(*e, hidden, n_rows, threshold, token, confidence, exit_flag, ws,
                                  static_cast<hipStream_t>(stream));
  g_prof_suspended = was;
  return st;
}

ee_status ee_profile_start(void) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  g_prof_records.clear();
  g_prof_used = 0;
  g_prof_on = true;
  return EE_OK;
}

int ee_profile_stop(ee_kernel_time *out, int capacity) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  g_prof_on = false;
  int count = 0;
  for (const ProfRecord &r : g_prof_records) {
    if (hipEventSynchronize(r.stop) != hipSuccess) {
      fail(EE_ERR_HIP, "event synchronize failed");
      return -1;
    }
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      fail(EE_ERR_HIP, "event elapsed time failed");
      return -1;
    }
    int k = 0;
    while (k < count && std::string(out[k].name) != r.name) ++k;
    if (k == count) {
      if (count == capacity) continue;
      out[k].name = r.name;
      out[k].launches = 0;
      out[k].total_ms = 0.0;
      ++count;
    }
    out[k].launches += 1;
    out[k].total_ms += ms;
  }
  g_prof_records.clear();
  g_prof_used = 0;
  return count;
}

ee_status ee_check_device_error(void *ws, size_t ws_bytes, void *stream) {
  g_last_error.clear();
  EE_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < kHeader) return fail(EE_ERR_WORKSPACE, "workspace smaller than its header");
  hipStream_t s = static_cast<hipStream_t>(stream);
  EE_HIP(hipStreamSynchronize(s), "stream synchronize");
  int flag = 0;
  EE_HIP(hipMemcpy(&flag, at(ws, kFlagOff), sizeof(int), hipMemcpyDeviceToHost), "read error flag");
  if (flag != 0) {
    const int zero = 0;
    EE_HIP(hipMemcpy(at(ws, kFlagOff), &zero, sizeof(int), hipMemcpyHostToDevice), "clear error flag");
    return fail(EE_ERR_TARGET, "a target token id was outside [0, V)");
  }
  return EE_OK;
}

}  // extern "C"
