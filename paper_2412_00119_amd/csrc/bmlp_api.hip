// C ABI of the train-step library: validation, state/workspace layout and the
// launch sequence of Algorithm 1 on the caller's stream.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "bmlp_internal.h"
#include "fp4.h"

// One run of consecutive launches of one kernel class on one stream, within
// one API call, bracketed by a single pair of events.
struct ProfRec {
  int kind;
  int launches;
  hipEvent_t t0, t1;
};

struct bmlp_ctx {
  bmlp::Plan plan;
  uint8_t *state;
  uint8_t *ws;
  int device = 0;               // the device current at bmlp_init / bmlp_attach
  bool prof_on = false;
  size_t prof_used = 0;
  long prof_open = -1;          // index of the run still open, or -1
  hipStream_t prof_stream = nullptr;
  std::vector<ProfRec> prof;
};

// The no-allocation entry point's scratch (its device address per device is
// kept in bmlp::g_scratch_ptr).
static __device__ __align__(256) uint8_t scratch[BMLP_NOALLOC_SCRATCH_BYTES];

namespace bmlp {
namespace {

thread_local char g_last_error[256] = "";

int hip_fail(hipError_t e, const char *where) {
  snprintf(g_last_error, sizeof(g_last_error), "%s: %s", where, hipGetErrorString(e));
  return BMLP_EHIP;
}

#define BMLP_LAUNCH(call)                                    \
  do {                                                       \
    hipError_t e_ = (call);                                  \
    if (e_ != hipSuccess) return hip_fail(e_, #call);        \
  } while (0)

// The static scratch of bmlp_forward_noalloc: one copy per device, held
// until the process ends.  Host code never uses the array's name as an
// address: it uses the device address hipGetSymbolAddress returns for the
// device, looked up once per device with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch_ptr[kMaxDevices] = {};

// Looks up (once) the scratch address on the current device.
int scratch_setup(int *dev_out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) {
    snprintf(g_last_error, sizeof(g_last_error), "device %d: the static scratch supports devices 0..%d", dev,
             kMaxDevices - 1);
    return BMLP_EHIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = static_cast<uint8_t *>(ptr);
  }
  if (dev_out) *dev_out = dev;
  return BMLP_OK;
}

// Ends the open profiling run (if any) with its closing event.
inline hipError_t prof_close(bmlp_ctx *ctx) {
  if (ctx->prof_open < 0) return hipSuccess;
  const hipError_t e = hipEventRecord(ctx->prof[ctx->prof_open].t1, ctx->prof_stream);
  ctx->prof_open = -1;
  return e;
}

// Closes the open profiling run when an API call returns, so that no run
// spans host time between calls.
struct ProfScope {
  bmlp_ctx *ctx;
  ~ProfScope() {
    if (ctx != nullptr) (void)prof_close(ctx);
  }
};

// Launch with optional event bracketing (profiling aid): a launch of another
// class or on another stream closes the open run and opens a new one.
#define BMLP_TIMED(ctx, kind_, s, call)                                         \
  do {                                                                         \
    if ((ctx)->prof_on) {                                                      \
      if ((ctx)->prof_open >= 0 &&                                             \
          ((ctx)->prof[(ctx)->prof_open].kind != (kind_) || (ctx)->prof_stream != (s))) { \
        hipError_t ee_ = prof_close(ctx);                                      \
        if (ee_ != hipSuccess) return hip_fail(ee_, "hipEventRecord");         \
      }                                                                        \
      if ((ctx)->prof_open < 0 && (ctx)->prof_used < (ctx)->prof.size()) {     \
        ProfRec &r_ = (ctx)->prof[(ctx)->prof_used];                           \
        r_.kind = (kind_);                                                     \
        r_.launches = 0;                                                       \
        hipError_t ee_ = hipEventRecord(r_.t0, (s));                           \
        if (ee_ != hipSuccess) return hip_fail(ee_, "hipEventRecord");         \
        (ctx)->prof_open = (long)(ctx)->prof_used++;                           \
        (ctx)->prof_stream = (s);                                              \
      }                                                                        \
    }                                                                          \
    BMLP_LAUNCH(call);                                                         \
    if ((ctx)->prof_on && (ctx)->prof_open >= 0) (ctx)->prof[(ctx)->prof_open].launches++; \
  } while (0)

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

bool use_mfma(const Plan &p) { return p.fwd_impl != BMLP_FWD_POPCOUNT; }

// y_hat = a_l P_l^T by the forward kernel, for class counts above what the
// classifier kernel takes, up to kMaxFwdSlices layers per launch (once every
// forward is done, so that the launch has the tiles of all of them): int32
// rows [n][c] into y32, or int16 rows [n][ldy16] into y16, per layer.
struct ClsGemm {
  FwdArgs g{};
  ClsGemm(const Plan &p, int n, bool wide) {
    g.M = n; g.N = p.c;
    g.abits = nullptr; g.words_out = 0;
    g.mode = wide ? kFwdWriteZ32 : kFwdWriteZ;
    g.ldz = wide ? p.c : p.ldy16;
  }
  // layer l: a_l rows a, classifier rows P, output rows y32 or y16; true
  // when the launch is full (flush it before the next add)
  bool add(const Plan &p, int l, const uint64_t *a, const uint64_t *P, int32_t *y32, int16_t *y16) {
    const LayerPlan &lp = p.layer[l - 1];
    g.sl[g.nslices++] = FwdSlice{a, P, lp.words_out, lp.k_out, y16, y32};
    return g.nslices == kMaxFwdSlices;
  }
  bool pending() const { return g.nslices > 0; }
  hipError_t flush(hipStream_t s) {
    if (g.nslices == 1) {   // the single-layer form
      const FwdSlice q = g.sl[0];
      g.A = q.A; g.B = q.B; g.lda = g.ldb = q.ld; g.K = q.K; g.z = q.z; g.z32 = q.z32;
      g.nslices = 0;
    }
    const hipError_t e = launch_fwd_fp4(g, s);
    g.nslices = 0;
    return e;
  }
};

// Forward of every layer for inference (y_hat out) or evaluation (counts:
// layer l adds to correct[cstride * (l - 1)]; with flags, each pattern's
// flag of layer l goes to flags[(l - 1) * max_batch + mu]).  a_rows, if set,
// replaces the workspace's a_l rows: layer l's n rows start at a_rows +
// a_rows_offset(p, n, l) (the no-allocation entry point).
int forward_layers(bmlp_ctx *ctx, const uint64_t *x, int n, hipStream_t s, int32_t *yhat_out,
                   const int32_t *y, int32_t *correct, int cstride = 1, uint8_t *flags = nullptr,
                   uint8_t *a_rows = nullptr) {
  ProfScope prof_scope{ctx};
  const Plan &p = ctx->plan;
  int32_t *yh_ws = reinterpret_cast<int32_t *>(ctx->ws + p.off_yhat);
  auto a_of = [&](int l) {
    return reinterpret_cast<uint64_t *>(a_rows ? a_rows + a_rows_offset(p, n, l) : ctx->ws + p.layer[l - 1].off_a);
  };
  if (use_mfma(p)) {
    const bool cls_gemm = p.c > kClsMaxClasses;
    int16_t *y16_ws = reinterpret_cast<int16_t *>(ctx->ws + p.off_yhat);
    ClsGemm gemm(p, n, correct == nullptr);
    const uint64_t *a_prev = x;
    for (int l = 1; l <= p.L; ++l) {
      const LayerPlan &lp = p.layer[l - 1];
      FwdArgs f{};
      f.A = a_prev; f.lda = lp.words_in;
      f.B = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_w); f.ldb = lp.words_in;
      f.M = n; f.N = lp.k_out; f.K = lp.k_in;
      f.abits = a_of(l); f.words_out = lp.words_out;
      f.mode = kFwdPlain;
      BMLP_TIMED(ctx, BMLP_KERNEL_FWD, s, launch_fwd_fp4(f, s));
      a_prev = f.abits;
    }
    if (cls_gemm) {   // y_hat of every layer
      for (int l = 1; l <= p.L; ++l)
        if (gemm.add(p, l, a_of(l), reinterpret_cast<const uint64_t *>(ctx->state + p.layer[l - 1].off_p),
                     correct ? nullptr : yhat_out + (size_t)(l - 1) * n * p.c,
                     correct ? y16_ws + (size_t)(l - 1) * p.max_batch * p.ldy16 : nullptr))
          BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, gemm.flush(s));
      if (gemm.pending()) BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, gemm.flush(s));
    }
    if (cls_gemm && !correct) return BMLP_OK;   // y_hat is the output
    // every layer's local classifier (or, after the products above, its
    // error signal) in one launch per kMaxClsLayers layers
    ClsBatch cb{};
    cb.n = n; cb.c = p.c; cb.y = y; cb.mode = correct ? kClsEval : kClsYhatOnly; cb.ldy = p.ldy16;
    for (int l = 1; l <= p.L; ++l) {
      const LayerPlan &lp = p.layer[l - 1];
      ClsLayer &c = cb.L[cb.nl++];
      c.A = a_of(l);
      c.P = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p);
      c.words = lp.words_out; c.K = lp.k_out; c.thr = lp.robust_thr;
      c.yhat = yhat_out ? yhat_out + (size_t)(l - 1) * n * p.c : nullptr;
      c.y16 = y16_ws + (size_t)(l - 1) * p.max_batch * p.ldy16;
      c.correct = correct ? correct + (size_t)cstride * (l - 1) : nullptr;
      c.flag = flags ? flags + (size_t)(l - 1) * p.max_batch : nullptr;
      if (cb.nl == kMaxClsLayers || l == p.L) {
        BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, cls_gemm ? launch_cls_argmax(cb, s) : launch_cls_fp4(cb, s));
        cb.nl = 0;
      }
    }
    return BMLP_OK;
  }
  const uint64_t *a_prev = x;
  for (int l = 1; l <= p.L; ++l) {
    const LayerPlan &lp = p.layer[l - 1];
    const uint64_t *W = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_w);
    const uint64_t *P = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p);
    uint64_t *a = a_of(l);
    BMLP_TIMED(ctx, BMLP_KERNEL_FWD, s,
               launch_fwd_popcount(a_prev, lp.words_in, lp.k_in, W, n, lp.k_out, nullptr, 0, a,
                                   lp.words_out, s));
    int32_t *yh = yhat_out ? yhat_out + (size_t)(l - 1) * n * p.c : yh_ws;
    BMLP_TIMED(ctx, BMLP_KERNEL_OTHER, s, launch_fill_i32(yh, n * p.c, lp.k_out, s));
    BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, launch_cls_popcount(a, lp.words_out, lp.k_out, P, n, p.c, yh, p.c, s));
    if (correct)
      BMLP_TIMED(ctx, BMLP_KERNEL_SELECT, s,
                 launch_eval_count(yh, p.c, y, n, correct + (size_t)cstride * (l - 1),
                                   flags ? flags + (size_t)(l - 1) * p.max_batch : nullptr, lp.robust_thr, s));
    a_prev = a;
  }
  return BMLP_OK;
}

int check_ctx_batch(bmlp_ctx *ctx, const void *x, int n) {
  if (ctx == nullptr) return BMLP_EINVAL;
  if (n < 0 || n > ctx->plan.max_batch) return BMLP_ESHAPE;
  if (n > 0 && x == nullptr) return BMLP_EINVAL;
  return BMLP_OK;
}

int setup(const bmlp_config *cfg, void *d_state, void *d_ws, void *stream, bmlp_ctx **out,
          bool from_h) {
  if (out == nullptr || d_state == nullptr || d_ws == nullptr) return BMLP_EINVAL;
  if ((reinterpret_cast<uintptr_t>(d_state) & 255) || (reinterpret_cast<uintptr_t>(d_ws) & 255))
    return BMLP_ESTATE;
  bmlp_ctx *ctx = new (std::nothrow) bmlp_ctx;
  if (ctx == nullptr) return BMLP_EINVAL;
  const int st = make_plan(cfg, &ctx->plan);
  if (st != BMLP_OK) {
    delete ctx;
    return st;
  }
  ctx->state = static_cast<uint8_t *>(d_state);
  ctx->ws = static_cast<uint8_t *>(d_ws);
  const int sst = scratch_setup(&ctx->device);
  if (sst != BMLP_OK) {
    delete ctx;
    return sst;
  }
  const Plan &p = ctx->plan;
  hipStream_t s = as_stream(stream);
  for (int l = 1; l <= p.L; ++l) {
    const LayerPlan &lp = p.layer[l - 1];
    uint8_t *H = ctx->state + lp.off_h;
    uint64_t *W = reinterpret_cast<uint64_t *>(ctx->state + lp.off_w);
    uint64_t *P = reinterpret_cast<uint64_t *>(ctx->state + lp.off_p);
    hipError_t e = launch_init_h(H, lp.ld_h, lp.h_ps, p.bound, W, lp.words_in, lp.k_in, lp.k_out, p.seed, l,
                                 from_h, s);
    const bool own_p = l == 1 || !(p.variants & BMLP_VARIANT_SHARED_CLASSIFIER);
    if (e == hipSuccess && !from_h && own_p) e = launch_init_p(P, lp.words_out, lp.k_out, p.c, p.seed, l, s);
    if (e != hipSuccess) {
      delete ctx;
      return hip_fail(e, "init");
    }
  }
  *out = ctx;
  return BMLP_OK;
}

}  // namespace
}  // namespace bmlp

using namespace bmlp;

extern "C" {





int bmlp_init(const bmlp_config *cfg, void *d_state, void *d_workspace, void *stream,
              bmlp_ctx **out) {
  return setup(cfg, d_state, d_workspace, stream, out, false);
}

int bmlp_attach(const bmlp_config *cfg, void *d_state, void *d_workspace, void *stream,
                bmlp_ctx **out) {
  return setup(cfg, d_state, d_workspace, stream, out, true);
}

int bmlp_pack(const int8_t *d_pm1, int32_t n, int32_t K, uint64_t *d_bits, void *stream) {
  if (n < 0 || K < 1 || n > 65535) return BMLP_ESHAPE;
  if (n > 0 && (d_pm1 == nullptr || d_bits == nullptr)) return BMLP_EINVAL;
  BMLP_LAUNCH(launch_pack(d_pm1, n, K, d_bits, as_stream(stream)));
  return BMLP_OK;
}

int bmlp_feature_median(const int8_t *d_x, int32_t n, int32_t K, int8_t *d_median, void *stream) {
  if (n < 1 || K < 1) return BMLP_ESHAPE;
  if (d_x == nullptr || d_median == nullptr) return BMLP_EINVAL;
  BMLP_LAUNCH(launch_feature_median(d_x, n, K, d_median, as_stream(stream)));
  return BMLP_OK;
}

int bmlp_binarize(const int8_t *d_x, int32_t n, int32_t K, const int8_t *d_median, uint64_t *d_bits,
                  void *stream) {
  if (n < 0 || K < 1 || n > 65535) return BMLP_ESHAPE;
  if (n > 0 && (d_x == nullptr || d_median == nullptr || d_bits == nullptr)) return BMLP_EINVAL;
  BMLP_LAUNCH(launch_binarize(d_x, n, K, d_median, d_bits, as_stream(stream)));
  return BMLP_OK;
}

int bmlp_expand(const int8_t *d_x, int32_t n, int32_t k_raw, int32_t k0, uint64_t seed, uint64_t *d_bits,
                void *stream) {
  if (n < 0 || k_raw < 1 || k_raw > BMLP_MAX_EXPAND_INPUTS || k0 < 1 || k0 > BMLP_MAX_WIDTH) return BMLP_ESHAPE;
  if (n > 0 && (d_x == nullptr || d_bits == nullptr)) return BMLP_EINVAL;
  BMLP_LAUNCH(launch_expand(d_x, n, k_raw, k0, seed, d_bits, as_stream(stream)));
  return BMLP_OK;
}

int bmlp_forward(bmlp_ctx *ctx, const uint64_t *d_x, int32_t n, int32_t *d_yhat, void *stream) {
  int st = check_ctx_batch(ctx, d_x, n);
  if (st != BMLP_OK) return st;
  if (n > 0 && d_yhat == nullptr) return BMLP_EINVAL;
  if (n == 0) return BMLP_OK;
  return forward_layers(ctx, d_x, n, as_stream(stream), d_yhat, nullptr, nullptr);
}

int bmlp_forward_noalloc(bmlp_ctx *ctx, const uint64_t *d_x, int32_t n, int32_t *d_yhat, void *stream) {
  int st = check_ctx_batch(ctx, d_x, n);
  if (st != BMLP_OK) return st;
  if (n > 0 && d_yhat == nullptr) return BMLP_EINVAL;
  if (n == 0) return BMLP_OK;
  const Plan &p = ctx->plan;
  const size_t need = a_rows_offset(p, n, p.L + 1);
  if (need > (size_t)BMLP_NOALLOC_SCRATCH_BYTES) {
    snprintf(g_last_error, sizeof(g_last_error),
             "bmlp_forward_noalloc: %zu bytes of activation rows for n = %d exceed the static scratch of %zu bytes",
             need, (int)n, (size_t)BMLP_NOALLOC_SCRATCH_BYTES);
    return BMLP_ESHAPE;
  }
  uint8_t *base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (ctx->device >= 0 && ctx->device < kMaxDevices) base = g_scratch_ptr[ctx->device];
  }
  if (base == nullptr) {   // not looked up at init: do it now, on the ctx's device
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != ctx->device && (e = hipSetDevice(ctx->device)) != hipSuccess) return hip_fail(e, "hipSetDevice");
    st = scratch_setup(nullptr);
    if (cur != ctx->device) (void)hipSetDevice(cur);
    if (st != BMLP_OK) return st;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    base = g_scratch_ptr[ctx->device];
  }
  return forward_layers(ctx, d_x, n, as_stream(stream), d_yhat, nullptr, nullptr, 1, nullptr, base);
}

int bmlp_eval(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
              int32_t *d_correct, void *stream) {
  int st = check_ctx_batch(ctx, d_x, n);
  if (st != BMLP_OK) return st;
  if (n > 0 && (d_y == nullptr || d_correct == nullptr)) return BMLP_EINVAL;
  if (n == 0) return BMLP_OK;
  return forward_layers(ctx, d_x, n, as_stream(stream), nullptr, d_y, d_correct);
}

int bmlp_eval_exit(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
                   int32_t *d_counts, void *stream) {
  int st = check_ctx_batch(ctx, d_x, n);
  if (st != BMLP_OK) return st;
  if (n > 0 && (d_y == nullptr || d_counts == nullptr)) return BMLP_EINVAL;
  if (n == 0) return BMLP_OK;
  const Plan &p = ctx->plan;
  hipStream_t s = as_stream(stream);
  uint8_t *flags = ctx->ws + p.off_flag;
  st = forward_layers(ctx, d_x, n, s, nullptr, d_y, d_counts, 3, flags);
  if (st != BMLP_OK) return st;
  BMLP_LAUNCH(launch_exit_count(flags, p.max_batch, p.L, n, d_counts, s));
  return BMLP_OK;
}



int bmlp_train_step(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
                    uint64_t step, double p_r, int32_t *d_stats, void *stream) {
  int st = check_ctx_batch(ctx, d_x, n);
  if (st != BMLP_OK) return st;
  if (d_stats == nullptr || (n > 0 && d_y == nullptr)) return BMLP_EINVAL;
  if (reinterpret_cast<uintptr_t>(d_stats) & 7) return BMLP_EINVAL;
  if (!(p_r >= 0.0) || !isfinite(p_r)) return BMLP_EINVAL;
  const Plan &p = ctx->plan;
  hipStream_t s = as_stream(stream);
  const bool mfma = use_mfma(p);
  ProfScope prof_scope{ctx};
  if (n == 0 || !mfma)
    BMLP_TIMED(ctx, BMLP_KERNEL_OTHER, s, launch_fill_i32(d_stats, BMLP_STATS_STRIDE * p.L, 0, s));
  if (n == 0) return BMLP_OK;
  int16_t *z = reinterpret_cast<int16_t *>(ctx->ws + p.off_z);
  int32_t *yh = reinterpret_cast<int32_t *>(ctx->ws + p.off_yhat);
  int16_t *y16 = reinterpret_cast<int16_t *>(ctx->ws + p.off_yhat);
  const bool cls_gemm = mfma && p.c > kClsMaxClasses;
  const bool reshuffle = p.variants & BMLP_VARIANT_RESHUFFLE_GROUPS;
  if (reshuffle) {   // this step's group order of every layer
    PermBatch pb{};
    pb.key0 = (uint32_t)p.seed; pb.key1 = (uint32_t)(p.seed >> 32); pb.step = (uint32_t)step;
    for (int l = 1; l <= p.L; ++l) {
      PermLayer &q = pb.L[pb.nl++];
      q.perm = reinterpret_cast<int32_t *>(ctx->ws + p.layer[l - 1].off_perm);
      q.k = p.layer[l - 1].k_out;
      q.ctr1 = (uint32_t)(l - 1);
      if (pb.nl == 8 || l == p.L) {
        BMLP_TIMED(ctx, BMLP_KERNEL_SELECT, s, launch_group_perm(pb, s));
        pb.nl = 0;
      }
    }
  }
  const uint64_t *a_prev = d_x;
  for (int l = 1; l <= p.L; ++l) {
    const LayerPlan &lp = p.layer[l - 1];
    const uint64_t *W = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_w);
    const uint64_t *P = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p);
    uint64_t *a = reinterpret_cast<uint64_t *>(ctx->ws + lp.off_a);
    uint8_t *err = ctx->ws + lp.off_err;
    uint8_t *upd = ctx->ws + lp.off_upd;
    int16_t *kstar = reinterpret_cast<int16_t *>(ctx->ws + lp.off_kstar);
    int32_t *stats = d_stats + BMLP_STATS_STRIDE * (l - 1);
    LossSelectArgs ls{};
    ls.c = p.c;
    ls.z = z; ls.ldz = p.ldz;
    ls.P = P; ls.words_out = lp.words_out;
    ls.y = d_y; ls.n = n;
    ls.k_out = lp.k_out; ls.gamma = lp.gamma; ls.groups = lp.groups; ls.thr = lp.robust_thr;
    ls.err = err; ls.upd = upd; ls.kstar = kstar; ls.ldk = p.max_batch; ls.stats = stats;
    // the selection's view of z: clipped to z_bits(K_{l-1}) bits as a variant
    int zlo = -65536, zhi = 65535;
    if (p.variants & BMLP_VARIANT_SATURATE_Z) {
      const int b = z_bits(lp.k_in);
      zlo = -(1 << (b - 1));
      zhi = (1 << (b - 1)) - 1;
    }
    ls.zlo = zlo; ls.zhi = zhi;
    const int32_t *perm = reshuffle ? reinterpret_cast<const int32_t *>(ctx->ws + lp.off_perm) : nullptr;
    ls.perm = perm;
    if (mfma) {
      // the fused selection takes contiguous groups of 64
      const bool fused = lp.gamma == 64 && !reshuffle;
      // Algorithm 1's pre-activation and sign, and Algorithm 2's choice when fused
      FwdArgs f{};
      f.A = a_prev; f.lda = lp.words_in;
      f.B = W; f.ldb = lp.words_in;
      f.M = n; f.N = lp.k_out; f.K = lp.k_in;
      f.abits = a; f.words_out = lp.words_out;
      f.mode = fused ? kFwdFusedSelect : kFwdWriteZ;
      f.kstar = kstar; f.ldk = p.max_batch;
      f.y = d_y; f.c = p.c; f.P = P; f.ldp = lp.words_out;
      f.zlo = (float)zlo; f.zhi = (float)zhi;
      f.z = z; f.ldz = p.ldz;
      if (l == 1) {   // the step statistics start at zero
        f.zero = d_stats; f.nzero = BMLP_STATS_STRIDE * p.L;
      }
      BMLP_TIMED(ctx, BMLP_KERNEL_FWD, s, launch_fwd_fp4(f, s));
      if (!fused) {   // Algorithm 2 from the stored z, before the next layer reuses it
        ls.yhat = nullptr;
        BMLP_TIMED(ctx, BMLP_KERNEL_SELECT, s, launch_loss_select(ls, s));
      }

    } else {
      BMLP_TIMED(ctx, BMLP_KERNEL_FWD, s,
                 launch_fwd_popcount(a_prev, lp.words_in, lp.k_in, W, n, lp.k_out, z, p.ldz, a,
                                     lp.words_out, s));
      BMLP_TIMED(ctx, BMLP_KERNEL_OTHER, s, launch_fill_i32(yh, n * p.c, lp.k_out, s));
      BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, launch_cls_popcount(a, lp.words_out, lp.k_out, P, n, p.c, yh, p.c, s));
      ls.yhat = yh;
      BMLP_TIMED(ctx, BMLP_KERNEL_SELECT, s, launch_loss_select(ls, s));
    }
    a_prev = a;
  }
  if (cls_gemm) {   // Algorithm 1's y_hat of every layer
    ClsGemm gemm(p, n, false);
    for (int l = 1; l <= p.L; ++l) {
      const LayerPlan &lp = p.layer[l - 1];
      if (gemm.add(p, l, reinterpret_cast<const uint64_t *>(ctx->ws + lp.off_a),
                   reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p), nullptr,
                   y16 + (size_t)(l - 1) * p.max_batch * p.ldy16))
        BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, gemm.flush(s));
    }
    if (gemm.pending()) BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, gemm.flush(s));
  }
  if (mfma) {
    // Algorithm 1's local output (or, after the products above, the error
    // signal from it), loss and robustness test for every layer, one launch
    // per kMaxClsLayers layers
    ClsBatch cb{};
    cb.n = n; cb.c = p.c; cb.y = d_y; cb.mode = kClsTrain; cb.ldy = p.ldy16;
    for (int l = 1; l <= p.L; ++l) {
      const LayerPlan &lp = p.layer[l - 1];
      ClsLayer &c = cb.L[cb.nl++];
      c.A = reinterpret_cast<const uint64_t *>(ctx->ws + lp.off_a);
      c.P = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p);
      c.words = lp.words_out; c.K = lp.k_out; c.thr = lp.robust_thr;
      c.y16 = y16 + (size_t)(l - 1) * p.max_batch * p.ldy16;
      c.err = ctx->ws + lp.off_err; c.upd = ctx->ws + lp.off_upd;
      c.stats = d_stats + BMLP_STATS_STRIDE * (l - 1);
      if (cb.nl == kMaxClsLayers || l == p.L) {
        BMLP_TIMED(ctx, BMLP_KERNEL_CLS, s, cls_gemm ? launch_cls_argmax(cb, s) : launch_cls_fp4(cb, s));
        cb.nl = 0;
      }
    }
  }
  // Algorithm 3 for every layer (each layer's forward above used its
  // pre-step weights; the updates touch only H_l and W_l).
  UpdateBatch ub{};
  ub.y = d_y; ub.n = n; ub.ldk = p.max_batch; ub.c = p.c; ub.bound = p.bound;
  ub.key0 = (uint32_t)p.seed; ub.key1 = (uint32_t)(p.seed >> 32); ub.step = (uint32_t)step;
  ub.sequential = (p.variants & BMLP_VARIANT_SEQUENTIAL_CLIP) ? 1 : 0;
  for (int l = 1; l <= p.L; ++l) {
    const LayerPlan &lp = p.layer[l - 1];
    UpdLayer &u = ub.L[ub.nl++];
    u.H = ctx->state + lp.off_h;
    u.W32 = reinterpret_cast<uint32_t *>(ctx->state + lp.off_w);
    u.a32 = reinterpret_cast<const uint32_t *>(l == 1 ? d_x : reinterpret_cast<const uint64_t *>(
                                                               ctx->ws + p.layer[l - 2].off_a));
    u.kstar = reinterpret_cast<const int16_t *>(ctx->ws + lp.off_kstar);
    u.upd = ctx->ws + lp.off_upd;
    u.P = reinterpret_cast<const uint64_t *>(ctx->state + lp.off_p);
    u.stats = d_stats + BMLP_STATS_STRIDE * (l - 1);
    u.ld_h = lp.ld_h; u.h_ps = lp.h_ps; u.nw32 = 2 * lp.words_in; u.words_out = lp.words_out;
    u.k_in = lp.k_in; u.groups = lp.groups; u.gamma = lp.gamma;
    // R11: K_l, or the fan-in K_{l-1} as a variant
    const uint64_t T = reinforce_threshold(p_r, (p.variants & BMLP_VARIANT_FAN_IN_REINFORCE) ? lp.k_in : lp.k_out);
    u.t_hi = (uint32_t)(T >> 24); u.t_lo = (uint32_t)(T & 0xFFFFFFu);
    u.ctr1 = (uint32_t)(l - 1);
    u.perm = reshuffle ? reinterpret_cast<const int32_t *>(ctx->ws + lp.off_perm) : nullptr;
    if (ub.nl == kMaxUpdLayers || l == p.L) {
      BMLP_TIMED(ctx, BMLP_KERNEL_UPDATE, s, launch_update(ub, s));
      ub.nl = 0;
    }
  }
  return BMLP_OK;
}

int bmlp_train_epoch(bmlp_ctx *ctx, const uint64_t *d_x_all, const int32_t *d_y_all, int32_t n_all,
                     const int32_t *d_order, int32_t n_order, int32_t batch, uint64_t step0, double p_r,
                     int32_t *d_stats, void *stream) {
  if (ctx == nullptr) return BMLP_EINVAL;
  const Plan &p = ctx->plan;
  if (batch < 1 || batch > p.max_batch || n_all < 0 || n_order < 0) return BMLP_ESHAPE;
  const int nb = n_order / batch;
  if (nb == 0) return BMLP_OK;
  if (n_all < 1 || d_x_all == nullptr || d_y_all == nullptr || d_order == nullptr || d_stats == nullptr)
    return BMLP_EINVAL;
  if (reinterpret_cast<uintptr_t>(d_stats) & 7) return BMLP_EINVAL;
  hipStream_t s = as_stream(stream);
  uint64_t *xb = reinterpret_cast<uint64_t *>(ctx->ws + p.off_xb);
  int32_t *yb = reinterpret_cast<int32_t *>(ctx->ws + p.off_yb);
  for (int b = 0; b < nb; ++b) {
    {
      ProfScope prof_scope{ctx};
      BMLP_TIMED(ctx, BMLP_KERNEL_OTHER, s,
                 launch_gather_batch(d_x_all, d_y_all, n_all, p.layer[0].words_in, d_order + (size_t)b * batch,
                                     batch, xb, yb, s));
    }
    const int st = bmlp_train_step(ctx, xb, yb, batch, step0 + (uint64_t)b, p_r,
                                   d_stats + (size_t)b * BMLP_STATS_STRIDE * p.L, stream);
    if (st != BMLP_OK) return st;
  }
  return BMLP_OK;
}

int bmlp_layer_views(bmlp_ctx *ctx, int32_t l, uint8_t **d_h, uint64_t **d_w, uint64_t **d_p) {
  if (ctx == nullptr) return BMLP_EINVAL;
  if (l < 1 || l > ctx->plan.L) return BMLP_ESHAPE;
  const LayerPlan &lp = ctx->plan.layer[l - 1];
  if (d_h) *d_h = ctx->state + lp.off_h;
  if (d_w) *d_w = reinterpret_cast<uint64_t *>(ctx->state + lp.off_w);
  if (d_p) *d_p = reinterpret_cast<uint64_t *>(ctx->state + lp.off_p);
  return BMLP_OK;
}

int bmlp_read_h(bmlp_ctx *ctx, int32_t l, int8_t *d_out, void *stream) {
  if (ctx == nullptr || d_out == nullptr) return BMLP_EINVAL;
  if (l < 1 || l > ctx->plan.L) return BMLP_ESHAPE;
  const LayerPlan &lp = ctx->plan.layer[l - 1];
  BMLP_LAUNCH(launch_read_h(ctx->state + lp.off_h, lp.ld_h, lp.h_ps, ctx->plan.bound, lp.k_in, lp.k_out, d_out,
                            as_stream(stream)));
  return BMLP_OK;
}

int bmlp_step_trace(bmlp_ctx *ctx, int32_t l, const uint64_t **d_a, const uint8_t **d_err,
                    const uint8_t **d_upd, const int16_t **d_kstar) {
  if (ctx == nullptr) return BMLP_EINVAL;
  if (l < 1 || l > ctx->plan.L) return BMLP_ESHAPE;
  const LayerPlan &lp = ctx->plan.layer[l - 1];
  if (d_a) *d_a = reinterpret_cast<const uint64_t *>(ctx->ws + lp.off_a);
  if (d_err) *d_err = ctx->ws + lp.off_err;
  if (d_upd) *d_upd = ctx->ws + lp.off_upd;
  if (d_kstar) *d_kstar = reinterpret_cast<const int16_t *>(ctx->ws + lp.off_kstar);
  return BMLP_OK;
}


const char *bmlp_last_error(void) { return g_last_error; }

static void prof_release(bmlp_ctx *ctx) {
  for (ProfRec &r : ctx->prof) {
    if (r.t0) (void)hipEventDestroy(r.t0);
    if (r.t1) (void)hipEventDestroy(r.t1);
  }
  ctx->prof.clear();
  ctx->prof_used = 0;
  ctx->prof_open = -1;
  ctx->prof_on = false;
}

int bmlp_profile_start(bmlp_ctx *ctx, int32_t max_launches) {
  if (ctx == nullptr) return BMLP_EINVAL;
  if (max_launches < 1 || max_launches > (1 << 20)) return BMLP_ESHAPE;
  prof_release(ctx);
  ctx->prof.resize((size_t)max_launches, ProfRec{0, 0, nullptr, nullptr});
  for (ProfRec &r : ctx->prof) {
    hipError_t e = hipEventCreate(&r.t0);
    if (e == hipSuccess) e = hipEventCreate(&r.t1);
    if (e != hipSuccess) {
      prof_release(ctx);
      return hip_fail(e, "hipEventCreate");
    }
  }
  ctx->prof_on = true;
  return BMLP_OK;
}

int bmlp_profile_stop(bmlp_ctx *ctx, double *h_ms, int64_t *h_launches) {
  if (ctx == nullptr) return BMLP_EINVAL;
  double ms[BMLP_KERNEL_KINDS] = {0};
  int64_t cnt[BMLP_KERNEL_KINDS] = {0};
  int status = BMLP_OK;
  if (ctx->prof_open >= 0) {
    const hipError_t e = prof_close(ctx);
    if (e != hipSuccess) status = hip_fail(e, "hipEventRecord");
  }
  if (status == BMLP_OK && ctx->prof_used > 0) {
    hipError_t e = hipEventSynchronize(ctx->prof[ctx->prof_used - 1].t1);
    if (e != hipSuccess) status = hip_fail(e, "hipEventSynchronize");
    for (size_t i = 0; status == BMLP_OK && i < ctx->prof_used; ++i) {
      float t = 0.f;
      e = hipEventElapsedTime(&t, ctx->prof[i].t0, ctx->prof[i].t1);
      if (e != hipSuccess) {
        status = hip_fail(e, "hipEventElapsedTime");
        break;
      }
      ms[ctx->prof[i].kind] += t;
      cnt[ctx->prof[i].kind] += ctx->prof[i].launches;
    }
  }
  prof_release(ctx);
  for (int k = 0; k < BMLP_KERNEL_KINDS; ++k) {
    if (h_ms) h_ms[k] = ms[k];
    if (h_launches) h_launches[k] = cnt[k];
  }
  return status;
}

void bmlp_destroy(bmlp_ctx *ctx) {
  if (ctx) prof_release(ctx);
  delete ctx;
}

}  // extern "C"
