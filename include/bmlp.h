/*
 * bmlp.h — C ABI of the MI355X train-step library for fully binary multi-layer
 * perceptrons trained with random local binary error signals (Colombo,
 * Pittorino, Roveri, arXiv 2412.00119).
 *
 * One call of bmlp_train_step is one mini-batch of the paper's Algorithm 1:
 * for every layer l the bit-packed XNOR-popcount forward z = a W^T and
 * a = sign(z), the fixed random local classifier y_hat = a P^T, the 01-loss
 * (Eq. 1) with the robustness margin that selects the patterns to update
 * (Section 3.2), the choice of the "easiest" wrong perceptron in each group of
 * gamma (Algorithm 2, Section 3.3), and the Clipped-Perceptron increments plus
 * stochastic reinforcement of the bounded integer hidden weights, re-binarised
 * by sign into the visible weights (Algorithm 3, Section 3.4).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Pointers named d_* are DEVICE pointers, h_* are HOST pointers.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call
 *    that takes a stream only enqueues work on it and returns without
 *    synchronising; results are visible after the stream is synchronised.
 *  - The library never allocates or frees device memory.  The caller owns the
 *    state and workspace buffers (sizes from bmlp_state_bytes and
 *    bmlp_workspace_bytes, 256-byte aligned) and every input/output buffer, and
 *    keeps them alive while a context uses them.
 *  - Bit rows: a row of K values in {-1,+1} is ceil(K/64) little-endian uint64
 *    words; value j is bit (j % 64) of word (j / 64), bit 1 means +1, and the
 *    bits past K in the last word are 0.  A uint32 view of the same memory is
 *    the same layout with 32-bit words.
 *  - Labels are int32 in [0, n_classes) (the paper numbers classes 1..c).
 *    A label outside that range is a precondition violation; the result is
 *    unspecified but stays within the buffers.
 *  - Return value: BMLP_OK or a negative status.  Argument, shape and
 *    configuration errors are detected on the host before anything is
 *    enqueued and leave every buffer untouched.  BMLP_EHIP reports a failed
 *    kernel launch; bmlp_last_error() then gives the HIP message.  Faults
 *    inside a kernel surface at the caller's next stream synchronisation.
 *  - One context is used from one host thread and one stream at a time.
 */
#ifndef BMLP_H_
#define BMLP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  BMLP_OK = 0,
  BMLP_EINVAL = -1,   /* bad argument: null pointer, unknown option          */
  BMLP_ESHAPE = -2,   /* size out of range: n > max_batch, widths, gamma      */
  BMLP_EHIP = -3,     /* a HIP call or kernel launch failed                   */
  BMLP_ESTATE = -4,   /* misaligned state/workspace buffer                    */
};

/* Forward GEMM implementation (the binary contraction z = a W^T). */
enum {
  BMLP_FWD_AUTO = 0,      /* the library's fastest implementation (MFMA_FP4)   */
  BMLP_FWD_POPCOUNT = 1,  /* XNOR-popcount over 32-bit words (v_xor + v_bcnt)  */
  BMLP_FWD_MFMA_FP4 = 2,  /* ±1 as e2m1 operands of the scaled fp4 MFMA: exact  */
};

/* Method variants (bmlp_config.variants, a bit set; 0 = the method as
 * printed). */
enum {
  /* q_l = p_r sqrt(2 / (pi K_{l-1})): the fan-in instead of K_l in the
   * reinforcement probability (Algorithm 3 prints K_l). */
  BMLP_VARIANT_FAN_IN_REINFORCE = 1,
  /* one classifier P for every layer, layer 1's (Section 3.1); needs every
   * K_l (l >= 1) equal.  The state then holds P once. */
  BMLP_VARIANT_SHARED_CLASSIFIER = 2,
  /* Algorithm 2 on z held in min(8, ceil(log2(2 K_{l-1}))) two's-complement
   * bits, i.e. clipped to [-2^(b-1), 2^(b-1) - 1] (Section 3.5); a_l keeps
   * the sign of the exact z. */
  BMLP_VARIANT_SATURATE_Z = 4,
  /* group membership drawn again every step (Section 4.3): layer l orders
   * its K_l perceptrons by a 32-bit key, word (k & 3) of Philox block
   * k >> 2 of stream 6 at counter (block, l - 1, t, 6), ties by index, and
   * group g is positions g*gamma .. g*gamma + gamma - 1 of that order.  k*
   * is then a position within the group; equal stabilities go to the
   * lowest perceptron index. */
  BMLP_VARIANT_RESHUFFLE_GROUPS = 8,
  /* the Clipped-Perceptron increments of a step applied pattern by pattern
   * in index order, each clipped to [-B, B] at once (Algorithm 3 gives no
   * clip; the default sums the batch's increments and clips once). */
  BMLP_VARIANT_SEQUENTIAL_CLIP = 16,
};

/* Limits of this build. */
#define BMLP_MAX_LAYERS 64
#define BMLP_MAX_WIDTH 32767      /* |z| <= K_{l-1} must fit in int16          */
#define BMLP_MAX_CLASSES 32767
#define BMLP_MAX_GROUP 4096       /* gamma, bounded by on-chip bucket storage  */
#define BMLP_MAX_BATCH 16384      /* pattern indices are kept in 15 bits on chip */
#define BMLP_MAX_EXPAND_INPUTS 65536   /* |sum| <= 128 K_raw stays far inside int32 */

/*
 * Network and hyper-parameters (Algorithm 1's variables and hyper-parameters;
 * Section 3.1 for the architecture).
 *   n_layers     L >= 1 hidden layers (1..BMLP_MAX_LAYERS).
 *   h_widths     host array of L+1 widths K_0..K_L, each 1..BMLP_MAX_WIDTH; K_0
 *                is the input width.  Copied by bmlp_init/bmlp_attach.
 *   n_classes    c, 2..BMLP_MAX_CLASSES.
 *   max_batch    largest n accepted by the batch calls, 1..BMLP_MAX_BATCH.
 *   bound        B: hidden weights live in [-B, B].  Odd, 1..127 (8-bit hidden
 *                weights, Table 4); B = 1 keeps only the visible weights.
 *   group_size   gamma; must divide every K_l (l >= 1) and be <= BMLP_MAX_GROUP.
 *                0 selects the paper's rule gamma* per layer (Section 4.3): the
 *                divisor of K_l closest to [75, 105], ties to the larger.
 *   robustness   r >= 0 (Section 3.2; the paper uses 0.25, Appendix A.1).  A
 *                pattern is updated when tau < ceil(r * K_l).
 *   seed         64-bit key of the Philox4x32-10 streams (init, reinforcement).
 *   fwd_impl     BMLP_FWD_* .
 *   variants     0 or a bit set of BMLP_VARIANT_* .
 */
typedef struct bmlp_config {
  int32_t n_layers;
  const int32_t *h_widths;
  int32_t n_classes;
  int32_t max_batch;
  int32_t bound;
  int32_t group_size;
  double robustness;
  uint64_t seed;
  int32_t fwd_impl;
  int32_t variants;
} bmlp_config;

/*
 * Derived per-layer plan (host-only query; no device work).
 *   k_in, k_out      K_{l-1}, K_l.
 *   gamma, groups    group size and G_l = K_l / gamma.
 *   words_in/out     uint64 words per bit row of a_{l-1} / a_l.
 *   h_planes, h_ps   H_l stores u = (h + B) / 2, an integer in [0, B] (h is
 *                    odd), in h_planes = bits(B) bit planes (5 for B = 31,
 *                    7 for B = 127) of h_ps 32-bit words each (h_ps >=
 *                    ceil(k_in / 32), a multiple of 16).
 *   ld_h             bytes per row of H_l: 4 * h_planes * h_ps.
 *   robust_thr       ceil(r * K_l), computed in IEEE double.
 *   off_h, off_w, off_p  byte offsets in the state buffer of
 *                    H_l  [k_out][ld_h bytes]  hidden weights, perceptron-major
 *                                                    (the transpose of the paper's
 *                                                    K_{l-1} x K_l, so h^k is a row),
 *                                                    stored bit-sliced: a row is
 *                                                    h_planes planes of h_ps uint32
 *                                                    words; bit i of word g of plane
 *                                                    p is bit p of u = (h + B) / 2
 *                                                    for column 32g + i.  Columns
 *                                                    past k_in hold u = 0.
 *                                                    bmlp_read_h unpacks it to int8;
 *                    W_l  uint64 [k_out][words_in]   visible weights sign(H_l), bits;
 *                    P_l  uint64 [n_classes][words_out]  fixed classifier, row y is rho^y.
 *   off_a, off_err, off_upd, off_kstar  byte offsets in the workspace of the
 *                    last train step's
 *                    a_l    uint64 [max_batch][words_out]
 *                    err_l  uint8  [max_batch]   01-loss
 *                    upd_l  uint8  [max_batch]   1 = pattern in M_l
 *                    kstar_l int16 [groups][max_batch]  easiest wrong
 *                           perceptron of each group as an offset in the
 *                           group (-1 when the group has none), for every
 *                           pattern; U_l (Algorithm 2) is its restriction to
 *                           the patterns with upd_l = 1
 */
typedef struct bmlp_layer_info {
  int32_t k_in, k_out, gamma, groups;
  int32_t words_in, words_out, ld_h, robust_thr;
  uint64_t off_h, off_w, off_p;
  uint64_t off_a, off_err, off_upd, off_kstar;
  int32_t h_planes, h_ps;
} bmlp_layer_info;

typedef struct bmlp_ctx bmlp_ctx;   /* opaque, host memory only */

/* Bytes of the state buffer (H, W, P of every layer), or 0 for an invalid
 * configuration.  A checkpoint is this buffer (or just H and P, see
 * bmlp_attach) plus the step counter, p_r, the seed and the configuration. */
size_t bmlp_state_bytes(const bmlp_config *cfg);

/* Bytes of the workspace buffer, or 0 for an invalid configuration. */
size_t bmlp_workspace_bytes(const bmlp_config *cfg);

/* Validates cfg and fills info for layer l (1..L).  Host only. */
int bmlp_describe(const bmlp_config *cfg, int32_t l, bmlp_layer_info *info);

/* The reinforcement threshold T_l = ceil(q * 2^32), q = p_r sqrt(2 / (pi K_l))
 * (Algorithm 3), computed in IEEE double in that order and clamped to
 * [0, 2^32].  A hidden weight is reinforced when its 32-bit draw is < T_l.
 * Host only. */
uint64_t bmlp_reinforce_threshold(double p_r, int32_t k_l);

/* Creates a context over caller-owned buffers and initialises the state:
 * H_l and P_l uniform on {-1,+1} from Philox streams 1 and 2 (Algorithm 1,
 * initialisation), W_l = sign(H_l).  d_state and d_workspace must be
 * 256-byte aligned and of the sizes above.  On success *out receives the
 * context (free it with bmlp_destroy). */
int bmlp_init(const bmlp_config *cfg, void *d_state, void *d_workspace, void *stream,
              bmlp_ctx **out);

/* Like bmlp_init but keeps H_l and P_l already in d_state (a restored
 * checkpoint) and only recomputes what derives from them: W_l = sign(H_l). */
int bmlp_attach(const bmlp_config *cfg, void *d_state, void *d_workspace, void *stream,
                bmlp_ctx **out);

/* Packs an int8 matrix [n][K] of {-1,+1} (any value > 0 counts as +1) into bit
 * rows [n][ceil(K/64)] (the step before the forward, Algorithm 1: the input
 * is already binarised).  n >= 0, K >= 1. */
int bmlp_pack(const int8_t *d_pm1, int32_t n, int32_t K, uint64_t *d_bits, void *stream);

/* The input side for integer features (Algorithm 1, its binarisation of the inputs; Section 3.2,
 * footnote 1).  Inputs are int8 rows [n][K], row-major; outputs are bit rows
 * as bmlp_pack's (bit = 1 <=> +1, tail bits 0).  No context is needed.
 *
 * bmlp_feature_median: d_median int8 [K] receives each feature's median
 * over the n >= 1 rows, the lower middle order statistic (element
 * floor((n-1)/2) of the sorted column), so the threshold is one of the
 * feature's values.
 * bmlp_binarize: median binarisation, bit = (x >= d_median[feature]).
 * 0 <= n <= 65535.
 * bmlp_expand: the fixed random ±1 expansion layer for integer inputs,
 * a_0[j] = sign(sum_i x_i R[j][i]) with sign(0) = +1, summed exactly in
 * int32; R [k0][k_raw] is fixed by seed: element e = j k_raw + i is +1 iff
 * bit (e & 127) of Philox4x32-10 block e >> 7 is set, counter (block,
 * 2^32 - 1, 0, 5), key = seed.  d_bits [n][words(k0)];
 * 1 <= k_raw <= BMLP_MAX_EXPAND_INPUTS, 1 <= k0 <= BMLP_MAX_WIDTH. */
int bmlp_feature_median(const int8_t *d_x, int32_t n, int32_t K, int8_t *d_median, void *stream);
int bmlp_binarize(const int8_t *d_x, int32_t n, int32_t K, const int8_t *d_median, uint64_t *d_bits,
                  void *stream);
int bmlp_expand(const int8_t *d_x, int32_t n, int32_t k_raw, int32_t k0, uint64_t seed, uint64_t *d_bits,
                void *stream);

/* Inference (Algorithm 1 forward and local outputs only): writes the local
 * output y_hat_l of every layer to d_yhat, int32 [L][n][n_classes].
 * d_x: bit rows [n][words(K_0)].  0 <= n <= max_batch. */
int bmlp_forward(bmlp_ctx *ctx, const uint64_t *d_x, int32_t n, int32_t *d_yhat, void *stream);

/* Bytes of the library's static device scratch (one copy per device the
 * library runs on, held until the process ends). */
#define BMLP_NOALLOC_SCRATCH_BYTES (48u << 20)

/* bmlp_forward for callers that cannot allocate device memory or touch the
 * workspace at call time (code under stream or graph capture, serving loops,
 * harnesses that forbid allocation): the same launches and the same d_yhat,
 * but the activation rows a_l go to the library's static scratch instead of
 * the context's workspace, so the workspace (and the trace of the last train
 * step in it) is left alone.  Allocates nothing: no hipMalloc, no hipFree.
 *   Sizes: the a_l rows need sum over l of n * 8 * ceil(K_l / 64) bytes, each
 *   layer rounded up to 256; more than BMLP_NOALLOC_SCRATCH_BYTES returns
 *   BMLP_ESHAPE before any launch (message in bmlp_last_error).
 *   The scratch is shared by every call on a device and keeps the last
 *   call's contents: calls that overlap on one device (two streams, two
 *   threads) race and must be ordered by the caller.  Its device address is
 *   looked up at bmlp_init / bmlp_attach on the then-current device (the
 *   context's device); other arguments and errors as bmlp_forward. */
int bmlp_forward_noalloc(bmlp_ctx *ctx, const uint64_t *d_x, int32_t n, int32_t *d_yhat, void *stream);

/* One training step on a mini-batch (Algorithm 1 body with Algorithms 2-3).
 *   d_x      bit rows [n][words(K_0)], d_y int32 [n].
 *   step     the global step counter t; keys the reinforcement draws, so a run
 *            restored from a checkpoint continues bit-exactly.
 *   p_r      reinforcement probability of this step (the epoch rescale
 *            p_r <- p_r sqrt(E^e) stays with the caller).
 *   d_stats  int32 [L][BMLP_STATS_STRIDE], 8-byte aligned; entries 0..3 of
 *            row l-1 are overwritten with layer l's counts: sum of the
 *            01-loss, |M_l|, |U_l| (selected pairs), and reinforcement draws
 *            that fired (0 when M_l is empty, as the layer is then untouched).
 *            The other entries of a row are scratch.  Each layer's counts
 *            sit in a 128-byte line of their own, so the work-groups adding
 *            to them do not queue on one cache line.
 * Every layer's forward uses the weights from before the step. */
int bmlp_train_step(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
                    uint64_t step, double p_r, int32_t *d_stats, void *stream);

/* Evaluation: adds to d_correct[l-1] the number of patterns whose layer-l
 * local classifier predicts the label (the last layer's classifier is the
 * network output; earlier ones are early exits, Section 3.1).  The caller
 * zeroes d_correct (int32 [L]) before the first batch. */
int bmlp_eval(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
              int32_t *d_correct, void *stream);

/* Early-exit evaluation.  Section 3.1 keeps the intermediate classifiers for
 * early exit without fixing a rule; here a pattern exits at the first layer
 * whose local output has a margin tau = top1 - top2 of at least
 * ceil(r K_l) (the training-time robustness test passed), else at the last
 * layer, and takes that layer's prediction.  Adds to d_counts, int32
 * [L][3] (zeroed by the caller before the first batch), per layer l:
 * [0] patterns whose layer-l classifier predicts the label (as bmlp_eval),
 * [1] patterns that exit at layer l, [2] those exits whose prediction is
 * the label.  0 <= n <= max_batch. */
int bmlp_eval_exit(bmlp_ctx *ctx, const uint64_t *d_x, const int32_t *d_y, int32_t n,
                   int32_t *d_counts, void *stream);

/* One epoch of Algorithm 1 (its loop over mini-batches) over a training set
 * resident on the device: d_x_all bit rows [n_all][words(K_0)], d_y_all
 * int32 [n_all].  d_order int32 [n_order] lists training-set indices (the
 * caller's shuffle; indices outside [0, n_all) are clamped into range).
 * The epoch trains the n_order / batch full batches
 * order[b * batch .. b * batch + batch), b = 0, 1, ..., with step counters
 * step0 + b, all at p_r (1 <= batch <= max_batch; the n_order % batch
 * leftover indices are not trained on).  Each batch is gathered into the
 * workspace and stepped exactly as bmlp_train_step; step b's counts go to
 * d_stats + b * L * BMLP_STATS_STRIDE (int32 [n_order / batch][L][stride],
 * 8-byte aligned).  Everything is enqueued on the stream; the call does not
 * wait for it.  The epoch's error fraction E^e is the sum over the steps of
 * the last layer's 01-loss count, divided by the trained samples; see
 * bmlp_epoch_rescale for the p_r of the next epoch. */
int bmlp_train_epoch(bmlp_ctx *ctx, const uint64_t *d_x_all, const int32_t *d_y_all, int32_t n_all,
                     const int32_t *d_order, int32_t n_order, int32_t batch, uint64_t step0, double p_r,
                     int32_t *d_stats, void *stream);

/* The rescale at the end of an epoch (Algorithm 1, the end of its epoch loop; Section 3.4):
 * p_r * sqrt(wrong / samples) in IEEE double, or p_r unchanged when no
 * sample was trained on.  Host only. */
double bmlp_epoch_rescale(double p_r, int64_t wrong, int64_t samples);

/* The end of an epoch from its step counts (Algorithm 1's epoch loop; Section
 * 3.4, reading R16): h_stats is a host copy of the d_stats that
 * bmlp_train_epoch filled, int32 [steps][n_layers][BMLP_STATS_STRIDE];
 * wrong = the sum over the steps of entry 0 (01-loss count) of the last
 * layer's row, samples = steps * batch.  Writes E^e = wrong / samples to
 * *h_error_fraction (NaN when steps = 0) and bmlp_epoch_rescale(p_r, wrong,
 * samples) to *h_p_r_next; either pointer may be NULL.  Host only; returns
 * BMLP_EINVAL for a NULL h_stats with steps > 0, BMLP_ESHAPE for negative
 * sizes or a layer count outside 1..BMLP_MAX_LAYERS. */
int bmlp_epoch_summary(const int32_t *h_stats, int32_t steps, int32_t n_layers, int32_t batch, double p_r,
                       double *h_error_fraction, double *h_p_r_next);

/* Device pointers to H_l (bit-sliced, see bmlp_layer_info), W_l and P_l of
 * layer l (1..L) in the state. */
int bmlp_layer_views(bmlp_ctx *ctx, int32_t l, uint8_t **d_h, uint64_t **d_w, uint64_t **d_p);

/* Unpacks the hidden weights of layer l (1..L) into plain int8
 * d_out[k_out][k_in] (caller-owned, k_out * k_in bytes), asynchronously on
 * stream.  For checkpoints in a portable form and for inspection. */
int bmlp_read_h(bmlp_ctx *ctx, int32_t l, int8_t *d_out, void *stream);

/* Device pointers to the last train step's per-layer trace in the workspace
 * (layouts in bmlp_layer_info).  bmlp_forward and bmlp_eval overwrite a_l. */
int bmlp_step_trace(bmlp_ctx *ctx, int32_t l, const uint64_t **d_a, const uint8_t **d_err,
                    const uint8_t **d_upd, const int16_t **d_kstar);

/* Static description of a status code. */
const char *bmlp_status_string(int status);

/* Message of the last BMLP_EHIP on this thread ("" if none). */
const char *bmlp_last_error(void);

/* int32 entries per layer row of bmlp_train_step's d_stats (128 bytes). */
#define BMLP_STATS_STRIDE 32

/* Kernel classes timed by the profiling aid below. */
enum {
  BMLP_KERNEL_FWD = 0,      /* hidden-layer forward contraction (z, a)       */
  BMLP_KERNEL_CLS = 1,      /* local classifier contraction (y_hat)          */
  BMLP_KERNEL_SELECT = 2,   /* 01-loss, margin, M_l, easiest perceptrons     */
  BMLP_KERNEL_UPDATE = 3,   /* CP increments, reinforcement, re-sign         */
  BMLP_KERNEL_OTHER = 4,    /* fills and the rest                            */
  BMLP_KERNEL_KINDS = 5
};

/* Profiling aid: times the kernel launches of this context with HIP events
 * on the launch's stream.  Consecutive launches of one kernel class on one
 * stream within one API call form a run that shares a single pair of events
 * (so the event overhead is paid once per run); at most max_launches runs
 * are recorded, later launches go untimed.  The events are host-created
 * objects; no device buffer is allocated.  Returns BMLP_EHIP if the events
 * cannot be created. */
int bmlp_profile_start(bmlp_ctx *ctx, int32_t max_launches);

/* Ends profiling: waits for the last recorded event, then writes per kernel
 * class the summed duration of its runs in milliseconds
 * (h_ms[BMLP_KERNEL_KINDS]) and the number of launches in those runs
 * (h_launches[BMLP_KERNEL_KINDS]), and releases the events.  Either output
 * may be NULL. */
int bmlp_profile_stop(bmlp_ctx *ctx, double *h_ms, int64_t *h_launches);

/* Frees the host-side context.  Device buffers stay with the caller. */
void bmlp_destroy(bmlp_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* BMLP_H_ */
