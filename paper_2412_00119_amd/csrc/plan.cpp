// Host-side planning of the train-step library (see plan.h) and the C ABI
// calls that need no device: sizes, layer descriptions, thresholds, the end
// of an epoch, status strings.
#include "plan.h"

#include <math.h>
#include <string.h>

#include <algorithm>

namespace bmlp {

// Group-size rule of Section 4.3: the divisor of K closest to any value of
// [75, 105]; among equally close divisors the largest.
int gamma_star(int k) {
  int best = 1, best_d = -1;
  for (int g = 1; g <= k; ++g) {
    if (k % g) continue;
    const int d = (g >= 75 && g <= 105) ? 0 : (g < 75 ? 75 - g : g - 105);
    if (best_d < 0 || d < best_d || (d == best_d && g > best)) {
      best = g;
      best_d = d;
    }
  }
  return best;
}

int make_plan(const bmlp_config *cfg, Plan *p) {
  if (cfg == nullptr || p == nullptr || cfg->h_widths == nullptr) return BMLP_EINVAL;
  if (cfg->n_layers < 1 || cfg->n_layers > BMLP_MAX_LAYERS) return BMLP_ESHAPE;
  if (cfg->n_classes < 2 || cfg->n_classes > BMLP_MAX_CLASSES) return BMLP_ESHAPE;
  if (cfg->max_batch < 1 || cfg->max_batch > BMLP_MAX_BATCH) return BMLP_ESHAPE;
  if (cfg->bound < 1 || cfg->bound > 127 || (cfg->bound & 1) == 0) return BMLP_EINVAL;
  if (cfg->group_size < 0 || cfg->group_size > BMLP_MAX_GROUP) return BMLP_ESHAPE;
  if (!(cfg->robustness >= 0.0) || !isfinite(cfg->robustness)) return BMLP_EINVAL;
  if (cfg->fwd_impl != BMLP_FWD_AUTO && cfg->fwd_impl != BMLP_FWD_POPCOUNT &&
      cfg->fwd_impl != BMLP_FWD_MFMA_FP4)
    return BMLP_EINVAL;
  constexpr int kAllVariants =
      BMLP_VARIANT_FAN_IN_REINFORCE | BMLP_VARIANT_SHARED_CLASSIFIER | BMLP_VARIANT_SATURATE_Z |
      BMLP_VARIANT_RESHUFFLE_GROUPS | BMLP_VARIANT_SEQUENTIAL_CLIP;
  if (cfg->variants & ~kAllVariants) return BMLP_EINVAL;
  memset(p, 0, sizeof(*p));
  p->variants = cfg->variants;
  p->L = cfg->n_layers;
  p->c = cfg->n_classes;
  p->max_batch = cfg->max_batch;
  p->bound = cfg->bound;
  p->fwd_impl = cfg->fwd_impl;
  p->r = cfg->robustness;
  p->seed = cfg->seed;
  int kmax = 0;
  for (int l = 0; l <= p->L; ++l) {
    const int k = cfg->h_widths[l];
    if (k < 1 || k > BMLP_MAX_WIDTH) return BMLP_ESHAPE;
    p->widths[l] = k;
    if (l > 0 && k > kmax) kmax = k;
    if ((p->variants & BMLP_VARIANT_SHARED_CLASSIFIER) && l > 1 && k != p->widths[1]) return BMLP_ESHAPE;
  }
  const int nb = p->max_batch;
  size_t so = 0;
  for (int l = 1; l <= p->L; ++l) {
    LayerPlan &lp = p->layer[l - 1];
    lp.k_in = p->widths[l - 1];
    lp.k_out = p->widths[l];
    lp.gamma = cfg->group_size > 0 ? cfg->group_size : gamma_star(lp.k_out);
    if (lp.gamma > BMLP_MAX_GROUP || lp.k_out % lp.gamma != 0) return BMLP_ESHAPE;
    lp.groups = lp.k_out / lp.gamma;
    lp.words_in = words64(lp.k_in);
    lp.words_out = words64(lp.k_out);
    lp.h_ps = (2 * lp.words_in + 15) / 16 * 16;
    lp.ld_h = 4 * h_planes(p->bound) * lp.h_ps;
    const double thr = ceil(p->r * (double)lp.k_out);
    if (thr > 2147483647.0) return BMLP_EINVAL;
    lp.robust_thr = (int)thr;
    lp.off_h = so;
    so = align256(so + (size_t)lp.k_out * lp.ld_h);
    lp.off_w = so;
    so = align256(so + (size_t)lp.k_out * lp.words_in * 8);
    if ((p->variants & BMLP_VARIANT_SHARED_CLASSIFIER) && l > 1) {
      lp.off_p = p->layer[0].off_p;   // layer 1's P serves every layer
    } else {
      lp.off_p = so;
      so = align256(so + (size_t)p->c * lp.words_out * 8);
    }
  }
  p->state_bytes = so;
  size_t wo = 0;
  for (int l = 1; l <= p->L; ++l) {
    LayerPlan &lp = p->layer[l - 1];
    lp.off_a = wo;
    wo = align256(wo + (size_t)nb * lp.words_out * 8);
    lp.off_err = wo;
    wo = align256(wo + (size_t)nb);
    lp.off_upd = wo;
    wo = align256(wo + (size_t)nb);
    lp.off_kstar = wo;
    wo = align256(wo + (size_t)nb * lp.groups * 2);
    lp.off_perm = wo;
    wo = align256(wo + (p->variants & BMLP_VARIANT_RESHUFFLE_GROUPS ? (size_t)lp.k_out * 4 : 0));
  }
  p->off_flag = wo;   // early-exit flags [L][max_batch]
  wo = align256(wo + (size_t)p->L * nb);
  p->off_xb = wo;     // a gathered batch: bit rows [max_batch][words(K_0)] and labels
  wo = align256(wo + (size_t)nb * p->layer[0].words_in * 8);
  p->off_yb = wo;
  wo = align256(wo + (size_t)nb * 4);
  p->ldz = 64 * words64(kmax);
  p->off_z = wo;
  wo = align256(wo + (size_t)nb * p->ldz * 2);
  p->off_yhat = wo;   // int32 [L][max_batch][c], or int16 [L][max_batch][ldy16]
  p->ldy16 = (p->c + 7) & ~7;
  wo = align256(wo + (size_t)p->L * nb * std::max((size_t)p->c * 4, (size_t)p->ldy16 * 2));
  p->ws_bytes = wo;
  return BMLP_OK;
}

uint64_t reinforce_threshold(double p_r, int k) {
  // q = p_r * sqrt(2 / (pi * K)), in this order, in IEEE double.
  const double pk = 3.14159265358979323846 * (double)k;
  const double q = p_r * sqrt(2.0 / pk);
  if (!(q > 0.0)) return 0;
  const double t = ceil(q * 4294967296.0);
  if (t >= 4294967296.0) return 4294967296ull;
  return (uint64_t)t;
}

// min(8, ceil(log2(2 K))) bits: the width of z in the saturating variant
int z_bits(int k) {
  int b = 0;
  while ((1 << b) < 2 * k) ++b;
  return b < 8 ? b : 8;
}

size_t a_rows_offset(const Plan &p, int n, int l) {
  size_t o = 0;
  for (int j = 1; j < l; ++j) o = align256(o + (size_t)n * p.layer[j - 1].words_out * 8);
  return o;
}

}  // namespace bmlp

using namespace bmlp;

extern "C" {

size_t bmlp_state_bytes(const bmlp_config *cfg) {
  Plan p;
  return make_plan(cfg, &p) == BMLP_OK ? p.state_bytes : 0;
}

size_t bmlp_workspace_bytes(const bmlp_config *cfg) {
  Plan p;
  return make_plan(cfg, &p) == BMLP_OK ? p.ws_bytes : 0;
}

int bmlp_describe(const bmlp_config *cfg, int32_t l, bmlp_layer_info *info) {
  if (info == nullptr) return BMLP_EINVAL;
  Plan p;
  const int st = make_plan(cfg, &p);
  if (st != BMLP_OK) return st;
  if (l < 1 || l > p.L) return BMLP_ESHAPE;
  const LayerPlan &lp = p.layer[l - 1];
  info->k_in = lp.k_in;
  info->k_out = lp.k_out;
  info->gamma = lp.gamma;
  info->groups = lp.groups;
  info->words_in = lp.words_in;
  info->words_out = lp.words_out;
  info->ld_h = lp.ld_h;
  info->h_planes = h_planes(p.bound);
  info->h_ps = lp.h_ps;
  info->robust_thr = lp.robust_thr;
  info->off_h = lp.off_h;
  info->off_w = lp.off_w;
  info->off_p = lp.off_p;
  info->off_a = lp.off_a;
  info->off_err = lp.off_err;
  info->off_upd = lp.off_upd;
  info->off_kstar = lp.off_kstar;
  return BMLP_OK;
}

uint64_t bmlp_reinforce_threshold(double p_r, int32_t k_l) {
  if (k_l < 1) return 0;
  return reinforce_threshold(p_r, k_l);
}

double bmlp_epoch_rescale(double p_r, int64_t wrong, int64_t samples) {
  if (samples <= 0) return p_r;
  return p_r * sqrt((double)wrong / (double)samples);
}

int bmlp_epoch_summary(const int32_t *h_stats, int32_t steps, int32_t n_layers, int32_t batch, double p_r,
                       double *h_error_fraction, double *h_p_r_next) {
  if (steps < 0 || batch < 0 || n_layers < 1 || n_layers > BMLP_MAX_LAYERS) return BMLP_ESHAPE;
  if (steps > 0 && h_stats == nullptr) return BMLP_EINVAL;
  int64_t wrong = 0;
  for (int32_t b = 0; b < steps; ++b)
    wrong += h_stats[((size_t)b * n_layers + (n_layers - 1)) * BMLP_STATS_STRIDE];
  const int64_t samples = (int64_t)steps * batch;
  if (h_error_fraction) *h_error_fraction = samples > 0 ? (double)wrong / (double)samples : NAN;
  if (h_p_r_next) *h_p_r_next = bmlp_epoch_rescale(p_r, wrong, samples);
  return BMLP_OK;
}

const char *bmlp_status_string(int status) {
  switch (status) {
    case BMLP_OK: return "ok";
    case BMLP_EINVAL: return "invalid argument";
    case BMLP_ESHAPE: return "size out of range";
    case BMLP_EHIP: return "HIP launch failed";
    case BMLP_ESTATE: return "misaligned state or workspace buffer";
    default: return "unknown status";
  }
}

}  // extern "C"
