// Host-only check of the library's planning code (plan.cpp): thousands of
// random configurations, valid and invalid, through make_plan and the C ABI
// calls that need no device, with the layout invariants checked on every
// valid plan.  Built and run under AddressSanitizer and UndefinedBehavior-
// Sanitizer by tests/test_host_sanitized.py; prints "ok" and exits 0 when
// every check holds.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <random>
#include <utility>
#include <vector>

#include "plan.h"

using namespace bmlp;

static int g_fail = 0;
#define CHECK(cond, ...)                                      \
  do {                                                        \
    if (!(cond)) {                                            \
      fprintf(stderr, "check failed: %s: ", #cond);           \
      fprintf(stderr, __VA_ARGS__);                           \
      fprintf(stderr, "\n");                                  \
      if (++g_fail > 20) exit(1);                             \
    }                                                         \
  } while (0)

// Every region of a valid plan starts on 256 bytes, lies inside its buffer,
// and no two regions of one buffer overlap (layer 1's classifier is shared
// by every layer with the shared-classifier variant).
static void check_layout(const bmlp_config &cfg, const Plan &p) {
  std::vector<std::pair<size_t, size_t>> st, ws;
  for (int l = 1; l <= p.L; ++l) {
    const LayerPlan &lp = p.layer[l - 1];
    CHECK(lp.k_in == cfg.h_widths[l - 1] && lp.k_out == cfg.h_widths[l], "widths of layer %d", l);
    CHECK(lp.gamma >= 1 && lp.k_out % lp.gamma == 0 && lp.groups * lp.gamma == lp.k_out, "groups of layer %d", l);
    if (cfg.group_size > 0) CHECK(lp.gamma == cfg.group_size, "gamma of layer %d", l);
    else CHECK(lp.gamma == gamma_star(lp.k_out), "gamma* of layer %d", l);
    CHECK(lp.words_in == (lp.k_in + 63) / 64 && lp.words_out == (lp.k_out + 63) / 64, "words of layer %d", l);
    CHECK(lp.h_ps % 16 == 0 && lp.h_ps >= 2 * lp.words_in, "h_ps of layer %d", l);
    CHECK(lp.ld_h == 4 * h_planes(p.bound) * lp.h_ps, "ld_h of layer %d", l);
    CHECK((double)lp.robust_thr == ceil(cfg.robustness * (double)lp.k_out), "robust_thr of layer %d", l);
    const size_t h_bytes = (size_t)lp.k_out * lp.ld_h, w_bytes = (size_t)lp.k_out * lp.words_in * 8;
    const size_t p_bytes = (size_t)p.c * lp.words_out * 8;
    st.push_back({lp.off_h, h_bytes});
    st.push_back({lp.off_w, w_bytes});
    const bool shared = (p.variants & BMLP_VARIANT_SHARED_CLASSIFIER) && l > 1;
    if (shared) CHECK(lp.off_p == p.layer[0].off_p, "shared P of layer %d", l);
    else st.push_back({lp.off_p, p_bytes});
    const size_t nb = (size_t)p.max_batch;
    ws.push_back({lp.off_a, nb * lp.words_out * 8});
    ws.push_back({lp.off_err, nb});
    ws.push_back({lp.off_upd, nb});
    ws.push_back({lp.off_kstar, nb * lp.groups * 2});
    if (p.variants & BMLP_VARIANT_RESHUFFLE_GROUPS) ws.push_back({lp.off_perm, (size_t)lp.k_out * 4});
  }
  int kmax = 0;
  for (int l = 1; l <= p.L; ++l) kmax = std::max(kmax, p.widths[l]);
  CHECK(p.ldz >= kmax && p.ldz % 64 == 0, "ldz");
  const size_t nb = (size_t)p.max_batch;
  ws.push_back({p.off_flag, (size_t)p.L * nb});
  ws.push_back({p.off_xb, nb * p.layer[0].words_in * 8});
  ws.push_back({p.off_yb, nb * 4});
  ws.push_back({p.off_z, nb * p.ldz * 2});
  ws.push_back({p.off_yhat, (size_t)p.L * nb * p.c * 4});
  for (auto *v : {&st, &ws}) {
    const size_t total = v == &st ? p.state_bytes : p.ws_bytes;
    CHECK(total % 256 == 0, "total %zu not aligned", total);
    std::sort(v->begin(), v->end());
    for (size_t i = 0; i < v->size(); ++i) {
      const auto &r = (*v)[i];
      CHECK(r.first % 256 == 0, "region at %zu not aligned", r.first);
      CHECK(r.first + r.second <= total, "region [%zu, +%zu) past the buffer (%zu)", r.first, r.second, total);
      if (i + 1 < v->size()) CHECK(r.first + r.second <= (*v)[i + 1].first, "regions overlap at %zu", r.first);
    }
  }
  CHECK(bmlp_state_bytes(&cfg) == p.state_bytes && bmlp_workspace_bytes(&cfg) == p.ws_bytes, "sizes");
  for (int l = 1; l <= p.L; ++l) {
    bmlp_layer_info info;
    CHECK(bmlp_describe(&cfg, l, &info) == BMLP_OK, "describe %d", l);
    const LayerPlan &lp = p.layer[l - 1];
    CHECK(info.gamma == lp.gamma && info.ld_h == lp.ld_h && info.off_h == lp.off_h && info.off_a == lp.off_a &&
              info.h_planes == h_planes(p.bound) && info.robust_thr == lp.robust_thr,
          "describe fields of layer %d", l);
  }
  bmlp_layer_info info;
  CHECK(bmlp_describe(&cfg, 0, &info) == BMLP_ESHAPE && bmlp_describe(&cfg, p.L + 1, &info) == BMLP_ESHAPE,
        "describe out of range");
  // the packed activation rows of the no-allocation forward
  for (int n : {1, 7, p.max_batch}) {
    size_t prev = 0;
    for (int l = 1; l <= p.L + 1; ++l) {
      const size_t o = a_rows_offset(p, n, l);
      CHECK(o % 256 == 0 && o >= prev, "a_rows_offset(%d, %d)", n, l);
      if (l > 1) CHECK(o >= prev + (size_t)n * p.layer[l - 2].words_out * 8, "a_rows_offset gap");
      prev = o;
    }
  }
}

int main() {
  std::mt19937_64 rng(20241130);
  auto pick = [&](int lo, int hi) { return (int)std::uniform_int_distribution<int>(lo, hi)(rng); };
  const int divisors_pool[] = {1, 2, 3, 4, 8, 13, 16, 32, 64, 96, 105, 128};
  int valid = 0, invalid = 0;
  std::vector<int32_t> widths(BMLP_MAX_LAYERS + 1);
  for (int it = 0; it < 20000; ++it) {
    bmlp_config cfg;
    cfg.n_layers = pick(0, 6) == 0 ? pick(-1, BMLP_MAX_LAYERS + 1) : pick(1, 12);
    const int L = std::max(1, std::min(cfg.n_layers, BMLP_MAX_LAYERS));
    cfg.group_size = pick(0, 3) == 0 ? 0 : divisors_pool[pick(0, 11)];
    for (int l = 0; l <= L; ++l) {
      int k;
      switch (pick(0, 5)) {
        case 0: k = pick(-2, 40); break;
        case 1: k = pick(1, BMLP_MAX_WIDTH + 2); break;
        case 2: k = 64 * pick(1, 64); break;
        default: k = (cfg.group_size > 0 ? cfg.group_size : 64) * pick(1, 40); break;
      }
      widths[l] = k;
    }
    if (pick(0, 7) == 0) for (int l = 2; l <= L; ++l) widths[l] = widths[1];
    cfg.h_widths = widths.data();
    cfg.n_classes = pick(0, 9) == 0 ? pick(-1, BMLP_MAX_CLASSES + 1) : pick(2, 1000);
    cfg.max_batch = pick(0, 9) == 0 ? pick(-1, BMLP_MAX_BATCH + 1) : pick(1, 4096);
    cfg.bound = pick(0, 9) == 0 ? pick(-1, 130) : 2 * pick(0, 63) + 1;
    const double rs[] = {0.0, 0.25, 1.0, 3.5, -0.5, NAN, INFINITY, 1e12};
    cfg.robustness = pick(0, 4) == 0 ? rs[pick(0, 7)] : std::uniform_real_distribution<double>(0.0, 2.0)(rng);
    cfg.seed = rng();
    cfg.fwd_impl = pick(0, 9) == 0 ? pick(-1, 4) : pick(0, 2);
    cfg.variants = pick(0, 9) == 0 ? pick(0, 64) : pick(0, 31);
    Plan p;
    const int st = make_plan(&cfg, &p);
    if (st == BMLP_OK) {
      ++valid;
      check_layout(cfg, p);
    } else {
      ++invalid;
      CHECK(st == BMLP_EINVAL || st == BMLP_ESHAPE, "status %d", st);
      CHECK(bmlp_state_bytes(&cfg) == 0 && bmlp_workspace_bytes(&cfg) == 0, "sizes of an invalid config");
    }
  }
  CHECK(valid > 1000 && invalid > 1000, "valid %d invalid %d", valid, invalid);

  // specific invalid configurations
  {
    int32_t w[3] = {64, 128, 128};
    bmlp_config base{2, w, 10, 32, 7, 64, 0.25, 1, 0, 0};
    Plan p;
    CHECK(make_plan(&base, &p) == BMLP_OK, "base config");
    bmlp_config c = base;
    c.bound = 8;
    CHECK(make_plan(&c, &p) == BMLP_EINVAL, "even bound");
    c = base;
    c.group_size = 48;
    CHECK(make_plan(&c, &p) == BMLP_ESHAPE, "gamma not dividing");
    c = base;
    c.h_widths = nullptr;
    CHECK(make_plan(&c, &p) == BMLP_EINVAL, "null widths");
    CHECK(make_plan(nullptr, &p) == BMLP_EINVAL && make_plan(&base, nullptr) == BMLP_EINVAL, "null pointers");
    c = base;
    c.variants = BMLP_VARIANT_SHARED_CLASSIFIER;
    w[2] = 192;
    CHECK(make_plan(&c, &p) == BMLP_ESHAPE, "shared classifier with unequal widths");
    CHECK(bmlp_describe(nullptr, 1, nullptr) == BMLP_EINVAL, "describe null");
  }

  // the group-size rule's worked examples (Section 4.3), and divisibility
  CHECK(gamma_star(525) == 105 && gamma_star(2025) == 81, "gamma* examples");
  for (int k = 1; k <= 5000; ++k) CHECK(k % gamma_star(k) == 0, "gamma*(%d) divides", k);

  // reinforcement thresholds: 0 for p_r = 0, monotone, at most 2^32
  for (int k : {1, 64, 784, 4096, 32767}) {
    uint64_t prev = 0;
    CHECK(reinforce_threshold(0.0, k) == 0 && bmlp_reinforce_threshold(0.0, k) == 0, "T(0)");
    for (double pr = 1e-6; pr < 1e4; pr *= 1.7) {
      const uint64_t t = reinforce_threshold(pr, k);
      CHECK(t >= prev && t <= (1ull << 32), "T(%g, %d)", pr, k);
      prev = t;
    }
    CHECK(reinforce_threshold(1e9, k) == (1ull << 32), "T saturates");
  }
  CHECK(bmlp_reinforce_threshold(0.5, 0) == 0, "T of an empty layer");
  for (int k = 1; k < 200; ++k) CHECK(z_bits(k) >= 1 && z_bits(k) <= 8 && (1 << z_bits(k)) >= std::min(2 * k, 256), "z_bits");

  // the end of an epoch
  for (int it = 0; it < 2000; ++it) {
    const int steps = pick(0, 20), L = pick(1, 6), batch = pick(1, 300);
    std::vector<int32_t> s((size_t)std::max(steps, 1) * L * BMLP_STATS_STRIDE);
    int64_t wrong = 0;
    for (int b = 0; b < steps; ++b) {
      for (int l = 0; l < L; ++l) s[((size_t)b * L + l) * BMLP_STATS_STRIDE] = pick(0, batch);
      wrong += s[((size_t)b * L + L - 1) * BMLP_STATS_STRIDE];
    }
    double e = -1.0, nxt = -1.0;
    CHECK(bmlp_epoch_summary(s.data(), steps, L, batch, 0.5, &e, &nxt) == BMLP_OK, "summary");
    if (steps > 0) {
      CHECK(e == (double)wrong / ((double)steps * batch), "E^e");
      CHECK(nxt == bmlp_epoch_rescale(0.5, wrong, (int64_t)steps * batch), "p_r");
    } else {
      CHECK(isnan(e) && nxt == 0.5, "empty epoch");
    }
  }
  CHECK(bmlp_epoch_summary(nullptr, 1, 1, 1, 0.5, nullptr, nullptr) == BMLP_EINVAL, "summary null");
  CHECK(bmlp_epoch_summary(nullptr, 0, 0, 1, 0.5, nullptr, nullptr) == BMLP_ESHAPE, "summary no layer");
  for (int code = -6; code <= 1; ++code) CHECK(bmlp_status_string(code) != nullptr, "status string %d", code);

  if (g_fail) {
    fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  printf("ok: %d valid and %d invalid configurations\n", valid, invalid);
  return 0;
}
