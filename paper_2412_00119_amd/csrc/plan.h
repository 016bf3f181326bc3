// Host-side planning of the train-step library: configuration checks, the
// group-size rule, the host scalars of the method (thresholds) and the
// layout of the state and workspace buffers.  Plain C++ with no HIP, so that
// it also builds and runs on the host alone (the sanitizer test does that).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "bmlp.h"

namespace bmlp {

// Bit planes of H: u = (h + B) / 2 lies in [0, B], B odd.
constexpr int h_planes(int bound) {
  int m = 1;
  while ((1 << m) <= bound) ++m;
  return m;
}

struct LayerPlan {
  int k_in, k_out, gamma, groups;
  int words_in, words_out;   // uint64 words per bit row of a_{l-1} / a_l
  int ld_h;                  // bytes per H row: h_planes planes of h_ps words
  int h_ps;                  // 32-bit words per plane of an H row, multiple of 16
  int robust_thr;            // ceil(r K_l)
  size_t off_h, off_w, off_p;                              // state
  size_t off_a, off_err, off_upd, off_kstar, off_perm;     // workspace
};

struct Plan {
  int L, c, max_batch, bound, fwd_impl, variants;
  double r;
  uint64_t seed;
  int widths[BMLP_MAX_LAYERS + 1];
  LayerPlan layer[BMLP_MAX_LAYERS];   // layer[l-1] describes layer l
  int ldz;                            // int16 elements per row of the z scratch
  size_t off_z, off_yhat;             // shared scratch in the workspace
  int ldy16;                          // y_hat as int16 rows [L][max_batch][ldy16] (in off_yhat)
  size_t off_flag, off_xb, off_yb;    // early-exit flags; a gathered batch (epoch driver)
  size_t state_bytes, ws_bytes;
};

// Validates cfg and fills plan; returns a BMLP_* status.
int make_plan(const bmlp_config *cfg, Plan *plan);

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }
inline int words64(int k) { return (k + 63) / 64; }

// Group-size rule of Section 4.3 (gamma* of a layer of k perceptrons).
int gamma_star(int k);

// ceil(q 2^32) for the reinforcement probability q = p_r sqrt(2 / (pi k))
// (Algorithm 3), at most 2^32.
uint64_t reinforce_threshold(double p_r, int k);

// min(8, ceil(log2(2 k))): the bits of z in the saturating variant.
int z_bits(int k);

// Byte offset of layer l's n activation rows when the rows of every layer
// are packed one after another, each layer from a 256-byte boundary
// (a_rows_offset(p, n, L + 1) is the total).
size_t a_rows_offset(const Plan &p, int n, int l);

}  // namespace bmlp
