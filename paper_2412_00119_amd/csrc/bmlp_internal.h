// Internal declarations shared by the host library and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bmlp.h"
#include "plan.h"

namespace bmlp {

// Philox stream ids of the method's random draws (counter word 3).
enum : uint32_t {
  kStreamHInit = 1,     // H_l initial signs
  kStreamPInit = 2,     // P_l entries
  kStreamCoarse = 3,    // reinforcement: top byte of the 32-bit draw
  kStreamFine = 4,      // reinforcement: low 24 bits of the 32-bit draw
  kStreamGroups = 6,    // per-step group order (reshuffle variant)
};

// The fourth word of a buffer descriptor for a raw (stride 0) buffer of
// 32-bit words on this architecture family: the kernels that read through
// buffer descriptors (scalar or per-lane offsets, bounds checked against the
// buffer's size) build theirs with it.
constexpr int kRawRsrcWord3 = 0x00020000;

// ---------------------------------------------------------------------------
// Launchers (each returns hipSuccess or the launch error).
// ---------------------------------------------------------------------------

hipError_t launch_pack(const int8_t *x, int n, int K, uint64_t *bits, hipStream_t s);

// H_l and W_l of one layer from Philox stream 1 (init) or W_l from the H_l in
// place (attach); P_l from stream 2.
hipError_t launch_read_h(const uint8_t *H, int ld_h, int h_ps, int bound, int k_in, int k_out,
                         int8_t *out, hipStream_t s);
hipError_t launch_init_h(uint8_t *H, int ld_h, int h_ps, int bound, uint64_t *W, int words_in, int k_in,
                         int k_out, uint64_t seed, int layer, bool from_h, hipStream_t s);
hipError_t launch_init_p(uint64_t *P, int words_out, int k_out, int c, uint64_t seed, int layer,
                         hipStream_t s);

hipError_t launch_fill_i32(int32_t *p, int count, int32_t value, hipStream_t s);
hipError_t launch_fill_rows_i32(int32_t *p, int rows, int cols, int ld, int32_t value,
                                hipStream_t s);

// Hidden layer forward: z = K_in - 2 popc(a_prev ^ W) -> z (int16 [n][ldz],
// optional) and a = (z >= 0) bits [n][words_out].
hipError_t launch_fwd_popcount(const uint64_t *a_prev, int words_in, int k_in, const uint64_t *W,
                               int n, int k_out, int16_t *z, int ldz, uint64_t *a_out,
                               int words_out, hipStream_t s);

// Local classifier: out[m][c] += -2 popc(a ^ P_c); out must hold K_l first.
hipError_t launch_cls_popcount(const uint64_t *a, int words, int k, const uint64_t *P, int n,
                               int c, int32_t *out, int ldo, hipStream_t s);

// Forward on the matrix cores: bit-row operands expanded to fp4 in registers.
// The same contraction gives the local classifier's y_hat = a_l P_l^T (A =
// a_l, B = P_l) when the classes are too many for the classifier kernel
// (kFwdWriteZ or kFwdWriteZ32, words_out = 0: no sign bits).
enum { kFwdFusedSelect = 0, kFwdWriteZ = 1, kFwdPlain = 2, kFwdWriteZ32 = 3 };
// One layer of a launch: its operands (A and B rows share the stride ld),
// K and z.  A launch of several slices (kFwdWriteZ or kFwdWriteZ32 only)
// runs the nt_m x nt_n tiles of each in turn; M, N and ldz are common.
struct FwdSlice {
  const uint64_t *A, *B;
  int ld, K;
  int16_t *z;
  int32_t *z32;
};
constexpr int kMaxFwdSlices = 8;
struct FwdArgs {
  const uint64_t *A; int lda;       // a_{l-1} bit rows [M][lda words]
  const uint64_t *B; int ldb;       // W_l bit rows [N][ldb words]
  int M, N, K;                      // K = K_{l-1} elements per row (lda, ldb >= ceil(K / 64))
  uint64_t *abits; int words_out;   // a_l bits [M][words_out]
  int mode;
  int16_t *kstar; int ldk;          // kFwdFusedSelect (gamma = 64): raw selection [groups][ldk]
  const int32_t *y; int c;          // kFwdFusedSelect: labels [M] and class count
  const uint64_t *P; int ldp;       // kFwdFusedSelect: P_l rows [c][ldp], rho^{y^mu} = P_l[y^mu]
  int16_t *z; int ldz;              // kFwdWriteZ: z int16 [M][ldz]
  int32_t *z32;                     // kFwdWriteZ32: z int32 [M][ldz]
  float zlo, zhi;                   // kFwdFusedSelect: the selection clips z to [zlo, zhi]
  int32_t *zero; int nzero;         // if set: zeroed by the first work-group (step statistics)
  int nslices;                      // > 1: sl[0 .. nslices) replace A, B, lda, ldb, K, z, z32
  FwdSlice sl[kMaxFwdSlices];       // (for one slice the launcher fills sl[0] from those fields)
  int nt_m, nt_n, xcd_remap;        // set by the launcher (xcd_remap: 1 = slices of B, 2 = of A)
  int pw_max, ystride;              // set by the launcher: last word of a P row; label stride
};
hipError_t launch_fwd_fp4(FwdArgs &a, hipStream_t s);

// Classifier on the matrix cores, then the local error signal, for up to
// kMaxClsLayers layers in one launch (ceil(n / 16) work-groups per layer),
// for up to kClsMaxClasses classes.  Above that, y_hat comes from the
// forward kernel (kFwdWriteZ) and launch_cls_argmax takes the error signal
// from it.
constexpr int kClsMaxClasses = 128;
enum { kClsTrain = 0, kClsYhatOnly = 1, kClsEval = 2 };
struct ClsLayer {
  const uint64_t *A;                // a_l bit rows [n][words]
  const uint64_t *P;                // P_l bit rows [c][words]
  int words, K, thr;                // words = ceil(K / 64)
  int32_t *yhat;                    // y_hat int32 [n][c]: output (kClsYhatOnly)
  const int16_t *y16;               // launch_cls_argmax: y_hat int16 [n][ldy]
  uint8_t *err, *upd;               // train
  int32_t *stats;                   // train: this layer's [4], adds [0] and [1]
  int32_t *correct;                 // eval: adds the correct count
  uint8_t *flag;                    // eval, if set: per pattern, 1 = correct, 2 = tau >= thr
};
constexpr int kMaxClsLayers = 8;
struct ClsBatch {
  ClsLayer L[kMaxClsLayers];
  int nl, n, c, mode;
  const int32_t *y;
  int ldy;                          // launch_cls_argmax: a multiple of 4, >= c
};
hipError_t launch_cls_fp4(const ClsBatch &a, hipStream_t s);
// The local error signal (kClsTrain or kClsEval) from stored int16 y_hat rows.
hipError_t launch_cls_argmax(const ClsBatch &a, hipStream_t s);

// 01-loss, margin and M (when yhat is given), and the easiest wrong
// perceptron of every group for every pattern (U_l is its restriction to the
// patterns in M, which the update kernel applies).
struct LossSelectArgs {
  const int32_t *yhat; int c;
  const int16_t *z; int ldz;
  const uint64_t *P; int words_out;
  const int32_t *y; int n;
  int k_out, gamma, groups, thr;
  uint8_t *err, *upd;
  int16_t *kstar; int ldk; // [groups][ldk]
  int32_t *stats;          // this layer's [4]
  int zlo, zhi;            // the selection clips z to [zlo, zhi]
  const int32_t *perm;     // group order [k_out] (reshuffle variant), or null: contiguous
};
hipError_t launch_loss_select(const LossSelectArgs &a, hipStream_t s);

// correct[0] += #(argmax yhat == y)
// flag, if set: per pattern, 1 = correct, 2 = the margin tau reaches thr
hipError_t launch_eval_count(const int32_t *yhat, int c, const int32_t *y, int n, int32_t *correct,
                             uint8_t *flag, int thr, hipStream_t s);
// Early exits from the per-layer flags [L][ldf] (see launch_eval_count):
// counts[l][1] += patterns whose first layer with flag & 2 (or the last
// layer) is l, counts[l][2] += those of them with flag & 1.
hipError_t launch_exit_count(const uint8_t *flags, int ldf, int L, int n, int32_t *counts, hipStream_t s);
// Rows order[0..n) of a training set gathered into a batch: xb [n][words],
// yb [n]; indices outside [0, n_all) are clamped into it.
hipError_t launch_gather_batch(const uint64_t *x_all, const int32_t *y_all, int n_all, int words,
                               const int32_t *order, int n, uint64_t *xb, int32_t *yb, hipStream_t s);

// The input side (int8 features): per-feature lower median over n rows;
// bit = (x >= thr) rows; the fixed random ±1 expansion layer sign(x R^T).
hipError_t launch_feature_median(const int8_t *x, int n, int K, int8_t *med, hipStream_t s);
hipError_t launch_binarize(const int8_t *x, int n, int K, const int8_t *thr, uint64_t *bits, hipStream_t s);
hipError_t launch_expand(const int8_t *x, int n, int k_raw, int k0, uint64_t seed, uint64_t *bits, hipStream_t s);

// Clipped-Perceptron increments + reinforcement + clip + re-sign of up to
// kMaxUpdLayers layers in one launch.
struct UpdLayer {
  uint8_t *H;              // bit-sliced [K_l][ld_h bytes]
  uint32_t *W32;
  const uint32_t *a32;     // a_{l-1} bit rows as 32-bit words [n][nw32]
  const int16_t *kstar;    // [groups][ldk], for every pattern
  const uint8_t *upd;      // [n]: only patterns in M_l are used
  const uint64_t *P;
  int32_t *stats;          // this layer's [4]; reads [1] (|M|), adds [2] and [3]
  int ld_h, h_ps, nw32, words_out, k_in, groups, gamma;
  int chunks, block0;      // filled by launch_update
  uint32_t t_hi, t_lo;     // T_l >> 24 (0..256) and T_l & 0xFFFFFF
  uint32_t ctr1;           // layer - 1
  const int32_t *perm;     // group order [k_out], or null: contiguous groups
};
constexpr int kMaxUpdLayers = 8;
struct UpdateBatch {
  UpdLayer L[kMaxUpdLayers];
  int nl;
  const int32_t *y;
  int n, ldk, c, bound;
  uint32_t key0, key1, step;
  int sequential;          // increments applied pattern by pattern, each clipped
};
hipError_t launch_update(UpdateBatch &b, hipStream_t s);

// The reshuffle variant's group order of each layer at one step: perm[i]
// is the perceptron at position i when the K perceptrons are sorted by
// their stream-6 keys, ties by index.
struct PermLayer {
  int32_t *perm;
  int k;
  uint32_t ctr1;           // layer - 1
  int block0;              // filled by launch_group_perm
};
struct PermBatch {
  PermLayer L[8];
  int nl;
  uint32_t key0, key1, step;
};
hipError_t launch_group_perm(PermBatch &b, hipStream_t s);

}  // namespace bmlp
