// Local classifiers and local error signals on the matrix cores, for every
// layer of a step in one launch (Algorithm 1: y_hat = a_l P_l^T, the 01-loss
// of Eq. 1 and the robustness test that builds M_l).  The layers are
// independent once every forward is done, so one launch covers them all.
//
// A work-group owns 16 patterns of one layer and all its classes, up to
// kClsMaxClasses of them: CB blocks of 16 classes (CB, a template parameter,
// is the exact block count).  Its four waves split K: wave w takes the
// super-blocks w, w + 4, ... of 512 elements, over every class block, so
// that a_l's rows are read once per work-group and each wave's a_l operand
// serves all CB blocks.  a_l and P_l are read as bit rows straight into
// registers, lane (r, q) holding the 16 bytes 16q .. 16q + 15 of the
// super-block's 64 bytes of row r (elements 128q .. 128q + 127: four 32-bit
// words); the loads of CH super-blocks are all issued before their MFMAs
// (for a 4096-wide layer with more than 64 classes, every load of the wave).
//
// Operands by K class (element k in class k mod 4, bit 4t + s of a word in
// class s): the MFMA of class s takes, from each of the lane's four words,
// the bits of class s in place (nibble t of dword d = bit 4t + s of word d;
// both operands use the same map, so every product pairs the same k).
//   * a_l as ±1 in every class (the e2m1 sign bit made from the element's
//     bit: a shift to bit 3 and one bit operation);
//   * P_l as ±1 in class 3 and, in classes 0..2, as the bit alone (0 or
//     2^(s-1)) with block scale 2^(2-s), so that a product is 2 (2a - 1) p
//     for bits a, p.
// The accumulator then holds y' = y_hat + 2 P_a - n_low, with P_a the
// pattern row's popcount over classes 0..2 and n_low = K - floor(K / 4)
// its class 0..2 elements (2 (2a - 1) p - (2a - 1)(2p - 1) = 2a - 1).  The
// offset is the same for every class of a pattern, so the argmax and the
// margin tau are those of y_hat; y_hat itself (kClsYhatOnly) subtracts it,
// with P_a counted from the same words.  Every value is an integer below
// 2^24, exact in fp32.  Elements past K_l become fp4 zeros in the P
// operand; rows past n or c repeat the last row and only feed entries that
// are never read.
//
// The accumulators go to LDS (the four K groups' partials are added when
// read), then sixteen lanes take each pattern: first argmax (lowest class on
// ties), the two largest values (tau = top1 - top2, 0 on a tie), err =
// (pred != y) and upd = err or tau < ceil(r K_l).
//
// With more classes, loading every class row for each 16 patterns would
// read P_l n / 16 times over; y_hat then comes from the forward kernel (a
// tiled contraction with P_l in place of W_l, which reads each operand tile
// once per output tile), and cls_argmax_kernel below takes the same error
// signal from the stored y_hat, one wave per pattern.
#include <limits.h>

#include <type_traits>

#include "bmlp_internal.h"
#include "fp4.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;

// the class-s operand of a pattern's words: ±1 from bit 4t + s of each word
__device__ __forceinline__ uint32_t pm1_class(uint32_t w, int s) {
  return fp4_sign_nibbles(s == 3 ? w : w << (3 - s));
}
__device__ __forceinline__ uint4 pm1_operand(const uint4 &w, int s) {
  return make_uint4(pm1_class(w.x, s), pm1_class(w.y, s), pm1_class(w.z, s), pm1_class(w.w, s));
}
__device__ __forceinline__ uint4 bit_operand(const uint4 &w, int s) {
  return make_uint4(class_bits(w.x, s), class_bits(w.y, s), class_bits(w.z, s), class_bits(w.w, s));
}
__device__ __forceinline__ uint4 bit_operand_masked(const uint4 &w, const uint32_t (&v)[4], int s) {
  return make_uint4(class_bits_masked(w.x, v[0], s), class_bits_masked(w.y, v[1], s),
                    class_bits_masked(w.z, v[2], s), class_bits_masked(w.w, v[3], s));
}

// lane l: A row / B column (l & 15), elements 32 (l >> 4) .. +31 of the
// 128-element K block; result element e of lane l is row 4 (l >> 4) + e,
// column (l & 15).  Operand formats 4 = e2m1; E8M0 block scales: 1 for the
// patterns, class_scale(s) for the classifier rows.
__device__ __forceinline__ v4f mfma_fp4(const uint4 &a, const uint4 &b, v4f c, int s) {
  const v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
  const v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 4, 4, 0, 127, 0, class_scale(s));
}

// 16 bytes at byte o of a bit row of rowbytes bytes (a multiple of 8), zero
// past its end; rows start on 16-byte boundaries when ALIGNED, else on
// 8-byte ones
template <bool ALIGNED>
__device__ __forceinline__ uint4 load16(const uint8_t *row, int o) {
  if constexpr (ALIGNED) {
    return *reinterpret_cast<const uint4 *>(row + o);
  } else {
    const uint2 lo = *reinterpret_cast<const uint2 *>(row + o);
    const uint2 hi = *reinterpret_cast<const uint2 *>(row + o + 8);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}
template <bool ALIGNED>
__device__ __forceinline__ uint4 load16_tail(const uint8_t *row, int o, int rowbytes) {
  if (o + 16 <= rowbytes) return load16<ALIGNED>(row, o);
  uint2 lo = make_uint2(0u, 0u);
  if (o + 8 <= rowbytes) lo = *reinterpret_cast<const uint2 *>(row + o);
  return make_uint4(lo.x, lo.y, 0u, 0u);
}

struct Top2 {
  int v1, i1, v2;
};

__device__ __forceinline__ Top2 merge(Top2 a, Top2 b) {
  Top2 r;
  if (a.v1 > b.v1 || (a.v1 == b.v1 && a.i1 < b.i1)) {
    r.v1 = a.v1;
    r.i1 = a.i1;
  } else {
    r.v1 = b.v1;
    r.i1 = b.i1;
  }
  r.v2 = max(min(a.v1, b.v1), max(a.v2, b.v2));   // second largest of the union
  return r;
}

// a lane's top-two as seen through DPP control CTRL (a partner in its row)
template <int CTRL>
__device__ __forceinline__ Top2 dpp_top2(const Top2 &t) {
  Top2 o;
  o.v1 = __builtin_amdgcn_update_dpp(0, t.v1, CTRL, 0xF, 0xF, false);
  o.i1 = __builtin_amdgcn_update_dpp(0, t.i1, CTRL, 0xF, 0xF, false);
  o.v2 = __builtin_amdgcn_update_dpp(0, t.v2, CTRL, 0xF, 0xF, false);
  return o;
}

template <int CB>
struct ClsShape {
  static constexpr int KG = kWaves;              // wave groups along K (each wave takes every class block)
  static constexpr int CH = CB > 4 ? 2 : 4;      // super-blocks per load round
  static constexpr int LD = CB * 16 + 4;         // LDS row stride of the partials
};

// ALIGNED: every row starts on a 16-byte boundary.  YHAT: y_hat is the
// output (kClsYhatOnly); otherwise the error signal (kClsTrain, kClsEval).
// The pattern count, the class count and the labels come first as scalars,
// preloaded into scalar registers when the wave starts, so that the layer
// lookup and the label loads do not wait for a read of the argument buffer.
template <int CB, bool ALIGNED, bool YHAT>
__global__ __launch_bounds__(64 * kWaves) void cls_fp4_kernel(int pn, int pc, const int32_t *py, ClsBatch p) {
  constexpr int KG = ClsShape<CB>::KG, CH = ClsShape<CB>::CH, LD = ClsShape<CB>::LD;
  __shared__ int red[KG][16][LD];        // y' partials of the K groups
  __shared__ int spa[KG][16];            // YHAT: P_a partials of the K groups
  __shared__ int cnt[3];                 // block totals of err, upd, correct

  const int tid = threadIdx.x, kg = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int bpl = (pn + 15) / 16;               // work-groups per layer
  const ClsLayer &Lr = p.L[blockIdx.x / bpl];
  const int m0 = (blockIdx.x % bpl) * 16;
  const int lr = lane & 15, q = lane >> 4;       // row / class, and which 16 bytes of a super-block
  const int K = Lr.K;
  if (tid < 3) cnt[tid] = 0;
  const int mu = m0 + 4 * kg + q;                // the argmax: waves 0..3 take 4 patterns each
  int label = 0;
  // Every argument the end of the kernel needs, read now: left to itself the
  // compiler loads them where they are used, one dependent scalar load after
  // another, each a miss that the argmax then waits for.
  const int mode = p.mode, thr = Lr.thr;
  uint8_t *const err_out = Lr.err, *const upd_out = Lr.upd, *const flag_out = Lr.flag;
  int32_t *const stats_out = Lr.stats, *const correct_out = Lr.correct, *const yhat_out = Lr.yhat;
  asm volatile("" ::"s"(mode), "s"(thr), "s"(err_out), "s"(upd_out), "s"(flag_out), "s"(stats_out),
               "s"(correct_out), "s"(yhat_out));

  // the lane's 16 bytes of each super-block start at row + 64 sb
  const uint8_t *rowA = reinterpret_cast<const uint8_t *>(Lr.A + (size_t)min(m0 + lr, pn - 1) * Lr.words) + 16 * q;
  const uint8_t *rowP[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j)
    rowP[j] = reinterpret_cast<const uint8_t *>(Lr.P + (size_t)min(j * 16 + lr, pc - 1) * Lr.words) + 16 * q;
  const int rowlim = 8 * Lr.words - 16 * q;      // bytes of the row from the lane's first byte

  v4f acc[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
  int pa = 0;   // YHAT: P_a over the lane's words
  auto popc_low = [](const uint4 &w) {
    return __popc(w.x & kLowClasses) + __popc(w.y & kLowClasses) + __popc(w.z & kLowClasses) +
           __popc(w.w & kLowClasses);
  };
  const int nfull = K / 512, nsb = (K + 511) / 512;
  const int nf = nfull > kg ? (nfull - kg + KG - 1) / KG : 0;   // the wave's whole super-blocks: kg + KG i
  // super-blocks i .. i + N - 1 of the wave: every load first, then the
  // MFMAs, each waiting only for its own operands
  auto run = [&](auto n_tag, int i) {
    constexpr int N = decltype(n_tag)::value;
    uint4 wa[N], wb[N][CB];
#pragma unroll
    for (int u = 0; u < N; ++u) {
      const int o = 64 * (kg + KG * (i + u));
      wa[u] = load16<ALIGNED>(rowA, o);
#pragma unroll
      for (int j = 0; j < CB; ++j) wb[u][j] = load16<ALIGNED>(rowP[j], o);
    }
    // the label of the lane's pattern in the argmax below, loaded behind
    // the first operands so that its latency hides under the contraction
    if (!YHAT && i == 0 && kg < 4 && mu < pn) label = py[mu];
#pragma unroll
    for (int u = 0; u < N; ++u) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const uint4 ea = pm1_operand(wa[u], s);
#pragma unroll
        for (int j = 0; j < CB; ++j) acc[j] = mfma_fp4(ea, bit_operand(wb[u][j], s), acc[j], s);
      }
      if constexpr (YHAT) pa += popc_low(wa[u]);
    }
  };
  int i = 0;
  for (; i + CH <= nf; i += CH) run(std::integral_constant<int, CH>{}, i);
  for (; i < nf; ++i) run(std::integral_constant<int, 1>{}, i);
  if (!YHAT && nf == 0 && kg < 4 && mu < pn) label = py[mu];
  if (nsb > nfull && (nsb - 1) % KG == kg) {   // the super-block that holds K's end
    const int sb = nsb - 1;
    const uint4 a = load16_tail<ALIGNED>(rowA, 64 * sb, rowlim);
    uint4 b[CB];
#pragma unroll
    for (int j = 0; j < CB; ++j) b[j] = load16_tail<ALIGNED>(rowP[j], 64 * sb, rowlim);
    uint32_t valid[4];   // elements of word d before K
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int nv = K - (512 * sb + 128 * q + 32 * d);
      valid[d] = nv >= 32 ? 0xFFFFFFFFu : nv <= 0 ? 0u : ((1u << nv) - 1u);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint4 ea = pm1_operand(a, s);
#pragma unroll
      for (int j = 0; j < CB; ++j) acc[j] = mfma_fp4(ea, bit_operand_masked(b[j], valid, s), acc[j], s);
    }
    if constexpr (YHAT)
      pa += __popc(a.x & kLowClasses & valid[0]) + __popc(a.y & kLowClasses & valid[1]) +
            __popc(a.z & kLowClasses & valid[2]) + __popc(a.w & kLowClasses & valid[3]);
  }
  // lane holds classes 16 j + lr of patterns 4q + e
#pragma unroll
  for (int j = 0; j < CB; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[kg][4 * q + e][j * 16 + lr] = (int)acc[j][e];
  if constexpr (YHAT) {
    pa += __shfl_xor(pa, 16);
    pa += __shfl_xor(pa, 32);
    if (q == 0) spa[kg][lr] = pa;
  }
  __syncthreads();
  if constexpr (YHAT) {
    const int nlow = K - K / 4;
    for (int i = tid; i < 16 * pc; i += 64 * kWaves) {
      const int r = i / pc, cl = i - r * pc, m = m0 + r;
      if (m < pn) {
        int v = 0, pr = 0;
#pragma unroll
        for (int k = 0; k < KG; ++k) {
          v += red[k][r][cl];
          pr += spa[k][r];
        }
        yhat_out[(size_t)m * pc + cl] = v - 2 * pr + nlow;
      }
    }
    return;
  } else {
    // Sixteen lanes per pattern (a DPP row): lane li takes classes li, li +
    // 16, ... in order (the K groups' partials added), then the row merges
    // its lanes' top-two with four DPP exchanges (xor 1 and 2 within quads,
    // then the half-row and row mirrors), after which every lane of the row
    // holds the pattern's first argmax and its two largest values.  Waves
    // 0..3 take the 16 patterns.
    if (kg < 4 && mu < pn) {
      const int r = mu - m0, li = lane & 15;
      int v[CB];
#pragma unroll
      for (int j = 0; j < CB; ++j) {   // every LDS read first (entries past c are read, not used)
        v[j] = 0;
#pragma unroll
        for (int k = 0; k < KG; ++k) v[j] += red[k][r][li + 16 * j];
      }
      Top2 t{INT_MIN, INT_MAX, INT_MIN};
#pragma unroll
      for (int j = 0; j < CB; ++j)
        if (li + 16 * j < pc) {
          if (v[j] > t.v1) {
            t.v2 = t.v1;
            t.v1 = v[j];
            t.i1 = li + 16 * j;
          } else if (v[j] > t.v2) {
            t.v2 = v[j];
          }
        }
      t = merge(t, dpp_top2<0xB1>(t));    // quad_perm [1,0,3,2]
      t = merge(t, dpp_top2<0x4E>(t));    // quad_perm [2,3,0,1]
      t = merge(t, dpp_top2<0x141>(t));   // row_half_mirror
      t = merge(t, dpp_top2<0x140>(t));   // row_mirror
      if (li == 0) {
        if (mode == kClsEval) {
          if (t.i1 == label) atomicAdd(&cnt[2], 1);
          if (flag_out != nullptr)
            flag_out[mu] = (uint8_t)((t.i1 == label ? 1 : 0) | ((t.v1 - t.v2) >= thr ? 2 : 0));
        } else {
          const bool err = t.i1 != label;
          const bool upd = err || (t.v1 - t.v2) < thr;
          err_out[mu] = err ? 1 : 0;
          upd_out[mu] = upd ? 1 : 0;
          if (err) atomicAdd(&cnt[0], 1);
          if (upd) atomicAdd(&cnt[1], 1);
        }
      }
    }
    // one global atomic per work-group (same-address atomics from every
    // pattern would serialise in L2): err and |M| are adjacent 32-bit counts
    // of the layer's stats row, added at once as one 64-bit value
    __syncthreads();
    if (tid == 0) {
      if (mode == kClsEval) {
        if (cnt[2]) atomicAdd(correct_out, cnt[2]);
      } else {
        const unsigned long long v = (unsigned long long)(uint32_t)cnt[0] | ((unsigned long long)(uint32_t)cnt[1] << 32);
        if (v) atomicAdd(reinterpret_cast<unsigned long long *>(stats_out), v);
      }
    }
  }
}

// One wave per pattern: lane l scans classes 4l .. 4l + 3, then 256 + 4l
// .., in order (one 8-byte load of four int16 entries per 256 classes), and
// the wave merges its lanes' top-two (DPP within rows of 16 lanes, then
// across rows).  The error signal and the counts are those of the
// classifier kernel above.
constexpr int kArgWaves = 8;

__global__ __launch_bounds__(64 * kArgWaves) void cls_argmax_kernel(ClsBatch p) {
  __shared__ int cnt[3];   // block totals of err, upd, correct
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int bpl = (p.n + kArgWaves - 1) / kArgWaves;   // work-groups per layer
  const ClsLayer &Lr = p.L[blockIdx.x / bpl];
  const int mu = (blockIdx.x % bpl) * kArgWaves + wave;
  if (tid < 3) cnt[tid] = 0;
  __syncthreads();
  if (mu < p.n) {
    // p.ldy is a multiple of 4 and rows start 8-byte aligned: a load that
    // starts below c stays inside the row
    const int16_t *row = Lr.y16 + (size_t)mu * p.ldy;
    Top2 t{INT_MIN, INT_MAX, INT_MIN};
#pragma unroll 4
    for (int c0 = 4 * lane; c0 < p.c; c0 += 256) {
      const uint2 w = *reinterpret_cast<const uint2 *>(row + c0);
      const int v4[4] = {(int)(int16_t)(w.x & 0xFFFFu), (int)(int16_t)(w.x >> 16),
                         (int)(int16_t)(w.y & 0xFFFFu), (int)(int16_t)(w.y >> 16)};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = c0 + e < p.c ? v4[e] : INT_MIN;
        if (v > t.v1) {
          t.v2 = t.v1;
          t.v1 = v;
          t.i1 = c0 + e;
        } else if (v > t.v2) {
          t.v2 = v;
        }
      }
    }
    t = merge(t, dpp_top2<0xB1>(t));    // quad_perm [1,0,3,2]
    t = merge(t, dpp_top2<0x4E>(t));    // quad_perm [2,3,0,1]
    t = merge(t, dpp_top2<0x141>(t));   // row_half_mirror
    t = merge(t, dpp_top2<0x140>(t));   // row_mirror
#pragma unroll
    for (int d = 16; d < 64; d *= 2) {
      Top2 o;
      o.v1 = __shfl_xor(t.v1, d);
      o.i1 = __shfl_xor(t.i1, d);
      o.v2 = __shfl_xor(t.v2, d);
      t = merge(t, o);
    }
    if (lane == 0) {
      const int label = p.y[mu];
      if (p.mode == kClsEval) {
        if (t.i1 == label) atomicAdd(&cnt[2], 1);
        if (Lr.flag != nullptr)
          Lr.flag[mu] = (uint8_t)((t.i1 == label ? 1 : 0) | ((t.v1 - t.v2) >= Lr.thr ? 2 : 0));
      } else {
        const bool err = t.i1 != label;
        const bool upd = err || (t.v1 - t.v2) < Lr.thr;
        Lr.err[mu] = err ? 1 : 0;
        Lr.upd[mu] = upd ? 1 : 0;
        if (err) atomicAdd(&cnt[0], 1);
        if (upd) atomicAdd(&cnt[1], 1);
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    if (p.mode == kClsEval) {
      if (cnt[2]) atomicAdd(Lr.correct, cnt[2]);
    } else {
      const unsigned long long v = (unsigned long long)(uint32_t)cnt[0] | ((unsigned long long)(uint32_t)cnt[1] << 32);
      if (v) atomicAdd(reinterpret_cast<unsigned long long *>(Lr.stats), v);
    }
  }
}

template <int CB>
void launch_cls_cb(const ClsBatch &a, bool aligned, bool yhat, dim3 grid, hipStream_t s) {
  const dim3 block(64 * kWaves);
  if (aligned) {
    if (yhat)
      hipLaunchKernelGGL((cls_fp4_kernel<CB, true, true>), grid, block, 0, s, a.n, a.c, a.y, a);
    else
      hipLaunchKernelGGL((cls_fp4_kernel<CB, true, false>), grid, block, 0, s, a.n, a.c, a.y, a);
  } else {
    if (yhat)
      hipLaunchKernelGGL((cls_fp4_kernel<CB, false, true>), grid, block, 0, s, a.n, a.c, a.y, a);
    else
      hipLaunchKernelGGL((cls_fp4_kernel<CB, false, false>), grid, block, 0, s, a.n, a.c, a.y, a);
  }
}

}  // namespace

hipError_t launch_cls_fp4(const ClsBatch &a, hipStream_t s) {
  if (a.n <= 0 || a.nl <= 0) return hipSuccess;
  if (a.c < 1 || a.c > kClsMaxClasses || a.nl > kMaxClsLayers) return hipErrorInvalidValue;
  const bool yhat = a.mode == kClsYhatOnly;
  bool aligned = true;
  for (int l = 0; l < a.nl; ++l) {
    const ClsLayer &L = a.L[l];
    if (L.A == nullptr || L.P == nullptr || L.K < 1 || L.words < (L.K + 63) / 64) return hipErrorInvalidValue;
    if (yhat ? L.yhat == nullptr
             : (a.mode == kClsEval ? L.correct == nullptr : (L.err == nullptr || L.upd == nullptr || L.stats == nullptr)))
      return hipErrorInvalidValue;
    // rows start on 16-byte boundaries when the bases are 16-byte aligned
    // and the stride is an even number of words
    aligned = aligned && L.words % 2 == 0 && (reinterpret_cast<uintptr_t>(L.A) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(L.P) & 15) == 0;
  }
  if (!yhat && a.y == nullptr) return hipErrorInvalidValue;
  const dim3 grid(a.nl * ((a.n + 15) / 16));
  switch ((a.c + 15) / 16) {   // class blocks
    case 1: launch_cls_cb<1>(a, aligned, yhat, grid, s); break;
    case 2: launch_cls_cb<2>(a, aligned, yhat, grid, s); break;
    case 3: launch_cls_cb<3>(a, aligned, yhat, grid, s); break;
    case 4: launch_cls_cb<4>(a, aligned, yhat, grid, s); break;
    case 5: launch_cls_cb<5>(a, aligned, yhat, grid, s); break;
    case 6: launch_cls_cb<6>(a, aligned, yhat, grid, s); break;
    case 7: launch_cls_cb<7>(a, aligned, yhat, grid, s); break;
    default: launch_cls_cb<8>(a, aligned, yhat, grid, s); break;
  }
  return hipGetLastError();
}

hipError_t launch_cls_argmax(const ClsBatch &a, hipStream_t s) {
  if (a.n <= 0 || a.nl <= 0) return hipSuccess;
  if (a.c < 1 || a.ldy < a.c || a.ldy % 4 != 0 || a.nl > kMaxClsLayers ||
      (a.mode != kClsTrain && a.mode != kClsEval))
    return hipErrorInvalidValue;
  for (int l = 0; l < a.nl; ++l)
    if (a.L[l].y16 == nullptr || (reinterpret_cast<uintptr_t>(a.L[l].y16) & 7) != 0) return hipErrorInvalidValue;
  const dim3 grid(a.nl * ((a.n + kArgWaves - 1) / kArgWaves)), block(64 * kArgWaves);
  hipLaunchKernelGGL(cls_argmax_kernel, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace bmlp
