// Local classifiers and local error signals on the matrix cores, for every
// layer of a step in one launch (Algorithm 1: y_hat = a_l P_l^T, the 01-loss
// of Eq. 1 and the robustness test that builds M_l).  The layers are
// independent once every forward is done, so one launch covers them all.
//
// A work-group owns 16 patterns of one layer and all its classes, up to
// kClsMaxClasses of them: CB blocks of 16 classes (CB is a template
// parameter sized to the class count).  a_l and P_l are read as bit rows:
// chunks of 4096 columns of the 16 pattern rows and the class rows are
// staged in LDS with coalesced loads (a load that touched 16 rows at once
// cost 16 cache-line requests, which bound the kernel), rows padded so that
// operand reads hit 64 banks.  A lane takes one 32-bit word (32 elements of
// a 128-element K step) of its row and expands it in registers to an fp4
// operand; the expansion permutes K inside the word, identically for a_l
// and P_l, which leaves every dot product unchanged.  Elements past K_l
// become fp4 zeros in the P operand.  Rows past n or c repeat the last row:
// they only feed y_hat entries that are never read.
//
// The waves form KG groups along K times kWaves / KG groups along the
// classes: a wave runs one v_mfma_scale_f32_16x16x128_f8f6f4 per K step for
// each of its PB class blocks, over the chunk's K steps kg, kg + KG, ....
// The partial sums are exact integers: each K group stores its int32
// partials in LDS (over the staged chunk) and every thread then adds the KG
// partials of its own y_hat entries, in a fixed order.
//
// Then sixteen lanes take each pattern: first argmax (lowest class on
// ties), the two largest values (tau = top1 - top2, 0 on a tie), err =
// (pred != y) and upd = err or tau < ceil(r K_l).
//
// With more classes, staging every class row for each 16 patterns would
// read P_l n / 16 times over; y_hat then comes from the forward kernel (a
// tiled contraction with P_l in place of W_l, which reads each operand tile
// once per output tile), and cls_argmax_kernel below takes the same error
// signal from the stored y_hat, one wave per pattern.
#include <limits.h>

#include "bmlp_internal.h"
#include "fp4.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;

__device__ __forceinline__ v4f mfma_fp4(const uint4 &a, const uint4 &b, v4f c) {
  const v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
  const v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 4, 4, 0, 127, 0, 127);
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
  static constexpr int PB = CB < 4 ? CB : 4;     // class blocks per wave
  static constexpr int CG = CB / PB;             // wave groups along the classes
  static constexpr int KG = kWaves / CG;         // wave groups along K
};

// K is staged through LDS in chunks of kChunk 32-bit words (4096 elements)
// per row; rows are padded to kStride words (kStride = 4 mod 64), so the
// lanes of an operand read (16 rows x 4 consecutive words) hit 64 banks.
constexpr int kChunk = 128, kStride = kChunk + 4;

template <int CB>
__global__ __launch_bounds__(64 * kWaves) void cls_fp4_kernel(ClsBatch p) {
  constexpr int PB = ClsShape<CB>::PB, KG = ClsShape<CB>::KG;
  constexpr int kRows = 16 + CB * 16;                      // staged rows: 16 patterns, CB*16 classes
  constexpr int kStage = kRows * kStride;                  // words
  constexpr int kRed = KG * 16 * CB * 16;                  // words of the partials
  __shared__ __align__(16) uint32_t lds[kStage > kRed ? kStage : kRed];
  uint32_t *const sA = lds, *const sP = lds + 16 * kStride;
  int (*red)[16][CB * 16] = reinterpret_cast<int (*)[16][CB * 16]>(lds);   // per K group; red[0] ends with y_hat
  __shared__ int cnt[3];                 // block totals of err, upd, correct

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int kg = wave % KG, cg = wave / KG;
  const int bpl = (p.n + 15) / 16;               // work-groups per layer
  const ClsLayer &Lr = p.L[blockIdx.x / bpl];
  const int m0 = (blockIdx.x % bpl) * 16;
  const int lr = lane & 15, q = lane >> 4;   // row / class, and which 32 of a K step's 128
  const int nb = (p.c + 15) / 16;                 // class blocks (<= CB)
  const uint32_t *A32 = reinterpret_cast<const uint32_t *>(Lr.A);
  const uint32_t *P32 = reinterpret_cast<const uint32_t *>(Lr.P);
  const int w32 = 2 * Lr.words;                  // 32-bit words per row
  if (tid < 3) cnt[tid] = 0;

  v4f acc[PB];
#pragma unroll
  for (int j = 0; j < PB; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
  for (int kw0 = 0; kw0 < w32; kw0 += kChunk) {
    // stage words kw0 .. kw0 + kChunk of the 16 pattern rows and the class
    // rows, 16 bytes per thread, coalesced along rows; rows past n or c
    // repeat the last row, words past the row are 0
    __syncthreads();   // the previous chunk is no longer read
    constexpr int kLoads = kRows * (kChunk / 4);                      // 16-byte pieces
    constexpr int kPer = (kLoads + 64 * kWaves - 1) / (64 * kWaves);    // per thread
    uint4 v[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {   // all loads in flight before any store
      const int t = min(tid + i * 64 * kWaves, kLoads - 1);
      const int row = t / (kChunk / 4), w = kw0 + (t % (kChunk / 4)) * 4;
      const uint32_t *src = row < 16 ? A32 + (size_t)min(m0 + row, p.n - 1) * w32
                                     : P32 + (size_t)min(row - 16, p.c - 1) * w32;
      // rows are whole u64 words (8-byte aligned), and w32 is even
      uint2 lo = make_uint2(0u, 0u), hi = make_uint2(0u, 0u);
      if (w < w32) lo = *reinterpret_cast<const uint2 *>(src + w);
      if (w + 2 < w32) hi = *reinterpret_cast<const uint2 *>(src + w + 2);
      v[i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int t = tid + i * 64 * kWaves;
      if (t < kLoads) *reinterpret_cast<uint4 *>(lds + (t / (kChunk / 4)) * kStride + (t % (kChunk / 4)) * 4) = v[i];
    }
    __syncthreads();
    const int nsteps = min(kChunk, w32 - kw0 + 3) / 4;   // K steps of 4 words in this chunk
    if (cg * PB < nb && nsteps == kChunk / 4) {
      // a whole chunk: every operand word of the wave's K steps is read
      // from LDS first, so the reads overlap instead of queueing behind
      // each step's MFMAs
      constexpr int kSteps = kChunk / 4 / KG;
      uint32_t wa[kSteps], wb[kSteps][PB];
#pragma unroll
      for (int s = 0; s < kSteps; ++s) {
        const int wl = 4 * (kg + s * KG) + q;
        wa[s] = sA[lr * kStride + wl];
#pragma unroll
        for (int j = 0; j < PB; ++j) wb[s][j] = sP[((cg * PB + j) * 16 + lr) * kStride + wl];
      }
#pragma unroll
      for (int s = 0; s < kSteps; ++s) {
        const int wl = 4 * (kg + s * KG) + q;
        const int nv = min(max(Lr.K - 32 * (kw0 + wl), 0), 32);
        const uint32_t valid = nv == 32 ? 0xFFFFFFFFu : ((1u << nv) - 1u);
        const uint4 av = fp4x32_permuted(wa[s]);
#pragma unroll
        for (int j = 0; j < PB; ++j)
          if (cg * PB + j < nb) {
            const uint4 bv = valid == 0xFFFFFFFFu ? fp4x32_permuted(wb[s][j]) : fp4x32_permuted_masked(wb[s][j], valid);
            acc[j] = mfma_fp4(av, bv, acc[j]);
          }
      }
    } else if (cg * PB < nb) {   // the wave has a class block in range
      for (int ks = kg; ks < nsteps; ks += KG) {
        const int wl = 4 * ks + q;   // the lane's word of the step, in the chunk
        // elements 32 (kw0 + wl) .. +31; those past K are padding (0 in fp4)
        const int nv = min(max(Lr.K - 32 * (kw0 + wl), 0), 32);
        const uint32_t valid = nv == 32 ? 0xFFFFFFFFu : ((1u << nv) - 1u);
        const uint4 av = fp4x32_permuted(sA[lr * kStride + wl]);
#pragma unroll
        for (int j = 0; j < PB; ++j)
          if (cg * PB + j < nb) {
            const uint32_t bw = sP[((cg * PB + j) * 16 + lr) * kStride + wl];
            const uint4 bv = valid == 0xFFFFFFFFu ? fp4x32_permuted(bw) : fp4x32_permuted_masked(bw, valid);
            acc[j] = mfma_fp4(av, bv, acc[j]);
          }
      }
    }
  }
  __syncthreads();   // the staged chunk is no longer read: red reuses it
  // lane holds classes (cg*PB + j)*16 + (lane & 15) of patterns
  // 4*(lane >> 4) + e; blocks past nb are never read
#pragma unroll
  for (int j = 0; j < PB; ++j)
    if (cg * PB + j < nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[kg][4 * (lane >> 4) + e][(cg * PB + j) * 16 + lr] = (int)acc[j][e];
  __syncthreads();
  for (int i = tid; i < 16 * CB * 16; i += 64 * kWaves) {
    int sum = 0;
#pragma unroll
    for (int k = 0; k < KG; ++k) sum += (&red[k][0][0])[i];
    (&red[0][0][0])[i] = sum;
  }
  __syncthreads();
  if (p.mode == kClsYhatOnly) {
    for (int i = tid; i < 16 * CB * 16; i += 64 * kWaves) {
      const int r = i / (CB * 16), cl = i % (CB * 16);
      const int m = m0 + r;
      if (m < p.n && cl < p.c) Lr.yhat[(size_t)m * p.c + cl] = red[0][r][cl];
    }
    return;
  }
  // Sixteen lanes per pattern (a DPP row): lane li scans classes li, li + 16,
  // ... in order, then the row merges its lanes' top-two with four DPP
  // exchanges (xor 1 and 2 within quads, then the half-row and row mirrors),
  // after which every lane of the row holds the pattern's first argmax and
  // its two largest values.  Waves 0..3 take the 16 patterns.
  if (wave < 4) {
    const int r = 4 * wave + (lane >> 4), li = lane & 15;
    const int mu = m0 + r;
    if (mu < p.n) {
      Top2 t{INT_MIN, INT_MAX, INT_MIN};
      for (int cl = li; cl < p.c; cl += 16) {
        const int v = red[0][r][cl];
        if (v > t.v1) {
          t.v2 = t.v1;
          t.v1 = v;
          t.i1 = cl;
        } else if (v > t.v2) {
          t.v2 = v;
        }
      }
      t = merge(t, dpp_top2<0xB1>(t));    // quad_perm [1,0,3,2]
      t = merge(t, dpp_top2<0x4E>(t));    // quad_perm [2,3,0,1]
      t = merge(t, dpp_top2<0x141>(t));   // row_half_mirror
      t = merge(t, dpp_top2<0x140>(t));   // row_mirror
      if (li == 0) {
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
  }
  // one global atomic per work-group (same-address atomics from every
  // pattern would serialise in L2): err and |M| are adjacent 32-bit counts of
  // the layer's stats row, added at once as one 64-bit value
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

}  // namespace

hipError_t launch_cls_fp4(const ClsBatch &a, hipStream_t s) {
  if (a.n <= 0 || a.nl <= 0) return hipSuccess;
  if (a.c < 1 || a.c > kClsMaxClasses || a.nl > kMaxClsLayers) return hipErrorInvalidValue;
  const int nblk = (a.c + 15) / 16;
  const dim3 grid(a.nl * ((a.n + 15) / 16)), block(64 * kWaves);
  if (nblk <= 1)
    hipLaunchKernelGGL(cls_fp4_kernel<1>, grid, block, 0, s, a);
  else if (nblk <= 2)
    hipLaunchKernelGGL(cls_fp4_kernel<2>, grid, block, 0, s, a);
  else if (nblk <= 4)
    hipLaunchKernelGGL(cls_fp4_kernel<4>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(cls_fp4_kernel<8>, grid, block, 0, s, a);
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
