// Local classifiers and local error signals on the matrix cores, for every
// layer of a step in one launch (Algorithm 1: y_hat = a_l P_l^T, the 01-loss
// of Eq. 1 and the robustness test that builds M_l).  The layers are
// independent once every forward is done, so one launch covers them all.
//
// A work-group owns 16 patterns of one layer and all classes, taken CB
// blocks of 16 classes per pass (CB is a template parameter sized to the
// class count).  Its sixteen waves form KG groups along K times 16 / KG
// groups along the classes: a wave runs one
// v_mfma_scale_f32_16x16x128_f8f6f4 per K step for each of its PB class
// blocks, over K steps kg, kg + KG, ..., with the operands of kU steps
// loaded together so that one memory latency covers them.  Loads are
// unconditional with clamped indices: a clamped row only feeds y_hat
// entries of patterns past n or classes past c, which are never read.  The partial sums are exact
// integers: each K group stores its int32 partials in LDS and every thread
// then adds the KG partials of its own y_hat entries, in a fixed order.
//
// Then each wave takes one pattern: first argmax (lowest class on ties), the
// two largest values (tau = top1 - top2, 0 on a tie), err = (pred != y) and
// upd = err or tau < ceil(r K_l).  When the classes fit one pass y_hat is
// read from LDS; otherwise each pass goes through the y_hat buffer.
#include <limits.h>

#include "bmlp_internal.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 16;

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

template <int CB>
struct ClsShape {
  static constexpr int PB = CB < 4 ? CB : 4;     // class blocks per wave
  static constexpr int CG = CB / PB;             // wave groups along the classes
  static constexpr int KG = kWaves / CG;         // wave groups along K
  static constexpr int kU = KG >= 16 ? 2 : 4;    // K steps loaded together
};

template <int CB>
__global__ __launch_bounds__(64 * kWaves) void cls_fp4_kernel(ClsBatch p) {
  constexpr int PB = ClsShape<CB>::PB, KG = ClsShape<CB>::KG, kU = ClsShape<CB>::kU;
  __shared__ int red[KG][16][CB * 16];   // per K group; red[0] ends with y_hat
  __shared__ int cnt[3];                 // block totals of err, upd, correct

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kg = wave % KG, cg = wave / KG;
  const int bpl = (p.n + 15) / 16;               // work-groups per layer
  const ClsLayer &Lr = p.L[blockIdx.x / bpl];
  const int m0 = (blockIdx.x % bpl) * 16;
  const int lr = lane & 15, lk = (lane >> 4) * 16;
  const int nblk = (p.c + 15) / 16;
  const bool one_pass = nblk <= CB;
  const int am = m0 + lr;
  // 32-bit byte offsets from the layer's base pointers (scalar base +
  // vector offset addressing; a_l and P_l are far below 4 GiB)
  const uint32_t aoff = (uint32_t)min(am, p.n - 1) * (uint32_t)Lr.lda + (uint32_t)lk;
  const int ksteps = Lr.ksteps;
  if (tid < 3) cnt[tid] = 0;

  for (int cb0 = 0; cb0 < nblk; cb0 += CB) {
    const int nb = min(CB, nblk - cb0);
    v4f acc[PB];
    uint32_t boff[PB];
#pragma unroll
    for (int j = 0; j < PB; ++j) {
      acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
      const int cls = (cb0 + cg * PB + j) * 16 + lr;
      boff[j] = (uint32_t)min(cls, p.c - 1) * (uint32_t)Lr.ldp + (uint32_t)lk;
    }
    const bool any = cg * PB < nb;   // wave-uniform: the wave has a class block in range
    for (int ks0 = kg; any && ks0 < ksteps; ks0 += KG * kU) {
      uint4 a[kU], b[kU][PB];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int ks = min(ks0 + u * KG, ksteps - 1);
        a[u] = *reinterpret_cast<const uint4 *>(Lr.A + (aoff + (uint32_t)ks * 64u));
#pragma unroll
        for (int j = 0; j < PB; ++j) b[u][j] = *reinterpret_cast<const uint4 *>(Lr.P + (boff[j] + (uint32_t)ks * 64u));
      }
#pragma unroll
      for (int u = 0; u < kU; ++u)
        if (ks0 + u * KG < ksteps) {
#pragma unroll
          for (int j = 0; j < PB; ++j)
            if (cg * PB + j < nb) acc[j] = mfma_fp4(a[u], b[u][j], acc[j]);
        }
    }
    // lane holds classes (cb0 + cg*PB + j)*16 + (lane & 15) of patterns
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
    if (!(one_pass && p.mode != kClsYhatOnly)) {
      for (int i = tid; i < 16 * CB * 16; i += 64 * kWaves) {
        const int r = i / (CB * 16), cl = i % (CB * 16);
        const int m = m0 + r, cls = cb0 * 16 + cl;
        if (m < p.n && cls < p.c) Lr.yhat[(size_t)m * p.c + cls] = red[0][r][cl];
      }
      __syncthreads();   // y_hat of this pass is in memory (same work-group)
    }
  }
  if (p.mode == kClsYhatOnly) return;

  for (int r = wave; r < 16; r += kWaves) {
    const int mu = m0 + r;
    if (mu >= p.n) break;
    Top2 t{INT_MIN, INT_MAX, INT_MIN};
    const int32_t *row = Lr.yhat + (size_t)mu * p.c;
    for (int cl = lane; cl < p.c; cl += 64) {
      const int v = one_pass ? red[0][r][cl] : row[cl];
      if (v > t.v1) {
        t.v2 = t.v1;
        t.v1 = v;
        t.i1 = cl;
      } else if (v > t.v2) {
        t.v2 = v;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      Top2 o;
      o.v1 = __shfl_xor(t.v1, off, 64);
      o.i1 = __shfl_xor(t.i1, off, 64);
      o.v2 = __shfl_xor(t.v2, off, 64);
      t = merge(t, o);
    }
    const int label = p.y[mu];
    if (lane == 0) {
      if (p.mode == kClsEval) {
        if (t.i1 == label) atomicAdd(&cnt[2], 1);
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

}  // namespace

hipError_t launch_cls_fp4(const ClsBatch &a, hipStream_t s) {
  if (a.n <= 0 || a.nl <= 0) return hipSuccess;
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

}  // namespace bmlp
