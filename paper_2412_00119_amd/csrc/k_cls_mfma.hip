// Local classifier and local error signal on the matrix cores (Algorithm 1:
// y_hat = a_l P_l^T, the 01-loss of Eq. 1 and the robustness test that
// builds M_l).
//
// A work-group owns 16 patterns and all classes: each wave takes every
// fourth block of 16 classes (at most 1024 classes per pass), walks K in
// steps of 128 fp4 elements with v_mfma_scale_f32_16x16x128_f8f6f4 and
// writes y_hat as int32.  After a barrier each wave takes four of the
// patterns: first argmax (lowest class on ties), the two largest values
// (tau = top1 - top2, 0 on a tie), err = (pred != y), upd = err or
// tau < ceil(r K_l).  Patterns outside M_l get no selected perceptron
// (kstar = -1 in every group); for patterns in M_l the selected ones are
// counted.
#include <limits.h>

#include "bmlp_internal.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int CPW = 16;   // class blocks per wave per pass -> 4 * 16 * 16 = 1024 classes

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
  r.v2 = max(min(a.v1, b.v1), max(a.v2, b.v2));
  return r;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__global__ __launch_bounds__(256) void cls_fp4_kernel(ClsArgs p) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m0 = blockIdx.x * 16;
  const int lr = lane & 15, lk = (lane >> 4) * 16;
  const int nblk = (p.c + 15) / 16;
  const int am = m0 + lr;
  const uint8_t *arow = am < p.n ? p.A + (size_t)am * p.lda : nullptr;

  for (int cb0 = 0; cb0 < nblk; cb0 += 4 * CPW) {
    v4f acc[CPW];
#pragma unroll
    for (int j = 0; j < CPW; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < p.ksteps; ++ks) {
      const uint4 a = arow ? *reinterpret_cast<const uint4 *>(arow + ks * 64 + lk) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        const int cb = cb0 + wave + 4 * j;
        if (cb < nblk) {   // uniform per wave
          const int cls = cb * 16 + lr;
          const uint4 b = cls < p.c ? *reinterpret_cast<const uint4 *>(p.P + (size_t)cls * p.ldp + ks * 64 + lk)
                                    : make_uint4(0, 0, 0, 0);
          acc[j] = mfma_fp4(a, b, acc[j]);
        }
      }
    }
    // y_hat: lane holds class cb*16 + (lane & 15), patterns m0 + 4*(lane >> 4) + e
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int cb = cb0 + wave + 4 * j;
      if (cb < nblk) {
        const int cls = cb * 16 + lr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + 4 * (lane >> 4) + e;
          if (m < p.n && cls < p.c) p.yhat[(size_t)m * p.ldo + cls] = (int32_t)acc[j][e];
        }
      }
    }
  }
  if (p.mode == kClsYhatOnly) return;
  __syncthreads();   // y_hat of the 16 patterns is complete (global writes, same work-group)

  for (int r = wave; r < 16; r += 4) {
    const int mu = m0 + r;
    if (mu >= p.n) break;
    Top2 t{INT_MIN, INT_MAX, INT_MIN};
    const int32_t *row = p.yhat + (size_t)mu * p.ldo;
    for (int cl = lane; cl < p.c; cl += 64) {
      const int v = row[cl];
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
    if (p.mode == kClsEval) {
      if (lane == 0 && t.i1 == label) atomicAdd(p.correct, 1);
      continue;
    }
    const bool err = t.i1 != label;
    const bool upd = err || (t.v1 - t.v2) < p.thr;
    int nsel = 0;
    if (p.kstar != nullptr) {
      int16_t *ks = p.kstar + mu;
      for (int g = lane; g < p.groups; g += 64) {
        if (upd)
          nsel += ks[(size_t)g * p.ldk] >= 0;
        else
          ks[(size_t)g * p.ldk] = (int16_t)-1;
      }
      nsel = wave_sum(nsel);
    }
    if (lane == 0) {
      p.err[mu] = err ? 1 : 0;
      p.upd[mu] = upd ? 1 : 0;
      if (err) atomicAdd(p.stats + 0, 1);
      if (upd) atomicAdd(p.stats + 1, 1);
      if (nsel) atomicAdd(p.stats + 2, nsel);
    }
  }
}

}  // namespace

hipError_t launch_cls_fp4(const ClsArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cls_fp4_kernel, dim3((a.n + 15) / 16), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bmlp
