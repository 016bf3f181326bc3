// Local classifier and local error signal on the matrix cores (Algorithm 1:
// y_hat = a_l P_l^T, the 01-loss of Eq. 1 and the robustness test that
// builds M_l).
//
// A work-group owns 16 patterns and all classes, taken CB blocks of 16
// classes per pass (CB is a template parameter sized to the class count).
// Its sixteen waves split K (wave w takes K steps w, w+16, ...); for each
// step a wave loads its operands, waits and runs one MFMA per class block,
// and the other fifteen waves on the CU hide that latency.  Loads are
// unconditional (indices clamped, data masked).  The partial sums are exact
// integers, so they are converted to int32 and added with integer LDS
// atomics (float LDS atomics are far slower), giving the same y_hat in any
// order.  After a barrier each wave takes one of the
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

constexpr int kWaves = 16;

template <int CB>
__global__ __launch_bounds__(64 * kWaves) void cls_fp4_kernel(ClsArgs p) {
  __shared__ int red[16][CB * 16];
  __shared__ int cnt[4];   // block totals of err, upd, selected, correct
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m0 = blockIdx.x * 16;
  const int lr = lane & 15, lk = (lane >> 4) * 16;
  const int nblk = (p.c + 15) / 16;
  const int am = m0 + lr;
  const uint32_t amask = am < p.n ? 0xFFFFFFFFu : 0u;
  const uint8_t *arow = p.A + (size_t)min(am, p.n - 1) * p.lda + lk;
  auto masked = [](const uint4 &v, uint32_t m) { return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m); };

  for (int cb0 = 0; cb0 < nblk; cb0 += CB) {
    const int nb = min(CB, nblk - cb0);
    for (int i = tid; i < 16 * CB * 16; i += 64 * kWaves) (&red[0][0])[i] = 0;
    v4f acc[CB];
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
    const uint8_t *brow[CB];
    uint32_t bmask[CB];
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int cls = (cb0 + j) * 16 + lr;
      bmask[j] = cls < p.c ? 0xFFFFFFFFu : 0u;
      brow[j] = p.P + (size_t)min(cls, p.c - 1) * p.ldp + lk;
    }
    for (int ks = wave; ks < p.ksteps; ks += kWaves) {
      const uint4 a = masked(*reinterpret_cast<const uint4 *>(arow + ks * 64), amask);
      uint4 b[CB];
#pragma unroll
      for (int j = 0; j < CB; ++j) b[j] = *reinterpret_cast<const uint4 *>(brow[j] + ks * 64);
#pragma unroll
      for (int j = 0; j < CB; ++j)
        if (j < nb) acc[j] = mfma_fp4(a, masked(b[j], bmask[j]), acc[j]);
    }
    __syncthreads();   // red is zeroed
    // lane holds classes (cb0 + j)*16 + (lane & 15) of patterns 4*(lane >> 4) + e
#pragma unroll
    for (int j = 0; j < CB; ++j)
      if (j < nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) atomicAdd(&red[4 * (lane >> 4) + e][j * 16 + lr], (int)acc[j][e]);
    __syncthreads();
    for (int i = tid; i < 16 * CB * 16; i += 64 * kWaves) {
      const int r = i / (CB * 16), cl = i % (CB * 16);
      const int m = m0 + r, cls = cb0 * 16 + cl;
      if (m < p.n && cls < p.c) p.yhat[(size_t)m * p.ldo + cls] = red[r][cl];
    }
    __syncthreads();
  }
  if (p.mode == kClsYhatOnly) return;
  if (tid < 4) cnt[tid] = 0;
  __syncthreads();   // y_hat of the 16 patterns is complete (global writes, same work-group)

  for (int r = wave; r < 16; r += kWaves) {
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
      if (lane == 0 && t.i1 == label) atomicAdd(&cnt[3], 1);
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
      if (err) atomicAdd(&cnt[0], 1);
      if (upd) atomicAdd(&cnt[1], 1);
      if (nsel) atomicAdd(&cnt[2], nsel);
    }
  }
  // one global atomic per counter and work-group: same-address atomics from
  // every pattern would serialise in L2
  __syncthreads();
  if (tid == 0) {
    if (p.mode == kClsEval) {
      if (cnt[3]) atomicAdd(p.correct, cnt[3]);
    } else {
      if (cnt[0]) atomicAdd(p.stats + 0, cnt[0]);
      if (cnt[1]) atomicAdd(p.stats + 1, cnt[1]);
      if (cnt[2]) atomicAdd(p.stats + 2, cnt[2]);
    }
  }
}

}  // namespace

hipError_t launch_cls_fp4(const ClsArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const int nblk = (a.c + 15) / 16;
  const dim3 grid((a.n + 15) / 16), block(64 * kWaves);
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
