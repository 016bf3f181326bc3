// Local error signal and perceptron selection (Algorithm 1 01-loss and
// robustness test, Eq. 1; Algorithm 2 easiest-perceptron choice).
//
// One wave per pattern.  Given y_hat, the wave finds the first argmax and the
// two largest values (tau = top1 - top2, 0 on a tie), sets err = (pred != y)
// and upd = err or tau < ceil(r K_l).  For every pattern it then takes, in
// every group of gamma perceptrons (contiguous, or consecutive in the
// reshuffle variant's per-step order), the one with the largest
// negative stability delta_k = z_k rho^{y}_k, i.e. the smallest |z_k| among
// those whose sign disagrees with rho^{y}_k, lowest k on ties; delta = 0 is
// not eligible.  The update keeps only the patterns in M.
#include <limits.h>

#include "bmlp_internal.h"
#include "philox.h"

namespace bmlp {
namespace {

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
  // second largest value of the union of the two multisets
  r.v2 = max(min(a.v1, b.v1), max(a.v2, b.v2));
  return r;
}

__device__ __forceinline__ Top2 wave_top2(const int32_t *row, int c, int lane) {
  Top2 t{INT_MIN, INT_MAX, INT_MIN};
  for (int cl = lane; cl < c; cl += 64) {
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
  return t;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Grid: ceil(n / 4) blocks of 256 threads, one wave per pattern.
__global__ __launch_bounds__(256) void loss_select_kernel(LossSelectArgs p) {
  __shared__ int cnt[2];
  if (threadIdx.x < 2) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int mu = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (mu < p.n) {
  const bool select_only = p.yhat == nullptr;
  const int label = p.y[mu];
  const int yl = min(max(label, 0), p.c - 1);      // stay inside P on a bad label
  bool err = false, upd = false;
  if (!select_only) {
    const Top2 t = wave_top2(p.yhat + (size_t)mu * p.c, p.c, lane);
    err = t.i1 != label;
    upd = err || (t.v1 - t.v2) < p.thr;
  }
  int16_t *ks = p.kstar + mu;   // column mu of kstar [groups][ldk]
  {
    const int16_t *zr = p.z + (size_t)mu * p.ldz;
    const uint64_t *rho = p.P + (size_t)yl * p.words_out;
    for (int g = lane; g < p.groups; g += 64) {
      int best = -1, bestabs = INT_MAX, bestk = INT_MAX;
      const int k0 = g * p.gamma;
      for (int e = 0; e < p.gamma; ++e) {
        const int k = p.perm ? p.perm[k0 + e] : k0 + e;
        const int zz = min(max((int)zr[k], p.zlo), p.zhi);   // z as the selection sees it
        const bool rpos = (rho[k >> 6] >> (k & 63)) & 1ull;
        const bool wrong = rpos ? (zz < 0) : (zz > 0);
        const int a = zz < 0 ? -zz : zz;
        if (wrong && (a < bestabs || (a == bestabs && k < bestk))) {   // ties: lowest k
          bestabs = a;
          bestk = k;
          best = e;
        }
      }
      ks[(size_t)g * p.ldk] = (int16_t)best;
    }
  }
  if (lane == 0 && !select_only) {
    p.err[mu] = err ? 1 : 0;
    p.upd[mu] = upd ? 1 : 0;
    if (err) atomicAdd(&cnt[0], 1);
    if (upd) atomicAdd(&cnt[1], 1);
  }
  }
  __syncthreads();
  if (threadIdx.x == 0) {   // one global atomic per counter and work-group
    if (cnt[0]) atomicAdd(p.stats + 0, cnt[0]);
    if (cnt[1]) atomicAdd(p.stats + 1, cnt[1]);
  }
}

__global__ __launch_bounds__(256) void eval_count_kernel(const int32_t *yhat, int c, const int32_t *y,
                                                         int n, int32_t *correct, uint8_t *flag, int thr) {
  __shared__ int cnt;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  const int mu = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (mu < n) {
    const Top2 t = wave_top2(yhat + (size_t)mu * c, c, lane);
    const bool ok = t.i1 == y[mu];
    if (lane == 0 && ok) atomicAdd(&cnt, 1);
    if (lane == 0 && flag != nullptr) flag[mu] = (uint8_t)((ok ? 1 : 0) | ((t.v1 - t.v2) >= thr ? 2 : 0));
  }
  __syncthreads();
  if (threadIdx.x == 0 && cnt) atomicAdd(correct, cnt);
}

// Early exit (one thread per pattern): the first layer whose flag has bit 1
// (margin reached), else the last layer.  Counts gather per work-group in
// LDS, then one atomic per nonzero counter.
__global__ __launch_bounds__(256) void exit_count_kernel(const uint8_t *flags, int ldf, int L, int n,
                                                         int32_t *counts) {
  __shared__ int cnt[BMLP_MAX_LAYERS][2];
  for (int i = threadIdx.x; i < L * 2; i += 256) cnt[i >> 1][i & 1] = 0;
  __syncthreads();
  const int mu = blockIdx.x * 256 + threadIdx.x;
  if (mu < n) {
    for (int l = 0; l < L; ++l) {
      const uint8_t f = flags[(size_t)l * ldf + mu];
      if ((f & 2) || l == L - 1) {
        atomicAdd(&cnt[l][0], 1);
        if (f & 1) atomicAdd(&cnt[l][1], 1);
        break;
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < L * 2; i += 256) {
    const int v = cnt[i >> 1][i & 1];
    if (v) atomicAdd(counts + 3 * (i >> 1) + 1 + (i & 1), v);
  }
}

// one thread per 64-bit word of the batch; the word-0 thread of a row also
// copies its label
__global__ __launch_bounds__(256) void gather_batch_kernel(const uint64_t *x_all, const int32_t *y_all,
                                                           int n_all, int words, const int32_t *order, int n,
                                                           uint64_t *xb, int32_t *yb) {
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  if (t >= (long long)n * words) return;
  const int i = (int)(t / words), w = (int)(t % words);
  const int src = min(max(order[i], 0), n_all - 1);
  xb[t] = x_all[(size_t)src * words + w];
  if (w == 0) yb[i] = y_all[src];
}

// The reshuffle variant's group order: perceptron k's key is word (k & 3)
// of stream-6 block k >> 2, and its position is its rank among all K keys
// (ties by index).  One thread per perceptron counts the keys below its
// own, with the keys staged through LDS kPermChunk at a time; every block
// makes each chunk's keys itself (a few Philox blocks per thread).
constexpr int kPermThreads = 256;
constexpr int kPermChunk = 2048;

__device__ __forceinline__ uint32_t word_of(const U32x4 &w, int i) {
  return i == 0 ? w.x : i == 1 ? w.y : i == 2 ? w.z : w.w;
}

__global__ __launch_bounds__(kPermThreads) void group_perm_kernel(PermBatch p) {
  __shared__ uint4 keys[kPermChunk / 4];
  int li = 0;
#pragma unroll 1
  for (int i = 1; i < p.nl; ++i)
    if ((int)blockIdx.x >= p.L[i].block0) li = i;
  const PermLayer &q = p.L[li];
  const int k = ((int)blockIdx.x - q.block0) * kPermThreads + (int)threadIdx.x;
  const bool on = k < q.k;
  uint32_t mine = 0;
  if (on) mine = word_of(philox4x32_10((uint32_t)k >> 2, q.ctr1, p.step, kStreamGroups, p.key0, p.key1), k & 3);
  int rank = 0;
#pragma unroll 1
  for (int j0 = 0; j0 < q.k; j0 += kPermChunk) {
    const int nj = min(kPermChunk, q.k - j0);
    __syncthreads();   // the previous chunk has been read
    for (int b = threadIdx.x; b < (nj + 3) / 4; b += kPermThreads) {
      const U32x4 w = philox4x32_10((uint32_t)(j0 / 4 + b), q.ctr1, p.step, kStreamGroups, p.key0, p.key1);
      keys[b] = make_uint4(w.x, w.y, w.z, w.w);
    }
    __syncthreads();
    if (on) {
      // keys of indices below k count on ties, the others only when smaller
      int j = 0;
#pragma unroll 4
      for (; j + 4 <= nj; j += 4) {
        const uint4 v = keys[j / 4];
        const int jj = j0 + j;
        rank += (v.x < mine) | ((v.x == mine) & (jj < k));
        rank += (v.y < mine) | ((v.y == mine) & (jj + 1 < k));
        rank += (v.z < mine) | ((v.z == mine) & (jj + 2 < k));
        rank += (v.w < mine) | ((v.w == mine) & (jj + 3 < k));
      }
      const uint32_t *tail = reinterpret_cast<const uint32_t *>(keys);
      for (; j < nj; ++j) rank += (tail[j] < mine) | ((tail[j] == mine) & (j0 + j < k));
    }
  }
  if (on) q.perm[rank] = k;
}

}  // namespace

hipError_t launch_loss_select(const LossSelectArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(loss_select_kernel, dim3((a.n + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_group_perm(PermBatch &b, hipStream_t s) {
  if (b.nl < 1 || b.nl > 8) return hipErrorInvalidValue;
  int blocks = 0;
  for (int i = 0; i < b.nl; ++i) {
    if (b.L[i].k < 1 || b.L[i].perm == nullptr) return hipErrorInvalidValue;
    b.L[i].block0 = blocks;
    blocks += (b.L[i].k + kPermThreads - 1) / kPermThreads;
  }
  hipLaunchKernelGGL(group_perm_kernel, dim3(blocks), dim3(kPermThreads), 0, s, b);
  return hipGetLastError();
}

hipError_t launch_eval_count(const int32_t *yhat, int c, const int32_t *y, int n, int32_t *correct,
                             uint8_t *flag, int thr, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(eval_count_kernel, dim3((n + 3) / 4), dim3(256), 0, s, yhat, c, y, n, correct, flag, thr);
  return hipGetLastError();
}

hipError_t launch_exit_count(const uint8_t *flags, int ldf, int L, int n, int32_t *counts, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (L < 1 || L > BMLP_MAX_LAYERS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(exit_count_kernel, dim3((n + 255) / 256), dim3(256), 0, s, flags, ldf, L, n, counts);
  return hipGetLastError();
}

hipError_t launch_gather_batch(const uint64_t *x_all, const int32_t *y_all, int n_all, int words,
                               const int32_t *order, int n, uint64_t *xb, int32_t *yb, hipStream_t s) {
  const long long total = (long long)n * words;
  if (total <= 0) return hipSuccess;
  if (n_all < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_batch_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, x_all, y_all,
                     n_all, words, order, n, xb, yb);
  return hipGetLastError();
}

}  // namespace bmlp
