// The input side of the step (Algorithm 1's binarisation of the inputs and Section 3.2,
// footnote 1), for integer features (int8):
//   * the median of every feature over a reference set (the lower middle
//     order statistic, so an element of the column and exact);
//   * median binarisation: bit = (x >= median);
//   * the fixed random ±1 expansion layer: bit = (sum_i x_i R[j][i] >= 0),
//     exact in int32, with R drawn from Philox stream 5 (counter layer word
//     2^32 - 1, t = 0): element e = j K_raw + i is bit (e & 127) of block
//     e >> 7.
#include "bmlp_internal.h"
#include "philox.h"

namespace bmlp {
namespace {

constexpr int kStreamExpand = 5;
constexpr int kFeat = 64;   // features per work-group of the median kernel

// One work-group per 64 features: a 256-bin histogram of each feature in
// LDS over all N rows (four rows per pass, 64 features each, one byte
// load per thread), then the first value whose running count reaches
// floor((N - 1) / 2) + 1.
__global__ __launch_bounds__(256) void feature_median_kernel(const int8_t *__restrict__ x, int n, int K,
                                                             int8_t *__restrict__ med) {
  __shared__ uint32_t hist[kFeat][256];
  const int f0 = blockIdx.x * kFeat;
  for (int i = threadIdx.x; i < kFeat * 256; i += 256) (&hist[0][0])[i] = 0u;
  __syncthreads();
  const int f = threadIdx.x & (kFeat - 1), r0 = threadIdx.x / kFeat;
  if (f0 + f < K) {
    for (int r = r0; r < n; r += 256 / kFeat) atomicAdd(&hist[f][x[(size_t)r * K + f0 + f] + 128], 1u);
  }
  __syncthreads();
  if (threadIdx.x < kFeat && f0 + threadIdx.x < K) {
    const uint32_t want = (uint32_t)((n - 1) / 2) + 1u;
    uint32_t run = 0u;
    int v = 0;
    for (; v < 256; ++v) {
      run += hist[threadIdx.x][v];
      if (run >= want) break;
    }
    med[f0 + threadIdx.x] = (int8_t)(v - 128);
  }
}

// one wave per 64-bit output word: lane i tests column 64 w + i
__global__ __launch_bounds__(256) void binarize_kernel(const int8_t *__restrict__ x, int n, int K, int words,
                                                       const int8_t *__restrict__ thr, uint64_t *__restrict__ bits) {
  const int row = blockIdx.y;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n || w >= words) return;   // whole wave leaves together
  const int col = w * 64 + lane;
  const bool pos = col < K && x[(size_t)row * K + col] >= thr[col];
  const uint64_t m = __ballot(pos);
  if (lane == 0) bits[(size_t)row * words + w] = m;
}

// bits e .. e + 31 of stream 5 (32 consecutive elements; they straddle at
// most two Philox blocks)
__device__ uint32_t expand_bits32(uint64_t e, uint32_t k0, uint32_t k1) {
  const uint32_t blk = (uint32_t)(e >> 7), off = (uint32_t)(e & 127);
  const U32x4 a = philox4x32_10(blk, 0xFFFFFFFFu, 0u, kStreamExpand, k0, k1);
  const uint32_t wi = off >> 5, sh = off & 31;
  const uint32_t lo = pick_word(a, wi);
  uint32_t hi;
  if (wi < 3) {
    hi = pick_word(a, wi + 1);
  } else {
    const U32x4 b = philox4x32_10(blk + 1u, 0xFFFFFFFFu, 0u, kStreamExpand, k0, k1);
    hi = b.x;
  }
  return sh ? (lo >> sh) | (hi << (32 - sh)) : lo;
}

constexpr int kXCols = 64;    // output columns (R rows) per work-group
constexpr int kXRows = 64;    // patterns per pass
constexpr int kXWords = 128;  // R words per column held in LDS (4096 inputs)

// Work-group: 64 output columns j0 .. j0 + 63 and a chunk of patterns.
// The columns' R rows are made once, as bits in LDS (in passes of 4096
// inputs); thread (pattern p, column group g) sums 16 columns with sdot4 on
// 4 int8 inputs and 4 ±1 bytes at a time.
__global__ __launch_bounds__(256) void expand_kernel(const int8_t *__restrict__ x, int n, int k_raw, int k0,
                                                     uint64_t seed, int rows_per_block, uint64_t *__restrict__ bits,
                                                     int words_out) {
  __shared__ uint32_t sR[kXCols][kXWords + 1];
  __shared__ int32_t sZ[kXRows][kXCols + 1];
  const int j0 = blockIdx.x * kXCols;
  const int p0 = blockIdx.y * rows_per_block;
  const int p1 = min(n, p0 + rows_per_block);
  const uint32_t key0 = (uint32_t)seed, key1 = (uint32_t)(seed >> 32);
  const int tid = threadIdx.x;
  const int pl = tid >> 2, cg = tid & 3;   // pattern in the pass, group of 16 columns
  for (int q0 = p0; q0 < p1; q0 += kXRows) {
    int32_t z[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) z[c] = 0;
    const int mu = q0 + pl;
    const int8_t *xr = x + (size_t)min(mu, n - 1) * k_raw;
    for (int i0 = 0; i0 < k_raw; i0 += 32 * kXWords) {
      const int nw = min(kXWords, (k_raw - i0 + 31) / 32);
      __syncthreads();   // the previous pass's R words are no longer read
      for (int t = tid; t < kXCols * nw; t += 256) {
        const int c = t / nw, w = t % nw;
        const int j = j0 + c, i = i0 + 32 * w;
        uint32_t r = 0u;
        if (j < k0) {
          r = expand_bits32((uint64_t)j * (uint64_t)k_raw + (uint64_t)i, key0, key1);
          const int valid = min(32, k_raw - i);   // past the row: no input, no weight
          if (valid < 32) r &= (1u << valid) - 1u;
        }
        sR[c][w] = r;
      }
      __syncthreads();
      for (int w = 0; w < nw; ++w) {
        const int i = i0 + 32 * w;
        // 32 inputs as 8 words of 4 int8 (zero past the row)
        int xs[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          uint32_t v = 0u;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int ii = i + 4 * q + b;
            if (ii < k_raw) v |= (uint32_t)(uint8_t)xr[ii] << (8 * b);
          }
          xs[q] = (int)v;
        }
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          const uint32_t r = sR[cg * 16 + c][w];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            // the 4 weights of inputs 4q .. 4q + 3 as bytes +1 / -1 (0xFF);
            // inputs past the row are 0, so their weight does not matter
            // bit b of the nibble to bit 0 of byte b (the four shifted
            // copies do not overlap), then 1 -> 0x01 and 0 -> 0xFF
            const uint32_t nib = (r >> (4 * q)) & 0xFu;
            const uint32_t spread = (nib * 0x00204081u) & 0x01010101u;
            const uint32_t wv = ~(spread * 0xFEu);
            z[c] = __builtin_amdgcn_sdot4(xs[q], (int)wv, z[c], false);
          }
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 16; ++c) sZ[pl][cg * 16 + c] = z[c];
    __syncthreads();
    // a_0 = sign(z), sign(0) = +1: one ballot per (pattern, 64 columns)
    const int wave = tid >> 6, lane = tid & 63;
    for (int r = wave; r < kXRows; r += 4) {
      const int m = q0 + r;
      const bool pos = j0 + lane < k0 && sZ[r][lane] >= 0;
      const uint64_t bal = __ballot(pos);
      if (lane == 0 && m < p1) bits[(size_t)m * words_out + (j0 >> 6)] = bal;
    }
  }
}

}  // namespace

hipError_t launch_feature_median(const int8_t *x, int n, int K, int8_t *med, hipStream_t s) {
  if (n <= 0 || K <= 0) return hipSuccess;
  hipLaunchKernelGGL(feature_median_kernel, dim3((K + kFeat - 1) / kFeat), dim3(256), 0, s, x, n, K, med);
  return hipGetLastError();
}

hipError_t launch_binarize(const int8_t *x, int n, int K, const int8_t *thr, uint64_t *bits, hipStream_t s) {
  if (n <= 0 || K <= 0) return hipSuccess;
  const int words = (K + 63) / 64;
  hipLaunchKernelGGL(binarize_kernel, dim3((words + 3) / 4, n), dim3(256), 0, s, x, n, K, words, thr, bits);
  return hipGetLastError();
}

hipError_t launch_expand(const int8_t *x, int n, int k_raw, int k0, uint64_t seed, uint64_t *bits, hipStream_t s) {
  if (n <= 0 || k0 <= 0) return hipSuccess;
  if (k_raw <= 0) return hipErrorInvalidValue;
  const int rows_per_block = 256;   // patterns per work-group (R made once per 256 patterns)
  const dim3 grid((k0 + kXCols - 1) / kXCols, (n + rows_per_block - 1) / rows_per_block);
  hipLaunchKernelGGL(expand_kernel, grid, dim3(256), 0, s, x, n, k_raw, k0, seed, rows_per_block, bits,
                     (k0 + 63) / 64);
  return hipGetLastError();
}

}  // namespace bmlp
