// Setup kernels: bit packing of ±1 inputs, state initialisation, fills.
#include "bmlp_internal.h"
#include "philox.h"

namespace bmlp {
namespace {

// One wave per 64-value chunk of a row: lane i tests value (w*64 + i) and the
// wave ballot is the packed word.  Grid: (ceil(words/4), n), 256 threads.
__global__ __launch_bounds__(256) void pack_kernel(const int8_t *__restrict__ x, int n, int K,
                                                   int words, uint64_t *__restrict__ bits) {
  const int row = blockIdx.y;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n || w >= words) return;     // whole wave leaves together
  const int col = w * 64 + lane;
  const bool pos = col < K && x[(size_t)row * K + col] > 0;
  const uint64_t m = __ballot(pos);
  if (lane == 0) bits[(size_t)row * words + w] = m;
}

// Bit (j & 127) of Philox block j >> 7 of the given layer/stream at step 0.
__device__ __forceinline__ bool stream_bit(uint64_t j, uint64_t seed, int layer, uint32_t stream) {
  const U32x4 v = philox4x32_10((uint32_t)(j >> 7), (uint32_t)(layer - 1), 0u, stream,
                                (uint32_t)seed, (uint32_t)(seed >> 32));
  const uint32_t b = (uint32_t)(j & 127);
  return (pick_word(v, b >> 5) >> (b & 31)) & 1u;
}

// Grid: (h_ps * 32 / 256, k_out).  Thread = one column of one H row (h_ps
// words per plane cover 32 * h_ps >= k_in columns, a multiple of 512, so
// waves stay whole).  H holds u = (h + B) / 2 in M = bits(B) planes: word
// p * h_ps + g of a row has bit p of u for the 32 columns of group g; a wave
// (two groups) ballots each plane and the W word.  Padding columns hold 0.
// from_h: H is kept and only W = sign(H), i.e. u >= (B + 1) / 2, is derived.
__global__ __launch_bounds__(256) void init_h_kernel(uint8_t *__restrict__ H, int ld_h, int h_ps, int B,
                                                     uint64_t *__restrict__ W, int words_in,
                                                     int k_in, int k_out, uint64_t seed, int layer,
                                                     int from_h) {
  const int k = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (k >= k_out || i >= h_ps * 32) return;
  const int lane = threadIdx.x & 63;
  const int M = h_planes(B);
  uint32_t *row = reinterpret_cast<uint32_t *>(H + (size_t)k * ld_h);
  const int g = i >> 5;
  bool pos;
  if (from_h) {
    int u = 0;
    for (int q = 0; q < M; ++q) u |= (int)((row[(size_t)q * h_ps + g] >> (i & 31)) & 1u) << q;
    pos = i < k_in && u >= (B + 1) / 2;
  } else {
    int u = 0;   // padding columns
    pos = false;
    if (i < k_in) {
      const uint64_t j = (uint64_t)k * (uint64_t)k_in + (uint64_t)i;
      pos = stream_bit(j, seed, layer, kStreamHInit);
      u = pos ? (B + 1) / 2 : (B - 1) / 2;   // h = +1 or -1
    }
    for (int q = 0; q < M; ++q) {
      const uint64_t b = __ballot((u >> q) & 1);
      if ((lane & 31) == 0) row[(size_t)q * h_ps + g] = (uint32_t)(b >> (lane & 32));
    }
  }
  const uint64_t m = __ballot(pos);
  const int w = i >> 6;
  if (lane == 0 && w < words_in) W[(size_t)k * words_in + w] = m;
}

// H planes [k_out][ld_h bytes] -> int8 h = 2u - B [k_out][k_in]; one thread per value
__global__ __launch_bounds__(256) void read_h_kernel(const uint8_t *__restrict__ H, int ld_h, int h_ps, int B,
                                                     int k_in, int k_out, int8_t *__restrict__ out) {
  const int k = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (k >= k_out || i >= k_in) return;
  const int M = h_planes(B);
  const uint32_t *row = reinterpret_cast<const uint32_t *>(H + (size_t)k * ld_h);
  int u = 0;
  for (int q = 0; q < M; ++q) u |= (int)((row[(size_t)q * h_ps + (i >> 5)] >> (i & 31)) & 1u) << q;
  out[(size_t)k * k_in + i] = (int8_t)(2 * u - B);
}

// Grid: (ceil(words_out / 4), c).  One wave per 64 classifier entries.
__global__ __launch_bounds__(256) void init_p_kernel(uint64_t *__restrict__ P, int words_out,
                                                     int k_out, int c, uint64_t seed, int layer) {
  const int cls = blockIdx.y;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (cls >= c || w >= words_out) return;
  const int k = w * 64 + lane;
  bool bit = false;
  if (k < k_out) {
    const uint64_t j = (uint64_t)cls * (uint64_t)k_out + (uint64_t)k;
    bit = stream_bit(j, seed, layer, kStreamPInit);
  }
  const uint64_t m = __ballot(bit);
  if (lane == 0) P[(size_t)cls * words_out + w] = m;
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t *p, int count, int32_t v) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < count) p[i] = v;
}

__global__ __launch_bounds__(256) void fill_rows_kernel(int32_t *p, int rows, int cols, int ld,
                                                        int32_t v) {
  const int r = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (r < rows && c < cols) p[(size_t)r * ld + c] = v;
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

hipError_t launch_pack(const int8_t *x, int n, int K, uint64_t *bits, hipStream_t s) {
  const int words = cdiv(K, 64);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3(cdiv(words, 4), n), dim3(256), 0, s, x, n, K, words, bits);
  return hipGetLastError();
}

hipError_t launch_init_h(uint8_t *H, int ld_h, int h_ps, int bound, uint64_t *W, int words_in, int k_in,
                         int k_out, uint64_t seed, int layer, bool from_h, hipStream_t s) {
  hipLaunchKernelGGL(init_h_kernel, dim3(h_ps * 32 / 256, k_out), dim3(256), 0, s, H, ld_h, h_ps, bound, W,
                     words_in, k_in, k_out, seed, layer, from_h ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_read_h(const uint8_t *H, int ld_h, int h_ps, int bound, int k_in, int k_out,
                         int8_t *out, hipStream_t s) {
  if (k_in <= 0 || k_out <= 0) return hipSuccess;
  hipLaunchKernelGGL(read_h_kernel, dim3(cdiv(k_in, 256), k_out), dim3(256), 0, s, H, ld_h, h_ps, bound, k_in,
                     k_out, out);
  return hipGetLastError();
}

hipError_t launch_init_p(uint64_t *P, int words_out, int k_out, int c, uint64_t seed, int layer,
                         hipStream_t s) {
  hipLaunchKernelGGL(init_p_kernel, dim3(cdiv(words_out, 4), c), dim3(256), 0, s, P, words_out,
                     k_out, c, seed, layer);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t *p, int count, int32_t value, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(cdiv(count, 256)), dim3(256), 0, s, p, count, value);
  return hipGetLastError();
}

hipError_t launch_fill_rows_i32(int32_t *p, int rows, int cols, int ld, int32_t value,
                                hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_rows_kernel, dim3(cdiv(cols, 256), rows), dim3(256), 0, s, p, rows, cols,
                     ld, value);
  return hipGetLastError();
}

}  // namespace bmlp
