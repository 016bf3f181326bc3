// Perceptron-level update of one layer (Algorithm 3, Section 3.4).
//
// For every perceptron k of group g, the Clipped-Perceptron increments of the
// batch are summed first:
//   dH[k][i] = 2 * sum over selected patterns mu of rho^{y^mu}_k a^mu_i,
// then h <- clip(h + dH, -B, B); then every hidden weight whose 32-bit
// Philox draw is below T_l moves one step away from zero, h <- clip(h +
// 2 sign(h), -B, B); finally W = sign(H) is re-packed into bits.  The layer
// is left untouched when no pattern is in M_l.
//
// Work decomposition: a work-group owns one group g and a chunk of 2048
// columns.  It first buckets the patterns that selected each perceptron of
// the group (a counting sort in LDS), then each wave walks whole rows: a
// lane owns 32 consecutive columns (one 32-bit word of a_{l-1}).  The sum of
// ±1 contributions is counted as  cnt_i = #(bit_i XOR [rho = -1]) over the
// row's selectors, so sum = 2 cnt_i - S and dH = 4 cnt_i - 2 S.  No two
// work-groups touch the same bytes of H, so the result does not depend on
// scheduling.
#include "bmlp_internal.h"
#include "philox.h"

namespace bmlp {
namespace {

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// spread the 4 bits of n (n < 16) into the low bit of the 4 bytes of a word
__device__ __forceinline__ uint32_t spread4(uint32_t n) { return (n * 0x00204081u) & 0x01010101u; }

__global__ __launch_bounds__(256) void update_kernel(UpdateArgs p) {
  extern __shared__ int smem[];
  __shared__ int part[256];
  if (p.stats[1] == 0) return;   // M_l empty: Algorithm 2 is not run for this layer

  const int tid = threadIdx.x;
  const int g = blockIdx.y;
  const int gamma = p.gamma;
  int *bucket = smem;                                            // [gamma]
  uint16_t *list = reinterpret_cast<uint16_t *>(smem + gamma);   // [n]

  // ---- bucket the selections of this group by perceptron -------------------
  for (int r = tid; r < gamma; r += 256) bucket[r] = 0;
  __syncthreads();
  for (int mu = tid; mu < p.n; mu += 256) {
    const int ks = p.kstar[(size_t)mu * p.groups + g];
    if (ks >= 0) atomicAdd(&bucket[ks], 1);
  }
  __syncthreads();
  {
    const int ch = (gamma + 255) / 256;
    const int b0 = min(gamma, tid * ch), b1 = min(gamma, b0 + ch);
    int s = 0;
    for (int r = b0; r < b1; ++r) s += bucket[r];
    part[tid] = s;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
      const int v = tid >= o ? part[tid - o] : 0;
      __syncthreads();
      part[tid] += v;
      __syncthreads();
    }
    int run = part[tid] - s;
    for (int r = b0; r < b1; ++r) {
      const int c = bucket[r];
      bucket[r] = run;
      run += c;
    }
  }
  __syncthreads();
  for (int mu = tid; mu < p.n; mu += 256) {
    const int ks = p.kstar[(size_t)mu * p.groups + g];
    if (ks >= 0) {
      const int k = g * gamma + ks;
      const int yl = min(max(p.y[mu], 0), p.c - 1);   // stay inside P on a bad label
      const bool rpos = (p.P[(size_t)yl * p.words_out + (k >> 6)] >> (k & 63)) & 1ull;
      const int pos = atomicAdd(&bucket[ks], 1);
      list[pos] = (uint16_t)(mu | (rpos ? 0 : 0x8000));
    }
  }
  __syncthreads();
  // now bucket[r] is the end of row r's selectors; row r starts at bucket[r-1]

  const int wave = tid >> 6, lane = tid & 63;
  const int nw32 = 2 * p.words_in;
  const int cw = blockIdx.x * 64 + lane;       // this lane's 32-bit column word
  const bool on = cw < nw32;
  const int nvalid = min(max(p.k_in - cw * 32, 0), 32);
  const uint32_t validmask = nvalid == 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
  const uint32_t *a32 = reinterpret_cast<const uint32_t *>(p.a_prev);
  uint32_t *W32 = reinterpret_cast<uint32_t *>(p.W);
  const uint32_t key0 = (uint32_t)p.seed, key1 = (uint32_t)(p.seed >> 32);
  const uint32_t ctr1 = (uint32_t)(p.layer - 1);
  int nreinf = 0;

  for (int r = wave; r < gamma; r += 4) {
    const int k = g * gamma + r;
    const int beg = r ? bucket[r - 1] : 0;
    const int S = bucket[r] - beg;

    // ---- count +1 contributions per column, 255 selectors per byte batch ----
    int cnt[32];
#pragma unroll
    for (int e = 0; e < 32; ++e) cnt[e] = 0;
    for (int s0 = 0; s0 < S; s0 += 255) {
      const int s1 = min(S, s0 + 255);
      uint32_t C[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) C[q] = 0u;
      for (int s = s0; s < s1; ++s) {
        const uint32_t ent = list[beg + s];
        const uint32_t mu = ent & 0x7FFFu;
        const uint32_t flip = (ent & 0x8000u) ? 0xFFFFFFFFu : 0u;
        const uint32_t x = (on ? a32[(size_t)mu * nw32 + cw] : 0u) ^ flip;
#pragma unroll
        for (int q = 0; q < 8; ++q) C[q] += spread4((x >> (4 * q)) & 0xFu);
      }
#pragma unroll
      for (int e = 0; e < 32; ++e) cnt[e] += (C[e >> 2] >> (8 * (e & 3))) & 0xFFu;
    }

    if (!on) continue;   // inactive lanes only took part in the uniform loop above

    // ---- reinforcement draws of the 32 weights (j0 .. j0+31) -------------------
    const uint32_t j0 = (uint32_t)k * (uint32_t)p.k_in + (uint32_t)(cw * 32);
    const uint32_t b0 = j0 >> 4, sh = j0 & 15u;
    const U32x4 v0 = philox4x32_10(b0, ctr1, p.step, kStreamCoarse, key0, key1);
    const U32x4 v1 = philox4x32_10(b0 + 1, ctr1, p.step, kStreamCoarse, key0, key1);
    uint32_t u[8];
    if (sh == 0) {
      u[0] = v0.x; u[1] = v0.y; u[2] = v0.z; u[3] = v0.w;
      u[4] = v1.x; u[5] = v1.y; u[6] = v1.z; u[7] = v1.w;
    } else {
      const U32x4 v2 = philox4x32_10(b0 + 2, ctr1, p.step, kStreamCoarse, key0, key1);
      const uint32_t src[12] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w,
                                v2.x, v2.y, v2.z, v2.w};
      const uint32_t ws = sh >> 2, bs = sh & 3u;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const uint32_t lo = ws == 0 ? src[q] : ws == 1 ? src[q + 1] : ws == 2 ? src[q + 2] : src[q + 3];
        const uint32_t hi = ws == 0 ? src[q + 1] : ws == 1 ? src[q + 2] : ws == 2 ? src[q + 3] : src[q + 4];
        u[q] = bs == 0 ? lo : (uint32_t)((((uint64_t)hi << 32) | lo) >> (8 * bs));
      }
    }
    uint32_t fire = 0u, need = 0u;
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const uint32_t u8 = (u[e >> 2] >> (8 * (e & 3))) & 0xFFu;
      fire |= (u8 < p.t_hi ? 1u : 0u) << e;
      need |= (u8 == p.t_hi ? 1u : 0u) << e;
    }
    fire &= validmask;
    need &= validmask;
    while (need) {
      const int e = __ffs(need) - 1;
      need &= need - 1u;
      const uint32_t j = j0 + (uint32_t)e;
      const U32x4 f = philox4x32_10(j >> 2, ctr1, p.step, kStreamFine, key0, key1);
      if ((pick_word(f, j & 3u) & 0xFFFFFFu) < p.t_lo) fire |= 1u << e;
    }
    nreinf += __popc(fire);

    // ---- apply to the 32 hidden weights ----------------------------------------
    int8_t *hrow = p.H + (size_t)k * p.ld_h + cw * 32;
    uint4 hv[2];
    hv[0] = reinterpret_cast<const uint4 *>(hrow)[0];
    hv[1] = reinterpret_cast<const uint4 *>(hrow)[1];
    uint32_t hw[8] = {hv[0].x, hv[0].y, hv[0].z, hv[0].w, hv[1].x, hv[1].y, hv[1].z, hv[1].w};
    uint32_t wbits = 0u;
    const int B = p.bound;
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      if (!((validmask >> e) & 1u)) continue;
      int h = (int)(int8_t)((hw[e >> 2] >> (8 * (e & 3))) & 0xFFu);
      h += 4 * cnt[e] - 2 * S;
      h = min(max(h, -B), B);
      if ((fire >> e) & 1u) {
        h += h > 0 ? 2 : -2;
        h = min(max(h, -B), B);
      }
      const uint32_t shift = 8 * (e & 3);
      hw[e >> 2] = (hw[e >> 2] & ~(0xFFu << shift)) | (((uint32_t)h & 0xFFu) << shift);
      wbits |= (h > 0 ? 1u : 0u) << e;
    }
    reinterpret_cast<uint4 *>(hrow)[0] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
    reinterpret_cast<uint4 *>(hrow)[1] = make_uint4(hw[4], hw[5], hw[6], hw[7]);
    W32[(size_t)k * nw32 + cw] = wbits;
  }

  nreinf = wave_sum(nreinf);
  if (lane == 0 && nreinf) atomicAdd(p.stats + 3, nreinf);
}

}  // namespace

hipError_t launch_update(const UpdateArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const int nw32 = 2 * a.words_in;
  const size_t lds = (size_t)a.gamma * sizeof(int) + (size_t)a.n * sizeof(uint16_t);
  hipLaunchKernelGGL(update_kernel, dim3((nw32 + 63) / 64, a.groups), dim3(256), lds, s, a);
  return hipGetLastError();
}

}  // namespace bmlp
