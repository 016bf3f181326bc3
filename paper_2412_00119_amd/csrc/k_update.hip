// Perceptron-level update (Algorithm 3, Section 3.4) of every layer of a step
// in one launch.
//
// For every perceptron k of group g, the Clipped-Perceptron increments of the
// batch are summed first:
//   dH[k][i] = 2 * sum over patterns mu that selected k of rho^{y^mu}_k a^mu_i,
// then h <- clip(h + dH, -B, B); then every hidden weight whose 32-bit
// Philox draw is below T_l moves one step away from zero, h <- clip(h +
// 2 sign(h), -B, B); finally W = sign(H) is re-packed into bits.  A layer
// whose M_l is empty is left untouched.
//
// Work item: (layer, group g, 2048-column chunk); a work-group of 8 waves.
// The group's selections U_l (each pattern in M_l with a wrong perceptron in
// the group) are bucketed by perceptron in LDS (counting sort),
// then each wave walks whole rows with a lane owning 32 consecutive columns
// (one 32-bit word of a_{l-1}).  With x = a-word XOR [rho = -1] the number
// of +1 contributions per column is counted in bit-sliced form (plane p holds
// bit p of the 32 counters), so one selector costs a short carry chain per
// word; the counts are then spread into byte lanes and the clip is done on
// packed 16-bit lanes: with cnt_i the count, sum_i = 2 cnt_i - S and
// dH_i = 4 cnt_i - 2 S.  No two work-groups write the same bytes of H or W.
#include "bmlp_internal.h"
#include "fp4.h"
#include "philox.h"

namespace bmlp {
namespace {

typedef short s16x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kPlanes = 15;   // counts up to 2^15 - 1 >= BMLP_MAX_BATCH

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// bit-sliced increment of the 32 counters by the bits of x, planes [0, NP)
template <int NP>
__device__ __forceinline__ void add_planes(uint32_t (&c)[kPlanes], uint32_t x) {
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const uint32_t t = c[p] & x;
    c[p] ^= x;
    x = t;
  }
}

struct SelCtx {
  const uint16_t *list;
  const uint32_t *a32;
  int nw32, cw;
  bool on;
};

// Adds selectors [s0, s1) of a row; after s selectors a counter is <= s, so
// the carry chain of selector s (0-based) stops at plane floor(log2(s+1)).
template <int NP>
__device__ __forceinline__ void count_segment(uint32_t (&c)[kPlanes], const SelCtx &sc, int beg,
                                              int s0, int s1) {
  for (int s = s0; s < s1; ++s) {
    const uint32_t ent = sc.list[beg + s];
    const uint32_t mu = ent & 0x7FFFu;
    const uint32_t flip = (ent & 0x8000u) ? 0xFFFFFFFFu : 0u;
    const uint32_t x = (sc.on ? sc.a32[(size_t)mu * sc.nw32 + sc.cw] : 0u) ^ flip;
    add_planes<NP>(c, x);
  }
}

// Per-byte flags of (byte < t) for t in [0, 128], as bit 7 of each byte.
__device__ __forceinline__ uint32_t bytes_lt(uint32_t x, uint32_t t) {
  const uint32_t y = (x | 0x80808080u) - t * 0x01010101u;
  return ~(y | x) & 0x80808080u;
}

// Gathers bit 7 of each byte into a 4-bit value (byte i -> bit i).
__device__ __forceinline__ uint32_t gather_msb(uint32_t m) {
  return (((m >> 7) * 0x01020408u) >> 24) & 0xFu;
}

// spread the 4 bits of n (n < 16) into bit 0 of the 4 bytes of a word
__device__ __forceinline__ uint32_t spread4(uint32_t n) { return (n * 0x00204081u) & 0x01010101u; }

__device__ __forceinline__ s16x2 as_s16x2(uint32_t v) { return __builtin_bit_cast(s16x2, v); }
__device__ __forceinline__ uint32_t as_u32(s16x2 v) { return __builtin_bit_cast(uint32_t, v); }

__global__ __launch_bounds__(kThreads) void update_kernel(UpdateBatch p) {
  extern __shared__ int smem[];
  __shared__ int part[kThreads];

  const int tid = threadIdx.x;
  // ---- which layer / group / chunk ------------------------------------------
  int li = 0;
#pragma unroll 1
  for (int i = 1; i < p.nl; ++i)
    if ((int)blockIdx.x >= p.L[i].block0) li = i;
  const UpdLayer &U = p.L[li];
  if (U.stats[1] == 0) return;   // M_l empty: Algorithm 2 is not run for this layer
  const int rel = (int)blockIdx.x - U.block0;
  const int g = rel / U.chunks;
  const int chunk = rel % U.chunks;
  const int gamma = U.gamma;
  int *bucket = smem;                                            // [gamma]
  uint16_t *list = reinterpret_cast<uint16_t *>(smem + gamma);   // [n]
  const int16_t *kcol = U.kstar + (size_t)g * p.ldk;

  // ---- bucket the selections of group g by perceptron (counting sort) -------
  __shared__ int s_sel;
  if (tid == 0) s_sel = 0;
  for (int r = tid; r < gamma; r += kThreads) bucket[r] = 0;
  __syncthreads();
  // U_l: the selections of the patterns in M_l
  int nsel = 0;
  for (int mu = tid; mu < p.n; mu += kThreads) {
    const int ks = U.upd[mu] ? kcol[mu] : -1;
    if (ks >= 0) {
      atomicAdd(&bucket[ks], 1);
      ++nsel;
    }
  }
  if (chunk == 0) {   // |U_l|, counted once per group
    nsel = wave_sum(nsel);
    if ((tid & 63) == 0 && nsel) atomicAdd(&s_sel, nsel);
  }
  __syncthreads();
  if (chunk == 0 && tid == 0 && s_sel) atomicAdd(U.stats + 2, s_sel);
  {
    const int ch = (gamma + kThreads - 1) / kThreads;
    const int b0 = min(gamma, tid * ch), b1 = min(gamma, b0 + ch);
    int s = 0;
    for (int r = b0; r < b1; ++r) s += bucket[r];
    part[tid] = s;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
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
  for (int mu = tid; mu < p.n; mu += kThreads) {
    const int ks = U.upd[mu] ? kcol[mu] : -1;
    if (ks >= 0) {
      const int k = g * gamma + ks;
      const int yl = min(max(p.y[mu], 0), p.c - 1);   // stay inside P on a bad label
      const bool rpos = (U.P[(size_t)yl * U.words_out + (k >> 6)] >> (k & 63)) & 1ull;
      const int pos = atomicAdd(&bucket[ks], 1);
      list[pos] = (uint16_t)(mu | (rpos ? 0 : 0x8000));
    }
  }
  __syncthreads();
  // bucket[r] is now the end of row r's selectors; row r starts at bucket[r-1]

  const int wave = tid >> 6, lane = tid & 63;
  SelCtx sc;
  sc.list = list;
  sc.a32 = U.a32;
  sc.nw32 = U.nw32;
  sc.cw = chunk * 64 + lane;
  sc.on = sc.cw < U.nw32;
  const int cw = sc.cw;
  const int nvalid = min(max(U.k_in - cw * 32, 0), 32);
  const uint32_t validmask = nvalid == 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
  const int B = p.bound;
  const uint32_t t_hi = U.t_hi, t_lo = U.t_lo;
  int nreinf = 0;

  for (int r = wave; r < gamma; r += kWaves) {
    const int k = g * gamma + r;
    const int beg = r ? bucket[r - 1] : 0;
    const int S = bucket[r] - beg;

    uint32_t hw[8];
    int8_t *hrow = U.H + (size_t)k * U.ld_h + cw * 32;
    if (sc.on) {
      const uint4 h0 = reinterpret_cast<const uint4 *>(hrow)[0];
      const uint4 h1 = reinterpret_cast<const uint4 *>(hrow)[1];
      hw[0] = h0.x; hw[1] = h0.y; hw[2] = h0.z; hw[3] = h0.w;
      hw[4] = h1.x; hw[5] = h1.y; hw[6] = h1.z; hw[7] = h1.w;
    }

    // ---- Clipped-Perceptron sum ---------------------------------------------
    if (S > 0) {
      uint32_t c[kPlanes];
#pragma unroll
      for (int q = 0; q < kPlanes; ++q) c[q] = 0u;
      count_segment<1>(c, sc, beg, 0, min(S, 1));
      count_segment<2>(c, sc, beg, 1, min(S, 3));
      count_segment<3>(c, sc, beg, 3, min(S, 7));
      count_segment<4>(c, sc, beg, 7, min(S, 15));
      count_segment<5>(c, sc, beg, 15, min(S, 31));
      count_segment<6>(c, sc, beg, 31, min(S, 63));
      count_segment<7>(c, sc, beg, 63, min(S, 127));
      count_segment<8>(c, sc, beg, 127, min(S, 255));
      if (S > 255) count_segment<kPlanes>(c, sc, beg, 255, S);

      if (sc.on) {
        if (S <= 255) {
          // counts as bytes, 4 columns per word
          const int np = 32 - __clz(S);   // planes in use
          const s16x2 lo2 = {(short)(128 - B), (short)(128 - B)};
          const s16x2 hi2 = {(short)(128 + B), (short)(128 + B)};
          const s16x2 m2 = {(short)(-2 * S), (short)(-2 * S)};
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            uint32_t cb = 0u;
#pragma unroll
            for (int pl = 0; pl < 8; ++pl)
              if (pl < np) cb |= spread4((c[pl] >> (4 * q)) & 0xFu) << pl;
            // biased bytes hb = h + 128 in 16-bit lanes: columns (4q, 4q+1), (4q+2, 4q+3)
            const uint32_t hb = hw[q] ^ 0x80808080u;
            s16x2 h01 = as_s16x2((hb & 0xFFu) | ((hb & 0xFF00u) << 8));
            s16x2 h23 = as_s16x2(((hb >> 16) & 0xFFu) | ((hb >> 8) & 0xFF0000u));
            const s16x2 c01 = as_s16x2((cb & 0xFFu) | ((cb & 0xFF00u) << 8));
            const s16x2 c23 = as_s16x2(((cb >> 16) & 0xFFu) | ((cb >> 8) & 0xFF0000u));
            h01 = h01 + c01 * (s16x2){4, 4} + m2;
            h23 = h23 + c23 * (s16x2){4, 4} + m2;
            h01 = __builtin_elementwise_min(__builtin_elementwise_max(h01, lo2), hi2);
            h23 = __builtin_elementwise_min(__builtin_elementwise_max(h23, lo2), hi2);
            const uint32_t u01 = as_u32(h01), u23 = as_u32(h23);
            const uint32_t nb = (u01 & 0xFFu) | ((u01 >> 8) & 0xFF00u) | ((u23 & 0xFFu) << 16) |
                                ((u23 << 8) & 0xFF000000u);
            // pad columns keep their bytes
            const uint32_t vm = spread4((validmask >> (4 * q)) & 0xFu) * 0xFFu;
            hw[q] = ((nb ^ 0x80808080u) & vm) | (hw[q] & ~vm);
          }
        } else {
          // more than 255 selectors: per-column integer counts
#pragma unroll
          for (int e = 0; e < 32; ++e) {
            if (!((validmask >> e) & 1u)) continue;
            int cnt = 0;
#pragma unroll
            for (int pl = 0; pl < kPlanes; ++pl) cnt |= (int)((c[pl] >> e) & 1u) << pl;
            const int q = e >> 2, sh = 8 * (e & 3);
            int h = (int)(int8_t)((hw[q] >> sh) & 0xFFu);
            h = min(max(h + 4 * cnt - 2 * S, -B), B);
            hw[q] = (hw[q] & ~(0xFFu << sh)) | (((uint32_t)h & 0xFFu) << sh);
          }
        }
      }
    }

    if (!sc.on) continue;   // lanes past the row took part in the uniform loops only

    // ---- reinforcement draws (Philox streams 3 and 4) -------------------------
    const uint32_t j0 = (uint32_t)k * (uint32_t)U.k_in + (uint32_t)(cw * 32);
    const uint32_t b0 = j0 >> 4, sh = j0 & 15u;
    const U32x4 v0 = philox4x32_10(b0, U.ctr1, p.step, kStreamCoarse, p.key0, p.key1);
    const U32x4 v1 = philox4x32_10(b0 + 1, U.ctr1, p.step, kStreamCoarse, p.key0, p.key1);
    uint32_t u[8];
    if (sh == 0) {
      u[0] = v0.x; u[1] = v0.y; u[2] = v0.z; u[3] = v0.w;
      u[4] = v1.x; u[5] = v1.y; u[6] = v1.z; u[7] = v1.w;
    } else {
      // weights j0.. start at byte sh of block b0: shift the 48 bytes of blocks
      // b0..b0+2 down by sh bytes (sh is the same for the whole wave)
      const U32x4 v2 = philox4x32_10(b0 + 2, U.ctr1, p.step, kStreamCoarse, p.key0, p.key1);
      uint32_t w[12] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w, v2.x, v2.y, v2.z, v2.w};
      if (sh & 4u) {
#pragma unroll
        for (int i = 0; i < 11; ++i) w[i] = w[i + 1];
      }
      if (sh & 8u) {
#pragma unroll
        for (int i = 0; i < 10; ++i) w[i] = w[i + 2];
      }
      const uint32_t bs = sh & 3u;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        u[q] = (uint32_t)((((uint64_t)w[q + 1] << 32) | w[q]) >> (8 * bs));
    }
    uint32_t fire = 0u, need = 0u;
    if (t_hi <= 127) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const uint32_t lt = bytes_lt(u[q], t_hi);
        const uint32_t le = bytes_lt(u[q], t_hi + 1);
        fire |= gather_msb(lt) << (4 * q);
        need |= gather_msb(le & ~lt) << (4 * q);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const uint32_t u8 = (u[e >> 2] >> (8 * (e & 3))) & 0xFFu;
        fire |= (u8 < t_hi ? 1u : 0u) << e;
        need |= (u8 == t_hi ? 1u : 0u) << e;
      }
    }
    fire &= validmask;
    need &= validmask;
    while (need) {
      const int e = __ffs(need) - 1;
      need &= need - 1u;
      const uint32_t j = j0 + (uint32_t)e;
      const U32x4 f = philox4x32_10(j >> 2, U.ctr1, p.step, kStreamFine, p.key0, p.key1);
      if ((pick_word(f, j & 3u) & 0xFFFFFFu) < t_lo) fire |= 1u << e;
    }
    nreinf += __popc(fire);

    // ---- h <- clip(h + 2 sign(h)) on the (rare) fired weights ---------------------
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      uint32_t m = (fire >> (4 * q)) & 0xFu;
      while (m) {
        const int b = __ffs(m) - 1;
        m &= m - 1u;
        const int shb = 8 * b;
        int h = (int)(int8_t)((hw[q] >> shb) & 0xFFu);
        h = min(max(h + (h > 0 ? 2 : -2), -B), B);
        hw[q] = (hw[q] & ~(0xFFu << shb)) | (((uint32_t)h & 0xFFu) << shb);
      }
    }

    // ---- store H and W = sign(H) (h is odd: positive iff the sign bit is clear) ----
    uint32_t wbits = 0u;
#pragma unroll
    for (int q = 0; q < 8; ++q) wbits |= gather_msb(~hw[q] & 0x80808080u) << (4 * q);
    wbits &= validmask;
    reinterpret_cast<uint4 *>(hrow)[0] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
    reinterpret_cast<uint4 *>(hrow)[1] = make_uint4(hw[4], hw[5], hw[6], hw[7]);
    U.W32[(size_t)k * U.nw32 + cw] = wbits;
    {
      uint32_t o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = fp4_from_bits8(wbits >> (8 * q), validmask >> (8 * q));
      *reinterpret_cast<uint4 *>(U.Wq + (size_t)k * U.ldq + cw * 16) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }

  nreinf = wave_sum(nreinf);
  if (lane == 0) part[wave] = nreinf;
  __syncthreads();
  if (tid == 0) {
    int t = 0;
    for (int w = 0; w < kWaves; ++w) t += part[w];
    if (t) atomicAdd(U.stats + 3, t);   // one atomic per work-group
  }
}

}  // namespace

size_t update_lds_bytes(int gamma, int n) {
  return (size_t)gamma * sizeof(int) + (size_t)n * sizeof(uint16_t);
}

hipError_t launch_update(UpdateBatch &b, hipStream_t s) {
  if (b.n <= 0 || b.nl <= 0) return hipSuccess;
  int blocks = 0;
  int gmax = 0;
  for (int i = 0; i < b.nl; ++i) {
    UpdLayer &u = b.L[i];
    u.chunks = (u.nw32 + 63) / 64;
    u.block0 = blocks;
    blocks += u.groups * u.chunks;
    gmax = max(gmax, u.gamma);
  }
  hipLaunchKernelGGL(update_kernel, dim3(blocks), dim3(kThreads), update_lds_bytes(gmax, b.n), s, b);
  return hipGetLastError();
}

}  // namespace bmlp
