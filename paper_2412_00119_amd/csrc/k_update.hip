// Perceptron-level update (Algorithm 3, Section 3.4) of every layer of a step
// in one launch.
//
// For every perceptron k of group g, the Clipped-Perceptron increments of the
// batch are summed first:
//   dH[k][i] = 2 * sum over patterns mu that selected k of rho^{y^mu}_k a^mu_i,
// then h <- clip(h + dH, -B, B); then every hidden weight whose 32-bit
// Philox draw is below T_l moves one step away from zero, h <- clip(h +
// 2 sign(h), -B, B); finally W = sign(H) is written as bits and as fp4.  A
// layer whose M_l is empty is left untouched.
//
// H is stored bit-sliced (see bmlp.h): each 32-column group of a row is eight
// words, word p holding bit p of the 32 two's-complement int8 values.  A lane
// owns one group, so every step below works on 32 columns with one bitwise
// operation per bit plane:
//   * the count cnt_i of +1 contributions (x = a-word XOR [rho = -1]) of the
//     S selectors of the row is accumulated bit-sliced (plane p = bit p of
//     the 32 counters), the loads of a-words issued eight at a time;
//   * h + 4 cnt - 2 S (= h + dH) and the clip to [-B, B] are ripple-carry
//     additions and comparisons on the planes, wide enough to be exact;
//   * the coarse reinforcement bytes arrive as bit planes (one Philox word
//     per plane), so "u8 < T >> 24" is an 8-step bit-sliced comparison; the
//     fine 24 bits are drawn only where u8 == T >> 24;
//   * h <- h + 2 sign(h) on the fired columns is one more planar addition,
//     and W = sign(H) is the complement of the sign plane.
//
// Work item: (layer, group g, 2048-column chunk); a work-group of 8 waves.
// The group's selections U_l (each pattern in M_l with a wrong perceptron in
// the group) are bucketed by perceptron in LDS (counting sort), then each
// wave walks whole rows, lane l owning 32-column group chunk * 64 + l.  No two
// work-groups write the same bytes of H or W.
#include "bmlp_internal.h"
#include "fp4.h"
#include "philox.h"

namespace bmlp {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kPlanes = 15;   // counts up to 2^15 - 1 >= BMLP_MAX_BATCH

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ uint32_t maj(uint32_t a, uint32_t b, uint32_t c) {
  return (a & b) | (c & (a ^ b));
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

template <int NP>
__device__ __forceinline__ void add_batch(uint32_t (&c)[kPlanes], const uint32_t (&x)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) add_planes<NP>(c, x[i]);
}

// Counts the +1 contributions of the row's S selectors (list[beg .. beg+S)),
// eight selectors per batch so that their loads are in flight together.  A
// batch past S loads a valid word (the row's last selector) and adds zero.
__device__ __forceinline__ void count_row(uint32_t (&c)[kPlanes], const uint16_t *list, int beg, int S,
                                          const uint32_t *a32, int nw32, int cw) {
#pragma unroll
  for (int q = 0; q < kPlanes; ++q) c[q] = 0u;
  for (int s0 = 0; s0 < S; s0 += 8) {
    uint32_t x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int s = s0 + i;
      const uint32_t ent = list[beg + min(s, S - 1)];
      const uint32_t mu = ent & 0x7FFFu;
      const uint32_t flip = (ent & 0x8000u) ? 0xFFFFFFFFu : 0u;
      const uint32_t v = a32[(size_t)mu * nw32 + cw];
      x[i] = s < S ? (v ^ flip) : 0u;
    }
    // planes in use after this batch: the counters are at most min(s0 + 8, S)
    switch (32 - __clz(min(s0 + 8, S))) {
      case 1: add_batch<1>(c, x); break;
      case 2: add_batch<2>(c, x); break;
      case 3: add_batch<3>(c, x); break;
      case 4: add_batch<4>(c, x); break;
      case 5: add_batch<5>(c, x); break;
      case 6: add_batch<6>(c, x); break;
      case 7: add_batch<7>(c, x); break;
      case 8: add_batch<8>(c, x); break;
      case 9: add_batch<9>(c, x); break;
      case 10: add_batch<10>(c, x); break;
      case 11: add_batch<11>(c, x); break;
      case 12: add_batch<12>(c, x); break;
      case 13: add_batch<13>(c, x); break;
      case 14: add_batch<14>(c, x); break;
      default: add_batch<15>(c, x); break;
    }
  }
}

// x += k (mod 2^NB) for a constant k, bit-sliced.
template <int NB>
__device__ __forceinline__ void add_const(uint32_t (&x)[NB], uint32_t k) {
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NB; ++p) {
    const uint32_t kb = ((k >> p) & 1u) ? 0xFFFFFFFFu : 0u;
    const uint32_t s = x[p] ^ kb ^ carry;
    carry = maj(x[p], kb, carry);
    x[p] = s;
  }
}

// Sign plane of x + k (mod 2^NB) for a constant k, bit-sliced (x unchanged).
template <int NB>
__device__ __forceinline__ uint32_t sign_of_sum(const uint32_t (&x)[NB], uint32_t k) {
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NB - 1; ++p) {
    const uint32_t kb = ((k >> p) & 1u) ? 0xFFFFFFFFu : 0u;
    carry = maj(x[p], kb, carry);
  }
  const uint32_t kb = ((k >> (NB - 1)) & 1u) ? 0xFFFFFFFFu : 0u;
  return x[NB - 1] ^ kb ^ carry;
}

// h <- clip(h + 4 cnt - 2 S, -B, B) on the 8 planes of h, computed in NB-bit
// two's complement (exact: |h| <= 127 and 4 cnt <= 4 S).
template <int NB>
__device__ __forceinline__ void cp_apply(uint32_t (&h)[8], const uint32_t (&c)[kPlanes], int S, int B) {
  // d = 4 cnt - 2 S
  uint32_t z[NB];
#pragma unroll
  for (int p = 0; p < NB; ++p) z[p] = (p >= 2 && p - 2 < kPlanes) ? c[p - 2] : 0u;
  add_const<NB>(z, (uint32_t)(-2 * S));
  // z = h + d, h sign-extended
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NB; ++p) {
    const uint32_t hp = h[p < 8 ? p : 7];
    const uint32_t s = z[p] ^ hp ^ carry;
    carry = maj(z[p], hp, carry);
    z[p] = s;
  }
  // z > B  <=>  z - (B + 1) >= 0 ;  z < -B  <=>  z + B < 0
  const uint32_t gt = ~sign_of_sum<NB>(z, (uint32_t)(-(B + 1)));
  const uint32_t lt = sign_of_sum<NB>(z, (uint32_t)B);
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const uint32_t bp = ((B >> p) & 1) ? 0xFFFFFFFFu : 0u;     // plane p of +B
    const uint32_t nbp = (((-B) >> p) & 1) ? 0xFFFFFFFFu : 0u;  // plane p of -B
    h[p] = (z[p] & ~(gt | lt)) | (bp & gt) | (nbp & lt);
  }
}

// Lanes where the 8-plane value equals the constant v.
__device__ __forceinline__ uint32_t equals(const uint32_t (&h)[8], int v) {
  uint32_t e = 0xFFFFFFFFu;
#pragma unroll
  for (int p = 0; p < 8; ++p) e &= ((v >> p) & 1) ? h[p] : ~h[p];
  return e;
}

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
  const int cw = chunk * 64 + lane;        // this lane's 32-column group
  const bool on = cw < U.nw32;
  const int cwc = min(cw, U.nw32 - 1);     // clamped: loads stay inside the rows
  const int nvalid = min(max(U.k_in - cw * 32, 0), 32);
  const uint32_t validmask = nvalid == 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
  const int B = p.bound;
  const uint32_t t_hi = U.t_hi, t_lo = U.t_lo;
  const int groups_in = (U.k_in + 31) >> 5;   // 32-column groups of a row holding columns
  int nreinf = 0;

  for (int r = wave; r < gamma; r += kWaves) {
    const int k = g * gamma + r;
    const int beg = r ? bucket[r - 1] : 0;
    const int S = bucket[r] - beg;

    uint8_t *hrow = U.H + (size_t)k * U.ld_h + (size_t)cwc * 32;
    uint32_t h[8];
    {
      const uint4 h0 = reinterpret_cast<const uint4 *>(hrow)[0];
      const uint4 h1 = reinterpret_cast<const uint4 *>(hrow)[1];
      h[0] = h0.x; h[1] = h0.y; h[2] = h0.z; h[3] = h0.w;
      h[4] = h1.x; h[5] = h1.y; h[6] = h1.z; h[7] = h1.w;
    }

    // ---- coarse reinforcement draws: plane p of the 32 bytes is word p of
    // Philox blocks 2 (k ceil(K/32) + group) and the one after (stream 3) ----
    const uint32_t blk = 2u * ((uint32_t)k * (uint32_t)groups_in + (uint32_t)cwc);
    const U32x4 v0 = philox4x32_10(blk, U.ctr1, p.step, kStreamCoarse, p.key0, p.key1);
    const U32x4 v1 = philox4x32_10(blk + 1u, U.ctr1, p.step, kStreamCoarse, p.key0, p.key1);

    // ---- Clipped-Perceptron sum and clip ------------------------------------
    if (S > 0) {
      uint32_t c[kPlanes];
      count_row(c, list, beg, S, U.a32, U.nw32, cwc);
      uint32_t hn[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) hn[q] = h[q];
      if (S <= 255)
        cp_apply<11>(hn, c, S, B);
      else
        cp_apply<18>(hn, c, S, B);
      // padding columns keep h = 0
#pragma unroll
      for (int q = 0; q < 8; ++q) h[q] = (hn[q] & validmask) | (h[q] & ~validmask);
    }

    // ---- which weights reinforce: u8 < T >> 24, or u8 == T >> 24 and the
    // fine 24 bits below T & 0xFFFFFF ---------------------------------------------
    uint32_t fire, need;
    if (t_hi >= 256u) {
      fire = 0xFFFFFFFFu;
      need = 0u;
    } else {
      const uint32_t rp[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
      uint32_t lt = 0u, eq = 0xFFFFFFFFu;
#pragma unroll
      for (int q = 7; q >= 0; --q) {
        if ((t_hi >> q) & 1u) {
          lt |= eq & ~rp[q];
          eq &= rp[q];
        } else {
          eq &= ~rp[q];
        }
      }
      fire = lt;
      need = eq;
    }
    fire &= validmask;
    need &= validmask;
    if (!on) {
      fire = 0u;
      need = 0u;
    }
    const uint32_t j0 = (uint32_t)k * (uint32_t)U.k_in + (uint32_t)(cwc * 32);
    while (need) {
      const int e = __ffs(need) - 1;
      need &= need - 1u;
      const uint32_t j = j0 + (uint32_t)e;
      const U32x4 f = philox4x32_10(j >> 2, U.ctr1, p.step, kStreamFine, p.key0, p.key1);
      if ((pick_word(f, j & 3u) & 0xFFFFFFu) < t_lo) fire |= 1u << e;
    }
    nreinf += __popc(fire);

    // ---- h <- clip(h + 2 sign(h)) on the fired weights: |h| = B stays ----------
    {
      const uint32_t gmask = fire & ~(equals(h, B) | equals(h, -B));
      const uint32_t neg = gmask & h[7];
      // add delta = +2 (0000 0010) or -2 (1111 1110) where gmask is set
      uint32_t carry = h[1] & gmask;
      h[1] ^= gmask;
#pragma unroll
      for (int q = 2; q < 8; ++q) {
        const uint32_t s = h[q] ^ neg ^ carry;
        carry = maj(h[q], neg, carry);
        h[q] = s;
      }
    }

    if (!on) continue;   // lanes past the row took part in the uniform loops only

    // ---- store H and W = sign(H) (h is odd, so the sign plane decides) -------
    const uint32_t wbits = ~h[7] & validmask;
    reinterpret_cast<uint4 *>(hrow)[0] = make_uint4(h[0], h[1], h[2], h[3]);
    reinterpret_cast<uint4 *>(hrow)[1] = make_uint4(h[4], h[5], h[6], h[7]);
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
