// Perceptron-level update (Algorithm 3, Section 3.4) of every layer of a step
// in one launch.
//
// For every perceptron k of group g, the Clipped-Perceptron increments of the
// batch are summed first:
//   dH[k][i] = 2 * sum over patterns mu that selected k of rho^{y^mu}_k a^mu_i,
// then h <- clip(h + dH, -B, B); then every hidden weight whose 32-bit
// Philox draw is below T_l moves one step away from zero, h <- clip(h +
// 2 sign(h), -B, B); finally W = sign(H) is written as bits.  A
// layer whose M_l is empty is left untouched.
//
// h is odd and |h| <= B (B odd), so H is stored as u = (h + B) / 2 in
// [0, B], in M = bits(B) planes (see bmlp.h): plane p of a row holds bit p of
// u for every column, one 32-bit word per 32-column group.  A lane owns one
// group, so every step below works on 32 columns with one bitwise operation
// per bit plane:
//   * the count cnt_i of +1 contributions (x = a-word XOR [rho = -1]) of the
//     S selectors of the row is accumulated bit-sliced (plane p = bit p of
//     the 32 counters) with carry-save adder trees, the loads of a row's
//     a-words issued sixteen at a time;
//   * u + 2 cnt - S (= (h + dH + B) / 2) and the clip to [0, B] are
//     ripple-carry additions and comparisons on the planes, wide enough to
//     be exact;
//   * the coarse reinforcement bytes arrive as bit planes (one Philox word
//     per plane), so "u8 < T >> 24" is an 8-step bit-sliced comparison; the
//     fine 24 bits are drawn only where u8 == T >> 24;
//   * h <- h + 2 sign(h) is u <- u +- 1 on the fired columns, one more planar
//     addition, and W = sign(H) is u >= (B + 1) / 2.
//
// Work-group: (layer, group g, half of g's rows), 12 waves.  The group's selections U_l (each
// pattern in M_l with a wrong perceptron in the group) are bucketed by
// perceptron in LDS (counting sort), then the waves take the group's (row,
// 2048-column chunk) items, lane l owning 32-column group chunk * 64 + l.  No
// two work-groups write the same bytes of H or W.
#include "bmlp_internal.h"
#include "philox.h"

namespace bmlp {
namespace {

// Two work-groups of 12 waves per group of perceptrons, each taking half
// of the group's rows: two of them fit a compute unit together (six waves
// per SIMD), which hides more of the H loads behind the draws than one
// work-group of 16 waves per compute unit did.
constexpr int kWaves = 12;
constexpr int kThreads = 64 * kWaves;
constexpr int kSplit = 2;
constexpr int kPre = 2;   // patterns per thread whose selection data the prologue loads up front
constexpr int kPlanes = 15;   // counts up to 2^15 - 1 >= BMLP_MAX_BATCH

// A wave-uniform word the compiler must treat as unknown and keep in a
// scalar register: bit-plane constants (0 or ~0) stay 32-bit operands of
// the bitwise ops instead of being turned into 64-bit lane masks and
// selects, and values made from it inside the item loop are not hoisted
// out of it (where they would no longer fit in scalar registers).
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+s"(v));
  return v;
}

// all-ones when bit p of k is set, else 0, as an opaque scalar
__device__ __forceinline__ uint32_t plane_of(uint32_t k, int p) { return opaque(0u - ((k >> p) & 1u)); }

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ uint32_t maj(uint32_t a, uint32_t b, uint32_t c) {
  return (a & b) | (c & (a ^ b));
}

// Carry-save compression: a full adder turns three bit-vectors of one
// weight into a sum of that weight and a carry of twice it (two 3-input
// bitwise operations), a half adder does the same for two.
__device__ __forceinline__ void fa(uint32_t a, uint32_t b, uint32_t c, uint32_t &s, uint32_t &cy) {
  s = a ^ b ^ c;
  cy = maj(a, b, c);
}
__device__ __forceinline__ void ha(uint32_t a, uint32_t b, uint32_t &s, uint32_t &cy) {
  s = a ^ b;
  cy = a & b;
}

// Per lane, the number of set bits among x[0..8) as 4 planes n[0..4).
__device__ __forceinline__ void compress8(const uint32_t (&x)[8], uint32_t (&n)[4]) {
  uint32_t a, b, c, d, e, f, s1, c1, s2, c2, t, u;
  fa(x[0], x[1], x[2], a, b);    // a:1 b:2
  fa(x[3], x[4], x[5], c, d);    // c:1 d:2
  fa(x[6], x[7], a, e, f);       // e:1 f:2
  ha(c, e, n[0], s1);            // n0:1 s1:2
  fa(b, d, f, s2, c1);           // s2:2 c1:4
  ha(s2, s1, n[1], c2);          // n1:2 c2:4
  ha(c1, c2, t, u);              // t:4 u:8
  n[2] = t;
  n[3] = u;
}

// Per lane, the number of set bits among x[0..16) as 5 planes n[0..5).
__device__ __forceinline__ void compress16(const uint32_t (&x)[16], uint32_t (&n)[5]) {
  // weight 1: 16 bits
  uint32_t s[6], c2[8];
  fa(x[0], x[1], x[2], s[0], c2[0]);
  fa(x[3], x[4], x[5], s[1], c2[1]);
  fa(x[6], x[7], x[8], s[2], c2[2]);
  fa(x[9], x[10], x[11], s[3], c2[3]);
  fa(x[12], x[13], x[14], s[4], c2[4]);
  uint32_t t0, t1;
  fa(s[0], s[1], s[2], t0, c2[5]);
  fa(s[3], s[4], x[15], t1, c2[6]);
  ha(t0, t1, n[0], c2[7]);
  // weight 2: 8 bits
  uint32_t w2a, w2b, w2c, c4[4];
  fa(c2[0], c2[1], c2[2], w2a, c4[0]);
  fa(c2[3], c2[4], c2[5], w2b, c4[1]);
  fa(c2[6], c2[7], w2a, w2c, c4[2]);
  ha(w2b, w2c, n[1], c4[3]);
  // weight 4: 4 bits
  uint32_t w4a, c8a, c8b;
  fa(c4[0], c4[1], c4[2], w4a, c8a);
  ha(w4a, c4[3], n[2], c8b);
  // weight 8: 2 bits
  ha(c8a, c8b, n[3], n[4]);
}

// c += n (n has NN planes), rippling the carry up to plane NP - 1.
template <int NN, int NP>
__device__ __forceinline__ void add_count(uint32_t (&c)[kPlanes], const uint32_t (&n)[NN]) {
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    if (p < NN) {
      const uint32_t sum = c[p] ^ n[p] ^ carry;
      carry = maj(c[p], n[p], carry);
      c[p] = sum;
    } else {
      const uint32_t sum = c[p] ^ carry;
      carry = c[p] & carry;
      c[p] = sum;
    }
  }
}

// The a_{l-1} rows are read through a buffer descriptor: the selector's row
// offset is a scalar (soffset) and the lane's word offset a vector register,
// so a load costs no vector address arithmetic.

__device__ __forceinline__ uint32_t load_word(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0);
}

// The 16 selector entries list[i .. i + 16) (i a multiple of 8, list 16-byte
// aligned): two 16-byte LDS reads at an address every lane shares, moved to
// scalar registers.
__device__ __forceinline__ void read_entries16(const uint16_t *list, int i, uint32_t (&e)[8]) {
  const uint4 a = *reinterpret_cast<const uint4 *>(list + i);
  const uint4 b = *reinterpret_cast<const uint4 *>(list + i + 8);
  e[0] = __builtin_amdgcn_readfirstlane(a.x);
  e[1] = __builtin_amdgcn_readfirstlane(a.y);
  e[2] = __builtin_amdgcn_readfirstlane(a.z);
  e[3] = __builtin_amdgcn_readfirstlane(a.w);
  e[4] = __builtin_amdgcn_readfirstlane(b.x);
  e[5] = __builtin_amdgcn_readfirstlane(b.y);
  e[6] = __builtin_amdgcn_readfirstlane(b.z);
  e[7] = __builtin_amdgcn_readfirstlane(b.w);
}

// x[i] = a-word of entry i of e, flipped where rho = -1, for i < N; with
// KEEP, entries i >= keep are zero (and read row 0, a valid address, since
// the list slots past the row's selectors hold no entry).
template <int N, bool KEEP>
__device__ __forceinline__ void load_selectors(uint32_t (&x)[N], const uint32_t (&e)[8], int keep,
                                               __amdgpu_buffer_rsrc_t rs, int rowbytes, int voff) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint32_t ent = (e[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    const bool live = !KEEP || i < keep;
    const int soff = live ? (int)(ent & 0x7FFFu) * rowbytes : 0;
    const uint32_t flip = (ent & 0x8000u) ? 0xFFFFFFFFu : 0u;
    const uint32_t w = load_word(rs, voff, soff) ^ flip;
    x[i] = live ? w : 0u;
  }
}

// c += n (NN planes) where the counters are at most `bound` afterwards: the
// carry ripples only through the planes in use (a uniform exit, so c stays
// in place).
template <int NN>
__device__ __forceinline__ void add_count_upto(uint32_t (&c)[kPlanes], const uint32_t (&n)[NN], int bound) {
  const int np = 32 - __clz(bound);
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) {
    if (p < NN) {
      const uint32_t sum = c[p] ^ n[p] ^ carry;
      carry = maj(c[p], n[p], carry);
      c[p] = sum;
    } else {
      if (p >= np) break;
      const uint32_t sum = c[p] ^ carry;
      carry = c[p] & carry;
      c[p] = sum;
    }
  }
}

// Counts the +1 contributions of the row's S >= 1 selectors (list[beg ..
// beg+S), beg a multiple of 8) into bit-sliced counters: batches of 16
// through a carry-save tree, all 16 loads in flight together, each batch's
// count added to the running one; the last batch (up to 15, or 8) masks
// the slots past S.
__device__ __forceinline__ void count_row(uint32_t (&c)[kPlanes], const uint16_t *list, int beg, int S,
                                          __amdgpu_buffer_rsrc_t rs, int rowbytes, int voff) {
#pragma unroll
  for (int q = 0; q < kPlanes; ++q) c[q] = 0u;
  int s0 = 0;
  for (; s0 + 16 <= S; s0 += 16) {
    uint32_t e[8], x[16], n[5];
    read_entries16(list, beg + s0, e);
    load_selectors<16, false>(x, e, 16, rs, rowbytes, voff);
    compress16(x, n);
    if (s0 == 0) {
#pragma unroll
      for (int q = 0; q < 5; ++q) c[q] = n[q];
    } else {
      add_count_upto<5>(c, n, s0 + 16);
    }
  }
  const int rem = S - s0;
  if (rem == 0) return;
  uint32_t e[8];
  read_entries16(list, beg + s0, e);
  if (rem <= 8) {
    uint32_t x[8], n[4];
    load_selectors<8, true>(x, e, rem, rs, rowbytes, voff);
    compress8(x, n);
    if (s0 == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = n[q];
    } else {
      add_count_upto<4>(c, n, S);
    }
  } else {
    uint32_t x[16], n[5];
    load_selectors<16, true>(x, e, rem, rs, rowbytes, voff);
    compress16(x, n);
    if (s0 == 0) {
#pragma unroll
      for (int q = 0; q < 5; ++q) c[q] = n[q];
    } else {
      add_count_upto<5>(c, n, S);
    }
  }
}

// x += k (mod 2^NB) for a constant k, bit-sliced.
template <int NB>
__device__ __forceinline__ void add_const(uint32_t (&x)[NB], uint32_t k) {
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NB; ++p) {
    const uint32_t kb = plane_of(k, p);
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
  for (int p = 0; p < NB - 1; ++p) carry = maj(x[p], plane_of(k, p), carry);
  return x[NB - 1] ^ plane_of(k, NB - 1) ^ carry;
}

// u <- clip(u + 2 cnt - S, 0, B) on the M planes of u, computed in NB-bit
// two's complement.  NB must hold z = u + 2 cnt - S, in [-S, B + S], and
// z - (B + 1): 9 bits for S <= 63, 10 for S <= 255, 17 for S <= 16384
// (B <= 127).
template <int M, int NB>
__device__ __forceinline__ void cp_apply(uint32_t (&u)[M], const uint32_t (&c)[kPlanes], int S, int B) {
  // z = 2 cnt - S
  uint32_t z[NB];
#pragma unroll
  for (int p = 0; p < NB; ++p) z[p] = (p >= 1 && p - 1 < kPlanes) ? c[p - 1] : 0u;
  add_const<NB>(z, (uint32_t)(-S));
  // z += u
  uint32_t carry = 0u;
#pragma unroll
  for (int p = 0; p < NB; ++p) {
    const uint32_t up = p < M ? u[p] : 0u;
    const uint32_t t = z[p] ^ up ^ carry;
    carry = maj(z[p], up, carry);
    z[p] = t;
  }
  // z > B  <=>  z - (B + 1) >= 0 ;  z < 0 is the sign plane
  const uint32_t gt = ~sign_of_sum<NB>(z, (uint32_t)(-(B + 1)));
  const uint32_t lt = z[NB - 1];
#pragma unroll
  for (int p = 0; p < M; ++p) u[p] = (z[p] & ~(gt | lt)) | (plane_of((uint32_t)B, p) & gt);
}

// Lanes where the M-plane value equals the constant v.
template <int M>
__device__ __forceinline__ uint32_t equals(const uint32_t (&u)[M], int v) {
  uint32_t e = 0xFFFFFFFFu;
#pragma unroll
  for (int p = 0; p < M; ++p) e &= ~(u[p] ^ plane_of((uint32_t)v, p));
  return e;
}

// The sequential reading of the increments: the row's S >= 1 selectors
// (list[beg .. beg+S), in pattern order) one at a time, each moving u by +1
// where a rho = +1 and -1 elsewhere, clipped to [0, B] at once.  Columns
// outside validmask keep their value.
template <int M>
__device__ __forceinline__ void cp_sequential(uint32_t (&u)[M], const uint16_t *list, int beg, int S, int B,
                                              uint32_t validmask, const uint32_t *a32, int nw32, int cw) {
  for (int s = 0; s < S; ++s) {
    const uint32_t ent = __builtin_amdgcn_readfirstlane(list[beg + s]);
    const uint32_t mu = ent & 0x7FFFu;
    const uint32_t x = a32[(size_t)mu * nw32 + cw] ^ ((ent & 0x8000u) ? 0xFFFFFFFFu : 0u);
    const uint32_t inc = x & validmask & ~equals<M>(u, B);
    const uint32_t dec = ~x & validmask & ~equals<M>(u, 0);
    const uint32_t g = inc | dec;
    // u + 1 on inc, u + (2^M - 1) = u - 1 on dec
    uint32_t carry = u[0] & g;
    u[0] ^= g;
#pragma unroll
    for (int q = 1; q < M; ++q) {
      const uint32_t sum = u[q] ^ dec ^ carry;
      carry = maj(u[q], dec, carry);
      u[q] = sum;
    }
  }
}

// Lanes where the M-plane value is at least the constant k (0 < k <= 2^M):
// the sign plane of u - k in M + 1 bits is clear.
template <int M>
__device__ __forceinline__ uint32_t at_least(const uint32_t (&u)[M], int k) {
  uint32_t x[M + 1];
#pragma unroll
  for (int p = 0; p < M; ++p) x[p] = u[p];
  x[M] = 0u;
  return ~sign_of_sum<M + 1>(x, (uint32_t)(-k));
}

// Lanes whose M-plane value has every plane set / any plane set.
template <int M>
__device__ __forceinline__ uint32_t all_planes(const uint32_t (&u)[M]) {
  uint32_t e = u[0];
#pragma unroll
  for (int q = 1; q < M; ++q) e &= u[q];
  return e;
}
template <int M>
__device__ __forceinline__ uint32_t any_plane(const uint32_t (&u)[M]) {
  uint32_t e = u[0];
#pragma unroll
  for (int q = 1; q < M; ++q) e |= u[q];
  return e;
}

__device__ __host__ __forceinline__ int round8(int v) { return (v + 7) & ~7; }

// Selector list slots: every row's selectors padded to a multiple of 8, and
// 16 more so that a batch read of 16 entries stays inside the list; a
// multiple of 8 slots, so that the bucket offsets after it stay aligned.
__device__ __host__ __forceinline__ int list_slots(int n, int gamma) { return round8(n + 7 * gamma) + 16; }

// FULL: B = 2^M - 1 (B = 1, 3, 7, 15, 31, 63, 127), so u = B is every plane
// set and u >= (B + 1) / 2 is the top plane; otherwise the planar
// comparisons with the constants of B.
// The layer lookup and the first load take their arguments from the
// leading scalars, which are preloaded into scalar registers when the wave
// starts: nl, the first work-group of layers 1..7 of the launch, and the
// stats row of its layer 0 (the rows of the launch's layers follow it at
// BMLP_STATS_STRIDE), so that |M_l| is requested before the argument
// buffer has been read.
template <int M, bool FULL>
__global__ __launch_bounds__(kThreads, kSplit * kWaves / 4) void update_kernel(
    int nl, int b1, int b2, int b3, int b4, int b5, int b6, int b7, const int32_t *stats0, UpdateBatch p) {
  extern __shared__ __align__(16) int smem[];
  __shared__ int wsum[kWaves];
  __shared__ int s_sel;

  const int tid = threadIdx.x;
  // the wave index is uniform: in a scalar register, so are the item indices
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  // ---- which layer / group ---------------------------------------------------
  const int bid = (int)blockIdx.x;
  int li = 0;
  li = (nl > 1 && bid >= b1) ? 1 : li;
  li = (nl > 2 && bid >= b2) ? 2 : li;
  li = (nl > 3 && bid >= b3) ? 3 : li;
  li = (nl > 4 && bid >= b4) ? 4 : li;
  li = (nl > 5 && bid >= b5) ? 5 : li;
  li = (nl > 6 && bid >= b6) ? 6 : li;
  li = (nl > 7 && bid >= b7) ? 7 : li;
  const int mcount = stats0[li * BMLP_STATS_STRIDE + 1];
  const UpdLayer &U = p.L[li];
  // what the bucketing reads first, requested together with |M_l| (one
  // wait for both instead of a second round trip after the check)
  const uint8_t *const upd = U.upd;
  const int16_t *const kstar = U.kstar;
  const int32_t *const labels = p.y;
  const int gamma = U.gamma, n = p.n, ldk = p.ldk;
  asm volatile("" ::"s"(mcount), "s"(upd), "s"(kstar), "s"(labels), "s"(gamma), "s"(n), "s"(ldk));
  const int block0 = li == 0 ? 0 : li == 1 ? b1 : li == 2 ? b2 : li == 3 ? b3 : li == 4 ? b4 : li == 5 ? b5 : li == 6 ? b6 : b7;
  const int g = (bid - block0) / kSplit;
  const int part = (bid - block0) % kSplit;
  const int16_t *kcol = kstar + (size_t)g * ldk;
  // The first kPre patterns of each thread: M_l flag, k* and label loaded
  // before |M_l| is known (in bounds: the index is clamped), so that they
  // arrive with it, and kept for the list fill below, which then loads only
  // the word of P_l that holds the selection's rho bit.
  int ks_pre[kPre], y_pre[kPre];
#pragma unroll
  for (int q = 0; q < kPre; ++q) {
    const int mu = tid + q * kThreads, muc = min(mu, n - 1);
    const int f = upd[muc], k16 = kcol[muc];
    y_pre[q] = labels[muc];
    ks_pre[q] = (mu < n && f) ? k16 : -1;
  }
  // used before the check, so that the compiler keeps the loads above it
  static_assert(kPre == 2, "one use of every preloaded value");
  asm volatile("" ::"v"(ks_pre[0]), "v"(y_pre[0]), "v"(ks_pre[1]), "v"(y_pre[1]));
  if (mcount == 0) return;   // M_l empty: Algorithm 2 is not run for this layer
  // the selector list first (16-byte aligned), then the bucket offsets
  uint16_t *list = reinterpret_cast<uint16_t *>(smem);               // [list_slots(n, gamma)]
  int *bucket = smem + list_slots(p.n, gamma) / 2;                     // [gamma]

  // ---- bucket the selections of group g by perceptron (counting sort) -------
  if (tid == 0) s_sel = 0;
  for (int r = tid; r < gamma; r += kThreads) bucket[r] = 0;
  __syncthreads();
  // U_l: the selections of the patterns in M_l
  int nsel = 0;
#pragma unroll
  for (int q = 0; q < kPre; ++q)
    if (ks_pre[q] >= 0) {
      atomicAdd(&bucket[ks_pre[q]], 1);
      ++nsel;
    }
  for (int mu = tid + kPre * kThreads; mu < n; mu += kThreads) {
    const int ks = upd[mu] ? kcol[mu] : -1;
    if (ks >= 0) {
      atomicAdd(&bucket[ks], 1);
      ++nsel;
    }
  }
  nsel = wave_sum(nsel);
  if (lane == 0 && nsel) atomicAdd(&s_sel, nsel);
  __syncthreads();

  {
    // exclusive prefix sum of the bucket sizes: thread t owns buckets
    // [t ch, t ch + ch); a scan inside each wave, then across the waves
    // (each row's slots padded to a multiple of 8, so that every row
    // starts on a 16-byte boundary)
    const int ch = (gamma + kThreads - 1) / kThreads;
    const int b0 = min(gamma, tid * ch), b1 = min(gamma, b0 + ch);
    int own = 0;
    for (int r = b0; r < b1; ++r) own += round8(bucket[r]);
    int inc = own;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(inc, d, 64);
      if (lane >= d) inc += v;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int run = inc - own;
    for (int w = 0; w < wave; ++w) run += wsum[w];
    for (int r = b0; r < b1; ++r) {
      const int c = bucket[r];
      bucket[r] = run;
      run += round8(c);
    }
  }
  __syncthreads();
  if (!p.sequential) {
    auto fill = [&](int mu, int ks, int y) {
      const int k = U.perm ? U.perm[g * gamma + ks] : g * gamma + ks;
      const int yl = min(max(y, 0), p.c - 1);   // stay inside P on a bad label
      const bool rpos = (U.P[(size_t)yl * U.words_out + (k >> 6)] >> (k & 63)) & 1ull;
      const int pos = atomicAdd(&bucket[ks], 1);
      list[pos] = (uint16_t)(mu | (rpos ? 0 : 0x8000));
    };
#pragma unroll
    for (int q = 0; q < kPre; ++q)
      if (ks_pre[q] >= 0) fill(tid + q * kThreads, ks_pre[q], y_pre[q]);
    for (int mu = tid + kPre * kThreads; mu < p.n; mu += kThreads) {
      const int ks = U.upd[mu] ? kcol[mu] : -1;
      if (ks >= 0) fill(mu, ks, p.y[mu]);
    }
  } else if (wave == 0) {
    // the same lists, each in pattern order: wave 0 walks the patterns 64
    // at a time, and the lanes that share a row take consecutive slots in
    // lane order
    for (int base = 0; base < p.n; base += 64) {
      const int mu = base + lane;
      const int ks = (mu < p.n && U.upd[mu]) ? kcol[mu] : -1;
      uint32_t ent = 0u;
      if (ks >= 0) {
        const int k = U.perm ? U.perm[g * gamma + ks] : g * gamma + ks;
        const int yl = min(max(p.y[mu], 0), p.c - 1);
        const bool rpos = (U.P[(size_t)yl * U.words_out + (k >> 6)] >> (k & 63)) & 1ull;
        ent = (uint32_t)mu | (rpos ? 0u : 0x8000u);
      }
      uint64_t pending = __ballot(ks >= 0);
      while (pending) {
        const int leader = __ffsll((unsigned long long)pending) - 1;
        const int key = __shfl(ks, leader, 64);
        const uint64_t same = __ballot(ks == key) & pending;
        const int start = bucket[key];
        if (lane == leader) bucket[key] = start + __popcll(same);
        if ((same >> lane) & 1ull) list[start + __popcll(same & ((1ull << lane) - 1ull))] = (uint16_t)ent;
        pending &= ~same;
      }
    }
  }
  __syncthreads();
  // bucket[r] is now the end of row r's selectors; row r starts at
  // round8(bucket[r - 1])

  const int B = p.bound;
  const uint32_t t_hi = U.t_hi, t_lo = U.t_lo;
  const int groups_in = (U.k_in + 31) >> 5;   // 32-column groups of a row holding columns
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t *>(U.a32), 0, p.n * U.nw32 * 4, kRawRsrcWord3);
  int nreinf = 0;

  // work items: (row r, 2048-column chunk); lane l owns 32-column group
  // chunk * 64 + l of the row
  // this work-group's rows: [r_lo, r_hi) of the group
  const int r_lo = part * gamma / kSplit, r_hi = (part + 1) * gamma / kSplit;
  const int items = (r_hi - r_lo) * U.chunks;
  for (int it = wave; it < items; it += kWaves) {
    const int r = r_lo + it / U.chunks, chunk = it % U.chunks;
    const int k = U.perm ? U.perm[g * gamma + r] : g * gamma + r;
    const int cw = chunk * 64 + lane;
    const bool on = cw < U.nw32;
    const int cwc = min(cw, U.nw32 - 1);     // clamped: loads stay inside the rows
    const int nvalid = min(max(U.k_in - cw * 32, 0), 32);
    const uint32_t validmask = nvalid == 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
    // the row's selector range is the same for every lane: scalars, so the
    // branches on S are scalar and its constants live in scalar registers
    const int beg = __builtin_amdgcn_readfirstlane(r ? round8(bucket[r - 1]) : 0);
    const int S = __builtin_amdgcn_readfirstlane(bucket[r]) - beg;

    // per-item copies of the uniform constants: what is made from them is
    // made again in each item, in scalar registers, instead of held across
    // the loop
    const uint32_t key0 = opaque(p.key0), key1 = opaque(p.key1);
    const int Bi = (int)opaque((uint32_t)B);
    const uint32_t thi = opaque(t_hi);

    // ---- Clipped-Perceptron sum and clip ------------------------------------
    // the counts first, then the H planes (loaded after the counting, so
    // that they hold no registers during it)
    const bool counted = S > 0 && !p.sequential;
    uint32_t c[kPlanes];
    if (counted) count_row(c, list, beg, S, rs, 4 * U.nw32, 4 * cwc);
    // plane p of the lane's group: word p * h_ps + cwc of the row
    uint32_t *urow = reinterpret_cast<uint32_t *>(U.H + (size_t)k * U.ld_h) + cwc;
    uint32_t u[M];
#pragma unroll
    for (int q = 0; q < M; ++q) u[q] = urow[(size_t)q * U.h_ps];
    if (S > 0 && p.sequential) {
      cp_sequential<M>(u, list, beg, S, Bi, validmask, U.a32, U.nw32, cwc);
    } else if (counted) {
      uint32_t un[M];
#pragma unroll
      for (int q = 0; q < M; ++q) un[q] = u[q];
      if (S <= 63)
        cp_apply<M, 9>(un, c, S, Bi);
      else if (S <= 255)
        cp_apply<M, 10>(un, c, S, Bi);
      else
        cp_apply<M, 17>(un, c, S, Bi);
      // padding columns keep u = 0
#pragma unroll
      for (int q = 0; q < M; ++q) u[q] = (un[q] & validmask) | (u[q] & ~validmask);
    }
    // sign(h) after the Clipped-Perceptron step; reinforcement keeps it
    const uint32_t pos = FULL ? u[M - 1] : at_least<M>(u, (Bi + 1) >> 1);

    // ---- coarse reinforcement draws: plane p of the 32 bytes is word p of
    // Philox blocks 2 (k ceil(K/32) + group) and the one after (stream 3)
    // (drawn after the counting, so that they hold no registers during it) ----
    const uint32_t blk = 2u * ((uint32_t)k * (uint32_t)groups_in + (uint32_t)cwc);
    const U32x4 v0 = philox4x32_10(blk, U.ctr1, p.step, kStreamCoarse, key0, key1);
    const U32x4 v1 = philox4x32_10(blk + 1u, U.ctr1, p.step, kStreamCoarse, key0, key1);

    // ---- which weights reinforce: u8 < T >> 24, or u8 == T >> 24 and the
    // fine 24 bits below T & 0xFFFFFF ---------------------------------------------
    uint32_t fire, need;
    if (thi >= 256u) {
      fire = 0xFFFFFFFFu;
      need = 0u;
    } else {
      const uint32_t rp[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
      uint32_t lt = 0u, eq = 0xFFFFFFFFu;
      // from the top bit: u8 < t_hi or still equal.  Bit q of t_hi is
      // uniform, so each plane takes a scalar branch and one or two
      // bitwise operations instead of three.
#pragma unroll
      for (int q = 7; q >= 0; --q) {
        if ((thi >> q) & 1u) {
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
      const U32x4 f = philox4x32_10(j >> 2, U.ctr1, p.step, kStreamFine, key0, key1);
      if ((pick_word(f, j & 3u) & 0xFFFFFFu) < t_lo) fire |= 1u << e;
    }
    nreinf += __popc(fire);

    // ---- h <- clip(h + 2 sign(h)) on the fired weights, i.e. u <- u + 1 where
    // h > 0 and u - 1 where h < 0; |h| = B (u = 0 or B) stays -------------------
    {
      const uint32_t at_bound = FULL ? (~any_plane<M>(u) | all_planes<M>(u)) : (equals<M>(u, 0) | equals<M>(u, Bi));
      const uint32_t gmask = fire & ~at_bound;
      const uint32_t dn = gmask & ~pos;   // delta -1 = all ones
      uint32_t carry = u[0] & gmask;
      u[0] ^= gmask;
#pragma unroll
      for (int q = 1; q < M; ++q) {
        const uint32_t sum = u[q] ^ dn ^ carry;
        carry = maj(u[q], dn, carry);
        u[q] = sum;
      }
    }

    if (!on) continue;   // lanes past the row took part in the uniform steps only

    // ---- store H and W = sign(H) ----------------------------------------------
    const uint32_t wbits = pos & validmask;
#pragma unroll
    for (int q = 0; q < M; ++q) urow[(size_t)q * U.h_ps] = u[q];
    U.W32[(size_t)k * U.nw32 + cw] = wbits;
  }

  nreinf = wave_sum(nreinf);
  __syncthreads();   // wsum is free again
  if (lane == 0) wsum[wave] = nreinf;
  __syncthreads();
  if (tid == 0) {
    int t = 0;
    for (int w = 0; w < kWaves; ++w) t += wsum[w];
    // |U_l| and the reinforced draws are adjacent 32-bit counts of the
    // layer's stats row: one 64-bit atomic per work-group adds both
    // |U_l| of the group once, from its first work-group
    const uint32_t sel = part == 0 ? (uint32_t)s_sel : 0u;
    const unsigned long long v = (unsigned long long)sel | ((unsigned long long)(uint32_t)t << 32);
    if (v) atomicAdd(reinterpret_cast<unsigned long long *>(U.stats + 2), v);
  }
}

template <int M>
void launch_planes(bool full, dim3 grid, dim3 block, size_t lds, hipStream_t s, const UpdateBatch &b) {
  int b0[kMaxUpdLayers] = {};
  for (int i = 0; i < b.nl; ++i) b0[i] = b.L[i].block0;
#define BMLP_UPD_ARGS b.nl, b0[1], b0[2], b0[3], b0[4], b0[5], b0[6], b0[7], b.L[0].stats, b
  if (full)
    hipLaunchKernelGGL((update_kernel<M, true>), grid, block, lds, s, BMLP_UPD_ARGS);
  else
    hipLaunchKernelGGL((update_kernel<M, false>), grid, block, lds, s, BMLP_UPD_ARGS);
#undef BMLP_UPD_ARGS
}

}  // namespace

size_t update_lds_bytes(int gamma, int n) {
  return (size_t)list_slots(n, gamma) * sizeof(uint16_t) + (size_t)gamma * sizeof(int);
}

hipError_t launch_update(UpdateBatch &b, hipStream_t s) {
  if (b.n <= 0 || b.nl <= 0) return hipSuccess;
  int blocks = 0;
  int gmax = 0;
  static_assert(kMaxUpdLayers == 8, "the kernel's leading arguments name layers 1..7");
  if (b.nl > kMaxUpdLayers) return hipErrorInvalidValue;
  for (int i = 0; i < b.nl; ++i) {
    UpdLayer &u = b.L[i];
    // the kernel finds the stats row of layer i at stats0 + i * BMLP_STATS_STRIDE
    if (u.stats != b.L[0].stats + (size_t)i * BMLP_STATS_STRIDE) return hipErrorInvalidValue;
    u.chunks = (u.nw32 + 63) / 64;
    u.block0 = blocks;
    blocks += u.groups * kSplit;
    gmax = max(gmax, u.gamma);
  }
  const dim3 grid(blocks), block(kThreads);
  const size_t lds = update_lds_bytes(gmax, b.n);
  const bool full = b.bound == (1 << h_planes(b.bound)) - 1;
  switch (h_planes(b.bound)) {
    case 1: launch_planes<1>(full, grid, block, lds, s, b); break;
    case 2: launch_planes<2>(full, grid, block, lds, s, b); break;
    case 3: launch_planes<3>(full, grid, block, lds, s, b); break;
    case 4: launch_planes<4>(full, grid, block, lds, s, b); break;
    case 5: launch_planes<5>(full, grid, block, lds, s, b); break;
    case 6: launch_planes<6>(full, grid, block, lds, s, b); break;
    default: launch_planes<7>(full, grid, block, lds, s, b); break;
  }
  return hipGetLastError();
}

}  // namespace bmlp
