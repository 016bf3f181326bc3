// XNOR-popcount binary GEMM on 32-bit words (the forward contraction of
// Algorithm 1: z = a_{l-1} W_l^T and y_hat = a_l P_l^T).
//
// For ±1 vectors stored as bits (1 = +1) with zero padding past K,
//   dot(u, v) = K - 2 * popcount(u XOR v),
// so each 32-bit word pair costs one v_xor_b32 and one v_bcnt_u32_b32 (which
// also accumulates).  Tiles of both operands are staged through LDS,
// K-major, double buffered; each thread keeps a TM x TN register tile of
// popcount accumulators.
#include "bmlp_internal.h"

namespace bmlp {
namespace {

constexpr int BK = 32;   // 32-bit words per K tile (1024 bits)

struct GemmArgs {
  const uint32_t *A; int lda;    // [M][lda] words
  const uint32_t *B; int ldb;    // [N][ldb] words
  int M, N, kw;                  // kw = ceil(kbits / 32)
  uint32_t tail;                 // valid-bit mask of word kw - 1
  int kbits;
  int ksplit;                    // words per split along K (multiple of BK)
  int16_t *z; int ldz;           // hidden layer: int16 pre-activations (may be null)
  uint64_t *abits; int ld_ab;    // hidden layer: sign bits
  int32_t *out; int ldo;         // classifier: atomically adds -2 * popcount
};

enum { kModeHidden = 0, kModeCls = 1 };

template <int BM, int BN, int TM, int TN, int MODE>
__global__ __launch_bounds__(256) void popc_gemm_kernel(GemmArgs p) {
  static_assert((BM / TM) * (BN / TN) == 256, "256 threads");
  constexpr int NTN = BN / TN;
  constexpr int LA = BM * BK / 256;   // words per thread of the A tile
  constexpr int LB = BN * BK / 256;
  static_assert(LA % 2 == 0 && LB % 2 == 0, "loads are 64-bit");
  __shared__ __align__(16) uint32_t As[2][BK][BM];
  __shared__ __align__(16) uint32_t Bs[2][BK][BN];

  const int tid = threadIdx.x;
  const int tn = tid % NTN, tm = tid / NTN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * p.ksplit;
  const int kend = min(p.kw, kbeg + p.ksplit);
  const int ntiles = (kend - kbeg + BK - 1) / BK;

  const int la_row = tid / (BK / LA), la_k = (tid % (BK / LA)) * LA;
  const int lb_row = tid / (BK / LB), lb_k = (tid % (BK / LB)) * LB;
  uint32_t ra[LA], rb[LB];

  auto gload = [&](int k0) {
    const int gm = m0 + la_row;
#pragma unroll
    for (int q = 0; q < LA; q += 2) {
      const int kk = k0 + la_k + q;   // even: 8-byte aligned (row pitch is even)
      uint2 v = make_uint2(0u, 0u);
      if (gm < p.M && kk < kend) v = *reinterpret_cast<const uint2 *>(p.A + (size_t)gm * p.lda + kk);
      if (kk + 1 >= kend) v.y = 0u;
      if (kk == p.kw - 1) v.x &= p.tail;
      if (kk + 1 == p.kw - 1) v.y &= p.tail;
      ra[q] = v.x;
      ra[q + 1] = v.y;
    }
    const int gn = n0 + lb_row;
#pragma unroll
    for (int q = 0; q < LB; q += 2) {
      const int kk = k0 + lb_k + q;
      uint2 v = make_uint2(0u, 0u);
      if (gn < p.N && kk < kend) v = *reinterpret_cast<const uint2 *>(p.B + (size_t)gn * p.ldb + kk);
      if (kk + 1 >= kend) v.y = 0u;
      if (kk == p.kw - 1) v.x &= p.tail;
      if (kk + 1 == p.kw - 1) v.y &= p.tail;
      rb[q] = v.x;
      rb[q + 1] = v.y;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < LA; ++q) As[buf][la_k + q][la_row] = ra[q];
#pragma unroll
    for (int q = 0; q < LB; ++q) Bs[buf][lb_k + q][lb_row] = rb[q];
  };

  uint32_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = 0u;

  if (ntiles > 0) {
    gload(kbeg);
    sstore(0);
  }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    if (t + 1 < ntiles) gload(kbeg + (t + 1) * BK);
#pragma unroll 4
    for (int k = 0; k < BK; ++k) {
      uint32_t a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; i += 4) {
        const uint4 v = *reinterpret_cast<const uint4 *>(&As[cur][k][tm * TM + i]);
        a[i] = v.x; a[i + 1] = v.y; a[i + 2] = v.z; a[i + 3] = v.w;
      }
      if constexpr (TN % 4 == 0) {
#pragma unroll
        for (int j = 0; j < TN; j += 4) {
          const uint4 v = *reinterpret_cast<const uint4 *>(&Bs[cur][k][tn * TN + j]);
          b[j] = v.x; b[j + 1] = v.y; b[j + 2] = v.z; b[j + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; j += 2) {
          const uint2 v = *reinterpret_cast<const uint2 *>(&Bs[cur][k][tn * TN + j]);
          b[j] = v.x; b[j + 1] = v.y;
        }
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] += __popc(a[i] ^ b[j]);
    }
    if (t + 1 < ntiles) sstore(cur ^ 1);
    __syncthreads();
  }

  if constexpr (MODE == kModeCls) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + tm * TM + i;
      if (m >= p.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + tn * TN + j;
        if (n < p.N && acc[i][j] != 0u) atomicAdd(p.out + (size_t)m * p.ldo + n, -2 * (int)acc[i][j]);
      }
    }
  } else {
    static_assert(MODE != kModeHidden || TN == 8, "one sign byte per thread row");
    // Sign bits go through LDS: byte [row][tn] holds columns tn*8 .. tn*8+7.
    uint8_t *sbytes = reinterpret_cast<uint8_t *>(&As[0][0][0]);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int rl = tm * TM + i;
      const int m = m0 + rl;
      uint32_t byte = 0u;
      int16_t zz[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + tn * TN + j;
        zz[j] = (int16_t)(p.kbits - 2 * (int)acc[i][j]);
        if (n < p.N && zz[j] >= 0) byte |= 1u << j;
      }
      sbytes[rl * (BN / 8) + tn] = (uint8_t)byte;
      if (p.z != nullptr && m < p.M) {
        int16_t *zrow = p.z + (size_t)m * p.ldz + n0 + tn * TN;
        if (n0 + tn * TN + TN <= p.N) {
          uint4 v;
          v.x = (uint16_t)zz[0] | ((uint32_t)(uint16_t)zz[1] << 16);
          v.y = (uint16_t)zz[2] | ((uint32_t)(uint16_t)zz[3] << 16);
          v.z = (uint16_t)zz[4] | ((uint32_t)(uint16_t)zz[5] << 16);
          v.w = (uint16_t)zz[6] | ((uint32_t)(uint16_t)zz[7] << 16);
          *reinterpret_cast<uint4 *>(zrow) = v;
        } else {
#pragma unroll
          for (int j = 0; j < TN; ++j)
            if (n0 + tn * TN + j < p.N) zrow[j] = zz[j];
        }
      }
    }
    __syncthreads();
    constexpr int WPR = BN / 64;   // u64 words of a per tile row
    for (int q = tid; q < BM * WPR; q += 256) {
      const int rl = q / WPR, wl = q % WPR;
      const int m = m0 + rl;
      const int wg = n0 / 64 + wl;
      if (m < p.M && wg < p.ld_ab && wg * 64 < p.N) {
        const uint64_t v = *reinterpret_cast<const uint64_t *>(sbytes + rl * (BN / 8) + wl * 8);
        p.abits[(size_t)m * p.ld_ab + wg] = v;
      }
    }
  }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

GemmArgs base_args(const uint64_t *A, int words_a, int kbits, const uint64_t *B, int M, int N) {
  GemmArgs g{};
  g.A = reinterpret_cast<const uint32_t *>(A);
  g.lda = 2 * words_a;
  g.B = reinterpret_cast<const uint32_t *>(B);
  g.ldb = 2 * words_a;
  g.M = M;
  g.N = N;
  g.kw = cdiv(kbits, 32);
  const int r = kbits & 31;
  g.tail = r == 0 ? 0xFFFFFFFFu : ((1u << r) - 1u);
  g.kbits = kbits;
  g.ksplit = cdiv(g.kw, BK) * BK;
  return g;
}

}  // namespace

hipError_t launch_fwd_popcount(const uint64_t *a_prev, int words_in, int k_in, const uint64_t *W,
                               int n, int k_out, int16_t *z, int ldz, uint64_t *a_out,
                               int words_out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  GemmArgs g = base_args(a_prev, words_in, k_in, W, n, k_out);
  g.z = z;
  g.ldz = ldz;
  g.abits = a_out;
  g.ld_ab = words_out;
  constexpr int BM = 128, BN = 128;
  hipLaunchKernelGGL((popc_gemm_kernel<BM, BN, 8, 8, kModeHidden>), dim3(cdiv(k_out, BN), cdiv(n, BM), 1),
                     dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_cls_popcount(const uint64_t *a, int words, int k, const uint64_t *P, int n, int c,
                               int32_t *out, int ldo, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  GemmArgs g = base_args(a, words, k, P, n, c);
  g.out = out;
  g.ldo = ldo;
  constexpr int BM = 64, BN = 32;
  const int tiles = cdiv(n, BM) * cdiv(c, BN);
  const int ktiles = cdiv(g.kw, BK);
  // split K so that the launch has a few hundred work-groups
  int splits = 1;
  while (splits < ktiles && tiles * splits < 512) ++splits;
  g.ksplit = cdiv(ktiles, splits) * BK;
  splits = cdiv(g.kw, g.ksplit);
  hipLaunchKernelGGL((popc_gemm_kernel<BM, BN, 4, 2, kModeCls>), dim3(cdiv(c, BN), cdiv(n, BM), splits),
                     dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace bmlp
