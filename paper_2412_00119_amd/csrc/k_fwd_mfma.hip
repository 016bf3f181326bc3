// Hidden-layer forward on the matrix cores (Algorithm 1: z = a_{l-1} W_l^T,
// a_l = sign(z)), with the layer-level selection of Algorithm 2 fused into
// the epilogue.
//
// Both operands are ±1 matrices stored as fp4 (see fp4.h), so z is computed
// exactly by v_mfma_scale_f32_16x16x128_f8f6f4 with fp32 accumulation.  A
// work-group computes a 128 x 128 tile of z (patterns x perceptrons) with
// four waves of 64 x 64; K is walked in steps of 128 elements through
// double-buffered LDS tiles.  The epilogue never writes z to memory:
//   * a_l as bit rows (wave ballots) and as fp4 rows for the next layer and
//     the classifier;
//   * for gamma = 64, the easiest wrong perceptron of each group: among the
//     columns k of the group with delta_k = z_k rho^{y}_k < 0, the smallest
//     |z_k|, lowest k on ties (key = |z| << 8 | k, min-reduced across lanes);
//   * for any other gamma, z as int16 for the generic selection kernel.
// Work-groups are mapped so that each XCD (work-group id mod 8) works on
// its own slice of W_l, which then stays in that XCD's L2.
#include "bmlp_internal.h"
#include "fp4.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int TM = 128, TN = 128;   // tile of z
constexpr int KB = 64;              // bytes per row per K step (128 fp4)

__device__ __forceinline__ v4f mfma_fp4(const uint4 &a, const uint4 &b, v4f c) {
  const v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
  const v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
  // operand formats 4 = e2m1 for A and B, unit (E8M0 127) block scales
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 4, 4, 0, 127, 0, 127);
}

__global__ __launch_bounds__(256) void fwd_fp4_kernel(FwdArgs p) {
  __shared__ __align__(16) uint8_t sA[2][TM * KB];
  __shared__ __align__(16) uint8_t sB[2][TN * KB];
  __shared__ uint64_t sP[TM][2];       // rho^{y^mu} bits of the tile's 128 columns

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  int mt, nt;
  {
    const int b = blockIdx.x;
    if (p.xcd_remap) {
      const int x = b & 7, idx = b >> 3, per = p.nt_n >> 3;
      nt = x * per + idx / p.nt_m;
      mt = idx % p.nt_m;
    } else {
      nt = b / p.nt_m;
      mt = b % p.nt_m;
    }
  }
  const int m0 = mt * TM, n0 = nt * TN;

  if (p.mode == kFwdFusedSelect) {
    // the classifier row of each pattern's label, for the tile's columns
    const int r = tid >> 1, w = tid & 1;
    const int m = m0 + r;
    const int wg = (n0 >> 6) + w;
    uint64_t v = 0;
    if (m < p.M && wg < p.words_out) {
      const int yl = min(max(p.y[m], 0), p.c - 1);
      v = p.Pbits[(size_t)yl * p.words_out + wg];
    }
    sP[r][w] = v;
  }

  // loader: 128 rows x 4 chunks of 16 bytes per operand; 2 rows per thread
  const int lrow = tid >> 2, lch = (tid & 3) * 16;
  uint4 ra[2], rb[2];
  auto gload = [&](int ks) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = lrow + 64 * h;
      const int gm = m0 + r, gn = n0 + r;
      ra[h] = gm < p.M ? *reinterpret_cast<const uint4 *>(p.A + (size_t)gm * p.lda + ks * KB + lch)
                       : make_uint4(0, 0, 0, 0);
      rb[h] = gn < p.N ? *reinterpret_cast<const uint4 *>(p.B + (size_t)gn * p.ldb + ks * KB + lch)
                       : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = lrow + 64 * h;
      *reinterpret_cast<uint4 *>(&sA[buf][r * KB + lch]) = ra[h];
      *reinterpret_cast<uint4 *>(&sB[buf][r * KB + lch]) = rb[h];
    }
  };

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  gload(0);
  sstore(0);
  __syncthreads();
  const int arow = lane & 15, achunk = (lane >> 4) * 16;
  for (int ks = 0; ks < p.ksteps; ++ks) {
    const int cur = ks & 1;
    if (ks + 1 < p.ksteps) gload(ks + 1);
    uint4 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] = *reinterpret_cast<const uint4 *>(&sA[cur][(wm * 64 + i * 16 + arow) * KB + achunk]);
      b[i] = *reinterpret_cast<const uint4 *>(&sB[cur][(wn * 64 + i * 16 + arow) * KB + achunk]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma_fp4(a[i], b[j], acc[i][j]);
    if (ks + 1 < p.ksteps) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue ---------------------------------------------------------------
  // lane holds z for column n0 + wn*64 + j*16 + (lane & 15) and rows
  // m0 + wm*64 + i*16 + 4*(lane >> 4) + e, e = 0..3, in acc[i][j][e]
  uint16_t *sbits = reinterpret_cast<uint16_t *>(&sA[0][0]);   // [128 rows][8 chunks of 16 columns]
  const int lg = lane >> 4, lc = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int col = n0 + wn * 64 + j * 16 + lc;
        const uint64_t bal = __ballot(col < p.N && acc[i][j][e] >= 0.f);
        if (lc == 0) {
          const int rl = wm * 64 + i * 16 + 4 * lg + e;
          sbits[rl * 8 + wn * 4 + j] = (uint16_t)(bal >> (16 * lg));
        }
      }

  if (p.mode == kFwdFusedSelect) {
    const int gcol0 = n0 + wn * 64;   // the wave's 64 columns are one group
    if (gcol0 < p.N) {
      const int g = gcol0 >> 6;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rl = wm * 64 + i * 16 + 4 * lg + e;
          const uint64_t rho = sP[rl][wn];
          uint32_t key = 0xFFFFFFFFu;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int kl = j * 16 + lc;              // column within the group
            const int zz = (int)acc[i][j][e];
            const bool rpos = (rho >> kl) & 1ull;
            const bool wrong = rpos ? (zz < 0) : (zz > 0);
            const uint32_t kk = ((uint32_t)(zz < 0 ? -zz : zz) << 8) | (uint32_t)kl;
            key = wrong ? min(key, kk) : key;
          }
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) key = min(key, (uint32_t)__shfl_xor((int)key, off, 64));
          const int m = m0 + rl;
          if (lc == 0 && m < p.M)
            p.kstar[(size_t)g * p.ldk + m] = key == 0xFFFFFFFFu ? (int16_t)-1 : (int16_t)(key & 0xFFu);
        }
    }
  } else if (p.mode == kFwdWriteZ) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + wm * 64 + i * 16 + 4 * lg + e;
          const int col = n0 + wn * 64 + j * 16 + lc;
          if (m < p.M && col < p.N) p.z[(size_t)m * p.ldz + col] = (int16_t)(int)acc[i][j][e];
        }
  }
  __syncthreads();

  // a_l bits: 128 rows x 2 words
  {
    const int r = tid >> 1, w = tid & 1;
    const int m = m0 + r, wg = (n0 >> 6) + w;
    if (m < p.M && wg < p.words_out) {
      const uint64_t v = *reinterpret_cast<const uint64_t *>(&sbits[r * 8 + w * 4]);
      p.abits[(size_t)m * p.words_out + wg] = v;
    }
  }
  // a_l fp4: 128 rows x 64 bytes; a thread converts 64 columns (32 bytes)
  {
    const int r = tid >> 1, h = tid & 1;
    const int m = m0 + r;
    if (m < p.M) {
      const uint64_t bits = *reinterpret_cast<const uint64_t *>(&sbits[r * 8 + h * 4]);
      const int cbase = n0 + h * 64;
      const int nv = min(max(p.N - cbase, 0), 64);
      const uint64_t valid = nv == 64 ? ~0ull : ((1ull << nv) - 1ull);
      uint32_t o[8];
#pragma unroll
      for (int q = 0; q < 8; ++q)
        o[q] = fp4_from_bits8((uint32_t)(bits >> (8 * q)), (uint32_t)(valid >> (8 * q)));
      uint4 *dst = reinterpret_cast<uint4 *>(p.afp4 + (size_t)m * p.ld_af + (cbase >> 1));
      dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
      dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
  }
}

// bit rows [R][words] -> fp4 rows [R][ldq]; one thread per output dword
// (8 columns).  Also zeroes `zero[0..nzero)` (the step statistics).
__global__ __launch_bounds__(256) void fp4_rows_kernel(const uint64_t *__restrict__ bits, int words,
                                                       int K, int R, uint8_t *__restrict__ q, int ldq,
                                                       int32_t *zero, int nzero) {
  const int dw_per_row = ldq >> 2;
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  if (zero != nullptr && t < nzero) zero[t] = 0;
  if (t >= (long long)R * dw_per_row) return;
  const int r = (int)(t / dw_per_row), d = (int)(t % dw_per_row);
  const int c0 = d * 8;                       // first column of this dword
  uint32_t b = 0u, valid = 0u;
  if (c0 < K) {
    const uint64_t w = bits[(size_t)r * words + (c0 >> 6)];
    b = (uint32_t)(w >> (c0 & 63)) & 0xFFu;
    const int nv = min(K - c0, 8);
    valid = (1u << nv) - 1u;
  }
  reinterpret_cast<uint32_t *>(q + (size_t)r * ldq)[d] = fp4_from_bits8(b, valid);
}

}  // namespace

hipError_t launch_fwd_fp4(FwdArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  a.nt_m = (a.M + TM - 1) / TM;
  a.nt_n = (a.N + TN - 1) / TN;
  a.xcd_remap = (a.nt_n % 8 == 0) ? 1 : 0;
  hipLaunchKernelGGL(fwd_fp4_kernel, dim3(a.nt_m * a.nt_n), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fp4_rows(const uint64_t *bits, int words, int K, int R, uint8_t *q, int ldq,
                           int32_t *zero, int nzero, hipStream_t s) {
  const long long total = (long long)R * (ldq >> 2);
  const long long need = total > nzero ? total : nzero;
  if (need <= 0) return hipSuccess;
  hipLaunchKernelGGL(fp4_rows_kernel, dim3((unsigned)((need + 255) / 256)), dim3(256), 0, s, bits, words,
                     K, R, q, ldq, zero, nzero);
  return hipGetLastError();
}

}  // namespace bmlp
