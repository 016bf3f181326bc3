// Hidden-layer forward on the matrix cores (Algorithm 1: z = a_{l-1} W_l^T,
// a_l = sign(z)), with the layer-level selection of Algorithm 2 fused into
// the epilogue.
//
// The operands are the bit rows the rest of the step keeps (bit 1 = +1):
// a_{l-1} (or the input) and W_l, made into OCP e2m1 (fp4) MFMA operands in
// registers by K class (element k is in class k mod 4; see class_bits): the
// sign class as ±1 (0x2 / 0xA), the other three as the bit alone, 0 or a
// power of two, which takes one bit operation per operand word instead of a
// shift and a merge.  The accumulators then hold z_3 + 4 C (C counting the
// elements of classes 0..2 where both bits are 1), and the epilogue adds
// n_low - 2 (P_a + P_w) from per-row popcounts with one fp32 MFMA per
// accumulator, which gives z exactly.  v_mfma_scale_f32_32x32x64_f8f6f4
// multiplies these values exactly and accumulates in fp32, exact below 2^24
// (on gfx950 the 32x32x64 shape runs fp4 at twice the rate of
// 16x16x128).  A wave issues its MFMAs and bit operations one after the
// other, so fewer VALU instructions per MFMA is a shorter K loop.
//
// A work-group computes a 128 x 128 tile of z (patterns x perceptrons) with
// four waves of 64 x 64.  K is walked in steps of 512 elements (64 bytes of
// each bit row) through a ring of kStages LDS buffers filled by
// direct-to-LDS buffer loads (16 bytes per lane, or 4 where rows are not
// 16-byte aligned) three steps ahead of the matrix cores, with one barrier
// per step; a step's operand words are read from LDS one step ahead, in
// between the MFMAs.  Rows past the matrix end are clamped into range; a
// load past the end of a row in the last step reads the next row, or zeros
// past the matrix (the buffer descriptors are sized to the operands): those
// bytes only feed outputs that are never stored, or elements past K, which
// are made fp4 zeros in the W_l operand.  The epilogue never writes z to
// memory:
//   * a_l as bit rows (wave ballots);
//   * for gamma = 64, the easiest wrong perceptron of each group: among the
//     columns k of the group with delta_k = z_k rho^{y}_k < 0, the smallest
//     |z_k|, lowest k on ties (key = |z| << 8 | k, min-reduced across lanes
//     with a butterfly reduce-scatter, so each lane ends with one row);
//   * for any other gamma, z as int16 for the generic selection kernel;
//   * for the local classifier of a layer with many classes (A = a_l, B =
//     P_l), y_hat as int16 or int32, and no sign bits.
// Work-groups are mapped so that each XCD (work-group id mod 8) works on
// its own slice of the larger operand (W_l in a hidden layer, a_l against
// a classifier matrix), which then stays in that XCD's L2.
#include <algorithm>
#include <type_traits>

#include "bmlp_internal.h"
#include "fp4.h"

namespace bmlp {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int TM = 128, TN = 128;   // tile of z
constexpr int KB = 64;              // bytes per row per K step (512 elements)
constexpr int kStages = 4;          // LDS ring depth (kStages - 1 steps in flight)

typedef __attribute__((address_space(3))) void lds_void;

// UNIT (16 or 4) bytes per lane from global memory to LDS at
// dst + UNIT * lane
template <int UNIT>
__device__ __forceinline__ void dma(const void *src, void *dst_wave_base) {
  static_assert(UNIT == 16 || UNIT == 4, "load size");
  if constexpr (UNIT == 16)
    __builtin_amdgcn_global_load_lds(src, (lds_void *)dst_wave_base, 16, 0, 0);
  else
    __builtin_amdgcn_global_load_lds(src, (lds_void *)dst_wave_base, 4, 0, 0);
}

// The same through a buffer descriptor: voff is the lane's byte offset from
// the buffer's base, which the hardware checks against the buffer's size (a
// load past the end reads zeros, no fault).  On this architecture family the
// scalar offset is left out of that check, so every offset goes into voff.
template <int UNIT>
__device__ __forceinline__ void bdma(__amdgpu_buffer_rsrc_t rs, uint32_t voff, void *dst_wave_base) {
  static_assert(UNIT == 16 || UNIT == 4, "load size");
  if constexpr (UNIT == 16)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)dst_wave_base, 16, voff, 0, 0, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)dst_wave_base, 4, voff, 0, 0, 0);
}

// v_writelane_b32: lane `lane` of the result takes the wave-uniform value
// `v`, every other lane keeps `old` (the compiler intrinsic, which this
// clang exposes under its LLVM name only)
extern "C" __device__ uint32_t bmlp_llvm_writelane(uint32_t v, uint32_t lane, uint32_t old)
    __asm("llvm.amdgcn.writelane.i32");
__device__ __forceinline__ uint32_t lane_write(uint32_t old, uint32_t v, int lane) {
  return bmlp_llvm_writelane(v, (uint32_t)lane, old);
}

// wait until at most n vector-memory operations of this wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  // vmcnt in bits 3:0 and 15:14; expcnt (6:4) and lgkmcnt (11:8) at their
  // maxima, i.e. not waited for
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0xF70);
}

// XOR swizzle of the 16-byte unit index within a 64-byte LDS row.  LDS has
// 64 banks of 4 bytes, so a 64-byte row spans a quarter of them, chosen by
// r & 3.  On gfx950 a ds_read_b128 is served in four passes of 16 lanes:
// the lanes that agree in bit 5 and in the parity of bits 2..4 (measured
// with the bank-conflict counter).  The operand reads give lane l row
// (l & 31) of a 32-row block, so a pass holds four rows per value of r & 3,
// whose bits 2..3 take four distinct values; XOR-ing the unit with them
// puts the pass on 64 distinct banks.
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

// lane l: A row / B column (l & 31), half (l >> 5) of the 64-element K
// block; result element i of lane l is row 8*(i>>2) + 4*(l>>5) + (i&3),
// column (l & 31)
// K classes (class_bits): the MFMA of class s over a 256-element chunk takes,
// from each of the lane's four words, the bits of class s in place (nibble t
// of dword d = bit 4t + s of word d); A and B use the same map, so every
// product pairs the same k.  So acc = z_3 + 4 C, and z = acc + n_low -
// 2 (P_a + P_w), where P_a and P_w are the rows' popcounts over classes 0..2
// and n_low = K - floor(K / 4) the class 0..2 elements of a row.  Every
// value is an integer below 2^24: exact in fp32.
__device__ __forceinline__ uint4 class_operand(const uint4 &w, int s) {
  return make_uint4(class_bits(w.x, s), class_bits(w.y, s), class_bits(w.z, s), class_bits(w.w, s));
}

// lane l: A row / B column (l & 31), half (l >> 5) of the 64-element K
// block; result element i of lane l is row 8*(i>>2) + 4*(l>>5) + (i&3),
// column (l & 31)
__device__ __forceinline__ v16f mfma_class(const uint4 &a, const uint4 &b, v16f c, int s) {
  const v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
  const v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
  // operand formats 4 = e2m1 for A and B; E8M0 block scales 2^(2-s) for
  // classes 0..2 (129, 128, 127), 1 for the sign class
  const int sc = class_scale(s);
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, 0, sc, 0, sc);
}

// acc + popcount(x) in one v_bcnt_u32_b32
__device__ __forceinline__ uint32_t bcnt_acc(uint32_t x, uint32_t acc) {
  uint32_t r;
  asm("v_bcnt_u32_b32 %0, %1, %2" : "=v"(r) : "v"(x), "v"(acc));
  return r;
}

// one reduce-scatter step at lane distance D, the partner given by DPP
// control CTRL: rows k + D move into slot k on lanes with bit D set
template <int D, int CTRL>
__device__ __forceinline__ void select_step(uint32_t (&v)[32], int lc) {
  const bool up = (lc & D) != 0;
#pragma unroll
  for (int k = 0; k < D; ++k) {
    const uint32_t send = up ? v[k] : v[k + D];
    const uint32_t keep = up ? v[k + D] : v[k];
    v[k] = min(keep, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)send, CTRL, 0xF, 0xF, false));
  }
}

// UNIT: bytes per lane of the direct-to-LDS loads, 16 when every operand
// row starts on a 16-byte boundary, else 4.  SLICED: the launch covers
// several layers (p.sl); a one-layer launch reads its fields directly, which
// keeps the slice lookup out of its prologue.
//
// The arguments the first loads depend on come first, as separate scalars:
// the leading 16 dwords of a kernel's arguments are preloaded into scalar
// registers when the wave starts (kernarg preloading), so the tile's first
// loads do not wait for a read of the argument buffer.
template <int UNIT, bool SLICED>
__global__ __launch_bounds__(256) void fwd_fp4_kernel(const uint64_t *pA, const uint64_t *pB, const int32_t *py, int pld,
                                                      int pK, int pM, int pN, int pnt_m, int pnt_n, int pxcd,
                                                      int pystride, int pmode, FwdArgs p) {
  // one LDS array per ring slot (A tile, then B tile): every access below
  // names its array, so the compiler can tell a slot being read from the
  // slots the direct-to-LDS loads are still filling (it tells apart at most
  // eight such arrays).  66 KB in all: two work-groups fit on a CU.
  constexpr int kSlot = (TM + TN) * KB;
  __shared__ __align__(16) uint8_t s0[kSlot], s1[kSlot], s2[kSlot], s3[kSlot];
  __shared__ uint64_t sP[2][TM];       // rho^{y^mu} bits of the tile's 128 columns, per group
  __shared__ int32_t sY[TM];           // labels of the tile's rows
  __shared__ uint32_t sPc[TM + TN];    // popcounts P_a (tile rows), then P_w (tile columns)
  static_assert(kStages == 4, "one named array per slot");
  constexpr int kRowsPerDma = 64 * UNIT / KB;     // rows per load instruction: 16 or 4
  constexpr int kDma = 32 / kRowsPerDma;          // instructions per operand per wave and step
  constexpr int kIssue = 2 * kDma;                // loads per wave and step
  static_assert(kIssue * (kStages - 2) < 64, "vmcnt range");

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // the slice (layer) of this work-group, then its tile
  FwdSlice S;   // a copy: kept in scalar registers
  int b = (int)blockIdx.x;
  if constexpr (SLICED) {
    const int tiles = pnt_m * pnt_n;
    const int sli = b / tiles;
    S = p.sl[sli];
    b -= sli * tiles;
  } else {
    S = FwdSlice{pA, pB, pld, pK, p.z, p.z32};
  }
  int mt, nt;
  {
    if (pxcd == 1) {   // XCD x takes the x-th eighth of B's tiles
      const int x = b & 7, idx = b >> 3, per = pnt_n >> 3;
      nt = x * per + idx / pnt_m;
      mt = idx % pnt_m;
    } else if (pxcd == 2) {   // the x-th eighth of A's tiles
      const int x = b & 7, idx = b >> 3, per = pnt_m >> 3;
      mt = x * per + idx / pnt_n;
      nt = idx % pnt_n;
    } else {
      nt = b / pnt_m;
      mt = b % pnt_m;
    }
  }
  const int m0 = mt * TM, n0 = nt * TN;

  // The step statistics start at zero (the first forward of a step zeroes
  // them; the classifiers add to them after every forward is done).
  if (p.zero != nullptr && blockIdx.x == 0)
    for (int i = tid; i < p.nzero; i += 256) p.zero[i] = 0;

  // For the fused selection thread (r, w) needs word w of the tile's
  // columns of rho^{y^mu} = P_l[y^mu] for tile row r (pattern m0 + r).  The
  // labels of the tile's rows come with the first operand loads, as a
  // direct-to-LDS load of wave 0 (a register load among the direct-to-LDS
  // loads would make the compiler wait for all of them before its use), and
  // the word of P_l is loaded once they have landed, to be used after the
  // K loop.  Both loads are unconditional (indices clamped; when the
  // selection is not fused the launcher points them at valid memory).
  const int pr = tid >> 1, pw = tid & 1;
  const int pm = m0 + pr, pwg = (n0 >> 6) + pw;
  const bool pvalid = pmode == kFwdFusedSelect && pm < pM && pwg < p.words_out;

  // Loads: a wave moves rows 32*wave .. 32*wave+31 of each operand.  Lane l
  // of instruction h fills LDS bytes UNIT*l of its kRowsPerDma rows: row
  // r = 32*wave + kRowsPerDma*h + (UNIT*l) / 64, physical 16-byte unit u,
  // which holds logical unit u ^ swz(r) of that row (the XOR swizzle keeps
  // the operand reads conflict-free).  Rows past the matrix are clamped to
  // its last row.  A source past the end of its row (only in the last step)
  // reads the next row's first bytes, elements past K that the last step
  // masks out, or, past the matrix, zeros: the loads go through buffer
  // descriptors sized to the matrices, so that a step costs one add per
  // load and no clamp.
  uint32_t voffA[kDma], voffB[kDma];
  const uint32_t rowbytes = 8u * (uint32_t)S.ld;
#pragma unroll
  for (int h = 0; h < kDma; ++h) {
    const int pos = UNIT * lane;   // byte in the instruction's rows
    const int r = 32 * wave + kRowsPerDma * h + pos / KB;
    const int inrow = pos % KB;
    const uint32_t off = 16 * ((inrow / 16) ^ swz(r)) + inrow % 16;
    voffA[h] = (uint32_t)min(m0 + r, pM - 1) * rowbytes + off;
    voffB[h] = (uint32_t)min(n0 + r, pN - 1) * rowbytes + off;
  }
  const __amdgpu_buffer_rsrc_t rsA =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(S.A), 0, (int)((uint32_t)pM * rowbytes), kRawRsrcWord3);
  const __amdgpu_buffer_rsrc_t rsB =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(S.B), 0, (int)((uint32_t)pN * rowbytes), kRawRsrcWord3);
  auto issue = [&](int ks, uint8_t *d) {
    const uint32_t so = (uint32_t)(ks * KB);
#pragma unroll
    for (int h = 0; h < kDma; ++h) {
      bdma<UNIT>(rsA, voffA[h] + so, d + (kDma * wave + h) * 64 * UNIT);
      bdma<UNIT>(rsB, voffB[h] + so, d + TM * KB + (kDma * wave + h) * 64 * UNIT);
    }
  };

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};

  // operand words of one K step: [c][i] for its two 256-element chunks;
  // lane (r, h) holds elements 256 c + 128 h .. +127 of row r
  struct Ops {
    uint4 a[2][2], b[2][2];
    uint4 bc[2];   // the B fragment this wave counts (fragment wm), per chunk
  };
  const int arow = lane & 31, ahalf = lane >> 5;
  // Register fragment i of a wave's A operands holds tile fragment i ^ wn
  // (rows wm*64 + (i ^ wn)*32 ..): the A fragment a wave counts in the row
  // popcounts below (fragment wn) is then always register fragment 0, with
  // no select per word.  acc[i][j] holds tile rows of fragment i ^ wn.  (The
  // same order for the B fragments by wm measured slower: the compiler then
  // waits for every LDS read early in each K step.)
  const int xa = wn;
  auto read = [&](Ops &o, const uint8_t *t) {
    const uint8_t *tA = t, *tB = t + TM * KB;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int u = 2 * c + ahalf;   // 16-byte unit of the 64-byte row
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ra_ = wm * 64 + (i ^ xa) * 32 + arow, rb_ = wn * 64 + i * 32 + arow;
        o.a[c][i] = *reinterpret_cast<const uint4 *>(&tA[ra_ * KB + ((u ^ swz(ra_)) * 16)]);
        o.b[c][i] = *reinterpret_cast<const uint4 *>(&tB[rb_ * KB + ((u ^ swz(rb_)) * 16)]);
      }
      const int rc_ = wn * 64 + wm * 32 + arow;
      o.bc[c] = *reinterpret_cast<const uint4 *>(&tB[rc_ * KB + ((u ^ swz(rc_)) * 16)]);
    }
  };
  // The expanded operands of one K block (c, q) of a step.  A step's MFMAs
  // take block 0 expanded beforehand (by the step before, or the prologue);
  // while the MFMAs of block b run, the operands of block b + 1 are expanded,
  // and during the last block those of block 0 of the next step, so that the
  // matrix core never waits for an expansion at the start of a step.
  struct Exp {
    uint4 a[2], b[2];
  };
  auto expand = [&](const Ops &o, int c, int cls, Exp &e) {
#pragma unroll
    for (int i = 0; i < 2; ++i) e.a[i] = class_operand(o.a[c][i], cls);
#pragma unroll
    for (int j = 0; j < 2; ++j) e.b[j] = class_operand(o.b[c][j], cls);
  };
  auto compute_pipe = [&](const Ops &o, const Exp &e0, const Ops &onext, Exp &e0next) {
    Exp e = e0;
#pragma unroll
    for (int blk = 0; blk < 8; ++blk) {
      Exp en;
      if (blk < 7)
        expand(o, (blk + 1) >> 2, (blk + 1) & 3, en);
      else
        expand(onext, 0, 0, e0next);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma_class(e.a[i], e.b[j], acc[i][j], blk & 3);
      if (blk < 7) e = en;
    }
  };
  // Row popcounts of classes 0..2 (P_a for the A rows, P_w for the B rows),
  // from operand words the lanes read anyway: wave (wm, wn) counts A
  // fragment wn (its register fragment 0) and B fragment wm (read from LDS
  // a second time, into bc, the choice made in the address: two more LDS
  // reads per step instead of a select per word),
  // so every tile row and column is counted once, lane l over half (l >> 5)
  // of the row.  m[q]: the bits of word q of a chunk that count.
  uint32_t pca = 0u, pcb = 0u;
  // each word's count added straight into the running total: left to
  // itself the compiler counts every word from zero and sums the counts
  // with three-input adds, half an instruction more per word
  auto popc4 = [](uint32_t acc, const uint4 &w, const uint32_t (&m)[4]) {
    acc = bcnt_acc(w.x & m[0], acc);
    acc = bcnt_acc(w.y & m[1], acc);
    acc = bcnt_acc(w.z & m[2], acc);
    return bcnt_acc(w.w & m[3], acc);
  };
  auto popc_ops = [&](const Ops &o, const uint32_t (&m0)[4], const uint32_t (&m1)[4]) {
    pca = popc4(popc4(pca, o.a[0][0], m0), o.a[1][0], m1);
    pcb = popc4(popc4(pcb, o.bc[0], m0), o.bc[1], m1);
  };
  const uint32_t kFull[4] = {kLowClasses, kLowClasses, kLowClasses, kLowClasses};
  // the last step when K is not a multiple of 512: elements past K become
  // fp4 zeros in the W_l operand
  auto compute_tail = [&](const Ops &o, int ks) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      uint32_t valid[4];   // valid bits of the lane's four words of chunk c
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int nv = S.K - (512 * ks + 256 * c + 128 * ahalf + 32 * q);
        valid[q] = nv >= 32 ? 0xFFFFFFFFu : nv <= 0 ? 0u : ((1u << nv) - 1u);
      }
      uint32_t mv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) mv[q] = valid[q] & kLowClasses;
      pca = popc4(pca, o.a[c][0], mv);
      pcb = popc4(pcb, o.bc[c], mv);
#pragma unroll
      for (int cls = 0; cls < 4; ++cls) {
        uint4 ea[2], eb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) ea[i] = class_operand(o.a[c][i], cls);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint4 w = o.b[c][j];
          eb[j] = make_uint4(class_bits_masked(w.x, valid[0], cls), class_bits_masked(w.y, valid[1], cls),
                             class_bits_masked(w.z, valid[2], cls), class_bits_masked(w.w, valid[3], cls));
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma_class(ea[i], eb[j], acc[i][j], cls);
      }
    }
  };



  // Pipeline of step ks: the loads of step ks+3 are issued into the slot of
  // step ks-1, the MFMAs of step ks run on operands read during step ks-1,
  // and the operands of step ks+1 are read from LDS in between the MFMAs, so
  // the reads complete under them.  The slot of step ks-1 is free: its
  // operands fed MFMAs issued before this step's barrier.
  //
  // Every step issues its loads, of step min(ks+3, nks-1): past the end they
  // repeat the last step into slots nobody reads.  So the count of loads in
  // flight is the same at every step and the code has no branches for the
  // compiler's wait-count tracking to merge over (a merge makes it wait for
  // every load before the next LDS read).  A partial last step is computed
  // after the loop.
  const int nks = (S.K + 511) / 512;
  const int nfull = S.K / 512;      // steps with no element past K
  const int klast = nks - 1;        // nks >= 1
  if (wave == 0) {   // labels first: the oldest loads, covered by the prologue's wait
#pragma unroll
    for (int h = 0; h < TM / 64; ++h)
      dma<4>(py + (size_t)min(m0 + 64 * h + lane, pM - 1) * pystride, sY + 64 * h);
  }
  issue(0, s0);
  issue(min(1, klast), s1);
  issue(min(2, klast), s2);
  __builtin_amdgcn_sched_barrier(0);
  Ops r0, r1;
  wait_vm<kIssue * (kStages - 2)>();   // this wave's loads of step 0 (and wave 0's labels) are done
  __builtin_amdgcn_s_barrier();        // every wave's loads of step 0 have landed
  read(r0, s0);
  Exp e0, e1;
  expand(r0, 0, 0, e0);
  const int yl = min(max(sY[pr], 0), p.c - 1);   // stay inside P on a bad label
  const uint64_t prow = p.P[(size_t)yl * p.ldp + min(pwg, p.pw_max)];
  __builtin_amdgcn_sched_barrier(0);
  // The sched_barrier(0) fences pin the order of the phases; otherwise the
  // scheduler sinks the read-ahead to its use and the LDS latency reappears.
  auto step = [&](int ks, Ops &cur, Ops &nxt, const Exp &ecur, Exp &enxt, const uint8_t *rs, uint8_t *ds) {
    __builtin_amdgcn_sched_barrier(0);
    wait_vm<kIssue * (kStages - 3)>();   // step ks+1 landed; ks+2 may still be in flight
    // A plain s_barrier: the fence of __syncthreads would also wait for the
    // loads still in flight for later steps.
    __builtin_amdgcn_s_barrier();
    issue(min(ks + kStages - 1, klast), ds);
    __builtin_amdgcn_sched_barrier(0);
    read(nxt, rs);   // past the last step this reads a slot nobody uses
    compute_pipe(cur, ecur, nxt, enxt);
    // The order of the step's instructions: each MFMA followed by a quarter
    // of the next K block's operands, so that the VALU work runs while the
    // matrix core works on the MFMA; one LDS read after each of the first
    // ten MFMAs (issued before them, the reads would share the wait-count
    // of the operands being consumed).
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      if (i < 10) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);   // VALU
    }
    __builtin_amdgcn_sched_barrier(0);
    popc_ops(cur, kFull, kFull);
  };
  // step ks reads slot (ks+1) % 4 and refills slot (ks+3) % 4
  int ks = 0;
  for (; ks + kStages <= nfull; ks += kStages) {
    step(ks + 0, r0, r1, e0, e1, s1, s3);
    step(ks + 1, r1, r0, e1, e0, s2, s0);
    step(ks + 2, r0, r1, e0, e1, s3, s1);
    step(ks + 3, r1, r0, e1, e0, s0, s2);
  }
  // the last nfull % 4 full steps; r0 then holds the next step's operands
  if (ks < nfull) {
    step(ks + 0, r0, r1, e0, e1, s1, s3);
    if (ks + 1 < nfull) {
      step(ks + 1, r1, r0, e1, e0, s2, s0);
      if (ks + 2 < nfull) {
        step(ks + 2, r0, r1, e0, e1, s3, s1);
        r0 = r1;
      }
    } else {
      r0 = r1;
    }
  }
  if (nfull < nks) compute_tail(r0, nfull);

  // ---- epilogue ---------------------------------------------------------------
  // The row popcounts and the rho words reach every wave through LDS.  A
  // plain barrier after the LDS writes: a __syncthreads fence would also
  // wait for the repeated loads of the last steps, which land during the
  // epilogue instead (and are waited for before the wave ends).
  {
    // the two halves of each row (lanes l and l + 32)
    const uint32_t ta = pca + (uint32_t)__shfl_xor((int)pca, 32, 64);
    const uint32_t tb = pcb + (uint32_t)__shfl_xor((int)pcb, 32, 64);
    if (lane < 32) {
      sPc[wm * 64 + wn * 32 + lane] = ta;
      sPc[TM + wn * 64 + wm * 32 + lane] = tb;
    }
  }
  sP[pw][pr] = pvalid ? prow : 0ull;
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0) only
  __builtin_amdgcn_s_barrier();

  // lane holds z for column n0 + wn*64 + j*32 + (lane & 31) and rows
  // m0 + wm*64 + i*32 + 8*(e >> 2) + 4*(lane >> 5) + (e & 3) in acc[i][j][e]
  const int lh = lane >> 5, lc = lane & 31;
  // z = acc + (n_low - 2 P_a[row]) + (-2 P_w[column]): a rank-2 term, added
  // exactly by one fp32 MFMA with K = 2 per accumulator (lane l holds A row
  // (l & 31) at k = l >> 5 and B column (l & 31) at k = l >> 5):
  // A = (n_low - 2 P_a, 1), B = (1, -2 P_w)
  {
    const float nlow = (float)(S.K - S.K / 4);
    float fa[2], fb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
      fa[i] = lh == 0 ? nlow - 2.f * (float)sPc[wm * 64 + (i ^ xa) * 32 + lc] : 1.f;
#pragma unroll
    for (int j = 0; j < 2; ++j)
      fb[j] = lh == 0 ? 1.f : -2.f * (float)sPc[TM + wn * 64 + j * 32 + lc];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i], fb[j], acc[i][j], 0, 0, 0);
  }
  // a_l = sign(z): the ballot of (i, j, e) holds the signs of 32 columns
  // (half j of the wave's 64) of two rows (lanes 0-31 and 32-63).  Ballot
  // k = 16 (2i + j) + e is moved to lane k, which then writes both rows' 32
  // bits: no LDS round trip, two stores per lane.
  uint32_t blo = 0u, bhi = 0u;
  uint64_t colok[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) colok[j] = __ballot(n0 + wn * 64 + j * 32 + lc < p.N);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint64_t bal = __ballot(acc[i][j][e] >= 0.f) & colok[j];
        const int k = (2 * i + j) * 16 + e;
        blo = lane_write(blo, (uint32_t)bal, k);
        bhi = lane_write(bhi, (uint32_t)(bal >> 32), k);
      }
  {
    const int i = lane >> 5, j = (lane >> 4) & 1, e = lane & 15;
    const int rl0 = wm * 64 + (i ^ xa) * 32 + 8 * (e >> 2) + (e & 3);   // the lanes-0-31 row; +4 for 32-63
    const int cw = ((n0 + wn * 64) >> 5) + j;                      // 32-bit word of the 32 columns
    uint32_t *ab32 = reinterpret_cast<uint32_t *>(p.abits);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int m = m0 + rl0 + 4 * h;
      // columns past N are 0 in the ballot
      if (m < p.M && cw < 2 * p.words_out) ab32[(size_t)m * 2 * p.words_out + cw] = h ? bhi : blo;
    }
  }

  if (p.mode == kFwdFusedSelect) {
    const int gcol0 = n0 + wn * 64;   // the wave's 64 columns are one group
    if (gcol0 < p.N) {
      const int g = gcol0 >> 6;
      // Key of each of the lane's 32 rows q = 16*i + e over its 2 columns,
      // formed on the bits of the exact fp32 z: with s = -z where the
      // classifier weight is +1 and s = z where it is -1, perceptron k is
      // wrong iff s >= 1.  s is an integer with |s| <= K_{l-1} <= 32767, so
      // the low 8 bits of bits(s) are zero, and key = bits(s) - bits(1.0f) +
      // k (mod 2^32) is below 2^27 exactly for the wrong perceptrons, in
      // the order (|z|, k); every right one (s = +0 wraps, s = -0 and s < 0
      // have the sign bit) gets a key of at least 2^30.
      const uint32_t sh = 31u - (uint32_t)lc;
      uint32_t v[32];
      // z as the selection sees it: clipped only where [zlo, zhi] is
      // narrower than every |z| <= 32767 (the saturating variant)
      auto keys = [&](auto clip_tag) {
        constexpr bool kClip = decltype(clip_tag)::value;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int rl = wm * 64 + (i ^ xa) * 32 + 8 * (e >> 2) + 4 * lh + (e & 3);
            const uint64_t rho = sP[wn][rl];
            uint32_t key[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const uint32_t r = (uint32_t)(rho >> (32 * j)) << sh;   // bit 31: rho of column j*32 + lc
              const float zc = kClip ? fminf(fmaxf(acc[i][j][e], p.zlo), p.zhi) : acc[i][j][e];
              const float sz = __uint_as_float(__float_as_uint(zc) ^ (r & 0x80000000u));
              key[j] = __float_as_uint(sz) + ((uint32_t)(j * 32 + lc) - 0x3F800000u);
            }
            v[i * 16 + e] = min(key[0], key[1]);
          }
      };
      if (p.zlo > -32767.f || p.zhi < 32767.f)
        keys(std::true_type{});
      else
        keys(std::false_type{});
      // Reduce-scatter over the 32 lanes of a half-wave: at each step a lane
      // keeps half of its rows (the upper half if the step's lane bit is
      // set) and takes the minimum with a partner's copy of those rows.
      // Lane bit 4: v_permlane16_swap trades the odd 16-lane rows of its
      // first operand for the even rows of its second, which leaves each
      // lane its own and its partner's copy of the rows it keeps.  Bits 3..0:
      // DPP row_mirror, row_half_mirror and two quad permutations, each of
      // which pairs a lane with one that differs in that bit.  Afterwards
      // lane lc holds the minimum over all 64 columns of row q = lc.
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const auto sw = __builtin_amdgcn_permlane16_swap(v[k], v[k + 16], false, false);
        v[k] = min((uint32_t)sw[0], (uint32_t)sw[1]);
      }
      select_step<8, 0x140>(v, lc);   // row_mirror: lane i <-> 15 - i
      select_step<4, 0x141>(v, lc);   // row_half_mirror: lane i <-> 7 - i
      select_step<2, 0x4E>(v, lc);    // quad_perm [2,3,0,1]
      select_step<1, 0xB1>(v, lc);    // quad_perm [1,0,3,2]
      const int i = lc >> 4, e = lc & 15;
      const int rl = wm * 64 + (i ^ xa) * 32 + 8 * (e >> 2) + 4 * lh + (e & 3);
      const int m = m0 + rl;
      if (m < p.M) p.kstar[(size_t)g * p.ldk + m] = (v[0] >= (1u << 27)) ? (int16_t)-1 : (int16_t)(v[0] & 0x3Fu);
    }
  } else if (p.mode == kFwdWriteZ || p.mode == kFwdWriteZ32) {
    const bool wide = p.mode == kFwdWriteZ32;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0 + wm * 64 + (i ^ xa) * 32 + 8 * (e >> 2) + 4 * lh + (e & 3);
          const int col = n0 + wn * 64 + j * 32 + lc;
          if (m < p.M && col < p.N) {
            const size_t o = (size_t)m * p.ldz + col;
            if (wide)
              S.z32[o] = (int)acc[i][j][e];
            else
              S.z[o] = (int16_t)(int)acc[i][j][e];
          }
        }
  }
  wait_vm<0>();   // the repeated loads write LDS: they land before the wave ends
}

}  // namespace

hipError_t launch_fwd_fp4(FwdArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const bool sliced = a.nslices > 1;
  if (!sliced) {   // one layer: its fields (checked as slice 0)
    if (a.lda != a.ldb) return hipErrorInvalidValue;
    a.nslices = 1;
    a.sl[0] = FwdSlice{a.A, a.B, a.lda, a.K, a.z, a.z32};
  } else if (a.nslices > kMaxFwdSlices || (a.mode != kFwdWriteZ && a.mode != kFwdWriteZ32)) {
    return hipErrorInvalidValue;
  }
  const bool zout = a.mode == kFwdWriteZ || a.mode == kFwdWriteZ32;
  if (a.N < 1 || (zout && a.ldz < a.N)) return hipErrorInvalidValue;
  if (a.words_out > 0 && a.abits == nullptr) return hipErrorInvalidValue;
  bool aligned = true;
  double bytes_a = 0.0, bytes_b = 0.0;
  for (int i = 0; i < a.nslices; ++i) {
    const FwdSlice &q = a.sl[i];
    if (q.A == nullptr || q.B == nullptr || q.K < 1 || q.ld < (q.K + 63) / 64) return hipErrorInvalidValue;
    if ((a.mode == kFwdWriteZ && q.z == nullptr) || (a.mode == kFwdWriteZ32 && q.z32 == nullptr))
      return hipErrorInvalidValue;
    // rows start on 16-byte boundaries when the bases are 16-byte aligned
    // and the stride is an even number of words
    aligned = aligned && q.ld % 2 == 0 && (reinterpret_cast<uintptr_t>(q.A) & 15) == 0 &&
              (reinterpret_cast<uintptr_t>(q.B) & 15) == 0;
    // the kernel's buffer descriptors hold each operand's size in bytes as a
    // 32-bit signed count
    if ((int64_t)a.M * q.ld * 8 > INT32_MAX || (int64_t)a.N * q.ld * 8 > INT32_MAX) return hipErrorInvalidValue;
    bytes_a += (double)a.M * q.ld;
    bytes_b += (double)a.N * q.ld;
  }
  a.nt_m = (a.M + TM - 1) / TM;
  a.nt_n = (a.N + TN - 1) / TN;
  // each XCD keeps its slice of the larger operand in its own L2 (W_l in a
  // hidden layer; a_l when B is a narrow classifier matrix P_l)
  if (a.nt_m % 8 == 0 && bytes_a > bytes_b)
    a.xcd_remap = 2;
  else
    a.xcd_remap = (a.nt_n % 8 == 0) ? 1 : 0;
  if (a.mode == kFwdFusedSelect) {
    if (a.y == nullptr || a.P == nullptr || a.c < 1) return hipErrorInvalidValue;
    a.pw_max = a.words_out - 1;
    a.ystride = 1;
  } else {   // the label and rho loads read slice 0's A instead (always valid)
    a.y = reinterpret_cast<const int32_t *>(a.sl[0].A);
    a.ystride = 0;
    a.P = a.sl[0].A;
    a.ldp = 0;
    a.c = 1;
    a.pw_max = 0;
  }
  const dim3 grid(a.nslices * a.nt_m * a.nt_n);
  const FwdSlice &s0 = a.sl[0];
#define BMLP_FWD_ARGS s0.A, s0.B, a.y, s0.ld, s0.K, a.M, a.N, a.nt_m, a.nt_n, a.xcd_remap, a.ystride, a.mode, a
  if (aligned && sliced)
    hipLaunchKernelGGL((fwd_fp4_kernel<16, true>), grid, dim3(256), 0, s, BMLP_FWD_ARGS);
  else if (aligned)
    hipLaunchKernelGGL((fwd_fp4_kernel<16, false>), grid, dim3(256), 0, s, BMLP_FWD_ARGS);
  else if (sliced)
    hipLaunchKernelGGL((fwd_fp4_kernel<4, true>), grid, dim3(256), 0, s, BMLP_FWD_ARGS);
  else
    hipLaunchKernelGGL((fwd_fp4_kernel<4, false>), grid, dim3(256), 0, s, BMLP_FWD_ARGS);
#undef BMLP_FWD_ARGS
  return hipGetLastError();
}

}  // namespace bmlp
