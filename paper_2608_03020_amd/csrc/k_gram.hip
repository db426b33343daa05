// k_gram.hip -- streaming statistics of one micro-batch (rows a3, a4 of the step).
//
// Eq. 9 / Section S7 with the identity projection: S += X^T X and the
// factored cross statistic K += -eta_bar X^T Y (Z = X^T T = K B~), where the
// micro-batch's eta_bar (Eq. 10) needs ||X||_F^2, taken from the diagonal of
// this micro-batch's own Gram tiles.
//
// bf16 mode: X is bf16, token-major (n x d).  Both MFMA operands of X^T X need
// 8 consecutive tokens per lane, i.e. the strided direction of X.  Tiles of X
// are copied to LDS in their natural [token][column] layout with 16-byte
// loads/stores and read back transposed with ds_read_b64_tr_b16, which feeds
// v_mfma_f32_32x32x16_bf16 directly.  Only tiles on or above the diagonal of S
// are computed.  Y (fp32) enters the cross product as two bf16 columns
// (hi = bf16(y), lo = bf16(y - hi)), so products stay exact and the sum of the
// two halves carries ~16 bits of y.  Every output element is owned by one
// workgroup and summed in a fixed order: results are deterministic.  With the
// overwrite flag (keep == 0 in the kernels; the first micro-batch of a step) S and K
// take this micro-batch's statistics without their old contents being read, which
// spares the caller a clearing pass over S and this call one read of it.
//
// Statistic weights a_t (Section S7's weighted form, S = X^T diag(a) X): in bf16 mode
// the second operand of every Gram product is scaled in registers, a_t x_tj as a
// float, and enters the matrix cores as two bf16 parts hi + lo (about 16 significant
// bits), so the weighted call does twice the MFMA work; the first operand stays the
// exact bf16 X.  The result is symmetric up to that rounding and only its upper
// triangle is formed, as without weights.
//
// fp32 mode: X is fp32 and the statistics are fp64 (v_mfma_f64_16x16x4f64).
#include <algorithm>
#include <cmath>

#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kThreads = 256;
constexpr int kBK = 32;  // tokens per pipeline stage (bf16)

// upper-triangular tile index -> (I, J), J >= I, T tiles per side
LOCA_DEV void upper_tile(int u, int T, int& I, int& J) {
  int i = 0;
  while (u >= T - i) { u -= T - i; ++i; }
  I = i;
  J = i + u;
}

// ------------------------------------------------------------------ statistic weights (bf16 mode)

// A Gram operand of lane l holds 8 consecutive tokens ks + 8 (l / 32) + e, e = 0..7, of
// one column.  weight_split scales them by the lanes' weights and splits each float
// product into bf16 hi and lo parts.
LOCA_DEV void weight_split(bf16x8_t b, const float (&w)[8], bf16x8_t& hi, bf16x8_t& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float f = (float)b[e] * w[e];
    const __bf16 h = (__bf16)f;  // round to nearest even
    hi[e] = h;
    lo[e] = (__bf16)(f - (float)h);
  }
}

typedef int32_t i32x16_t __attribute__((ext_vector_type(16)));
// Sixteen consecutive floats at the wave-uniform address p into scalar registers,
// asynchronously: sload_wait must run before the values are used.
LOCA_DEV i32x16_t sload16(const float* p) {
  i32x16_t v;
  asm volatile("s_load_dwordx16 %0, %1, 0x0" : "=s"(v) : "s"(p));
  return v;
}
// Waits for the outstanding scalar (and LDS) loads.  The values pass through the
// statement, so no use of them can be scheduled ahead of the wait.
LOCA_DEV void sload_wait(i32x16_t& v) { asm volatile("s_waitcnt lgkmcnt(0)" : "+s"(v)::"memory"); }
// The weights of a lane's 8 operand tokens from those of 16 consecutive tokens, as a
// bit select with a per-lane mask (kept opaque so that it is not rewritten into an
// indexed read of the 16 values).
LOCA_DEV void lane_weights(const i32x16_t& v, int lane, float (&w)[8]) {
  int m = -(lane >> 5);  // 0 for lanes 0..31, all ones for lanes 32..63
  asm("" : "+v"(m));
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e] = __int_as_float((v[e] & ~m) | (v[8 + e] & m));
}

// ------------------------------------------------------------------ bf16 tile staging

// One stage = kBK token rows x BM columns of X starting at column c0, loaded by NT threads
// with 16-byte vector loads (8 columns per chunk) and zero fill outside [0, n) x [0, d).
template <int BM, int NT>
struct XStage {
  static constexpr int kChunksPerRow = BM / 8;
  static constexpr int kChunks = kBK * kChunksPerRow;
  static constexpr int kPerThread = kChunks / NT;
  static_assert(kChunks % NT == 0, "stage must split evenly over the threads");
  uint4 r[kPerThread];

  LOCA_DEV void load(const uint16_t* __restrict__ X, int64_t ldx, int64_t n, int64_t d, int64_t t0,
                     int64_t c0) {
    // full 16-byte chunks: one unconditional vector load from a valid address, then select
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      const int e = threadIdx.x + q * NT;
      const int row = e / kChunksPerRow, ch = e % kChunksPerRow;
      const int64_t t = t0 + row, col = c0 + 8 * ch;
      const bool full = (t < n) && (col + 8 <= d);
      const uint4 v = *(const uint4*)(X + (full ? t * ldx + col : 0));
      r[q] = full ? v : make_uint4(0, 0, 0, 0);
    }
    // the ragged last chunk of each row (only when d % 8 != 0)
    if (d & 7) {
#pragma unroll
      for (int q = 0; q < kPerThread; ++q) {
        const int e = threadIdx.x + q * NT;
        const int row = e / kChunksPerRow, ch = e % kChunksPerRow;
        const int64_t t = t0 + row, col = c0 + 8 * ch;
        if (t < n && col < d && col + 8 > d) {
          const uint16_t* p = X + t * ldx + col;
          uint16_t h[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) h[u] = (col + u < d) ? p[u] : (uint16_t)0;
          r[q].x = h[0] | ((uint32_t)h[1] << 16);
          r[q].y = h[2] | ((uint32_t)h[3] << 16);
          r[q].z = h[4] | ((uint32_t)h[5] << 16);
          r[q].w = h[6] | ((uint32_t)h[7] << 16);
        }
      }
    }
  }
  LOCA_DEV void store(uint16_t* s, int ld) const {
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      const int e = threadIdx.x + q * NT;
      const int row = e / kChunksPerRow, ch = e % kChunksPerRow;
      *(uint4*)(s + row * ld + 8 * ch) = r[q];
    }
  }
};

// ------------------------------------------------------------------ S += X^T X (bf16)

// BM x BM tiles of S on or above the diagonal; WGM x WGN waves, each owning a
// (BM/WGM) x (BM/WGN) block of 32 x 32 MFMA tiles.
// WT: statistic weights from `wpad` (zero past n, readable up to the next multiple of kBK).
template <int BM, int WGM, int WGN, bool WT>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gram_bf16(int64_t n, int64_t d,
                                                             const uint16_t* __restrict__ Xall, int64_t ldx,
                                                             int64_t x_bstride, float* __restrict__ Sall,
                                                             int64_t s_bstride, double* __restrict__ diag_part,
                                                             const float* __restrict__ wpad, int keep) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BM / WGN;
  constexpr int NBM = WM / 32, NBN = WN / 32;
  constexpr int LDT = BM + 16;         // padded row (conflict-free transpose reads)
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][kBK * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][kBK * LDT];
  __shared__ double sred[NT / 64];

  const int T = (int)((d + BM - 1) / BM);
  int I, J;
  upper_tile(blockIdx.x, T, I, J);
  const bool diag = (I == J);
  const int64_t b = blockIdx.y;
  const uint16_t* X = Xall + b * x_bstride;
  float* S = Sall + b * s_bstride;

  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wi = wid / WGN, wj = wid % WGN;
  // a wave tile entirely below the diagonal of a diagonal tile has nothing to do
  const bool active = !(diag && (wj + 1) * WN <= wi * WM);

  f32x16_t acc[NBM][NBN];
#pragma unroll
  for (int m = 0; m < NBM; ++m)
#pragma unroll
    for (int q = 0; q < NBN; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][q][r] = 0.f;

  XStage<BM, NT> ra, rb;
  const int64_t cI = (int64_t)I * BM, cJ = (int64_t)J * BM;
  const int nk = (int)((n + kBK - 1) / kBK);
  ra.load(X, ldx, n, d, 0, cI);
  if (!diag) rb.load(X, ldx, n, d, 0, cJ);
  ra.store(sA[0], LDT);
  if (!diag) rb.store(sB[0], LDT);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      ra.load(X, ldx, n, d, (int64_t)(kt + 1) * kBK, cI);
      if (!diag) rb.load(X, ldx, n, d, (int64_t)(kt + 1) * kBK, cJ);
    }
    if (active) {
      const uint16_t* tA = sA[cur];
      const uint16_t* tB = diag ? sA[cur] : sB[cur];
#pragma unroll
      for (int ks = 0; ks < kBK; ks += 16) {
        bf16x8_t fb[NBN], fl[NBN];
#pragma unroll
        for (int q = 0; q < NBN; ++q) fb[q] = frag32_tr(tB, LDT, wj * WN + 32 * q, ks, lane);
        if (WT) {
          const float* wl = wpad + (int64_t)kt * kBK + ks + 8 * (lane >> 5);
          const float4 w0 = *(const float4*)wl, w1 = *(const float4*)(wl + 4);
          const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
          for (int q = 0; q < NBN; ++q) weight_split(fb[q], wv, fb[q], fl[q]);
        }
#pragma unroll
        for (int m = 0; m < NBM; ++m) {
          const bf16x8_t fa = frag32_tr(tA, LDT, wi * WM + 32 * m, ks, lane);
#pragma unroll
          for (int q = 0; q < NBN; ++q) acc[m][q] = mfma32(fa, fb[q], acc[m][q]);
          if (WT)
#pragma unroll
            for (int q = 0; q < NBN; ++q) acc[m][q] = mfma32(fa, fl[q], acc[m][q]);
        }
      }
    }
    if (kt + 1 < nk) {
      ra.store(sA[cur ^ 1], LDT);
      if (!diag) rb.store(sB[cur ^ 1], LDT);
    }
    __syncthreads();
  }

  double dsum = 0.0;
  if (active) {
#pragma unroll
    for (int m = 0; m < NBM; ++m)
#pragma unroll
      for (int q = 0; q < NBN; ++q) {
        // read the 16 old values of this MFMA block together, then add and store
        float old[16];
        int64_t idx[16];
        bool ok[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = cI + wi * WM + 32 * m + mfma32_row(lane, r);
          const int64_t col = cJ + wj * WN + 32 * q + mfma32_col(lane);
          ok[r] = row < d && col < d;
          idx[r] = row * d + col;
          old[r] = ld_or_zero(S, idx[r], keep && ok[r]);
          if (diag && ok[r] && row == col) dsum += (double)acc[m][q][r];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (ok[r]) S[idx[r]] = old[r] + acc[m][q][r];
      }
  }
  if (diag) {
    const double tot = block_sum(dsum, sred);
    if (threadIdx.x == 0) diag_part[b * T + I] = tot;
  }
}

// ------------------------------------------------------------------ S += X^T X, direct-to-LDS pipeline

// Same tiles and waves as k_gram_bf16, fed by global_load_lds_dwordx4: each lane's
// 16-byte chunk goes straight from HBM/L2 into LDS, so a 4-stage ring can run three
// stages ahead without holding anything in registers.  A stage is 32 tokens x 256
// columns of a panel (16 KB, rows of 512 B).  A wave's load instruction fills 1 KB of
// consecutive LDS, so the conflict-free layout for the transpose reads comes from an
// XOR swizzle of the 16-byte chunks instead of padding: chunk c of row r sits at
// c ^ 4(r & 3), so the four rows x four chunks that half a wave reads in one LDS
// cycle land on 16 distinct chunk positions (all 64 banks).  Rows past n and columns past d are read from a zeroed 16-byte area of the
// workspace.  Requires d % 8 == 0.
constexpr int kDLStages = 4;
constexpr int kDLRowBytes = 512;

// WGM x WGN waves of (256 / WGM) x (256 / WGN) columns each: 2 x 4 waves (two per SIMD)
// or 2 x 2 waves of 128 x 128 (one per SIMD, a third fewer LDS reads per MFMA).
//
// Cross statistic in the same launch (Yhl != nullptr): a diagonal tile needs one panel
// only, so its second ring panel carries the split target rows Yhl = [Y_hi | Y_lo | 0]
// (n x w2p bf16 per block, w2p = 2k rounded up to 8 <= 64) instead of a second copy of
// its panel, and its two waves that lie below the diagonal (no Gram output) form
// Kraw = X_I^T [Y_hi | Y_lo] for the panel's 256 columns, 128 each.
//
// Cross tiles (ncross > 0, for split targets wider than the fused path's 64 columns): the
// launch has ncross = T extra tiles per block after its Gram tiles, tile T(T+1)/2 + I being
// row panel I of X against the split targets: an off-diagonal tile whose second ring panel
// comes from Yhl (columns past w2p read as zero, so the waves wholly past them multiply
// zeros) and whose result is Kraw = X_I^T [Y_hi | Y_lo] (columns < w2).
//
// WT: statistic weights, padded in `wpad` (zero past n, readable up to kBK floats past
// the last stage).  The second operand (X_J, or the split targets of a cross wave) is
// scaled and split in registers, and each row of MFMAs runs on both parts.  The split
// of a half stage's operands runs in the middle of the other half's MFMA rows, so that
// its vector work overlaps them; the weights reach scalar registers a quarter stage
// before that.
template <int WGM, int WGN, bool BUF, bool WT>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gram_bf16_dl(int64_t n, int64_t d, const uint16_t* __restrict__ Xall,
                                                                int64_t ldx, int64_t x_bstride, float* __restrict__ Sall,
                                                                int64_t s_bstride, double* __restrict__ diag_part,
                                                                const uint16_t* __restrict__ zero16, int64_t b0,
                                                                const uint16_t* __restrict__ Yhl_all, int64_t w2,
                                                                int64_t w2p, float* __restrict__ Kraw_all,
                                                                const float* __restrict__ wpad, int ncross, int run,
                                                                int per, int gx, int nblk, int keep) {
  constexpr int BM = 256, NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BM / WGN, NBM = WM / 32, NBN = WN / 32;
  constexpr int TILE_ELEMS = kBK * BM;            // one panel stage (bf16 elements)
  constexpr int NQ = TILE_ELEMS * 2 / 16 / NT;    // 16-byte copies per thread per panel
  constexpr int NCP = 2 * NQ;                     // copies per thread per stage
  constexpr int NSLOT = 2 * NBM;                  // fragment rows of MFMAs per stage
  static_assert(NCP <= NSLOT, "at most one copy between two fragment rows");
  // one LDS object per ring slot: the loop below touches each through a static name,
  // so the in-flight loads into one slot are not mistaken for writes to the slot read
  __shared__ __attribute__((aligned(1024))) uint16_t sb0[2 * TILE_ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sb1[2 * TILE_ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sb2[2 * TILE_ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sb3[2 * TILE_ELEMS];
  __shared__ double sred[NT / 64];
  static_assert(kDLStages == 4, "the ring below is written out for four slots");

  const int T = (int)((d + BM - 1) / BM);
  const int ntile = T * (T + 1) / 2, ntot = ntile + ncross;
  // Tile order.  per == 0: the XCD-aware order over all blocks of the launch (each XCD runs
  // its own run of blocks).  per > 0: the XCDs form 8 / gx groups of gx, each block is cut
  // into gx runs (run tiles each, the last one the rest, at most per), and XCD x takes run
  // x % gx of every (8 / gx)-th block, from block x / gx on, in slots of per (the slots past
  // a run, or past the last block, exit): the XCDs of a group work on the same block at the
  // same time, so that the blocks in flight, 8 / gx of them, keep their X in the last-level
  // cache and read it from HBM about once; taken when a run still fills most of an XCD's 32
  // compute units.
  int logical;
  if (per > 0) {
    const int L = (int)blockIdx.x, x = L & 7, i = L >> 3;
    const int xs = x % gx, u = i % per;
    const int t = xs * run + u;
    const int blk = (i / per) * (8 / gx) + x / gx;
    if ((xs < gx - 1 && u >= run) || t >= ntot || blk >= nblk) return;
    logical = blk * ntot + t;
  } else {
    logical = xcd_logical((int)blockIdx.x, (int)gridDim.x);
  }
  const int tl = logical % ntot;
  const bool ctile = tl >= ntile;  // a cross tile: row panel tl - ntile against the split targets
  int I, J;
  if (ctile) {
    I = tl - ntile;
    J = -1;
  } else {
    upper_tile_banded(tl, T, I, J);
  }
  const bool diag = (I == J);
  const int64_t b = b0 + logical / ntot;
  const uint16_t* X = Xall + b * x_bstride;
  float* S = Sall + b * s_bstride;
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);  // uniform
  int wi = wid / WGN, wj = wid % WGN;
  // The waves of a cross tile whose columns lie wholly past the split targets' w2p would
  // multiply zeros: they take the last wave slots and skip their fragments and products, so
  // that with at most two column blocks of targets each SIMD (waves w and w + 4) holds one
  // wave with products.  (The waves of a diagonal tile below its diagonal keep computing:
  // skipping their products made the c5 call about 1% slower.)
  const int ncb = (int)((w2p + WN - 1) / WN);
  if (WGM == 2 && WGN == 4 && ctile && ncb < WGN) {
    if (wid < 2 * ncb) {
      wi = wid / ncb;
      wj = wid % ncb;
    } else {
      const int u = wid - 2 * ncb, ni = WGN - ncb;
      wi = u / ni;
      wj = ncb + u % ni;
    }
  }
  const bool mm_on = !(ctile && wj * WN >= w2p);
  const bool active = !(diag && (wj + 1) * WN <= wi * WM);
  const bool fuse = diag && Yhl_all != nullptr && ncross == 0;  // this tile also forms the cross statistic
  const bool cross = fuse && !active && WGM == 2 && wj < 2;     // ... in this wave
  const bool ysec = fuse || ctile;                              // the second ring panel holds Yhl
  const uint16_t* Yhl = ysec ? Yhl_all + b * n * w2p : zero16;
  const int64_t cI = (int64_t)I * BM, cJ = (int64_t)J * BM;
  const int nk = (int)((n + kBK - 1) / kBK);
  // fragment sources: Gram waves of a diagonal tile read both operands from the first
  // panel; cross waves take rows 128 wj.. of the panel and the split targets
  const int arow0 = cross ? 128 * wj : wi * WM;
  const int bcol0 = cross ? 0 : wj * WN;
  const int boff = (diag && !cross) ? 0 : TILE_ELEMS;

  // per-thread source chunks: copy q of wave w fills LDS chunks (NQ w + q) * 64 + lane
  int lrow[NQ], lcol[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int slot = (NQ * wid + q) * 64 + lane;
    lrow[q] = slot >> 5;
    lcol[q] = 8 * ((slot & 31) ^ dl_swz(slot >> 5));
  }
  // Copy j (0 .. NCP-1) of a stage: panel j / NQ (a diagonal tile loads its panel twice), chunk j % NQ.
  // buffer path: one resource for the block's X, one for its split targets
  const i32x4_t rsX = buffer_rsrc(X, (uint32_t)(n * ldx * 2));
  const i32x4_t rsY = buffer_rsrc(Yhl, ysec ? (uint32_t)(n * w2p * 2) : 0u);
  auto issue = [&](uint16_t* buf, int kt, int j) {
    const int pnl = j / NQ, q = j % NQ;
    const int64_t t = (int64_t)kt * kBK + lrow[q], col = (pnl == 0 ? cI : cJ) + lcol[q];
    const bool ysrc = ysec && pnl == 1;
    if (BUF) {
      const bool ok = t < n && (ysrc ? lcol[q] < w2p : col < d);
      const uint32_t off = ok ? (uint32_t)(2 * (ysrc ? t * w2p + lcol[q] : t * ldx + col)) : kBufOutside;
      const uint32_t dst = (uint32_t)(uintptr_t)(LOCA_LDS void*)buf + pnl * TILE_ELEMS * 2 + (NQ * wid + q) * 1024;
      lds_dma16_buf(off, ysrc ? rsY : rsX, __builtin_amdgcn_readfirstlane(dst));
      return;
    }
    // both addresses are formed and one selected, without a branch
    const uint64_t in_x = ysrc ? (uint64_t)(uintptr_t)Yhl + 2 * (uint64_t)(t * w2p + lcol[q])
                               : (uint64_t)(uintptr_t)X + 2 * (uint64_t)(t * ldx + col);
    const bool ok = t < n && (ysrc ? lcol[q] < w2p : col < d);
    const uint64_t src = ok ? in_x : (uint64_t)(uintptr_t)zero16;
    const uint32_t dst = (uint32_t)(uintptr_t)(LOCA_LDS void*)buf + pnl * TILE_ELEMS * 2 + (NQ * wid + q) * 1024;
    lds_dma16((const void*)(uintptr_t)src, __builtin_amdgcn_readfirstlane(dst));
  };

  f32x16_t acc[NBM][NBN];
#pragma unroll
  for (int m = 0; m < NBM; ++m)
#pragma unroll
    for (int q = 0; q < NBN; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][q][r] = 0.f;

  // Fragments are double-buffered in registers across the two 16-token halves of a
  // stage and across stages: the operands of the next half (or of the next stage's
  // first half) are read from LDS while the MFMAs of the current half run.  Reading
  // stage kt + 1 during stage kt needs it landed too, so each step waits until at most
  // one stage of copies is in flight and refills the slot of kt + 3.
  // The copies of a step are spread between its rows of MFMAs: a wave issues in order,
  // and copies issued back to back would queue at the address unit and hold up the
  // MFMAs behind them.  Every wave runs the same instruction stream (waves of a
  // diagonal tile below its diagonal compute too and only skip the write-back; the
  // cross-tile waves past the targets skip fragments and products on a branch that is
  // uniform in the wave), so the loop has no divergent branches.
  bf16x8_t fa0[NBM], fb0[NBN], fa1[NBM], fb1[NBN], fl0[NBN], fl1[NBN];
  auto load_frags = [&](const uint16_t* buf, int ks, bf16x8_t (&fa)[NBM], bf16x8_t (&fb)[NBN]) {
#pragma unroll
    for (int q = 0; q < NBN; ++q) fb[q] = frag32_tr_swz(buf + boff, bcol0 + 32 * q, ks, lane);
#pragma unroll
    for (int m = 0; m < NBM; ++m) fa[m] = frag32_tr_swz(buf, arow0 + 32 * m, ks, lane);
  };
  auto mma_row = [&](const bf16x8_t (&fa)[NBM], const bf16x8_t (&fb)[NBN], const bf16x8_t (&fl)[NBN], int m) {
#pragma unroll
    for (int q = 0; q < NBN; ++q) acc[m][q] = mfma32(fa[m], fb[q], acc[m][q]);
    if (WT)
#pragma unroll
      for (int q = 0; q < NBN; ++q) acc[m][q] = mfma32(fa[m], fl[q], acc[m][q]);
  };
  i32x16_t wsc;
  if (WT) wsc = sload16(wpad);  // stage 0, first half
  // scale and split the second operands with the weights loaded one half stage ago,
  // and start the load of the next half stage's weights
  auto weigh = [&](bf16x8_t (&fb)[NBN], bf16x8_t (&fl)[NBN], const float* next) {
    sload_wait(wsc);
    float wv[8];
    lane_weights(wsc, lane, wv);
    wsc = sload16(next);
#pragma unroll
    for (int q = 0; q < NBN; ++q) weight_split(fb[q], wv, fb[q], fl[q]);
  };
  auto step = [&](uint16_t* cur, uint16_t* nxt, uint16_t* fill, int kt) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(NCP));  // stage kt + 1 landed (this thread's copies)
    barrier_nofence();                           // ... everyone's; slot `fill` no longer read
    if (!mm_on) {  // copies only
#pragma unroll
      for (int j = 0; j < NCP; ++j) issue(fill, kt + kDLStages - 1, j);
      return;
    }
#pragma unroll
    for (int sl = 0; sl < NSLOT; ++sl) {
      if ((sl * NCP) % NSLOT == 0) {
        __builtin_amdgcn_sched_barrier(0);
        issue(fill, kt + kDLStages - 1, sl * NCP / NSLOT);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (sl == 0) load_frags(cur, 16, fa1, fb1);
      if (WT && sl == NBM / 2) weigh(fb1, fl1, wpad + (int64_t)(kt + 1) * kBK);  // this stage, second half
      if (sl == NBM) load_frags(nxt, 0, fa0, fb0);
      if (WT && sl == NBM + NBM / 2) weigh(fb0, fl0, wpad + (int64_t)(kt + 1) * kBK + 16);  // next stage, first half
      if (sl < NBM) mma_row(fa0, fb0, fl0, sl);
      else mma_row(fa1, fb1, fl1, sl - NBM);
    }
  };
  // stages past nk read zeros: harmless
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb0, 0, j);
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb1, 1, j);
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb2, 2, j);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * NCP));  // stage 0 landed
  barrier_nofence();
  load_frags(sb0, 0, fa0, fb0);
  if (WT) weigh(fb0, fl0, wpad + 16);  // stage 0, second half next
  for (int kt = 0; kt < nk; kt += 4) {
    step(sb0, sb1, sb3, kt);
    if (kt + 1 < nk) step(sb1, sb2, sb0, kt + 1);
    if (kt + 2 < nk) step(sb2, sb3, sb1, kt + 2);
    if (kt + 3 < nk) step(sb3, sb0, sb2, kt + 3);
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // drain the look-ahead loads before the workgroup ends

  double dsum = 0.0;
  if (active && !ctile) {
#pragma unroll
    for (int m = 0; m < NBM; ++m)
#pragma unroll
      for (int q = 0; q < NBN; ++q) {
        // the 16 old values of this MFMA block are read together, then added and stored
        const int64_t col = cJ + wj * WN + 32 * q + mfma32_col(lane);
        const int64_t rb = cI + wi * WM + 32 * m;
        float old[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = rb + mfma32_row(lane, r);
          old[r] = ld_or_zero(S, row * d + col, keep && row < d && col < d);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = rb + mfma32_row(lane, r);
          if (row < d && col < d) {
            S[row * d + col] = old[r] + acc[m][q][r];
            if (diag && row == col) dsum += (double)acc[m][q][r];
          }
        }
      }
  }
  if (cross || (ctile && mm_on)) {  // Kraw rows cI + arow0 + .., columns kc0 + .. < w2 (row stride w2)
    float* Kraw = Kraw_all + b * d * w2;
    const int kc0 = ctile ? bcol0 : 0;
#pragma unroll
    for (int m = 0; m < NBM; ++m)
#pragma unroll
      for (int q = 0; q < NBN; ++q) {
        const int64_t col = kc0 + 32 * q + mfma32_col(lane);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = cI + arow0 + 32 * m + mfma32_row(lane, r);
          if (row < d && col < w2) Kraw[row * w2 + col] = acc[m][q][r];
        }
      }
  }
  if (diag) {
    const double tot = block_sum(dsum, sred);
    if (threadIdx.x == 0) diag_part[b * T + I] = tot;
  }
}

// ------------------------------------------------------------------ Kraw = X^T [Y_hi | Y_lo] (bf16)

// Rows: a 256-column panel of X; columns: the 2k split columns of Y padded to YB.
// 4 waves stacked along the rows (64 rows each).
template <int YB>
__global__ __launch_bounds__(kThreads) void k_cross_bf16(int64_t n, int64_t d, int64_t k,
                                                         const uint16_t* __restrict__ Xall, int64_t ldx,
                                                         int64_t x_bstride, const float* __restrict__ Yall,
                                                         int64_t y_bstride, float* __restrict__ Kraw,
                                                         const float* __restrict__ aw) {
  constexpr int BM = 256;
  constexpr int LDT = BM + 16;
  constexpr int LDY = YB + 16;
  constexpr int NQ = YB / 32;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][kBK * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t sY[2][kBK * LDY];
  const int64_t b = blockIdx.y;
  const int I = blockIdx.x;
  const uint16_t* X = Xall + b * x_bstride;
  const float* Y = Yall + b * y_bstride;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t cI = (int64_t)I * BM;

  f32x16_t acc[2][NQ];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][q][r] = 0.f;

  XStage<BM, kThreads> ra;
  // Y staging: kBK rows x k floats, converted to hi/lo bf16 columns [0,k) and [k,2k)
  auto load_y = [&](int64_t t0, int buf) {
    // columns [0, k): hi = bf16(y), [k, 2k): lo = bf16(y - hi), [2k, YB): zero
    constexpr int PER = (kBK * YB + kThreads - 1) / kThreads;
    float v[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int row = e / YB, c = e % YB;
      const int64_t t = t0 + row;
      const int cc = c < k ? c : c - (int)k;
      const bool ok = e < kBK * YB && t < n && c < 2 * k;
      v[q] = ld_or_zero(Y, t * k + cc, ok);
      if (aw) v[q] *= ld_or_zero(aw, t, ok);  // statistic weight, before the split
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = threadIdx.x + q * kThreads;
      if (e < kBK * YB) {
        const int row = e / YB, c = e % YB;
        const uint16_t hi = f32_to_bf16(v[q]);
        sY[buf][row * LDY + c] = (c < k) ? hi : f32_to_bf16(v[q] - bf16_to_f32(hi));
      }
    }
  };
  const int nk = (int)((n + kBK - 1) / kBK);
  ra.load(X, ldx, n, d, 0, cI);
  ra.store(sA[0], LDT);
  load_y(0, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) ra.load(X, ldx, n, d, (int64_t)(kt + 1) * kBK, cI);
#pragma unroll
    for (int ks = 0; ks < kBK; ks += 16) {
      bf16x8_t fa[2], fb[NQ];
#pragma unroll
      for (int m = 0; m < 2; ++m) fa[m] = frag32_tr(sA[cur], LDT, wid * 64 + 32 * m, ks, lane);
#pragma unroll
      for (int q = 0; q < NQ; ++q) fb[q] = frag32_tr(sY[cur], LDY, 32 * q, ks, lane);
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int q = 0; q < NQ; ++q) acc[m][q] = mfma32(fa[m], fb[q], acc[m][q]);
    }
    if (kt + 1 < nk) {
      ra.store(sA[cur ^ 1], LDT);
      load_y((int64_t)(kt + 1) * kBK, cur ^ 1);
    }
    __syncthreads();
  }
  float* Kb = Kraw + b * d * 2 * k;
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = cI + wid * 64 + 32 * m + mfma32_row(lane, r);
        const int64_t col = 32 * q + mfma32_col(lane);
        if (row < d && col < 2 * k) Kb[row * 2 * k + col] = acc[m][q][r];
      }
}

// ------------------------------------------------------------------ fp64 path (fp32 mode)

// 64 x 64 tiles, 4 waves of 32 x 32 (2 x 2 blocks of 16 x 16), 16 tokens per stage.
// Jobs [0, nS) are upper tiles of S (Q = X); jobs [nS, nS + nK) are tiles of
// Kraw = X^T Y (Q = Y, k columns).
constexpr int kBM64 = 64, kBK64 = 16, kLD64 = kBM64 + 1;

__global__ __launch_bounds__(kThreads) void k_gram_f64(int64_t n, int64_t d, int64_t k,
                                                       const float* __restrict__ Xall, int64_t ldx,
                                                       int64_t x_bstride, const float* __restrict__ Yall,
                                                       int64_t y_bstride, double* __restrict__ Sall,
                                                       int64_t s_bstride, double* __restrict__ Kraw,
                                                       double* __restrict__ diag_part, int nS,
                                                       const float* __restrict__ aw, int keep) {
  __shared__ double sP[kBK64 * kLD64];
  __shared__ double sQ[kBK64 * kLD64];
  __shared__ double sred[kThreads / 64];
  const int64_t b = blockIdx.y;
  const int T = (int)((d + kBM64 - 1) / kBM64);
  const bool kjob = (int)blockIdx.x >= nS;
  int I, J;
  if (!kjob) {
    upper_tile(blockIdx.x, T, I, J);
  } else {
    const int u = blockIdx.x - nS;
    const int TK = (int)((k + kBM64 - 1) / kBM64);
    I = u / TK;
    J = u % TK;
  }
  const bool diag = !kjob && I == J;
  const float* X = Xall + b * x_bstride;
  const float* Y = Yall + b * y_bstride;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wi = wid >> 1, wj = wid & 1;
  const int64_t cI = (int64_t)I * kBM64, cJ = (int64_t)J * kBM64;
  const int64_t qcols = kjob ? k : d;

  f64x4_t acc[2][2];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < 2; ++q) acc[m][q] = (f64x4_t){0.0, 0.0, 0.0, 0.0};

  for (int64_t t0 = 0; t0 < n; t0 += kBK64) {
    __syncthreads();
    for (int e = threadIdx.x; e < kBK64 * kBM64; e += kThreads) {
      const int row = e / kBM64, c = e % kBM64;
      const int64_t t = t0 + row;
      const int64_t ci = cI + c, cj = cJ + c;
      sP[row * kLD64 + c] = (t < n && ci < d) ? (double)X[t * ldx + ci] : 0.0;
      double qv = 0.0;
      if (t < n && cj < qcols) {
        qv = kjob ? (double)Y[t * k + cj] : (double)X[t * ldx + cj];
        if (aw) qv *= (double)aw[t];  // statistic weight (an exact product in fp64)
      }
      sQ[row * kLD64 + c] = qv;
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < kBK64; ks += 4) {
      double fa[2], fb[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) fa[m] = sP[(ks + (lane >> 4)) * kLD64 + wi * 32 + 16 * m + (lane & 15)];
#pragma unroll
      for (int q = 0; q < 2; ++q) fb[q] = sQ[(ks + (lane >> 4)) * kLD64 + wj * 32 + 16 * q + (lane & 15)];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[m][q] = mfma_f64(fa[m], fb[q], acc[m][q]);
    }
  }
  double dsum = 0.0;
  double* S = Sall + b * s_bstride;
  double* Kb = Kraw + b * d * k;
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = cI + wi * 32 + 16 * m + (lane >> 4) + 4 * r;
        const int64_t col = cJ + wj * 32 + 16 * q + (lane & 15);
        if (row < d && col < qcols) {
          if (kjob) {
            Kb[row * k + col] = acc[m][q][r];
          } else {
            S[row * d + col] = (keep ? S[row * d + col] : 0.0) + acc[m][q][r];
            if (diag && row == col) dsum += acc[m][q][r];
          }
        }
      }
  if (diag) {
    const double tot = block_sum(dsum, sred);
    if (threadIdx.x == 0) diag_part[b * T + I] = tot;
  }
}

// ------------------------------------------------------------------ finalize: eta_bar and K

// One workgroup per (block, 256 V entries of K); its first wave forms ||X||^2 from the
// diagonal tiles' partials (lane l sums partials l, l + 64, ... in order, then a fixed
// butterfly across the lanes: deterministic) and eta-bar once for the workgroup.  A thread
// takes V consecutive entries of a row of K (V = 4: 16-byte accesses, k % 4 == 0 and K's
// rows 16-byte aligned), each formed alike.  keep == 0: K is overwritten (its old
// contents are not read).
// dev_info (may be null) gets, per block, 0 or LOCA_INFO_NONFINITE when ||X||^2 or ||Q||^2
// is not finite (a NaN or infinite entry of X, an entry whose square overflows, or a
// non-finite error row in the head call).
template <typename AccT, int V = 1>
__global__ void k_stats_finalize(int64_t n, int64_t d, int64_t k, int ntile, const double* __restrict__ diag_part,
                                 loca_mb* __restrict__ mb, double eta, const AccT* __restrict__ Kraw, int split,
                                 AccT* __restrict__ Kall, int64_t k_bstride, int32_t* __restrict__ dev_info,
                                 int keep) {
  __shared__ double s_eb;
  const int64_t b = blockIdx.y;
  if (threadIdx.x < 64) {
    double part = 0.0;
    for (int i = (int)threadIdx.x; i < ntile; i += 64) part += diag_part[b * ntile + i];
    const double sx = wave_sum(part);
    if (threadIdx.x == 0) {
      const double sq = mb[b].sum_q2;
      const double eb = (sq > 0.0) ? eta * sqrt(sx / sq) : 0.0;
      s_eb = eb;
      if (blockIdx.x == 0) {
        mb[b].sum_x2 = sx;
        mb[b].eta_bar = eb;
        mb[b].n = n;
        if (dev_info)
          dev_info[b] = (__builtin_isfinite(sx) && __builtin_isfinite(sq)) ? 0 : (int32_t)LOCA_INFO_NONFINITE;
      }
    }
  }
  __syncthreads();
  const double eb = s_eb;
  const uint32_t e = V * (blockIdx.x * blockDim.x + threadIdx.x);  // d k < 2^31 (d, k <= 65535, 128)
  if (e >= (uint32_t)(d * k)) return;
  const uint32_t ku = (uint32_t)k, i = e / ku, c = e - i * ku;
  AccT* K = Kall + b * k_bstride;
  const uint32_t w = split ? 2 * ku : ku;
  const AccT* kr = Kraw + b * d * w + (int64_t)i * w;
  if constexpr (V == 4) {
    static_assert(sizeof(AccT) == 4, "16-byte accesses of floats");
    const float4 k0 = *(const float4*)(kr + c);
    const float4 k1 = split ? *(const float4*)(kr + c + ku) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 o = keep ? *(const float4*)(K + e) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float a0[4] = {k0.x, k0.y, k0.z, k0.w}, a1[4] = {k1.x, k1.y, k1.z, k1.w}, ov[4] = {o.x, o.y, o.z, o.w};
    float r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      double v = (double)a0[u];
      if (split) v += (double)a1[u];
      r[u] = (float)((double)ov[u] - eb * v);
    }
    *(float4*)(K + e) = make_float4(r[0], r[1], r[2], r[3]);
  } else {
    double v = (double)kr[c];
    if (split) v += (double)kr[c + ku];
    K[e] = (AccT)((keep ? (double)K[e] : 0.0) - eb * v);
  }
}

}  // namespace

__global__ void k_zero_bytes(uint32_t* p, int cnt) {
  if ((int)threadIdx.x < cnt) p[threadIdx.x] = 0u;
}

// Yhl[b][t] = [bf16(y) | bf16(y - bf16(y)) | 0] (w2p columns, w2p % 8 == 0) from the float
// targets, and the 256 zero bytes at the head of the workspace.  One thread per 8 columns of a
// row (one 16-byte store); IT is the index type (32-bit while n w2p / 8 fits).
// k_split_y8 (k % 8 == 0, so w2p = 2k, and Y's rows 32-byte aligned): a thread reads 8
// consecutive targets of a row once (two 16-byte loads) and writes their high and low
// parts (two 16-byte stores); the values are those of k_split_y.
template <typename IT>
__global__ void k_split_y8(int64_t n, int64_t k, const float* __restrict__ Yall, int64_t y_bstride,
                           uint16_t* __restrict__ Yhl, uint32_t* __restrict__ zero_area) {
  const int64_t b = blockIdx.y;
  if (b == 0 && blockIdx.x == 0 && threadIdx.x < 64) zero_area[threadIdx.x] = 0u;
  const IT g8 = (IT)(k / 8);
  const IT e = (IT)blockIdx.x * (IT)blockDim.x + (IT)threadIdx.x;
  if (e >= (IT)n * g8) return;
  const IT t = e / g8;
  const int c0 = 8 * (int)(e - t * g8);
  const float* yr = Yall + b * y_bstride + (int64_t)t * k + c0;
  const float4 v0 = *(const float4*)yr, v1 = *(const float4*)(yr + 4);
  const float y[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
  uint32_t wh[4], wl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t h2[2], l2[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const float x = y[2 * i + u];
      const __bf16 hi = (__bf16)x;  // round to nearest even
      const __bf16 lo = (__bf16)(x - (float)hi);
      h2[u] = (uint32_t)__builtin_bit_cast(uint16_t, hi);
      l2[u] = (uint32_t)__builtin_bit_cast(uint16_t, lo);
    }
    wh[i] = h2[0] | (h2[1] << 16);
    wl[i] = l2[0] | (l2[1] << 16);
  }
  uint16_t* row = Yhl + b * n * 2 * k + (int64_t)t * 2 * k;
  *(uint4*)(row + c0) = make_uint4(wh[0], wh[1], wh[2], wh[3]);
  *(uint4*)(row + k + c0) = make_uint4(wl[0], wl[1], wl[2], wl[3]);
}

template <typename IT>
__global__ void k_split_y(int64_t n, int64_t k, int64_t w2p, const float* __restrict__ Yall, int64_t y_bstride,
                          uint16_t* __restrict__ Yhl, uint32_t* __restrict__ zero_area) {
  const int64_t b = blockIdx.y;
  if (b == 0 && blockIdx.x == 0 && threadIdx.x < 64) zero_area[threadIdx.x] = 0u;
  const IT g8 = (IT)(w2p / 8);
  const IT e = (IT)blockIdx.x * (IT)blockDim.x + (IT)threadIdx.x;
  if (e >= (IT)n * g8) return;
  const IT t = e / g8;
  const int c0 = 8 * (int)(e - t * g8);
  const float* yr = Yall + b * y_bstride + (int64_t)t * k;
  const int kk = (int)k;
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t h2[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = c0 + 2 * i + u;
      __bf16 v = (__bf16)0.f;
      if (c < 2 * kk) {
        const float y = yr[c < kk ? c : c - kk];
        const __bf16 hi = (__bf16)y;  // round to nearest even
        v = c < kk ? hi : (__bf16)(y - (float)hi);
      }
      h2[u] = (uint32_t)__builtin_bit_cast(uint16_t, v);
    }
    w[i] = h2[0] | (h2[1] << 16);
  }
  *(uint4*)(Yhl + b * n * w2p + (int64_t)t * w2p + c0) = make_uint4(w[0], w[1], w[2], w[3]);
}

// wpad[i] = a_w[i] for i < n, 0 up to npad (the padded weights of the bf16 Gram kernels)
__global__ void k_pad_weights(int64_t n, int64_t npad, const float* __restrict__ aw, float* __restrict__ wpad) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < npad) wpad[i] = i < n ? aw[i] : 0.f;
}

// padded length of the weights: every stage the kernels compute, plus one stage of look-ahead
static int64_t weights_pad(int64_t n) { return ((n + kBK - 1) / kBK + 1) * kBK; }

size_t accumulate_stats_ws(int64_t nb, int64_t n, int64_t d, int64_t k, loca_dtype acc) {
  const int64_t T = acc == LOCA_F64 ? (d + kBM64 - 1) / kBM64 : (d + 127) / 128;
  const int64_t Tmax = (d + kBM64 - 1) / kBM64;  // generous: covers every tile size used
  size_t s = 256 + align256(sizeof(double) * nb * (T > Tmax ? T : Tmax));  // zeros + tile partials
  if (acc == LOCA_F64) s += align256(sizeof(double) * nb * d * k);
  else s += align256(sizeof(float) * nb * d * 2 * k) + align256(sizeof(uint16_t) * nb * n * ((2 * k + 7) / 8 * 8)) +
            align256(sizeof(float) * weights_pad(n));
  return s;
}

template <bool BUF, bool WT>
static void launch_gram_dl(const StatsArgs& a, int64_t ntile, int64_t b0, int64_t nbc, const uint16_t* zero16,
                           double* diag_part, const uint16_t* Yhl, int64_t w2, int64_t w2p, float* Kraw,
                           const float* wpad, int ncross) {
  // block-synchronous order with XCD groups of four (else two) whose runs hold at least 24
  // tiles, if there are blocks enough for every group; else the XCD-aware order.  Groups of
  // eight (every XCD on one block) were slower where runs of 24 allowed them (d = 5120:
  // statistics call +0.4%; two blocks' X of 84 MB each still fit the last-level cache).  The
  // runs split a block's cost: a cross tile whose targets span at most two of the four
  // column blocks (four waves with products, one per SIMD) is counted as 0.6 of a Gram tile,
  // and the cross tiles, last in a block, go to the last run of its group.
  const int64_t ntot = ntile + ncross;
  int gx = 0;
  for (int g = 4; g >= 2 && gx == 0; g /= 2)
    if ((ntot + g - 1) / g >= 24 && nbc >= 8 / g) gx = g;
  int64_t run = 0, per = 0;
  if (gx > 0) {
    const double cost = (double)ntile + (w2p <= 128 ? 0.6 : 1.0) * (double)ncross;
    run = std::min<int64_t>((int64_t)std::ceil(cost / gx), gx > 1 ? ntot / (gx - 1) : ntot);
    per = std::max<int64_t>(run, ntot - (gx - 1) * run);
  }
  const int64_t rounds = gx > 0 ? (nbc + 8 / gx - 1) / (8 / gx) : 0;
  const int64_t grid = gx > 0 ? 8 * per * rounds : ntot * nbc;
  k_gram_bf16_dl<2, 4, BUF, WT><<<dim3((unsigned)grid), 512, 0, a.stream>>>(
      a.n, a.d, (const uint16_t*)a.x, a.ldx, a.x_bstride, (float*)a.S, a.s_bstride, diag_part, zero16, b0, Yhl, w2,
      w2p, Kraw, wpad, ncross, (int)run, (int)per, gx > 0 ? gx : 8, (int)nbc, a.overwrite ? 0 : 1);
}

hipError_t launch_accumulate_stats(const StatsArgs& a) {
  const int64_t Tmax = (a.d + kBM64 - 1) / kBM64;
  const uint16_t* zero16 = (const uint16_t*)a.ws;  // 256 zeroed bytes
  double* diag_part = (double*)(a.ws + 256);
  char* p = a.ws + 256 + align256(sizeof(double) * a.nb * Tmax);
  if (a.acc == LOCA_F64) {
    double* Kraw = (double*)p;
    const int T = (int)((a.d + kBM64 - 1) / kBM64);
    const int nS = T * (T + 1) / 2;
    const int nK = T * (int)((a.k + kBM64 - 1) / kBM64);
    dim3 grid((unsigned)(nS + nK), (unsigned)a.nb);
    k_gram_f64<<<grid, kThreads, 0, a.stream>>>(a.n, a.d, a.k, (const float*)a.x, a.ldx, a.x_bstride, a.y,
                                                a.y_bstride, (double*)a.S, a.s_bstride, Kraw, diag_part, nS, a.a_w,
                                                a.overwrite ? 0 : 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((unsigned)((a.d * a.k + 255) / 256), (unsigned)a.nb);
    k_stats_finalize<double><<<g2, 256, 0, a.stream>>>(a.n, a.d, a.k, T, diag_part, a.mb, a.eta, Kraw, 0,
                                                       (double*)a.K, a.k_bstride, a.dev_info, a.overwrite ? 0 : 1);
    return hipGetLastError();
  }
  float* Kraw = (float*)p;
  uint16_t* Yhl = (uint16_t*)(p + align256(sizeof(float) * a.nb * a.d * 2 * a.k));
  float* wpad = (float*)((char*)Yhl + align256(sizeof(uint16_t) * a.nb * a.n * ((2 * a.k + 7) / 8 * 8)));
  const uint16_t* X = (const uint16_t*)a.x;
  const bool wt = a.a_w != nullptr;
  if (wt) {
    const int64_t npad = weights_pad(a.n);
    k_pad_weights<<<(unsigned)((npad + 255) / 256), 256, 0, a.stream>>>(a.n, npad, a.a_w, wpad);
  }
  // Tile size: 256 x 256 when the matrix is wide enough to fill the GPU with such tiles.
  const bool big = a.d >= 1024;
  const int BM = big ? 256 : 128;
  const int T = (int)((a.d + BM - 1) / BM);
  dim3 grid((unsigned)(T * (T + 1) / 2), (unsigned)a.nb);
  const int64_t w2 = 2 * a.k, w2p = (w2 + 7) / 8 * 8;
  // buffer-path copies when a block's X (and its split targets) fit 31-bit byte offsets
  const bool buf = (a.n * a.ldx * 2) < ((int64_t)1 << 31);
  // direct-to-LDS kernel; with weights only on the buffer path (the global-address
  // variant runs out of scalar registers with the weights, so blocks of X over 2 GB
  // take the register-staged kernel when weighted)
  const bool dl = big && (a.d % 8) == 0 && (buf || !wt);
  const bool fused = dl && w2p <= 64;
  // wider split targets: cross tiles in the same launch (one per row panel of each block)
  const bool ctiles = dl && !fused;
  if (dl) {
    if (fused || ctiles) {
      const bool v8 = a.k % 8 == 0 && a.y_bstride % 8 == 0 && ((uintptr_t)a.y & 31) == 0;
      const int64_t groups = v8 ? a.n * (a.k / 8) : a.n * (w2p / 8);
      dim3 gy((unsigned)((groups + 255) / 256), (unsigned)a.nb);
      if (v8 && groups < ((int64_t)1 << 31))
        k_split_y8<uint32_t><<<gy, 256, 0, a.stream>>>(a.n, a.k, a.y, a.y_bstride, Yhl, (uint32_t*)a.ws);
      else if (v8)
        k_split_y8<int64_t><<<gy, 256, 0, a.stream>>>(a.n, a.k, a.y, a.y_bstride, Yhl, (uint32_t*)a.ws);
      else if (groups < ((int64_t)1 << 31))
        k_split_y<uint32_t><<<gy, 256, 0, a.stream>>>(a.n, a.k, w2p, a.y, a.y_bstride, Yhl, (uint32_t*)a.ws);
      else
        k_split_y<int64_t><<<gy, 256, 0, a.stream>>>(a.n, a.k, w2p, a.y, a.y_bstride, Yhl, (uint32_t*)a.ws);
    } else {
      k_zero_bytes<<<1, 64, 0, a.stream>>>((uint32_t*)a.ws, 64);
    }
    // one-dimensional grid (the XCD-aware order spans the blocks), in chunks of blocks
    // small enough that the grid stays far below the launch limits
    const int64_t ntile = (int64_t)T * (T + 1) / 2;
    const int ncross = ctiles ? T : 0;
    const int64_t chunk = std::max<int64_t>(1, ((int64_t)1 << 22) / (ntile + ncross));
    for (int64_t b0 = 0; b0 < a.nb; b0 += chunk) {
      const int64_t nbc = std::min<int64_t>(chunk, a.nb - b0);
      const bool use_buf = buf;
      const uint16_t* yf = (fused || ctiles) ? Yhl : nullptr;
      if (use_buf && wt)
        launch_gram_dl<true, true>(a, ntile, b0, nbc, zero16, diag_part, yf, w2, w2p, Kraw, wpad, ncross);
      else if (use_buf)
        launch_gram_dl<true, false>(a, ntile, b0, nbc, zero16, diag_part, yf, w2, w2p, Kraw, nullptr, ncross);
      else
        launch_gram_dl<false, false>(a, ntile, b0, nbc, zero16, diag_part, yf, w2, w2p, Kraw, nullptr, ncross);
    }
  } else if (big) {
    if (wt)
      k_gram_bf16<256, 2, 4, true><<<grid, 512, 0, a.stream>>>(a.n, a.d, X, a.ldx, a.x_bstride, (float*)a.S,
                                                               a.s_bstride, diag_part, wpad, a.overwrite ? 0 : 1);
    else
      k_gram_bf16<256, 2, 4, false><<<grid, 512, 0, a.stream>>>(a.n, a.d, X, a.ldx, a.x_bstride, (float*)a.S,
                                                                a.s_bstride, diag_part, nullptr, a.overwrite ? 0 : 1);
  } else {
    if (wt)
      k_gram_bf16<128, 2, 2, true><<<grid, 256, 0, a.stream>>>(a.n, a.d, X, a.ldx, a.x_bstride, (float*)a.S,
                                                               a.s_bstride, diag_part, wpad, a.overwrite ? 0 : 1);
    else
      k_gram_bf16<128, 2, 2, false><<<grid, 256, 0, a.stream>>>(a.n, a.d, X, a.ldx, a.x_bstride, (float*)a.S,
                                                                a.s_bstride, diag_part, nullptr, a.overwrite ? 0 : 1);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gc((unsigned)((a.d + 255) / 256), (unsigned)a.nb);
  if (!fused && !ctiles) {  // the cross statistic in a launch of its own
    if (w2 <= 32)
      k_cross_bf16<32><<<gc, kThreads, 0, a.stream>>>(a.n, a.d, a.k, X, a.ldx, a.x_bstride, a.y, a.y_bstride, Kraw,
                                                       a.a_w);
    else if (w2 <= 64)
      k_cross_bf16<64><<<gc, kThreads, 0, a.stream>>>(a.n, a.d, a.k, X, a.ldx, a.x_bstride, a.y, a.y_bstride, Kraw,
                                                        a.a_w);
    else if (w2 <= 128)
      k_cross_bf16<128><<<gc, kThreads, 0, a.stream>>>(a.n, a.d, a.k, X, a.ldx, a.x_bstride, a.y, a.y_bstride, Kraw,
                                                        a.a_w);
    else
      k_cross_bf16<256><<<gc, kThreads, 0, a.stream>>>(a.n, a.d, a.k, X, a.ldx, a.x_bstride, a.y, a.y_bstride, Kraw,
                                                        a.a_w);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.k % 4 == 0 && a.k_bstride % 4 == 0 && ((uintptr_t)a.K & 15) == 0) {
    dim3 g4((unsigned)((a.d * a.k / 4 + 255) / 256), (unsigned)a.nb);
    k_stats_finalize<float, 4><<<g4, 256, 0, a.stream>>>(a.n, a.d, a.k, T, diag_part, a.mb, a.eta, Kraw, 1,
                                                         (float*)a.K, a.k_bstride, a.dev_info,
                                                         a.overwrite ? 0 : 1);
  } else {
    dim3 g2((unsigned)((a.d * a.k + 255) / 256), (unsigned)a.nb);
    k_stats_finalize<float><<<g2, 256, 0, a.stream>>>(a.n, a.d, a.k, T, diag_part, a.mb, a.eta, Kraw, 1,
                                                      (float*)a.K, a.k_bstride, a.dev_info, a.overwrite ? 0 : 1);
  }
  return hipGetLastError();
}

}  // namespace loca
