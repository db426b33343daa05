// k_fused.hip -- the fused LM head ("Local Targets", Eq. 4; Lemma S3.1's head error; the
// head applied once per top error, Section S11).  From the final hidden states h (n x d) and
// the frozen head W_u (V x d), for a right operand Vm (V x c):
//   out_t = w_t ( sum_v softmax(z_t)_v Vm[v, :] - Vm[y_t, :] ),   z_t = W_u h_t,
// i.e. out = E Vm with E_t = w_t (softmax(z_t) - onehot(y_t)).  Vm = W_u gives the top error
// e_t = W_u^T E_t of the paper's order (then V_k^T e_t per block); Vm = [A~_1 | ... | A~_L]
// gives every block's credit coordinates Y_b = E A~_b at once.
//
// The logits are never stored.  A workgroup (8 waves) owns 128 tokens, a tile of at most 64
// columns of Vm and a contiguous range of the vocabulary, and walks that range in chunks
// of 256:
//   1. z^T (256 x 128) = W_u[chunk] h_rows^T on the matrix cores (v_mfma_f32_32x32x16_bf16,
//      fp32 accumulation), both operands copied straight into LDS (buffer loads to LDS) in
//      32-wide slices of d through a four-slot ring that runs across chunk boundaries;
//   2. an online softmax per token, in registers: the running maximum m and sum s (fp32)
//      are updated with the chunk, the accumulated output is rescaled by exp(m_old - m_new),
//      and P = exp(z - m_new) is split into bf16 hi + lo parts (about 16 significant bits);
//   3. out += (P_hi + P_lo) Vm[chunk] on the matrix cores (Vm exact in bf16), P taken from
//      the registers of step 1 and the Vm^T slice from LDS.
// Each vocabulary range leaves (m, s) per token and its partial output; a second kernel
// combines the ranges in a fixed order in float64 and subtracts the label term.  Columns of
// Vm beyond one 64-wide tile recompute the logits (c / 64 passes over W_u).
#include "loca_bf16.h"
#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kFT = 512;        // threads: 8 waves, (vocabulary quarter wv) x (token half wt)
constexpr int kFR = 128;        // tokens per tile
constexpr int kFV = 256;        // vocabulary per chunk
constexpr int kFC = 64;         // columns of Vm per tile
constexpr int kFK = 32;         // hidden width per stage
constexpr int kFStages = 4;     // ring slots: three stages in flight while one is read
constexpr int kFLA = kFStages - 1;
constexpr int kFStage = (kFV + kFR) * kFK * 2;  // bytes per stage: W_u rows, then h rows (64 B each)
constexpr int kFCopies = kFStage / 16 / kFT;     // 16-byte copies per thread per stage (3)
constexpr int kFVt = kFC * kFV * 2;              // bytes of the Vm^T slice
constexpr int kFNV = kFVt / 16 / kFT;            // its copies per thread (4)

// A stage holds 384 rows of 64 bytes (32 bf16 of d): rows 0..255 the chunk's W_u rows,
// rows 256..383 the tile's h rows.  Chunk c (16 bytes) of row r sits at position
// c ^ ((r >> 2) & 3), so that the 16 lanes of a half wave reading one chunk of 16
// consecutive rows hit 16 distinct bank groups.
LOCA_DEV int fz_swz(int r) { return (r >> 2) & 3; }
// The Vm^T slice: 64 rows (columns of Vm) of 512 bytes (256 vocabulary entries), chunk c
// of row r at position c ^ (r & 15).
LOCA_DEV int fv_swz(int r) { return r & 15; }

// (m, s) of two disjoint parts of a row, combined
LOCA_DEV void fz_combine(float& m, float& s, float m2, float s2) {
  if (s2 == 0.f) return;
  if (s == 0.f) {
    m = m2;
    s = s2;
    return;
  }
  const float mm = fmaxf(m, m2);
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

// s_waitcnt vmcnt(a) for a run-time a in 0..31
LOCA_DEV void wait_vm(int a) {
  switch (a) {
#define LOCA_W(N) case N: __builtin_amdgcn_s_waitcnt(vmcnt_imm(N)); break;
    LOCA_W(0) LOCA_W(1) LOCA_W(2) LOCA_W(3) LOCA_W(4) LOCA_W(5) LOCA_W(6) LOCA_W(7) LOCA_W(8) LOCA_W(9)
    LOCA_W(10) LOCA_W(11) LOCA_W(12) LOCA_W(13) LOCA_W(14) LOCA_W(15) LOCA_W(16) LOCA_W(17) LOCA_W(18)
    LOCA_W(19) LOCA_W(20) LOCA_W(21) LOCA_W(22) LOCA_W(23) LOCA_W(24) LOCA_W(25) LOCA_W(26) LOCA_W(27)
    LOCA_W(28) LOCA_W(29) LOCA_W(30)
#undef LOCA_W
    default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;
  }
}

// The logits are formed transposed, z^T = W_u[chunk] h_tile^T (vocabulary x tokens), so
// that lane l of a 32 x 32 result block holds token l % 32 and 16 vocabulary entries:
// the softmax statistics of a token stay within a lane pair (l, l ^ 32) and the four
// waves that split the chunk's vocabulary, and the exponentials of a block are already
// the matrix-core operand of the product with Vm (the sum over the vocabulary taken in
// the order the result layout gives).
//
// Copy accounting: stage s is issued kFLA iterations ahead of its use (the prologue issues
// stages 0 .. kFLA - 1); the Vm^T slice of chunk j is issued at the top of iteration j nks,
// before that iteration's stage.  Every wait counts the copies issued after the one it
// needs, and vector-memory operations complete in order.
__global__ __launch_bounds__(kFT) void k_fused_head(int64_t n, int64_t V, int64_t d, int64_t c,
                                                    const uint16_t* __restrict__ h, int64_t ldh,
                                                    const uint16_t* __restrict__ wu,
                                                    const uint16_t* __restrict__ vmt, int64_t ldvt, int ntr, int nct,
                                                    int64_t vper, float* __restrict__ part_o,
                                                    float2* __restrict__ part_ms) {
  __shared__ __attribute__((aligned(1024))) uint8_t ring[kFStages * kFStage];
  __shared__ __attribute__((aligned(1024))) uint8_t sVt[kFVt];
  __shared__ float2 sEx[4][kFR];
  constexpr int NQ = kFC / 32;  // 32-column output blocks per wave
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, wv = wid >> 1, wt = wid & 1;
  const int l32 = lane & 31, lh = lane >> 5;
  // tiles that share a vocabulary range are consecutive within an XCD (W_u read once there)
  const int logical = xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int rt = logical % ntr, ct = (logical / ntr) % nct, sp = logical / (ntr * nct);
  const int64_t r0 = (int64_t)rt * kFR, c0 = (int64_t)ct * kFC;
  const int64_t vb = (int64_t)sp * vper, ve = (vb + vper < V) ? vb + vper : V;
  const int nks = (int)((d + kFK - 1) / kFK);
  const int nch = (int)((ve - vb + kFV - 1) / kFV);
  const int total = nch * nks;  // stages of this workgroup

  const int64_t nrow = (n - r0 < kFR) ? n - r0 : kFR;
  const i32x4_t rsH = buffer_rsrc(h + r0 * ldh, (uint32_t)(nrow * ldh * 2));
  const int64_t ncol = (c - c0 < kFC) ? c - c0 : kFC;
  const i32x4_t rsV = buffer_rsrc(vmt + c0 * ldvt, (uint32_t)(ncol * ldvt * 2));
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(LOCA_LDS void*)ring;
  const uint32_t vt_lds = (uint32_t)(uintptr_t)(LOCA_LDS void*)sVt;
  const int wq = __builtin_amdgcn_readfirstlane(wid);

  // stage g = (chunk g / nks, slice g % nks) into ring slot g % kFStages: 24 blocks of 1 KB
  // (16 rows each), blocks 0..15 the W_u rows, 16..23 the h rows; byte offsets fit 31 bits
  // (V, d, ldh <= 2^23 are checked by the caller)
  auto issue_stage = [&](int g) {
    const int64_t v0 = vb + (int64_t)(g / nks) * kFV;
    const int k0 = (g % nks) * kFK;
    const uint32_t slot = ring_lds + (uint32_t)((g % kFStages) * kFStage);
    const int64_t nvr = (V - v0 < kFV) ? V - v0 : kFV;
    const i32x4_t rsW = buffer_rsrc(wu + v0 * d, (uint32_t)(nvr * d * 2));
#pragma unroll
    for (int j = 0; j < kFCopies; ++j) {
      const int blk = wq * kFCopies + j;
      const int row = 16 * blk + (lane >> 2);
      const int k = k0 + 8 * ((lane & 3) ^ fz_swz(row));
      if (blk < kFV / 16) {
        const uint32_t off = k < (int)d ? 2u * (uint32_t)(row * (int)d + k) : kBufOutside;
        lds_dma16_buf(off, rsW, slot + (uint32_t)blk * 1024u);
      } else {
        const uint32_t off = k < (int)d ? 2u * (uint32_t)((row - kFV) * (int)ldh + k) : kBufOutside;
        lds_dma16_buf(off, rsH, slot + (uint32_t)blk * 1024u);
      }
    }
  };
  // the chunk's Vm^T slice (64 columns of Vm x 256 vocabulary entries; zero past V)
  auto issue_vt = [&](int64_t v0) {
#pragma unroll
    for (int j = 0; j < kFNV; ++j) {
      const int blk = wq * kFNV + j;  // 1 KB: rows 2 blk, 2 blk + 1
      const int row = 2 * blk + (lane >> 5);
      const uint32_t off = 2u * (uint32_t)(row * (int)ldvt + (int)v0 + 8 * ((lane & 31) ^ fv_swz(row)));
      lds_dma16_buf(off, rsV, vt_lds + (uint32_t)blk * 1024u);
    }
  };
  // copies issued before the top of iteration g, and up to and including stage s
  auto issued_before = [&](int g) {
    const int st = (g + kFLA < total) ? g + kFLA : total;
    return kFCopies * st + kFNV * (g >= 1 ? (g - 1) / nks + 1 : 0);
  };
  auto through_stage = [&](int s) {
    return kFCopies * (s + 1) + kFNV * (s >= kFLA ? (s - kFLA) / nks + 1 : 0);
  };

  f32x16_t o[2][NQ];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[mt][q][r] = 0.f;
  float m_run[2] = {-__builtin_inff(), -__builtin_inff()}, s_run[2] = {0.f, 0.f};  // token l32 of block mt
  f32x16_t z[2][2];

  for (int s = 0; s < kFLA && s < total; ++s) issue_stage(s);
  for (int g = 0; g < total; ++g) {
    const int ks = g % nks;
    wait_vm(issued_before(g) - through_stage(g));
    __syncthreads();  // every thread's copies of stage g landed; the slot refilled below is free
    if (ks == 0) {
      issue_vt(vb + (int64_t)(g / nks) * kFV);
#pragma unroll
      for (int mv = 0; mv < 2; ++mv)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) z[mv][mt][r] = 0.f;
    }
    if (g + kFLA < total) issue_stage(g + kFLA);
    // 1. z^T += W_u[chunk, slice] h[tile, slice]^T
    const uint8_t* st = ring + (g % kFStages) * kFStage;
#pragma unroll
    for (int kk = 0; kk < kFK / 16; ++kk) {
      bf16x8_t a[2], b[2];
      const int ch = 2 * kk + lh;  // 16-byte chunk of the row: k = 16 kk + 8 lh
#pragma unroll
      for (int mv = 0; mv < 2; ++mv) {
        const int row = wv * 64 + 32 * mv + l32;
        a[mv] = *(const bf16x8_t*)(st + row * 64 + 16 * (ch ^ fz_swz(row)));
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const int row = kFV + wt * 64 + 32 * mt + l32;
        b[mt] = *(const bf16x8_t*)(st + row * 64 + 16 * (ch ^ fz_swz(row)));
      }
#pragma unroll
      for (int mv = 0; mv < 2; ++mv)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) z[mv][mt] = mfma32(a[mv], b[mt], z[mv][mt]);
    }
    if (ks != nks - 1) continue;

    // 2. online softmax over the chunk.  Entry r of lane l in block (mv, mt): vocabulary
    // v0 + 64 wv + 32 mv + 8 (r >> 2) + 4 lh + (r & 3), token 64 wt + 32 mt + l32.
    const int j = g / nks;
    const int64_t v0 = vb + (int64_t)j * kFV;
    const int nv = (V - v0 < kFV) ? (int)(V - v0) : kFV;
    const bool full = nv == kFV;
    auto valid = [&](int mv, int r) { return full || 64 * wv + 32 * mv + 8 * (r >> 2) + 4 * lh + (r & 3) < nv; };
    float lm[2], ls[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      float mx = -__builtin_inff();
#pragma unroll
      for (int mv = 0; mv < 2; ++mv)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (valid(mv, r)) mx = fmaxf(mx, z[mv][mt][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      float sm = 0.f;
      if (mx > -__builtin_inff()) {
#pragma unroll
        for (int mv = 0; mv < 2; ++mv)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (valid(mv, r)) sm += __expf(z[mv][mt][r] - mx);
      }
      sm += __shfl_xor(sm, 32);
      lm[mt] = mx;
      ls[mt] = sm;
    }
    if (lh == 0)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) sEx[wv][wt * 64 + 32 * mt + l32] = make_float2(lm[mt], ls[mt]);
    // the Vm^T slice of this chunk: covered by the stage waits when a later stage was issued
    // after it and has been waited for (nks > kFLA), else waited for here
    if (nks <= kFLA) {
      const int g0 = j * nks;
      const int after_vt = kFCopies * ((g + kFLA + 1 < total ? g + kFLA + 1 : total) -
                                       (g0 + kFLA < total ? g0 + kFLA : total));
      wait_vm(after_vt);
    }
    __syncthreads();
    float al[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int tk = wt * 64 + 32 * mt + l32;
      float cm = sEx[0][tk].x, cs = sEx[0][tk].y;
#pragma unroll
      for (int u = 1; u < 4; ++u) fz_combine(cm, cs, sEx[u][tk].x, sEx[u][tk].y);  // the same order in all waves
      const float mn = fmaxf(m_run[mt], cm);
      al[mt] = __expf(m_run[mt] - mn);
      s_run[mt] = s_run[mt] * al[mt] + cs * __expf(cm - mn);
      m_run[mt] = mn;
    }
    // rescale the output rows: row r of an output block is token 8 (r >> 2) + 4 lh + (r & 3)
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float a_r = __shfl(al[mt], 8 * (r >> 2) + 4 * lh + (r & 3));
#pragma unroll
        for (int q = 0; q < NQ; ++q) o[mt][q][r] *= a_r;
      }
    // 3. out += (P_hi + P_lo) Vm[chunk]: k step (mv, ks2) takes the entries r = 8 ks2 .. 8 ks2 + 7
#pragma unroll
    for (int mv = 0; mv < 2; ++mv)
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2) {
        bf16x8_t phi[2], plo[2], bv[NQ];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          uint32_t hv[4], lv[4];
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2) {
            // hi and lo parts rounded to nearest even by the hardware conversion, in pairs
            const int r = 8 * ks2 + 2 * e2;
            const float p0 = valid(mv, r) ? __expf(z[mv][mt][r] - m_run[mt]) : 0.f;
            const float p1 = valid(mv, r + 1) ? __expf(z[mv][mt][r + 1] - m_run[mt]) : 0.f;
            const uint32_t h2 = cvt_pk_bf16(p0, p1);
            hv[e2] = h2;
            lv[e2] = cvt_pk_bf16(p0 - bf16_lo(h2), p1 - bf16_hi(h2));
          }
          phi[mt] = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
          plo[mt] = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
        }
        // B entry e of lane (col, lh): vocabulary 64 wv + 32 mv + 16 ks2 + 8 (e >> 2) + 4 lh + (e & 3)
        const int va = 64 * wv + 32 * mv + 16 * ks2 + 4 * lh, vc = va + 8;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int row = 32 * q + l32;
          const uint8_t* rp = sVt + row * (2 * kFV);
          const uint2 lo4 = *(const uint2*)(rp + 16 * ((va >> 3) ^ fv_swz(row)) + 2 * (va & 7));
          const uint2 hi4 = *(const uint2*)(rp + 16 * ((vc >> 3) ^ fv_swz(row)) + 2 * (vc & 7));
          bv[q] = __builtin_bit_cast(bf16x8_t, make_uint4(lo4.x, lo4.y, hi4.x, hi4.y));
        }
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            o[mt][q] = mfma32(phi[mt], bv[q], o[mt][q]);
            o[mt][q] = mfma32(plo[mt], bv[q], o[mt][q]);
          }
      }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();  // the ring is free: the four vocabulary quarters' outputs meet there
  // partial outputs summed as (O_0 + O_2) + (O_1 + O_3), in a fixed order
  float* red = (float*)ring;  // 2 x 128 tokens x (64 + 4) floats
  constexpr int RLD = kFC + 4;
  auto put = [&](int slot) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          red[(slot * kFR + wt * 64 + 32 * mt + 8 * (r >> 2) + 4 * lh + (r & 3)) * RLD + 32 * q + l32] = o[mt][q][r];
  };
  auto add = [&](int slot) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          o[mt][q][r] += red[(slot * kFR + wt * 64 + 32 * mt + 8 * (r >> 2) + 4 * lh + (r & 3)) * RLD + 32 * q + l32];
  };
  if (wv >= 2) put(wv - 2);
  __syncthreads();
  if (wv < 2) add(wv);
  __syncthreads();
  if (wv == 1) put(0);
  __syncthreads();
  if (wv == 0) {
    add(0);
    float* po = part_o + (int64_t)sp * n * c;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int tr = wt * 64 + 32 * mt + 8 * (r >> 2) + 4 * lh + (r & 3);
          const int64_t row = r0 + tr, col = c0 + 32 * q + l32;
          if (row < n && col < c) po[row * c + col] = o[mt][q][r];
        }
    if (ct == 0 && lh == 0)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const int64_t row = r0 + wt * 64 + 32 * mt + l32;
        if (row < n) part_ms[(int64_t)sp * n + row] = make_float2(m_run[mt], s_run[mt]);
      }
  }
}

// dev_info protocol: INT32_MAX while nothing is wrong; atomicMin with 1 + a bad row or with
// LOCA_INFO_NONFINITE (which therefore takes precedence); INT32_MAX becomes 0 at the end
__global__ void k_fused_info_init(int32_t* p) {
  if (threadIdx.x == 0) *p = INT32_MAX;
}
__global__ void k_fused_info_finish(int32_t* p) {
  if (threadIdx.x == 0 && *p == INT32_MAX) *p = 0;
}

// Vm^T (c x ldvt, bf16, zero past V) from Vm given as column groups of kc: entry (v, j) at
// vm[(j / kc) gstride + v ld_vm + j % kc] (one group: kc = c); 32 x 32 tiles via LDS
__global__ void k_vm_transpose(int64_t V, int64_t c, const uint16_t* __restrict__ vm, int64_t ld_vm, int64_t kc,
                               int64_t gstride, uint16_t* __restrict__ vmt, int64_t ldvt) {
  __shared__ uint16_t t[32][33];
  const int64_t v0 = (int64_t)blockIdx.x * 32, j0 = (int64_t)blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int64_t v = v0 + r, j = j0 + tx;
    t[r][tx] = (v < V && j < c) ? vm[(j / kc) * gstride + v * ld_vm + j % kc] : (uint16_t)0;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int64_t j = j0 + r, v = v0 + tx;
    if (j < c && v < ldvt) vmt[j * ldvt + v] = t[tx][r];
  }
}

// out_t = w_t (sum_i O_i[t] e^{m_i - M} / S - Vm[y_t]), S = sum_i s_i e^{m_i - M}: the ranges
// in order, float64.  One workgroup per token.  Column j of Vm and of the output is column
// j % kc of group j / kc (Vm entries as for k_vm_transpose; output at
// out[(j / kc) o_gstride + t ld_out + j % kc]).  A bad label drops the label term and is
// reported; a sum that is not finite or not positive is reported as non-finite data.  With
// ms_out the token's (M, S) are also written as floats (ms_out[2 t], ms_out[2 t + 1]).
__global__ __launch_bounds__(256) void k_fused_combine(int64_t n, int64_t c, int64_t V, int nsp,
                                                       const float* __restrict__ part_o,
                                                       const float2* __restrict__ part_ms,
                                                       const int32_t* __restrict__ labels, const float* __restrict__ w,
                                                       const uint16_t* __restrict__ vm, int64_t ld_vm, int64_t kc,
                                                       int64_t gstride, float* __restrict__ out, int64_t ld_out,
                                                       int64_t o_gstride, float* __restrict__ ms_out,
                                                       int32_t* __restrict__ info) {
  __shared__ double sc[kMaxFusedSplits];
  const int64_t t = blockIdx.x;
  // every range holds a valid chunk, so each finite s_i is at least 1
  double M = -__builtin_inf();
  for (int i = 0; i < nsp; ++i) M = fmax(M, (double)part_ms[(int64_t)i * n + t].x);
  double S = 0.0;
  for (int i = 0; i < nsp; ++i) {
    const float2 ms = part_ms[(int64_t)i * n + t];
    const double e = exp((double)ms.x - M);
    S += (double)ms.y * e;
    if ((int)threadIdx.x == i) sc[i] = e;
  }
  __syncthreads();
  const int32_t y = labels[t];
  const bool bad = y < 0 || (int64_t)y >= V;
  const bool nonfin = !isfinite(M) || !isfinite(S) || !(S > 0.0);
  if (threadIdx.x == 0) {
    if (bad) atomicMin(info, (int32_t)(t + 1));
    if (nonfin) atomicMin(info, (int32_t)LOCA_INFO_NONFINITE);
    if (ms_out) {
      ms_out[2 * t] = (float)M;
      ms_out[2 * t + 1] = (float)S;
    }
  }
  const double wt = w ? (double)w[t] : 1.0;
  const double inv = nonfin ? 0.0 : 1.0 / S;
  for (int64_t j = threadIdx.x; j < c; j += blockDim.x) {
    double acc = 0.0;
    for (int i = 0; i < nsp; ++i) acc += (double)part_o[((int64_t)i * n + t) * c + j] * sc[i];
    const int64_t g = j / kc, jc = j - g * kc;
    const double lab = bad ? 0.0 : (double)__uint_as_float((uint32_t)vm[g * gstride + (int64_t)y * ld_vm + jc] << 16);
    out[g * o_gstride + t * ld_out + jc] = (float)(wt * (acc * inv - lab));
  }
}

// ------------------------------------------------------------------ single pass over stored logits
// The head error of Lemma S3.1 applied to a right operand from stored logits in one pass
// (what k_softmax_stats and k_top_error_gemm compute in two): a wave owns 32 tokens and the
// 64 columns of a tile of Vm, a workgroup 128 tokens, and walks a range of the vocabulary
// in steps of 16 entries, one k step of v_mfma_f32_32x32x16_bf16.  The logits enter as the
// A operand (lane l: token l % 32, the 8 entries 8 (l / 32) .. 8 (l / 32) + 7 of the step),
// under an online softmax whose running maximum is raised only when a chunk of 64 entries
// exceeds it (the accumulated rows are then rescaled); P = exp(z - m) is split into bf16
// hi + lo against the bf16 Vm^T slice.  Both are copied straight into LDS by buffer loads:
// the logits through a three-slot ring, two chunks ahead, and the Vm^T slice (read from L2,
// where the tiles of one vocabulary range on an XCD share it) double-buffered one chunk
// ahead; one barrier per chunk.  ZT: bf16 (uint16_t, ld % 8 == 0) or float (ld % 4 == 0) logits with
// 16-byte aligned rows; entries past V are masked, reads stay inside the row's stride.
constexpr int kOnlineChunk = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kOnlineStages = 3;  // logits ring slots: two chunks in flight while one is read
// LDS staging of a chunk's logits: 128 token rows of 64 entries (bf16: 128 bytes, 8 chunks of
// 16 bytes; float: 256 bytes, 16 chunks), chunk c of row r at position c ^ swz(r), so that the
// 16 lanes of a half wave reading one chunk of 16 consecutive rows hit distinct bank groups.
template <typename ZT> LOCA_DEV int zo_swz(int r) { return sizeof(ZT) == 2 ? ((r >> 1) & 7) : (r & 15); }
// the Vm^T slice of a chunk: 64 rows (columns of Vm) of 64 entries (128 bytes), swizzled alike
LOCA_DEV int bo_swz(int r) { return (r >> 1) & 7; }
template <typename ZT>
__global__ __launch_bounds__(256) void k_head_online(int64_t n, int64_t V, const ZT* __restrict__ z, int64_t ldz,
                                                     const uint16_t* __restrict__ vmt, int64_t ldvt, int64_t c,
                                                     int ntr, int nct, int64_t vper, float* __restrict__ part_o,
                                                     float2* __restrict__ part_ms) {
  constexpr int RB = kOnlineChunk * (int)sizeof(ZT);   // bytes per staged logits row
  constexpr int CPR = RB / 16;                         // 16-byte chunks per row
  constexpr int STAGE = 128 * RB;                      // bytes per stage
  constexpr int NA = STAGE / 16 / 256;                 // copies per thread per stage (4 or 8)
  constexpr int RPB = 1024 / RB;                       // rows per 1 KB copy block
  constexpr int KS = kOnlineChunk / 16;
  __shared__ __attribute__((aligned(1024))) uint8_t ring[kOnlineStages * STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t sB[2][64 * 128];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, l32 = lane & 31, lh = lane >> 5;
  const int wq = __builtin_amdgcn_readfirstlane(wid);
  const int logical = xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int rt = logical % ntr, ct = (logical / ntr) % nct, sp = logical / (ntr * nct);
  const int64_t r0 = (int64_t)rt * 128;
  const int64_t tok0 = r0 + 32 * wid;
  const int64_t t = tok0 + l32;
  const int64_t c0 = (int64_t)ct * 64;
  const int64_t vb = (int64_t)sp * vper, ve = (vb + vper < V) ? vb + vper : V;
  const int nchunk = (int)((ve - vb + kOnlineChunk - 1) / kOnlineChunk);
  // byte offsets fit 31 bits: 128 rows x ldz and 64 rows x ldvt (V <= 2^23 is checked)
  const int64_t nrow = (n - r0 < 128) ? n - r0 : 128;
  const i32x4_t rsZ = buffer_rsrc(z + r0 * ldz, (uint32_t)(nrow * ldz * sizeof(ZT)));
  const int64_t ncol = (c - c0 < 64) ? c - c0 : 64;
  const i32x4_t rsB = buffer_rsrc(vmt + c0 * ldvt, (uint32_t)(ncol * ldvt * 2));
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(LOCA_LDS void*)ring;
  const uint32_t sb_lds = (uint32_t)(uintptr_t)(LOCA_LDS void*)sB;
  auto issue_a = [&](int g) {  // chunk g's logits into ring slot g % 3 (entries past the row's data masked later)
    const int64_t v0 = vb + (int64_t)g * kOnlineChunk;
    const uint32_t slot = ring_lds + (uint32_t)((g % kOnlineStages) * STAGE);
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      const int blk = wq * NA + j;
      const int row = RPB * blk + lane / CPR, pos = lane % CPR;
      const int ch = pos ^ zo_swz<ZT>(row);
      const uint32_t off = (uint32_t)((row * ldz + v0) * (int64_t)sizeof(ZT)) + 16u * (uint32_t)ch;
      lds_dma16_buf(off, rsZ, slot + (uint32_t)blk * 1024u);
    }
  };
  auto issue_b = [&](int g) {  // chunk g's Vm^T slice into sB[g & 1] (rows of 64 entries, zero past V and c)
    const int64_t v0 = vb + (int64_t)g * kOnlineChunk;
    const uint32_t base = sb_lds + (uint32_t)((g & 1) * 64 * 128);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int blk = wq * 2 + j;  // 1 KB = 8 rows of 128 bytes
      const int row = 8 * blk + (lane >> 3), pos = lane & 7;
      const uint32_t off = 2u * (uint32_t)(row * ldvt + v0 + 8 * (pos ^ bo_swz(row)));
      lds_dma16_buf(off, rsB, base + (uint32_t)blk * 1024u);
    }
  };
  auto wait_vm = [&](int a) {
    if (a == NA) __builtin_amdgcn_s_waitcnt(vmcnt_imm(NA));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };
  f32x16_t o[2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[q][r] = 0.f;
  float m_run = -__builtin_inff(), s_lane = 0.f;
  // prologue: chunks 0 .. kOnlineStages - 2 and the first Vm^T slice
  for (int g = 0; g < kOnlineStages - 1 && g < nchunk; ++g) issue_a(g);
  issue_b(0);
  const int arow = 32 * wid + l32;
  for (int g = 0; g < nchunk; ++g) {
    // chunk g's logits (issued kOnlineStages - 1 iterations ago) and its Vm^T slice (issued at
    // the top of iteration g - 1, before chunk g + 1's logits): only that copy may be pending
    wait_vm(g >= 1 && g + kOnlineStages - 2 < nchunk ? NA : 0);
    __syncthreads();  // every thread's copies landed; the slots refilled below are free
    if (g + 1 < nchunk) issue_b(g + 1);
    if (g + kOnlineStages - 1 < nchunk) issue_a(g + kOnlineStages - 1);
    const int64_t v0 = vb + (int64_t)g * kOnlineChunk;
    const uint8_t* st = ring + (g % kOnlineStages) * STAGE;
    const uint8_t* sb = sB[g & 1];
    // the chunk's logits of this lane's token: entry e of step ks is vocabulary v0 + 16 ks + 8 lh + e
    float zv[KS][8];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if constexpr (sizeof(ZT) == 2) {
        const int ch = 2 * ks + lh;
        const uint4 u = *(const uint4*)(st + arow * RB + 16 * (ch ^ zo_swz<ZT>(arow)));
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          zv[ks][2 * e] = __uint_as_float(w4[e] << 16);
          zv[ks][2 * e + 1] = __uint_as_float(w4[e] & 0xffff0000u);
        }
      } else {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int ch = 4 * ks + 2 * lh + h;
          const uint4 u = *(const uint4*)(st + arow * RB + 16 * (ch ^ zo_swz<ZT>(arow)));
          zv[ks][4 * h] = __uint_as_float(u.x);
          zv[ks][4 * h + 1] = __uint_as_float(u.y);
          zv[ks][4 * h + 2] = __uint_as_float(u.z);
          zv[ks][4 * h + 3] = __uint_as_float(u.w);
        }
      }
    }
    if (v0 + kOnlineChunk > ve) {  // the range's ragged last chunk: entries past ve out (p = 0)
      const int rem = (int)(ve - v0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (16 * ks + 8 * lh + e >= rem) zv[ks][e] = -__builtin_inff();
    }
    float cm = -__builtin_inff();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) cm = fmaxf(cm, zv[ks][e]);
    cm = fmaxf(cm, __shfl_xor(cm, 32));
    if (__any(cm > m_run)) {  // raise the running maximum of the tokens that need it
      const float mn = fmaxf(m_run, cm);
      const float al = __expf(m_run - mn);
      s_lane *= al;
      m_run = mn;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float a_r = __shfl(al, 8 * (r >> 2) + 4 * lh + (r & 3));
#pragma unroll
        for (int q = 0; q < 2; ++q) o[q][r] *= a_r;
      }
    }
    const float m2 = m_run * kLog2e;  // exp(z - m) = 2^(z log2(e) - m log2(e))
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint32_t hv[4], lv[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        // p = exp(z - m), 0 for the masked entries (m_run is finite); hi and lo parts rounded
        // to nearest even by the hardware conversion, two values per instruction
        const float p0 = __builtin_amdgcn_exp2f(fmaf(zv[ks][2 * e2], kLog2e, -m2)),
                    p1 = __builtin_amdgcn_exp2f(fmaf(zv[ks][2 * e2 + 1], kLog2e, -m2));
        s_lane += p0;
        s_lane += p1;
        const uint32_t h2 = cvt_pk_bf16(p0, p1);
        hv[e2] = h2;
        lv[e2] = cvt_pk_bf16(p0 - bf16_lo(h2), p1 - bf16_hi(h2));
      }
      const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
      const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        // B lane l: Vm[v0 + 16 ks + 8 lh + e][c0 + 32 q + l % 32] = Vm^T row 32 q + l % 32
        const int row = 32 * q + l32, ch = 2 * ks + lh;
        const bf16x8_t bq = *(const bf16x8_t*)(sb + row * 128 + 16 * (ch ^ bo_swz(row)));
        o[q] = mfma32(phi, bq, o[q]);
        o[q] = mfma32(plo, bq, o[q]);
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  const float s_tok = s_lane + __shfl_xor(s_lane, 32);
  float* po = part_o + (int64_t)sp * n * c;
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = tok0 + 8 * (r >> 2) + 4 * lh + (r & 3), col = c0 + 32 * q + l32;
      if (row < n && col < c) po[row * c + col] = o[q][r];
    }
  if (ct == 0 && lh == 0 && t < n) part_ms[(int64_t)sp * n + t] = make_float2(m_run, s_tok);
}

struct FusedPlan {
  int ct, ntr, nct, nsp;
  int64_t vper, ldvt;
};

FusedPlan fused_plan(int64_t n, int64_t V, int64_t c) {
  FusedPlan p;
  p.ct = kFC;  // a wider column tile holds more accumulators than the register file keeps
  p.ntr = (int)((n + kFR - 1) / kFR);
  p.nct = (int)((c + p.ct - 1) / p.ct);
  const int64_t tiles = (int64_t)p.ntr * p.nct, nchunk = (V + kFV - 1) / kFV;
  int64_t want = (1024 + tiles - 1) / tiles;  // about four workgroups per compute unit
  if (want > kMaxFusedSplits) want = kMaxFusedSplits;
  if (want > nchunk) want = nchunk;
  if (want < 1) want = 1;
  p.vper = ((nchunk + want - 1) / want) * kFV;
  p.nsp = (int)((V + p.vper - 1) / p.vper);  // every range holds at least one chunk
  p.ldvt = nchunk * kFV;
  return p;
}

}  // namespace

namespace {
struct OnlinePlan {
  int ntr, nct, nsp;
  int64_t vper, ldvt;
};
OnlinePlan online_plan(int64_t n, int64_t V, int64_t cols) {
  OnlinePlan p;
  p.ntr = (int)((n + 127) / 128);
  p.nct = (int)((cols + 63) / 64);
  const int64_t tiles = (int64_t)p.ntr * p.nct, nchunk = (V + kOnlineChunk - 1) / kOnlineChunk;
  int64_t want = (512 + tiles - 1) / tiles;  // about two workgroups per compute unit
  if (want > kMaxFusedSplits) want = kMaxFusedSplits;
  if (want > nchunk) want = nchunk;
  if (want < 1) want = 1;
  p.vper = ((nchunk + want - 1) / want) * kOnlineChunk;
  p.nsp = (int)((V + p.vper - 1) / p.vper);
  p.ldvt = nchunk * kOnlineChunk;
  return p;
}
}  // namespace

size_t softmax_product_online_ws(int64_t n, int64_t V, int64_t cols) {
  const OnlinePlan p = online_plan(n, V, cols);
  size_t s = align256(sizeof(float) * 2 * n);  // (m, s) per token, first (the e_out writer reads it there)
  s += align256(sizeof(float) * p.nsp * n * cols);
  s += align256(sizeof(float2) * p.nsp * n);
  s += align256(sizeof(uint16_t) * cols * p.ldvt);
  return s;
}

hipError_t launch_softmax_product_online(const SoftmaxProductArgs& a) {
  const int64_t cols = a.groups * a.kc;
  const OnlinePlan p = online_plan(a.n, a.V, cols);
  char* w = a.ws;
  float* ms = (float*)w; w += align256(sizeof(float) * 2 * a.n);
  float* part_o = (float*)w; w += align256(sizeof(float) * p.nsp * a.n * cols);
  float2* part_ms = (float2*)w; w += align256(sizeof(float2) * p.nsp * a.n);
  uint16_t* vmt = (uint16_t*)w;
  hipStream_t st = a.stream;
  k_vm_transpose<<<dim3((unsigned)((p.ldvt + 31) / 32), (unsigned)((cols + 31) / 32)), 256, 0, st>>>(
      a.V, cols, a.W, a.kc, a.kc, a.w_bstride, vmt, p.ldvt);
  const unsigned grid = (unsigned)((int64_t)p.ntr * p.nct * p.nsp);
  if (a.logits_dtype == LOCA_BF16)
    k_head_online<uint16_t><<<grid, 256, 0, st>>>(a.n, a.V, (const uint16_t*)a.logits, a.ld_logits, vmt, p.ldvt,
                                                   cols, p.ntr, p.nct, p.vper, part_o, part_ms);
  else
    k_head_online<float><<<grid, 256, 0, st>>>(a.n, a.V, (const float*)a.logits, a.ld_logits, vmt, p.ldvt, cols,
                                                p.ntr, p.nct, p.vper, part_o, part_ms);
  k_fused_combine<<<(unsigned)a.n, 256, 0, st>>>(a.n, cols, a.V, p.nsp, part_o, part_ms, a.labels, a.w, a.W, a.kc,
                                                 a.kc, a.w_bstride, a.out, a.ld_o, a.o_bstride, ms, a.dev_info);
  return hipGetLastError();
}

size_t fused_head_ws(int64_t n, int64_t V, int64_t c) {
  const FusedPlan p = fused_plan(n, V, c);
  size_t s = align256(sizeof(float) * p.nsp * n * c);
  s += align256(sizeof(float2) * p.nsp * n);
  s += align256(sizeof(uint16_t) * c * p.ldvt);
  return s;
}

hipError_t launch_fused_head(const FusedArgs& a) {
  const FusedPlan p = fused_plan(a.n, a.V, a.c);
  char* w = a.ws;
  float* part_o = (float*)w; w += align256(sizeof(float) * p.nsp * a.n * a.c);
  float2* part_ms = (float2*)w; w += align256(sizeof(float2) * p.nsp * a.n);
  uint16_t* vmt = (uint16_t*)w;
  hipStream_t st = a.stream;
  k_fused_info_init<<<1, 64, 0, st>>>(a.dev_info);
  k_vm_transpose<<<dim3((unsigned)((p.ldvt + 31) / 32), (unsigned)((a.c + 31) / 32)), 256, 0, st>>>(
      a.V, a.c, a.vm, a.ld_vm, a.c, 0, vmt, p.ldvt);
  const unsigned grid = (unsigned)((int64_t)p.ntr * p.nct * p.nsp);
  k_fused_head<<<grid, kFT, 0, st>>>(a.n, a.V, a.d, a.c, a.h, a.ldh, a.wu, vmt, p.ldvt, p.ntr, p.nct, p.vper,
                                          part_o, part_ms);
  k_fused_combine<<<(unsigned)a.n, 256, 0, st>>>(a.n, a.c, a.V, p.nsp, part_o, part_ms, a.labels, a.w, a.vm, a.ld_vm,
                                                 a.c, 0, a.out, a.ld_out, 0, nullptr, a.dev_info);
  k_fused_info_finish<<<1, 64, 0, st>>>(a.dev_info);
  return hipGetLastError();
}

}  // namespace loca
