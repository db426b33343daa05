// k_error.hip -- head error and credit coordinates (rows a1, a2 of the step).
//
// Lemma S3.1: E_t = w_t (softmax(z_t) - onehot(y_t)).  Sections S3 / S11: the
// feedback is applied through the rank-k factors, Y = E A~, and the
// denominator of the scale-normalised step (Eq. 10) is
// ||Q||_F^2 = sum_t Y_t (B~ B~^T) Y_t^T, so Q = Y B~ is never formed.
//
// Two kernels:
//  * small label sets (C <= 64): one thread per token; A~ and G = B~ B~^T are
//    staged in LDS; softmax in fp32 with the row maximum subtracted.
//  * large vocabularies: one workgroup per group of tokens streams the logits
//    once with an online (running-max) softmax, accumulating the rescaled
//    sum of exp(z - m) A~[c] alongside; Y = acc / s - A~[y].
// Both write per-workgroup partial sums of ||Q||^2 (fp64) that a finalize
// kernel adds in a fixed order, so results are bitwise reproducible.
#include <mutex>

#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kSmallThreads = 256;
constexpr int kSmallMaxC = 64;
constexpr int kSmallMaxK = 64;
constexpr int kMaxK = 128;

// G_b = B~_b B~_b^T (k x k, float64) in two passes.  k_credit_gram_part: one workgroup per
// (one of kCGSplit ranges of the width d, block): the k rows of B~ over the range stream
// through LDS in 64-column chunks (each load instruction one row's 64 consecutive columns;
// the next chunk held in registers while the current one is used), and the four waves take
// the 16 x 16 blocks on or above the diagonal in turn (block u to wave u % 4), each formed on
// the fp64 matrix cores in the order of the columns; every row of B~ is read once.
// k_credit_gram_sum adds the kCGSplit partials of an entry in a fixed order and writes it
// and its mirror: deterministic.
constexpr int kCGSplit = 8, kCGC = 64, kCGLd = kCGC + 4;  // row stride 68: conflict-free MFMA reads
template <int KR>  // rows staged: k rounded up to a multiple of 16 (at most 128)
__global__ __launch_bounds__(256) void k_credit_gram_part(int64_t k, int64_t d, const float* __restrict__ B,
                                                          int64_t b_bstride, double* __restrict__ part) {
  constexpr int NB16 = KR / 16, NUP = NB16 * (NB16 + 1) / 2, PER = (NUP + 3) / 4, RPT = KR / 4;
  __shared__ float sB[KR * kCGLd];
  const int64_t s = blockIdx.x, b = blockIdx.y;
  const float* Bb = B + b * b_bstride;
  const int64_t chunk = ((d + kCGSplit - 1) / kCGSplit + kCGC - 1) / kCGC * kCGC;
  const int64_t i0 = s * chunk, i1 = i0 + chunk < d ? i0 + chunk : d;
  const int t = threadIdx.x, lc = t & 63, wv = t >> 6, kr = (t & 63) >> 4, cr = t & 15;
  // this wave's blocks (I, J), I <= J, in row-major order of the upper triangle
  int bI[PER], bJ[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    int u = wv + 4 * q, I = 0;
    while (I < NB16 && u >= NB16 - I) { u -= NB16 - I; ++I; }
    bI[q] = I;
    bJ[q] = I + u;  // I == NB16 past the last block: no such block
  }
  f64x4_t acc[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) acc[q] = f64x4_t{0.0, 0.0, 0.0, 0.0};
  float v[RPT];  // rows wv + 4 e, column lc of the chunk
  auto load = [&](int64_t j0) {
    const int64_t col = j0 + lc;
#pragma unroll
    for (int e = 0; e < RPT; ++e) {
      const int r = wv + 4 * e;
      v[e] = (r < k && col < i1) ? Bb[r * d + col] : 0.f;
    }
  };
  if (i0 < i1) load(i0);
  for (int64_t j0 = i0; j0 < i1; j0 += kCGC) {
    __syncthreads();  // the previous chunk is no longer read
#pragma unroll
    for (int e = 0; e < RPT; ++e) sB[(wv + 4 * e) * kCGLd + lc] = v[e];
    __syncthreads();
    if (j0 + kCGC < i1) load(j0 + kCGC);
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      if (bI[q] >= NB16) break;
      const float* ra = sB + (16 * bI[q] + cr) * kCGLd + kr;  // A[i][x] = B~[16 I + i][x]
      const float* rc = sB + (16 * bJ[q] + cr) * kCGLd + kr;  // B[x][j] = B~[16 J + j][x]
#pragma unroll
      for (int kk = 0; kk < kCGC; kk += 4) acc[q] = mfma_f64((double)ra[kk], (double)rc[kk], acc[q]);
    }
  }
  double* P = part + ((s * (int64_t)gridDim.y + b) * k) * k;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    if (bI[q] >= NB16) break;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = 16 * bI[q] + kr + 4 * r, col = 16 * bJ[q] + cr;
      if (row < k && col < k) P[row * k + col] = acc[q][r];
    }
  }
}
// G is written with row stride ldg >= k, zero in the rows and columns past k.
__global__ void k_credit_gram_sum(int64_t k, int64_t ldg, int64_t nb, const double* __restrict__ part,
                                  double* __restrict__ G) {
  const int64_t b = blockIdx.y, e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= ldg * ldg) return;
  const int64_t a = e / ldg, c = e % ldg;
  if (a > c) return;  // written as the mirror of (c, a)
  double v = 0.0;
  if (c < k)
    for (int s = 0; s < kCGSplit; ++s) v += part[((s * nb + b) * k + a) * k + c];
  G[(b * ldg + a) * ldg + c] = v;
  G[(b * ldg + c) * ldg + a] = v;
}
static void launch_credit_gram(hipStream_t st, int64_t nb, int64_t k, int64_t d, const float* B, int64_t b_bstride,
                               double* part, double* G, int64_t ldg) {
  const dim3 g((unsigned)kCGSplit, (unsigned)nb);
  if (k <= 16) k_credit_gram_part<16><<<g, 256, 0, st>>>(k, d, B, b_bstride, part);
  else if (k <= 32) k_credit_gram_part<32><<<g, 256, 0, st>>>(k, d, B, b_bstride, part);
  else if (k <= 64) k_credit_gram_part<64><<<g, 256, 0, st>>>(k, d, B, b_bstride, part);
  else k_credit_gram_part<128><<<g, 256, 0, st>>>(k, d, B, b_bstride, part);
  k_credit_gram_sum<<<dim3((unsigned)((ldg * ldg + 255) / 256), (unsigned)nb), 256, 0, st>>>(k, ldg, nb, part, G);
}
static size_t credit_gram_part_ws(int64_t nb, int64_t k) { return align256(sizeof(double) * kCGSplit * nb * k * k); }

// One thread per token; A~ (C x k, [c][j]) sits in LDS.  Each wave then stages its 64 rows of
// Y (KB columns, zero past k and past n) in an LDS tile, from which it
//   * writes Y to HBM as whole rows of consecutive tokens, and
//   * forms its share of ||Q||^2 = sum_t a_t y_t G y_t^T = <G, sum_t a_t y_t y_t^T> with the
//     fp64 matrix cores: M_w = sum over its tokens of (a_t y_t) y_t^T in 16 x 16 blocks on or
//     above the diagonal (v_mfma_f64_16x16x4f64, products of floats exact in fp64), then
//     each lane multiplies its entries of M_w by those of G (KB x KB, zero past k; blocks off
//     the diagonal count twice).
// The tile reuses the A~ area once it is consumed.
// HC > 0 (label sets of C <= HC classes): since y_t = e_t A~, the same sum is
// sum_t a_t e_t H e_t^T with the C x C matrix H = A~ G A~^T (fp64, formed in LDS by every
// workgroup), HC^2 fp64 FMAs per token in place of the matrix-core pass over the tile.
static int64_t small_kb(int64_t k) { return k <= 16 ? 16 : k <= 32 ? 32 : 64; }
template <int KB>
struct SmallLds {
  static constexpr int WST = 64 * (KB + 1);            // floats of a wave's tile (odd row stride)
  static constexpr int IN = kSmallMaxC * KB * 4;
  static constexpr int ST = 4 * WST * 4;
  static constexpr int BYTES = IN > ST ? IN : ST;
};

template <typename LT, typename AT, int KB, int HC>
__global__ __launch_bounds__(kSmallThreads) void k_error_small(
    int64_t n, int64_t C, int64_t k, const LT* __restrict__ logits, int64_t ld,
    const int32_t* __restrict__ labels, const float* __restrict__ w, const float* __restrict__ aw,
    const AT* __restrict__ A, int64_t a_bstride, const double* __restrict__ G, float* __restrict__ y_out,
    int64_t y_bstride, float* __restrict__ e_out, double* __restrict__ partial, int32_t* __restrict__ dev_info) {
  using L = SmallLds<KB>;
  static_assert(kSmallThreads == 256, "four waves");
  constexpr int NB = KB / 16;  // 16-column blocks
  __shared__ __attribute__((aligned(16))) unsigned char lds[L::BYTES];
  __shared__ float sW[kSmallThreads];  // statistic weight of each token (0 past n)
  __shared__ double sred[kSmallThreads / 64];
  __shared__ double sAG[HC > 0 ? HC * KB : 1];  // A~ G (HC x KB)
  __shared__ double sH[HC > 0 ? HC * HC : 1];   // A~ G A~^T, zero past C
  float* sA = (float*)lds;  // C x KB, zero past k (the products below need no bound)
  const int64_t b = blockIdx.y;
  const AT* Ab = A + b * a_bstride;
  const double* Gb = G + b * KB * KB;
  for (int64_t e = threadIdx.x; e < C * KB; e += blockDim.x) {
    const int64_t c = e / KB, j = e % KB;
    sA[e] = j < k ? load_as_f32(Ab + c * k + j) : 0.f;
  }
  __syncthreads();
  if constexpr (HC > 0) {
    // A~ G: thread (j, iq) = (tid / 4, tid % 4) reads G[i][j] for its quarter of i once (the
    // loads issued together) and adds it into all HC rows; the quarters meet by shuffles
    static_assert(kSmallThreads == 4 * 64, "64 columns x 4 quarters");
    const int j = (int)threadIdx.x >> 2, iq = (int)threadIdx.x & 3;
    constexpr int IQ = KB / 4;
    if (j < KB) {
      double g[IQ];
#pragma unroll
      for (int ii = 0; ii < IQ; ++ii) g[ii] = Gb[(iq * IQ + ii) * KB + j];
      double v[HC];
#pragma unroll
      for (int c = 0; c < HC; ++c) {
        v[c] = 0.0;
#pragma unroll
        for (int ii = 0; ii < IQ; ++ii) v[c] = fma((double)sA[(c < C ? c : 0) * KB + iq * IQ + ii], g[ii], v[c]);
      }
#pragma unroll
      for (int c = 0; c < HC; ++c) {
        v[c] += __shfl_xor(v[c], 1, 64);
        v[c] += __shfl_xor(v[c], 2, 64);
        if (iq == 0) sAG[c * KB + j] = c < C ? v[c] : 0.0;
      }
    }
    __syncthreads();
    for (int e = (int)threadIdx.x; e < HC * HC; e += kSmallThreads) {
      const int c = e / HC, c2 = e % HC;
      double v = 0.0;
      if (c < C && c2 < C)
        for (int j = 0; j < KB; ++j) v = fma(sAG[c * KB + j], (double)sA[c2 * KB + j], v);
      sH[e] = v;
    }
    // sH is read after the barrier below that retires the reads of sA
  }

  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  float y[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) y[j] = 0.f;
  float wq = 0.f;  // weight of this token in ||Q||^2
  float ev[HC > 0 ? HC : 1];  // this token's error row (HC > 0), zero past C
#pragma unroll
  for (int c = 0; c < (HC > 0 ? HC : 1); ++c) ev[c] = 0.f;
  if (t < n) {
    const LT* zt = logits + t * ld;
    const int32_t yt = labels[t];
    if (yt < 0 || yt >= C) {
      atomicMin(dev_info, (int32_t)(t + 1));
    } else {
      // the logits in chunks of 8 classes, each chunk's loads issued together (held in
      // registers for the three passes when C <= 8)
      float zc[8];
      auto chunk = [&](int64_t c0) {
#pragma unroll
        for (int u = 0; u < 8; ++u) zc[u] = c0 + u < C ? load_as_f32(zt + c0 + u) : -INFINITY;
      };
      chunk(0);
      float m = zc[0];
      for (int64_t c0 = 0; c0 < C; c0 += 8) {
        if (c0 > 0) chunk(c0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (c0 + u < C) m = fmaxf(m, zc[u]);
      }
      float s = 0.f;
      for (int64_t c0 = 0; c0 < C; c0 += 8) {
        if (c0 > 0 || C > 8) chunk(c0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (c0 + u < C) s += __expf(zc[u] - m);
      }
      const float inv = 1.0f / s;
      const float wt = w ? w[t] : 1.0f;
      if constexpr (HC > 0) {  // the chunks unrolled, so that ev is indexed by constants
#pragma unroll
        for (int c0 = 0; c0 < HC; c0 += 8) {
          if (c0 >= C) break;
          if (c0 > 0 || C > 8) chunk(c0);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int c = c0 + u;
            if (c >= C) break;
            const float e = wt * (__expf(zc[u] - m) * inv - (c == yt ? 1.0f : 0.0f));
            if (e_out) e_out[t * C + c] = e;
            ev[c] = e;
#pragma unroll
            for (int j = 0; j < KB; ++j) y[j] = fmaf(e, sA[c * KB + j], y[j]);
          }
        }
      } else {
        for (int64_t c0 = 0; c0 < C; c0 += 8) {
          if (c0 > 0 || C > 8) chunk(c0);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int64_t c = c0 + u;
            if (c >= C) break;
            const float e = wt * (__expf(zc[u] - m) * inv - (c == yt ? 1.0f : 0.0f));
            if (e_out) e_out[t * C + c] = e;
#pragma unroll
            for (int j = 0; j < KB; ++j) y[j] = fmaf(e, sA[c * KB + j], y[j]);
          }
        }
      }
      wq = aw ? aw[t] : 1.0f;  // statistic weight of the position
    }
  }
  __syncthreads();  // every read of sA retired: the area becomes the waves' tiles

  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  float* sT = (float*)lds + wv * L::WST;  // [token of the wave][KB + 1]
#pragma unroll
  for (int j = 0; j < KB; ++j) sT[lane * (KB + 1) + j] = y[j];
  sW[threadIdx.x] = wq;
  wave_lds_sync();

  // Y rows to HBM: each store instruction covers consecutive tokens' whole rows (with k = KB
  // and 16-byte aligned rows, 16-byte stores of 256 / KB tokens, every value read from the
  // tile before the first store)
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + 64 * wv;
  float* yb = y_out + b * y_bstride;
  if (k == KB && (y_bstride & 3) == 0 && ((uintptr_t)y_out & 15) == 0) {
    constexpr int R4 = KB / 4;  // 16-byte chunks per row, and per lane
    float4 v[R4];
#pragma unroll
    for (int i = 0; i < R4; ++i) {
      const int e = lane + 64 * i, p = e / R4, c4 = 4 * (e % R4);
      const float* src = sT + p * (KB + 1) + c4;
      v[i] = make_float4(src[0], src[1], src[2], src[3]);
    }
#pragma unroll
    for (int i = 0; i < R4; ++i) {
      const int e = lane + 64 * i, p = e / R4, c4 = 4 * (e % R4);
      const int64_t tp = t0 + p;
      if (tp < n) *(float4*)(yb + tp * KB + c4) = v[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < KB; ++i) {
      const int e = lane + 64 * i, p = e / KB, c = e % KB;
      const int64_t tp = t0 + p;
      if (tp < n && c < k) yb[tp * k + c] = sT[p * (KB + 1) + c];
    }
  }

  if constexpr (HC > 0) {  // a_t e_t H e_t^T of this thread's token (ev and wq zero past n)
    double q = 0.0;
#pragma unroll
    for (int c = 0; c < HC; ++c) {
      double u = 0.0;
#pragma unroll
      for (int c2 = 0; c2 < HC; ++c2) u = fma(sH[c * HC + c2], (double)ev[c2], u);
      q = fma((double)ev[c], u, q);
    }
    const double tot = block_sum((double)wq * q, sred);
    if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
    return;
  }

  // this wave's part of ||Q||^2
  const float* sWw = sW + 64 * wv;
  const int kr = lane >> 4, cr = lane & 15;
  double q = 0.0;
#pragma unroll
  for (int ab = 0; ab < NB; ++ab)
#pragma unroll
    for (int cb = ab; cb < NB; ++cb) {
      f64x4_t acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int tt = 0; tt < 64; tt += 4) {
        const int p = tt + kr;
        const double av = (double)sWw[p] * (double)sT[p * (KB + 1) + 16 * ab + cr];  // A[i][kk] = a_t y_t[i]
        const double bv = (double)sT[p * (KB + 1) + 16 * cb + cr];                  // B[kk][j] = y_t[j]
        acc = mfma_f64(av, bv, acc);
      }
      const double mult = ab == cb ? 1.0 : 2.0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * ab + kr + 4 * r, col = 16 * cb + cr;
        q += mult * acc[r] * Gb[row * KB + col];
      }
    }
  const double tot = block_sum(q, sred);
  if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
}

// Large vocabulary (or k > 64): TOK tokens per workgroup, 256 threads = TOK x LPT
// lanes per token; lane ln of a token owns credit columns j = ln + q * LPT.
constexpr int kLargeThreads = 256;
constexpr int kLargeTok = 16;
constexpr int kLargeChunk = 256;
constexpr int kLargeLPT = kLargeThreads / kLargeTok;        // 16
constexpr int kLargeKPL = kMaxK / kLargeLPT;                // 8

template <typename LT, typename AT>
__global__ __launch_bounds__(kLargeThreads) void k_error_large(
    int64_t n, int64_t C, int64_t k, const LT* __restrict__ logits, int64_t ld,
    const int32_t* __restrict__ labels, const float* __restrict__ w, const float* __restrict__ aw,
    const AT* __restrict__ A, int64_t a_bstride, const double* __restrict__ G, int64_t ldg, float* __restrict__ y_out,
    int64_t y_bstride, float* __restrict__ ms_out, double* __restrict__ partial, int32_t* __restrict__ dev_info) {
  constexpr int LPT = kLargeLPT;
  __shared__ float sZ[kLargeTok][kLargeChunk];
  __shared__ float sAc[kLargeChunk][kMaxK];
  __shared__ float sY[kLargeTok][kMaxK];
  __shared__ double sred[kLargeThreads / 64];
  const int64_t b = blockIdx.y;
  const AT* Ab = A + b * a_bstride;
  const int tid = threadIdx.x;
  const int tk = tid / LPT, ln = tid % LPT;
  const int64_t t0 = (int64_t)blockIdx.x * kLargeTok;
  const int64_t t = t0 + tk;
  float acc[kLargeKPL];
#pragma unroll
  for (int q = 0; q < kLargeKPL; ++q) acc[q] = 0.f;
  float m_run = -INFINITY, s_run = 0.f;  // identical in all lanes of a token
  for (int64_t c0 = 0; c0 < C; c0 += kLargeChunk) {
    const int cw = (int)((C - c0) < kLargeChunk ? (C - c0) : kLargeChunk);
    __syncthreads();  // previous chunk fully consumed
    for (int e = tid; e < kLargeTok * kLargeChunk; e += kLargeThreads) {
      const int r = e / kLargeChunk, c = e % kLargeChunk;
      const int64_t tr = t0 + r;
      sZ[r][c] = (tr < n && c < cw) ? load_as_f32(logits + tr * ld + c0 + c) : -INFINITY;
    }
    for (int64_t e = tid; e < (int64_t)cw * k; e += kLargeThreads) {
      const int c = (int)(e / k), j = (int)(e % k);
      sAc[c][j] = load_as_f32(Ab + (c0 + c) * k + j);
    }
    __syncthreads();
    float cm = -INFINITY;
    for (int c = ln; c < cw; c += LPT) cm = fmaxf(cm, sZ[tk][c]);
    for (int off = LPT / 2; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, kWave));
    const float m_new = fmaxf(m_run, cm);
    const float scale = (m_run == -INFINITY) ? 0.f : __expf(m_run - m_new);
    float ps = 0.f;
    for (int c = ln; c < cw; c += LPT) {
      const float p = (m_new == -INFINITY) ? 0.f : __expf(sZ[tk][c] - m_new);
      sZ[tk][c] = p;
      ps += p;
    }
    for (int off = LPT / 2; off > 0; off >>= 1) ps += __shfl_xor(ps, off, kWave);
    s_run = s_run * scale + ps;
    m_run = m_new;
    __syncthreads();  // sZ now holds exp(z - m_new)
#pragma unroll
    for (int q = 0; q < kLargeKPL; ++q) acc[q] *= scale;
    for (int c = 0; c < cw; ++c) {
      const float p = sZ[tk][c];
#pragma unroll
      for (int q = 0; q < kLargeKPL; ++q) {
        const int j = ln + q * LPT;
        if (j < k) acc[q] = fmaf(p, sAc[c][j], acc[q]);
      }
    }
  }
  double qv = 0.0;
  if (t < n) {
    const int32_t yt = labels[t];
    const bool ok = (yt >= 0 && yt < C);
    if (!ok && ln == 0) atomicMin(dev_info, (int32_t)(t + 1));
    const float inv = 1.0f / s_run;
    const float wt = w ? w[t] : 1.0f;
#pragma unroll
    for (int q = 0; q < kLargeKPL; ++q) {
      const int j = ln + q * LPT;
      if (j < k) {
        const float ay = ok ? load_as_f32(Ab + (int64_t)yt * k + j) : 0.f;
        const float yv = wt * (acc[q] * inv - ay);
        sY[tk][j] = yv;
        y_out[b * y_bstride + t * k + j] = yv;
      }
    }
    if (ms_out && ln == 0) { ms_out[2 * t] = m_run; ms_out[2 * t + 1] = s_run; }
  }
  __syncthreads();
  if (t < n) {
    const double* Gb = G + b * ldg * ldg;
    for (int a2 = ln; a2 < k; a2 += LPT) {
      double r = 0.0;
      for (int c = 0; c < k; ++c) r += Gb[a2 * ldg + c] * (double)sY[tk][c];
      qv += (double)sY[tk][a2] * r;
    }
    if (aw) qv *= (double)aw[t];  // statistic weight of the position
  }
  const double tot = block_sum(qv, sred);
  if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
}

// E rows for the large-vocabulary path (optional output), from the saved (m, s).
// Tokens t = blockIdx.y, blockIdx.y + gridDim.y, ... (any n with gridDim.y <= 65535).
template <typename LT>
__global__ void k_error_write_e(int64_t n, int64_t C, const LT* __restrict__ logits, int64_t ld,
                                const int32_t* __restrict__ labels, const float* __restrict__ w,
                                const float* __restrict__ ms, float* __restrict__ e_out) {
  for (int64_t t = blockIdx.y; t < n; t += gridDim.y) {
    const float m = ms[2 * t], inv = 1.0f / ms[2 * t + 1];
    const float wt = w ? w[t] : 1.0f;
    const int32_t yt = labels[t];
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < C; c += (int64_t)gridDim.x * blockDim.x)
      e_out[t * C + c] = wt * (__expf(load_as_f32(logits + t * ld + c) - m) * inv - (c == yt ? 1.f : 0.f));
  }
}
static unsigned write_e_rows(int64_t n) { return (unsigned)(n < 65535 ? n : 65535); }

// On entry dev_info holds INT32_MAX (no bad label) or 1 + the smallest bad row.  A block
// whose ||Q||^2 is not finite (a non-finite logit, loss or statistic weight, or credit
// factor: NaN and infinities propagate into every product that uses them) lowers it to
// LOCA_INFO_NONFINITE; INT32_MAX then becomes 0.  The exchange leaves a code another block
// has already written in place, whatever the order of the blocks.
__global__ void k_error_finalize(int64_t n, int64_t nparts, const double* __restrict__ partial,
                                 loca_mb* __restrict__ mb, int32_t* __restrict__ dev_info) {
  // one wave: lane l adds partials l, l + 64, ... in order, then a fixed butterfly across
  // the lanes (deterministic)
  const int64_t b = blockIdx.x;
  double part = 0.0;
  for (int64_t i = threadIdx.x; i < nparts; i += 64) part += partial[b * nparts + i];
  const double s = wave_sum(part);
  if (threadIdx.x != 0) return;
  if (dev_info) {
    if (!__builtin_isfinite(s)) atomicMin(dev_info, (int32_t)LOCA_INFO_NONFINITE);
    if (b == 0) atomicCAS(dev_info, INT32_MAX, 0);
  }
  mb[b].sum_q2 = s;
  mb[b].sum_x2 = 0.0;
  mb[b].eta_bar = 0.0;
  mb[b].n = n;
}

// Paper-order credit coordinates (Section S11): Y_b = e V_k,b (n x k) from the top errors
// e (n x d) and sum_q2 partials as in the error kernels.  64 tokens per workgroup, d in
// chunks of 64 through LDS; thread t owns token t % 64 and the columns t / 64 + 4u (u < KQ),
// fp64 accumulation.
template <int KQ>
__global__ __launch_bounds__(256) void k_credit_project(int64_t n, int64_t d, int64_t k, const float* __restrict__ e,
                                                        int64_t ld_e, const float* __restrict__ Vk, int64_t v_bstride,
                                                        const double* __restrict__ G, const float* __restrict__ aw,
                                                        float* __restrict__ y_out, int64_t y_bstride,
                                                        double* __restrict__ partial) {
  constexpr int KW = 4 * KQ;
  __shared__ float sE[64][65];
  __shared__ float sV[64][KW];
  __shared__ double sY[64][KW + 1];
  __shared__ double sred[4];
  const int64_t b = blockIdx.y;
  const int64_t t0 = (int64_t)blockIdx.x * 64;
  const int tid = threadIdx.x, r = tid & 63, q = tid >> 6;
  const float* V = Vk + b * v_bstride;
  double acc[KQ];
#pragma unroll
  for (int u = 0; u < KQ; ++u) acc[u] = 0.0;
  for (int64_t c0 = 0; c0 < d; c0 += 64) {
    __syncthreads();
    for (int x = tid; x < 64 * 64; x += 256) {
      const int rr = x / 64, cc = x % 64;
      sE[rr][cc] = (t0 + rr < n && c0 + cc < d) ? e[(t0 + rr) * ld_e + c0 + cc] : 0.f;
    }
    for (int x = tid; x < 64 * KW; x += 256) {
      const int cc = x / KW, j = x % KW;
      sV[cc][j] = (c0 + cc < d && j < k) ? V[(c0 + cc) * k + j] : 0.f;
    }
    __syncthreads();
    for (int cc = 0; cc < 64; ++cc) {
      const double ev = (double)sE[r][cc];
#pragma unroll
      for (int u = 0; u < KQ; ++u) acc[u] += ev * (double)sV[cc][q + 4 * u];
    }
  }
  const int64_t t = t0 + r;
#pragma unroll
  for (int u = 0; u < KQ; ++u) {
    const int j = q + 4 * u;
    const float yv = (float)acc[u];
    sY[r][j] = (double)yv;
    if (t < n && j < k) y_out[b * y_bstride + t * k + j] = yv;
  }
  __syncthreads();
  // q_t = Y_t G Y_t^T of the stored (float) coordinates, weighted by the statistic weight
  double qv = 0.0;
  if (tid < 64 && t0 + tid < n) {
    const double* Gb = G + b * k * k;
    for (int a2 = 0; a2 < k; ++a2) {
      double rr = 0.0;
      for (int c = 0; c < k; ++c) rr += Gb[a2 * k + c] * sY[tid][c];
      qv += sY[tid][a2] * rr;
    }
    if (aw) qv *= (double)aw[t0 + tid];
  }
  const double tot = block_sum(qv, sred);
  if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
}

// sum_q2 partials from stored credit coordinates: one thread per token, q_t = Y_t G Y_t^T
// (fp64) times the statistic weight; grid (ceil(n / 256), nb).
__global__ __launch_bounds__(256) void k_q2_rows(int64_t n, int64_t k, const float* __restrict__ Y, int64_t y_bstride,
                                                 const double* __restrict__ G, const float* __restrict__ aw,
                                                 double* __restrict__ partial) {
  __shared__ double sred[4];
  const int64_t b = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double qv = 0.0;
  if (t < n) {
    const float* yt = Y + b * y_bstride + t * k;
    const double* Gb = G + b * k * k;
    for (int64_t a2 = 0; a2 < k; ++a2) {
      double r = 0.0;
      for (int64_t c = 0; c < k; ++c) r += Gb[a2 * k + c] * (double)yt[c];
      qv += (double)yt[a2] * r;
    }
    if (aw) qv *= (double)aw[t];
  }
  const double tot = block_sum(qv, sred);
  if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
}

// The same for k <= KB with G padded to KB x KB (zero past k): 16 lanes per token, lane p
// forming r_a = sum_c G[a][c] y_c for its KB / 16 rows a = p + 16 u (G transposed in LDS,
// so that the 16 lanes read consecutive a), then y_a r_a summed over its rows and over the
// 16 lanes by a fixed butterfly (fp64); 16 tokens per workgroup.
template <int KB>
__global__ __launch_bounds__(256) void k_q2_rows_kb(int64_t n, int64_t k, const float* __restrict__ Y,
                                                    int64_t y_bstride, const double* __restrict__ G,
                                                    const float* __restrict__ aw, double* __restrict__ partial) {
  constexpr int RPL = KB / 16;  // rows a per lane
  __shared__ double sG[KB * KB];  // [c][a]
  __shared__ double sred[4];
  const int64_t b = blockIdx.y;
  const double* Gb = G + b * KB * KB;
  for (int e = threadIdx.x; e < KB * KB; e += 256) sG[(e % KB) * KB + e / KB] = Gb[e];
  __syncthreads();
  const int p = threadIdx.x & 15;
  const int64_t t = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  double qv = 0.0;
  if (t < n) {
    const float* yt = Y + b * y_bstride + t * k;
    double r[RPL];
#pragma unroll
    for (int u = 0; u < RPL; ++u) r[u] = 0.0;
    for (int c = 0; c < (int)k; ++c) {
      const double yc = (double)yt[c];
#pragma unroll
      for (int u = 0; u < RPL; ++u) r[u] += sG[c * KB + p + 16 * u] * yc;
    }
#pragma unroll
    for (int u = 0; u < RPL; ++u) {
      const int a = p + 16 * u;
      if (a < k) qv += (double)yt[a] * r[u];
    }
  }
  // the 16 lanes of a token, in a fixed order
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) qv += __shfl_xor(qv, off, 16);
  if (aw && t < n) qv *= (double)aw[t];
  if (p != 0) qv = 0.0;
  const double tot = block_sum(qv, sred);
  if (threadIdx.x == 0) partial[b * gridDim.x + blockIdx.x] = tot;
}

__global__ void k_fill_i32(int32_t* p, int64_t cnt, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cnt) p[i] = v;
}

}  // namespace

static bool use_small(int64_t C, int64_t k) { return C <= kSmallMaxC && k <= kSmallMaxK; }

// Large vocabulary with bf16 A~ (k % 8 == 0, aligned operands): Y = E A~ of every block as one
// matrix-core product over the vocabulary (launch_softmax_product), A~ of the blocks side by side.
static bool use_product(const ErrorArgs& a) {
  if (use_small(a.C, a.k) || a.a_dtype != LOCA_BF16 || a.k % 8 != 0) return false;
  if (((uintptr_t)a.credit_a % 16) != 0 || (a.nb > 1 && a.a_bstride % 8 != 0)) return false;
  if (((uintptr_t)a.logits % 16) != 0 || a.ld_logits % (a.logits_dtype == LOCA_BF16 ? 8 : 4) != 0) return false;
  return true;
}

// Row stride of G for every path: the padded width of the register kernels (16, 32 or 64)
// for k <= 64, else k.
static int64_t g_ld_max(int64_t k) { return k <= kSmallMaxK ? small_kb(k) : k; }

size_t error_targets_ws(int64_t nb, int64_t n, int64_t C, int64_t k) {
  const int64_t lg = g_ld_max(k);
  size_t s = align256(sizeof(double) * nb * lg * lg);  // G
  s += credit_gram_part_ws(nb, k);                   // partials of G
  const int64_t parts = use_small(C, k) ? (n + kSmallThreads - 1) / kSmallThreads : (n + kLargeTok - 1) / kLargeTok;
  s += align256(sizeof(double) * nb * parts);          // partials
  if (!use_small(C, k)) {
    const size_t large = align256(sizeof(float) * 2 * n);  // (m, s) per token
    const size_t prod = (k % 8 == 0) ? softmax_product_ws(n, C, nb * k) : 0;
    s += large > prod ? large : prod;
  }
  return s;
}

template <typename LT, typename AT>
static hipError_t dispatch_error(const ErrorArgs& a, double* G, double* partial, float* ms) {
  const LT* z = (const LT*)a.logits;
  const AT* A = (const AT*)a.credit_a;
  if (use_small(a.C, a.k)) {
    dim3 grid((unsigned)((a.n + kSmallThreads - 1) / kSmallThreads), (unsigned)a.nb);
    // ||Q||^2 through the C x C matrix A~ G A~^T for label sets of at most 16 classes,
    // else on the fp64 matrix cores from the tile of Y
#define LOCA_SMALL(KB, HC)                                                                          \
  k_error_small<LT, AT, KB, HC><<<grid, kSmallThreads, 0, a.stream>>>(                              \
      a.n, a.C, a.k, z, a.ld_logits, a.labels, a.w, a.a_w, A, a.a_bstride, G, a.y_out, a.y_bstride, a.e_out, \
      partial, a.dev_info)
#define LOCA_SMALL_KB(KB)                      \
  if (a.C <= 8) LOCA_SMALL(KB, 8);             \
  else if (a.C <= 16) LOCA_SMALL(KB, 16);      \
  else LOCA_SMALL(KB, 0);
    if (a.k <= 16) { LOCA_SMALL_KB(16) }
    else if (a.k <= 32) { LOCA_SMALL_KB(32) }
    else { LOCA_SMALL_KB(64) }
#undef LOCA_SMALL_KB
#undef LOCA_SMALL
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_error_finalize<<<(unsigned)a.nb, 64, 0, a.stream>>>(a.n, grid.x, partial, a.mb_out, a.dev_info);
  } else {
    dim3 grid((unsigned)((a.n + kLargeTok - 1) / kLargeTok), (unsigned)a.nb);
    k_error_large<LT, AT><<<grid, kLargeThreads, 0, a.stream>>>(
        a.n, a.C, a.k, z, a.ld_logits, a.labels, a.w, a.a_w, A, a.a_bstride, G, g_ld_max(a.k), a.y_out, a.y_bstride,
        a.e_out ? ms : nullptr, partial, a.dev_info);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_error_finalize<<<(unsigned)a.nb, 64, 0, a.stream>>>(a.n, grid.x, partial, a.mb_out, a.dev_info);
    if (a.e_out) {
      dim3 g2((unsigned)((a.C + 255) / 256 < 64 ? (a.C + 255) / 256 : 64), write_e_rows(a.n));
      k_error_write_e<LT><<<g2, 256, 0, a.stream>>>(a.n, a.C, z, a.ld_logits, a.labels, a.w, ms, a.e_out);
    }
  }
  return hipGetLastError();
}

hipError_t launch_error_targets(const ErrorArgs& a) {
  char* p = a.ws;
  // B~ B~^T of every block, row stride g_ld_max(k) (zero past k): from the caller
  // (loca_credit_gram) when given, else formed here
  double* G = a.credit_gram ? (double*)a.credit_gram : (double*)p;
  const int64_t lg = g_ld_max(a.k);
  p += align256(sizeof(double) * a.nb * g_ld_max(a.k) * g_ld_max(a.k));
  double* gpart = (double*)p;
  p += credit_gram_part_ws(a.nb, a.k);
  double* partial = (double*)p;
  const int64_t parts = use_small(a.C, a.k) ? (a.n + kSmallThreads - 1) / kSmallThreads : (a.n + kLargeTok - 1) / kLargeTok;
  p += align256(sizeof(double) * a.nb * parts);
  float* ms = use_small(a.C, a.k) ? nullptr : (float*)p;

  k_fill_i32<<<1, 64, 0, a.stream>>>(a.dev_info, 1, INT32_MAX);
  if (!a.credit_gram) launch_credit_gram(a.stream, a.nb, a.k, a.d, a.credit_b, a.b_bstride, gpart, G, lg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (use_product(a)) {
    // partials of k_q2_rows_kb: one per 16 tokens (as many as the large kernel's, which the
    // workspace holds; k_q2_rows, for k > 64: one per 256); the product's statistics and
    // partial sums after them
    char* pw = (char*)partial + align256(sizeof(double) * a.nb * parts);
    SoftmaxProductArgs sp{a.stream, a.n, a.C, a.logits, a.logits_dtype, a.ld_logits, a.labels, a.w,
                          (const uint16_t*)a.credit_a, a.nb, a.k, a.nb > 1 ? a.a_bstride : 0, a.y_out, a.k,
                          a.y_bstride, a.dev_info, pw};
    if ((e = launch_softmax_product(sp)) != hipSuccess) return e;
    const bool kb = a.k <= kSmallMaxK;  // 16 tokens per workgroup, else 256
    dim3 gq((unsigned)(kb ? (a.n + 15) / 16 : (a.n + 255) / 256), (unsigned)a.nb);
    if (!kb)
      k_q2_rows<<<gq, 256, 0, a.stream>>>(a.n, a.k, a.y_out, a.y_bstride, G, a.a_w, partial);
    else if (lg == 16)
      k_q2_rows_kb<16><<<gq, 256, 0, a.stream>>>(a.n, a.k, a.y_out, a.y_bstride, G, a.a_w, partial);
    else if (lg == 32)
      k_q2_rows_kb<32><<<gq, 256, 0, a.stream>>>(a.n, a.k, a.y_out, a.y_bstride, G, a.a_w, partial);
    else
      k_q2_rows_kb<64><<<gq, 256, 0, a.stream>>>(a.n, a.k, a.y_out, a.y_bstride, G, a.a_w, partial);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    k_error_finalize<<<(unsigned)a.nb, 64, 0, a.stream>>>(a.n, gq.x, partial, a.mb_out, a.dev_info);
    if (a.e_out) {
      const float* msv = (const float*)pw;  // (m, s) per token, first in the product's workspace
      dim3 g2((unsigned)((a.C + 255) / 256 < 64 ? (a.C + 255) / 256 : 64), write_e_rows(a.n));
      if (a.logits_dtype == LOCA_BF16)
        k_error_write_e<uint16_t><<<g2, 256, 0, a.stream>>>(a.n, a.C, (const uint16_t*)a.logits, a.ld_logits,
                                                             a.labels, a.w, msv, a.e_out);
      else
        k_error_write_e<float><<<g2, 256, 0, a.stream>>>(a.n, a.C, (const float*)a.logits, a.ld_logits, a.labels,
                                                          a.w, msv, a.e_out);
    }
    return hipGetLastError();
  }
  const bool zb = a.logits_dtype == LOCA_BF16, ab = a.a_dtype == LOCA_BF16;
  if (!zb && !ab) return dispatch_error<float, float>(a, G, partial, ms);
  if (!zb && ab) return dispatch_error<float, uint16_t>(a, G, partial, ms);
  if (zb && !ab) return dispatch_error<uint16_t, float>(a, G, partial, ms);
  return dispatch_error<uint16_t, uint16_t>(a, G, partial, ms);
}

int64_t credit_gram_ld(int64_t k) { return g_ld_max(k); }
size_t credit_gram_ws(int64_t nb, int64_t k) { return credit_gram_part_ws(nb, k); }
hipError_t launch_credit_gram_only(hipStream_t st, int64_t nb, int64_t k, int64_t d, const float* B,
                                   int64_t b_bstride, double* G, char* ws) {
  launch_credit_gram(st, nb, k, d, B, b_bstride, (double*)ws, G, g_ld_max(k));
  return hipGetLastError();
}

// ------------------------------------------------------------------ allocation-free variant
// loca_error_targets_noalloc takes its scratch from a fixed device array instead of a
// caller workspace.  The runtime gives each device its own copy of the array; its device
// address is looked up once per device, with that device current, and kept.  Nothing in
// the head-error workspace has to start at zero (every kernel writes what it later reads),
// so the array is never cleared; calls on one device share it and must not overlap.

namespace {
constexpr size_t kScratchBytes = (size_t)16 << 20;  // 16 MiB
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};
}  // namespace

size_t error_targets_scratch_bytes() { return kScratchBytes; }

hipError_t error_targets_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> hold(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// ------------------------------------------------------------------ paper-order credit

size_t credit_from_top_error_ws(int64_t nb, int64_t n, int64_t k) {
  return align256(sizeof(double) * nb * k * k) + credit_gram_part_ws(nb, k) +
         align256(sizeof(double) * nb * ((n + 63) / 64));
}

hipError_t launch_credit_from_top_error(const CreditArgs& a) {
  double* G = (double*)a.ws;
  double* gpart = (double*)(a.ws + align256(sizeof(double) * a.nb * a.k * a.k));
  double* partial = (double*)((char*)gpart + credit_gram_part_ws(a.nb, a.k));
  launch_credit_gram(a.stream, a.nb, a.k, a.d, a.credit_b, a.b_bstride, gpart, G, a.k);
  dim3 g((unsigned)((a.n + 63) / 64), (unsigned)a.nb);
#define LOCA_PROJ(KQ)                                                                                          \
  k_credit_project<KQ><<<g, 256, 0, a.stream>>>(a.n, a.d, a.k, a.e, a.ld_e, a.vk, a.v_bstride, G, a.a_w, a.y_out, \
                                                 a.y_bstride, partial)
  if (a.k <= 16) LOCA_PROJ(4);
  else if (a.k <= 32) LOCA_PROJ(8);
  else if (a.k <= 64) LOCA_PROJ(16);
  else LOCA_PROJ(32);
#undef LOCA_PROJ
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_error_finalize<<<(unsigned)a.nb, 64, 0, a.stream>>>(a.n, g.x, partial, a.mb_out, nullptr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ dense targets (tests)

namespace {
__global__ void k_dense_targets(int64_t n, int64_t k, int64_t d, const float* __restrict__ y,
                                int64_t y_bstride, const loca_mb* __restrict__ mb,
                                const float* __restrict__ B, int64_t b_bstride,
                                float* __restrict__ T, int64_t t_bstride) {
  const int64_t b = blockIdx.z;
  const int64_t t = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= d) return;
  const double eb = mb[b].eta_bar;
  const float* yt = y + b * y_bstride + t * k;
  const float* Bb = B + b * b_bstride;
  double s = 0.0;
  for (int64_t j = 0; j < k; ++j) s += (double)yt[j] * (double)Bb[j * d + i];
  T[b * t_bstride + t * d + i] = (float)(-eb * s);
}
}  // namespace

hipError_t launch_dense_targets(hipStream_t s, int64_t nb, int64_t n, int64_t k, int64_t d,
                                const float* y, int64_t y_bstride, const loca_mb* mb,
                                const float* credit_b, int64_t b_bstride, float* t_out,
                                int64_t t_bstride) {
  dim3 grid((unsigned)((d + 255) / 256), (unsigned)n, (unsigned)nb);
  k_dense_targets<<<grid, 256, 0, s>>>(n, k, d, y, y_bstride, mb, credit_b, b_bstride, t_out, t_bstride);
  return hipGetLastError();
}

}  // namespace loca
