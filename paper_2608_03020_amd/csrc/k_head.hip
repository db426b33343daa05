// k_head.hip -- the head in the paper's order (Section S11): the top-layer error taken
// to the hidden width once for all blocks,
//   e_t = W_u^T E_t,   E_t = w_t (softmax(z_t) - onehot(y_t))   (the target's error term,
//                                                               Lemma S3.1's head error),
// so that each block then applies only V_k^T e_t (loca_credit_from_top_error).  It pays
// off when the blocks' folded factors A~ = W_u V_k together are wider than the hidden
// width (L k > d).
//
//   1. k_softmax_stats: per token the row maximum m_t and s_t = sum_c exp(z_tc - m_t)
//      (one workgroup per token, fixed-order combination of the partial pairs);
//   2. k_top_error_gemm: part_z = P W_u over the vocabulary chunk z, P_tc = w_t exp(z_tc -
//      m_t) / s_t formed while the logits tile is staged, split into bf16 hi + lo parts
//      (about 16 significant bits), each multiplied by the exact bf16 W_u on the matrix
//      cores (v_mfma_f32_32x32x16_bf16; W_u read transposed from LDS);
//   3. k_top_error_reduce: e = sum_z part_z in a fixed order (fp64), minus w_t W_u[y_t].
// With at most 64 columns the product takes one pass over the logits instead (an online
// softmax feeding the matrix cores, launch_softmax_product_online in k_fused.hip).
//
// The same product serves the folded order for a large vocabulary (loca_error_targets
// with bf16 A~): the right operand is then the blocks' A~ side by side (column j of
// group j / kc), so one launch forms Y_b = E A~_b for every block.
#include <algorithm>

#include "loca_launch.h"
#include "loca_bf16.h"

namespace loca {

namespace {

constexpr int kHT = 256;
constexpr int kHM = 128, kHK = 32;  // token rows, vocabulary per stage
constexpr int kLDA = kHK + 8;                  // bf16 per LDS row of P (80 bytes)

// dev_info: INT32_MAX while no bad label is seen, then 1 + the smallest bad row, or
// LOCA_INFO_NONFINITE once a row's softmax sum is not finite; INT32_MAX becomes 0 at the end
__global__ void k_fill_i32_head(int32_t* p) {
  if (threadIdx.x == 0) *p = INT32_MAX;
}
__global__ void k_finish_info_head(int32_t* p) {
  if (threadIdx.x == 0 && *p == INT32_MAX) *p = 0;
}

// (m, s) of two disjoint parts of a row combined into one
LOCA_DEV void ms_combine(float& m, float& s, float m2, float s2) {
  if (s2 == 0.f) return;
  if (s == 0.f) { m = m2; s = s2; return; }
  const float mm = fmaxf(m, m2);
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

// 8 consecutive logits as floats (a 16-byte aligned bf16 chunk or two float4)
LOCA_DEV void load8(const uint16_t* p, float (&v)[8]) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
LOCA_DEV void load8(const float* p, float (&v)[8]) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// One workgroup per token.  A 16-byte aligned row is read in chunks of 8 logits, two
// chunks in flight per thread: each chunk's maximum first rescales the running sum once,
// then its 8 terms are added.  Other rows (and the tail past a multiple of 8) go one
// logit at a time.
template <typename LT>
__global__ __launch_bounds__(kHT) void k_softmax_stats(int64_t n, int64_t V, const LT* __restrict__ z, int64_t ld,
                                                       const int32_t* __restrict__ labels, float* __restrict__ ms,
                                                       int32_t* __restrict__ dev_info) {
  __shared__ float sm[kHT], ss[kHT];
  const int64_t t = blockIdx.x;
  const LT* zt = z + t * ld;
  float m = -INFINITY, s = 0.f;  // s == 0: nothing seen yet
  auto add8 = [&](const float (&v)[8]) {
    float mx = v[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, v[i]);
    if (mx > m) {
      s *= __expf(m - mx);
      m = mx;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) s += __expf(v[i] - m);
  };
  int64_t c0 = 0;
  if ((((uintptr_t)zt) & 15) == 0) {
    const int64_t nch = V / 8;
    int64_t c = threadIdx.x;
    for (; c + kHT < nch; c += 2 * kHT) {
      float va[8], vb[8];
      load8(zt + 8 * c, va);
      load8(zt + 8 * (c + kHT), vb);
      add8(va);
      add8(vb);
    }
    for (; c < nch; c += kHT) {
      float va[8];
      load8(zt + 8 * c, va);
      add8(va);
    }
    c0 = nch * 8;
  }
  for (int64_t c = c0 + threadIdx.x; c < V; c += kHT) {
    const float v = load_as_f32(zt + c);
    if (v > m) {
      s = s * __expf(m - v) + 1.f;
      m = v;
    } else {
      s += __expf(v - m);
    }
  }
  sm[threadIdx.x] = m;
  ss[threadIdx.x] = s;
  __syncthreads();
  for (int h = kHT / 2; h > 0; h >>= 1) {  // pairs (i, i + h): a fixed tree
    if ((int)threadIdx.x < h) {
      float a = sm[threadIdx.x], b = ss[threadIdx.x];
      ms_combine(a, b, sm[threadIdx.x + h], ss[threadIdx.x + h]);
      sm[threadIdx.x] = a;
      ss[threadIdx.x] = b;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    ms[2 * t] = sm[0];
    ms[2 * t + 1] = ss[0];
    const int32_t yt = labels[t];
    if (yt < 0 || yt >= V) atomicMin(dev_info, (int32_t)(t + 1));
    // a NaN or +inf logit makes the sum NaN (a -inf logit is an excluded class and is fine)
    if (!__builtin_isfinite(ss[0])) atomicMin(dev_info, (int32_t)LOCA_INFO_NONFINITE);
  }
}

// Tiles of 128 tokens x HN columns (HN = 128, or 64 when there are at most 64 columns), one
// vocabulary chunk per grid.z; four waves of 64 columns each: 2 x 2 waves of 64 x 64 (HN =
// 128) or 4 x 1 of 32 x 64 (HN = 64).  Column j of the right operand is column j % kc of
// group j / kc: W + (j / kc) w_bstride (V x kc bf16 each).  d = total columns.  Requires
// ld % 8 == 0 (bf16) or % 4 == 0 (f32), kc % 8 == 0, d % kc == 0, kchunk % 32 == 0.
template <typename LT, int HN>
__global__ __launch_bounds__(kHT) void k_top_error_gemm(int64_t n, int64_t V, int64_t d, const LT* __restrict__ z,
                                                        int64_t ld, const float* __restrict__ w,
                                                        const float* __restrict__ ms, const uint16_t* __restrict__ wu,
                                                        int64_t kc, int64_t w_bstride, int64_t kchunk,
                                                        float* __restrict__ part) {
  constexpr int WGN = HN / 64, WGM = 4 / WGN, WM = kHM / WGM, NBM = WM / 32;
  constexpr int LDB = HN + 16;                  // bf16 per LDS row of W (conflict-free transpose reads)
  constexpr int NQB = HN * kHK / 8 / kHT;       // 16-byte chunks of the W stage per thread
  __shared__ __attribute__((aligned(16))) uint16_t sAh[2][kHM * kLDA];
  __shared__ __attribute__((aligned(16))) uint16_t sAl[2][kHM * kLDA];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][kHK * LDB];
  const int64_t t0 = (int64_t)blockIdx.x * kHM, j0 = (int64_t)blockIdx.y * HN;
  const int64_t cb = (int64_t)blockIdx.z * kchunk;
  const int64_t ce = std::min<int64_t>(V, cb + kchunk);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wi = wid / WGN, wj = wid % WGN;

  // staging: A chunk q of this thread = row (tid + 256 q) / 4, vocabulary 8 ((tid + 256 q) % 4);
  // B chunk q = vocabulary row (tid + 256 q) / (HN / 8), columns 8 ((tid + 256 q) % (HN / 8))
  int arow[2], acol[2], brow[NQB], bcol[NQB];
  float rmax[2], rscale[2];
  const LT* zrow[2];  // this thread's logits rows (row 0 for rows past n: never read)
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int e = tid + kHT * q;
    arow[q] = e >> 2;
    acol[q] = 8 * (e & 3);
    const int64_t t = t0 + arow[q];
    const bool ok = t < n;
    zrow[q] = z + (ok ? t : 0) * ld;
    rmax[q] = ok ? ms[2 * t] : 0.f;
    const float st = ok ? ms[2 * t + 1] : 1.f;
    rscale[q] = ok ? (w ? w[t] : 1.f) / st : 0.f;
  }
#pragma unroll
  for (int q = 0; q < NQB; ++q) {
    const int e = tid + kHT * q;
    brow[q] = e / (HN / 8);
    bcol[q] = 8 * (e % (HN / 8));
  }
  uint4 ph[2], pl[2], wb[NQB];
  auto load_stage = [&](int64_t c0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int64_t t = t0 + arow[q], c = c0 + acol[q];
      float v[8];
      if (t < n && c + 8 <= ce) {
        load8(zrow[q] + c, v);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (t < n && c + i < ce) ? load_as_f32(zrow[q] + c + i) : -INFINITY;
      }
      // P = w exp(z - m) / s split into bf16 hi + lo (packed hardware conversions, loca_bf16.h)
      uint32_t h[4], l[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p0 = __expf(v[2 * i] - rmax[q]) * rscale[q];
        const float p1 = __expf(v[2 * i + 1] - rmax[q]) * rscale[q];
        h[i] = cvt_pk_bf16(p0, p1);
        l[i] = cvt_pk_bf16(p0 - bf16_lo(h[i]), p1 - bf16_hi(h[i]));
      }
      ph[q] = make_uint4(h[0], h[1], h[2], h[3]);
      pl[q] = make_uint4(l[0], l[1], l[2], l[3]);
    }
#pragma unroll
    for (int q = 0; q < NQB; ++q) {
      const int64_t cr = c0 + brow[q], j = j0 + bcol[q];
      const int64_t grp = j / kc, jc = j - grp * kc;
      wb[q] = (cr < ce && j < d) ? *(const uint4*)(wu + grp * w_bstride + cr * kc + jc) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      *(uint4*)&sAh[buf][arow[q] * kLDA + acol[q]] = ph[q];
      *(uint4*)&sAl[buf][arow[q] * kLDA + acol[q]] = pl[q];
    }
#pragma unroll
    for (int q = 0; q < NQB; ++q) *(uint4*)&sB[buf][brow[q] * LDB + bcol[q]] = wb[q];
  };

  f32x16_t acc[NBM][2];
#pragma unroll
  for (int m = 0; m < NBM; ++m)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][q][r] = 0.f;

  const int nk = (int)((ce - cb + kHK - 1) / kHK);
  if (nk > 0) {
    load_stage(cb);
    store_stage(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_stage(cb + (int64_t)(kt + 1) * kHK);
#pragma unroll
    for (int ks = 0; ks < kHK; ks += 16) {
      bf16x8_t fh[NBM], fl[NBM], fb[2];
#pragma unroll
      for (int m = 0; m < NBM; ++m) {
        const int row = wi * WM + 32 * m + (lane & 31);
        const int off = row * kLDA + ks + 8 * (lane >> 5);
        fh[m] = __builtin_bit_cast(bf16x8_t, *(const uint4*)&sAh[cur][off]);
        fl[m] = __builtin_bit_cast(bf16x8_t, *(const uint4*)&sAl[cur][off]);
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) fb[q] = frag32_tr(sB[cur], LDB, wj * 64 + 32 * q, ks, lane);
#pragma unroll
      for (int m = 0; m < NBM; ++m)
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[m][q] = mfma32(fh[m], fb[q], acc[m][q]);
#pragma unroll
      for (int m = 0; m < NBM; ++m)
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[m][q] = mfma32(fl[m], fb[q], acc[m][q]);
    }
    if (kt + 1 < nk) store_stage(cur ^ 1);
    __syncthreads();
  }
  float* out = part + (int64_t)blockIdx.z * n * d;
#pragma unroll
  for (int m = 0; m < NBM; ++m)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t t = t0 + wi * WM + 32 * m + mfma32_row(lane, r);
        const int64_t j = j0 + wj * 64 + 32 * q + mfma32_col(lane);
        if (t < n && j < d) out[t * d + j] = acc[m][q][r];
      }
}

// out[(j / kc) o_bstride + t ld_o + j % kc] = sum_z part_z[t][j] (fp64, in order) - w_t W[y_t][j]
__global__ void k_top_error_reduce(int64_t n, int64_t d, int nsplit, const float* __restrict__ part,
                                   const float* __restrict__ w, const int32_t* __restrict__ labels, int64_t V,
                                   const uint16_t* __restrict__ wu, int64_t kc, int64_t w_bstride,
                                   float* __restrict__ out, int64_t ld_o, int64_t o_bstride) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n * d) return;
  const int64_t t = e / d, j = e % d;
  const int64_t grp = j / kc, jc = j - grp * kc;
  double s = 0.0;
  for (int zc = 0; zc < nsplit; ++zc) s += (double)part[(int64_t)zc * n * d + e];
  const int32_t yt = labels[t];
  if (yt >= 0 && yt < V)
    s -= (double)(w ? w[t] : 1.f) * (double)bf16_to_f32(wu[grp * w_bstride + (int64_t)yt * kc + jc]);
  out[grp * o_bstride + t * ld_o + jc] = (float)s;
}

// columns per tile of the product: 64 when there are at most 64, else 128
int head_hn(int64_t d) { return d <= 64 ? 64 : 128; }

int head_splits(int64_t n, int64_t V, int64_t d) {
  const int64_t tiles = ((n + kHM - 1) / kHM) * ((d + head_hn(d) - 1) / head_hn(d));
  int64_t s = (2048 + tiles - 1) / tiles;
  s = std::max<int64_t>(1, std::min<int64_t>(s, 32));
  s = std::min<int64_t>(s, std::max<int64_t>(1, (V + 255) / 256));  // at least 256 vocabulary entries a chunk
  return (int)s;
}

}  // namespace

// At most 64 columns (one tile of the single-pass kernel) the logits are read once, by the
// online-softmax product; wider products keep the statistics pass and a product pass per
// 128 columns.
// (Its buffer loads take 31-bit byte offsets within 128 rows of logits and 64 rows of the
// right operand.)
static bool product_online(const SoftmaxProductArgs& a) {
  const int64_t zb = a.logits_dtype == LOCA_BF16 ? 2 : 4;
  return a.groups * a.kc <= 64 && 128 * a.ld_logits * zb < ((int64_t)1 << 31) &&
         64 * ((a.V + 63) / 64) * 64 * 2 < ((int64_t)1 << 31);
}

static size_t two_pass_ws(int64_t n, int64_t V, int64_t cols) {
  return align256(sizeof(float) * 2 * n) + align256(sizeof(float) * (size_t)head_splits(n, V, cols) * n * cols);
}

size_t softmax_product_ws(int64_t n, int64_t V, int64_t cols) {
  const size_t two = two_pass_ws(n, V, cols);
  if (cols > 64) return two;
  const size_t one = softmax_product_online_ws(n, V, cols);
  return one > two ? one : two;  // the path is chosen at the launch (it also depends on the strides)
}

hipError_t launch_softmax_product(const SoftmaxProductArgs& a) {
  if (product_online(a)) return launch_softmax_product_online(a);
  float* ms = (float*)a.ws;
  float* part = (float*)(a.ws + align256(sizeof(float) * 2 * a.n));
  const int64_t cols = a.groups * a.kc;
  const int ns = head_splits(a.n, a.V, cols);
  const int64_t kchunk = ((a.V + ns - 1) / ns + kHK - 1) / kHK * kHK;
  hipStream_t st = a.stream;
  const int hn = head_hn(cols);
  dim3 g((unsigned)((a.n + kHM - 1) / kHM), (unsigned)((cols + hn - 1) / hn), (unsigned)ns);
  if (a.logits_dtype == LOCA_BF16) {
    const uint16_t* zb = (const uint16_t*)a.logits;
    k_softmax_stats<uint16_t><<<(unsigned)a.n, kHT, 0, st>>>(a.n, a.V, zb, a.ld_logits, a.labels, ms, a.dev_info);
    if (hn == 64)
      k_top_error_gemm<uint16_t, 64><<<g, kHT, 0, st>>>(a.n, a.V, cols, zb, a.ld_logits, a.w, ms, a.W, a.kc,
                                                        a.w_bstride, kchunk, part);
    else
      k_top_error_gemm<uint16_t, 128><<<g, kHT, 0, st>>>(a.n, a.V, cols, zb, a.ld_logits, a.w, ms, a.W, a.kc,
                                                         a.w_bstride, kchunk, part);
  } else {
    const float* zf = (const float*)a.logits;
    k_softmax_stats<float><<<(unsigned)a.n, kHT, 0, st>>>(a.n, a.V, zf, a.ld_logits, a.labels, ms, a.dev_info);
    if (hn == 64)
      k_top_error_gemm<float, 64><<<g, kHT, 0, st>>>(a.n, a.V, cols, zf, a.ld_logits, a.w, ms, a.W, a.kc,
                                                     a.w_bstride, kchunk, part);
    else
      k_top_error_gemm<float, 128><<<g, kHT, 0, st>>>(a.n, a.V, cols, zf, a.ld_logits, a.w, ms, a.W, a.kc,
                                                      a.w_bstride, kchunk, part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_top_error_reduce<<<(unsigned)((a.n * cols + 255) / 256), 256, 0, st>>>(
      a.n, cols, ns, part, a.w, a.labels, a.V, a.W, a.kc, a.w_bstride, a.out, a.ld_o, a.o_bstride);
  return hipGetLastError();
}

size_t top_error_ws(int64_t n, int64_t V, int64_t d) { return softmax_product_ws(n, V, d); }

hipError_t launch_top_error(const TopErrorArgs& a) {
  hipStream_t st = a.stream;
  k_fill_i32_head<<<1, 64, 0, st>>>(a.dev_info);
  SoftmaxProductArgs p{st, a.n, a.V, a.logits, a.logits_dtype, a.ld_logits, a.labels, a.w, (const uint16_t*)a.wu,
                       1, a.d, 0, a.e_out, a.ld_e, 0, a.dev_info, a.ws};
  hipError_t e = launch_softmax_product(p);
  if (e != hipSuccess) return e;
  k_finish_info_head<<<1, 64, 0, st>>>(a.dev_info);
  return hipGetLastError();
}

}  // namespace loca
