// k_fused.hip -- the fused LM head ("Local Targets", Eq. 4; Lemma S3.1's head error; the
// head applied once per top error, Section S11).  From the final hidden states h (n x d) and
// the frozen head W_u (V x d), for a right operand Vm (V x c):
//   out_t = w_t ( sum_v softmax(z_t)_v Vm[v, :] - Vm[y_t, :] ),   z_t = W_u h_t,
// i.e. out = E Vm with E_t = w_t (softmax(z_t) - onehot(y_t)).  Vm = W_u gives the top error
// e_t = W_u^T E_t of the paper's order (then V_k^T e_t per block); Vm = [A~_1 | ... | A~_L]
// gives every block's credit coordinates Y_b = E A~_b at once.
//
// The logits are never stored.  A workgroup owns 128 tokens, a tile of at most CT columns
// of Vm and a contiguous range of the vocabulary, and walks that range in chunks of 128:
//   1. z (128 x 128) = h_rows W_u[chunk]^T on the matrix cores (v_mfma_f32_32x32x16_bf16,
//      fp32 accumulation), the two operands staged through LDS in 32-wide slices of d;
//   2. an online softmax per token: the running maximum m and sum s (fp32) are updated with
//      the chunk, the accumulated output is rescaled by exp(m_old - m_new), and
//      P = exp(z - m_new) is split into bf16 hi + lo parts (about 16 significant bits);
//   3. out += (P_hi + P_lo) Vm[chunk] on the matrix cores (Vm exact in bf16).
// Each vocabulary range leaves (m, s) per token and its partial output; a second kernel
// combines the ranges in a fixed order in float64 and subtracts the label term.  Columns of
// Vm beyond one tile recompute the logits (c / CT passes over W_u).
#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kFT = 256;       // threads: 4 waves as 2 x 2
constexpr int kFR = 128;       // token rows per workgroup
constexpr int kFV = 128;       // vocabulary per chunk
constexpr int kFK = 32;        // hidden width per staging slice
constexpr int kFLD = kFK + 8;  // bf16 per LDS row of an h / W_u slice (80 bytes)
constexpr int kZLD = kFV + 4;  // 32-bit words per LDS row of the logits / packed P tile
constexpr int kVLD = kFV + 8;  // bf16 per LDS row of the transposed right operand

LOCA_DEV uint16_t rne_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <int CT>
__global__ __launch_bounds__(kFT) void k_fused_head(int64_t n, int64_t V, int64_t d, int64_t c,
                                                    const uint16_t* __restrict__ h, int64_t ldh,
                                                    const uint16_t* __restrict__ wu,
                                                    const uint16_t* __restrict__ vmt, int64_t ldvt, int ntr, int nct,
                                                    int64_t vper, float* __restrict__ part_o,
                                                    float2* __restrict__ part_ms) {
  __shared__ __attribute__((aligned(16))) uint16_t sH[2][kFR * kFLD];
  __shared__ __attribute__((aligned(16))) uint16_t sW[2][kFV * kFLD];
  __shared__ __attribute__((aligned(16))) uint32_t sZ[kFR * kZLD];
  __shared__ __attribute__((aligned(16))) uint16_t sVt[CT * kVLD];
  __shared__ float sAl[kFR];
  constexpr int NQ = CT / 64;                  // 32-column output blocks per wave
  constexpr int NPV = CT * kFV / 8 / kFT;      // 16-byte chunks of the Vm^T slice per thread
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, wi = wid >> 1, wj = wid & 1;
  const int l32 = lane & 31, lh = lane >> 5;
  // tiles that share a vocabulary range are consecutive within an XCD (W_u read once there)
  const int logical = xcd_logical((int)blockIdx.x, (int)gridDim.x);
  const int rt = logical % ntr, ct = (logical / ntr) % nct, sp = logical / (ntr * nct);
  const int64_t r0 = (int64_t)rt * kFR, c0 = (int64_t)ct * CT;
  const int64_t vb = (int64_t)sp * vper, ve = (vb + vper < V) ? vb + vper : V;
  const int nks = (int)((d + kFK - 1) / kFK);

  f32x16_t o[2][NQ];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[m][q][r] = 0.f;
  float m_run = -__builtin_inff(), s_run = 0.f;  // of token row tid >> 1 (both threads of the pair)

  uint4 ph[2], pw[2];
  auto gload = [&](int64_t v0, int ks) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + kFT * i, row = q >> 2;
      const int64_t k = (int64_t)ks * kFK + 8 * (q & 3);
      const bool kin = k < d;
      ph[i] = (r0 + row < n && kin) ? *(const uint4*)(h + (r0 + row) * ldh + k) : make_uint4(0, 0, 0, 0);
      pw[i] = (v0 + row < V && kin) ? *(const uint4*)(wu + (v0 + row) * d + k) : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + kFT * i, row = q >> 2, part = q & 3;
      *(uint4*)&sH[buf][row * kFLD + 8 * part] = ph[i];
      *(uint4*)&sW[buf][row * kFLD + 8 * part] = pw[i];
    }
  };

  for (int64_t v0 = vb; v0 < ve; v0 += kFV) {
    // the chunk's slice of Vm^T (CT x 128; padded rows of Vm^T hold zeros past V)
    uint4 pv[NPV];
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      const int q = tid + kFT * i, row = q >> 4, part = q & 15;
      pv[i] = (c0 + row < c) ? *(const uint4*)(vmt + (c0 + row) * ldvt + v0 + 8 * part) : make_uint4(0, 0, 0, 0);
    }
    // 1. logits of the chunk
    f32x16_t z[2][2];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r) z[m][q][r] = 0.f;
    gload(v0, 0);
    lstore(0);
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
      const int buf = ks & 1;
      if (ks + 1 < nks) gload(v0, ks + 1);
#pragma unroll
      for (int kk = 0; kk < kFK; kk += 16) {
        bf16x8_t a[2], b[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) a[m] = *(const bf16x8_t*)&sH[buf][(wi * 64 + 32 * m + l32) * kFLD + kk + 8 * lh];
#pragma unroll
        for (int q = 0; q < 2; ++q) b[q] = *(const bf16x8_t*)&sW[buf][(wj * 64 + 32 * q + l32) * kFLD + kk + 8 * lh];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
          for (int q = 0; q < 2; ++q) z[m][q] = mfma32(a[m], b[q], z[m][q]);
      }
      if (ks + 1 < nks) lstore(buf ^ 1);
      __syncthreads();
    }
    // the previous chunk's readers of sZ and sVt have passed the syncs above
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sZ[(wi * 64 + 32 * m + mfma32_row(lane, r)) * kZLD + wj * 64 + 32 * q + l32] = __float_as_uint(z[m][q][r]);
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      const int q = tid + kFT * i, row = q >> 4, part = q & 15;
      *(uint4*)&sVt[row * kVLD + 8 * part] = pv[i];
    }
    __syncthreads();
    // 2. online softmax: two threads per token, interleaved 4-column groups
    {
      const int row = tid >> 1, half = tid & 1;
      const int nv = (V - v0 < kFV) ? (int)(V - v0) : kFV;
      uint32_t* zr = sZ + row * kZLD;
      float cm = -__builtin_inff();
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int col = 8 * g + 4 * half;
        const uint4 u = *(const uint4*)(zr + col);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < nv) cm = fmaxf(cm, __uint_as_float(w4[e]));
      }
      cm = fmaxf(cm, __shfl_xor(cm, 1));
      const float mn = fmaxf(m_run, cm);
      const float al = __expf(m_run - mn);
      float ps = 0.f;
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int col = 8 * g + 4 * half;
        const uint4 u = *(const uint4*)(zr + col);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = (col + e < nv) ? __expf(__uint_as_float(w4[e]) - mn) : 0.f;
          ps += p;
          const uint16_t hi = rne_bf16(p);
          const uint16_t lo = rne_bf16(p - __uint_as_float((uint32_t)hi << 16));
          pk[e] = (uint32_t)hi | ((uint32_t)lo << 16);
        }
        *(uint4*)(zr + col) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
      }
      ps += __shfl_xor(ps, 1);
      s_run = s_run * al + ps;
      m_run = mn;
      if (half == 0) sAl[row] = al;
    }
    __syncthreads();
    // 3. rescale the output rows and add (P_hi + P_lo) Vm[chunk]
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float al = sAl[wi * 64 + 32 * m + mfma32_row(lane, r)];
#pragma unroll
        for (int q = 0; q < NQ; ++q) o[m][q][r] *= al;
      }
#pragma unroll
    for (int kv = 0; kv < kFV; kv += 16) {
      bf16x8_t phi[2], plo[2], b[NQ];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const uint32_t* src = sZ + (wi * 64 + 32 * m + l32) * kZLD + kv + 8 * lh;
        const uint4 u0 = *(const uint4*)src, u1 = *(const uint4*)(src + 4);
        const uint32_t wv[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
        uint32_t hv[4], lv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hv[e] = (wv[2 * e] & 0xffffu) | (wv[2 * e + 1] << 16);
          lv[e] = (wv[2 * e] >> 16) | (wv[2 * e + 1] & 0xffff0000u);
        }
        phi[m] = __builtin_bit_cast(bf16x8_t, make_uint4(hv[0], hv[1], hv[2], hv[3]));
        plo[m] = __builtin_bit_cast(bf16x8_t, make_uint4(lv[0], lv[1], lv[2], lv[3]));
      }
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        b[q] = *(const bf16x8_t*)&sVt[(wj * (CT / 2) + 32 * q + l32) * kVLD + kv + 8 * lh];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          o[m][q] = mfma32(phi[m], b[q], o[m][q]);
          o[m][q] = mfma32(plo[m], b[q], o[m][q]);
        }
    }
  }
  // this range's partial output and (m, s)
  float* po = part_o + (int64_t)sp * n * c;
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = r0 + wi * 64 + 32 * m + mfma32_row(lane, r);
        const int64_t col = c0 + wj * (CT / 2) + 32 * q + l32;
        if (row < n && col < c) po[row * c + col] = o[m][q][r];
      }
  if (ct == 0 && (tid & 1) == 0 && r0 + (tid >> 1) < n) part_ms[(int64_t)sp * n + r0 + (tid >> 1)] = make_float2(m_run, s_run);
}

// dev_info protocol: INT32_MAX while nothing is wrong; atomicMin with 1 + a bad row or with
// LOCA_INFO_NONFINITE (which therefore takes precedence); INT32_MAX becomes 0 at the end
__global__ void k_fused_info_init(int32_t* p) {
  if (threadIdx.x == 0) *p = INT32_MAX;
}
__global__ void k_fused_info_finish(int32_t* p) {
  if (threadIdx.x == 0 && *p == INT32_MAX) *p = 0;
}

// Vm^T (c x ldvt, bf16) from Vm (V x c, row stride ld_vm), zero past V; 32 x 32 tiles via LDS
__global__ void k_vm_transpose(int64_t V, int64_t c, const uint16_t* __restrict__ vm, int64_t ld_vm,
                               uint16_t* __restrict__ vmt, int64_t ldvt) {
  __shared__ uint16_t t[32][33];
  const int64_t v0 = (int64_t)blockIdx.x * 32, j0 = (int64_t)blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int64_t v = v0 + r, j = j0 + tx;
    t[r][tx] = (v < V && j < c) ? vm[v * ld_vm + j] : (uint16_t)0;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int64_t j = j0 + r, v = v0 + tx;
    if (j < c && v < ldvt) vmt[j * ldvt + v] = t[tx][r];
  }
}

// out_t = w_t (sum_i O_i[t] e^{m_i - M} / S - Vm[y_t]), S = sum_i s_i e^{m_i - M}: the ranges
// in order, float64.  One workgroup per token.  A bad label drops the label term and is
// reported; a sum that is not finite or not positive is reported as non-finite data.
__global__ __launch_bounds__(256) void k_fused_combine(int64_t n, int64_t c, int64_t V, int nsp,
                                                       const float* __restrict__ part_o,
                                                       const float2* __restrict__ part_ms,
                                                       const int32_t* __restrict__ labels, const float* __restrict__ w,
                                                       const uint16_t* __restrict__ vm, int64_t ld_vm,
                                                       float* __restrict__ out, int64_t ld_out, int32_t* __restrict__ info) {
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
  }
  const double wt = w ? (double)w[t] : 1.0;
  const double inv = nonfin ? 0.0 : 1.0 / S;
  for (int64_t j = threadIdx.x; j < c; j += blockDim.x) {
    double acc = 0.0;
    for (int i = 0; i < nsp; ++i) acc += (double)part_o[((int64_t)i * n + t) * c + j] * sc[i];
    const double lab = bad ? 0.0 : (double)__uint_as_float((uint32_t)vm[(int64_t)y * ld_vm + j] << 16);
    out[t * ld_out + j] = (float)(wt * (acc * inv - lab));
  }
}

struct FusedPlan {
  int ct, ntr, nct, nsp;
  int64_t vper, ldvt;
};

FusedPlan fused_plan(int64_t n, int64_t V, int64_t c) {
  FusedPlan p;
  p.ct = c <= 64 ? 64 : 128;
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
      a.V, a.c, a.vm, a.ld_vm, vmt, p.ldvt);
  const unsigned grid = (unsigned)((int64_t)p.ntr * p.nct * p.nsp);
  if (p.ct == 64)
    k_fused_head<64><<<grid, kFT, 0, st>>>(a.n, a.V, a.d, a.c, a.h, a.ldh, a.wu, vmt, p.ldvt, p.ntr, p.nct, p.vper,
                                            part_o, part_ms);
  else
    k_fused_head<128><<<grid, kFT, 0, st>>>(a.n, a.V, a.d, a.c, a.h, a.ldh, a.wu, vmt, p.ldvt, p.ntr, p.nct, p.vper,
                                             part_o, part_ms);
  k_fused_combine<<<(unsigned)a.n, 256, 0, st>>>(a.n, a.c, a.V, p.nsp, part_o, part_ms, a.labels, a.w, a.vm, a.ld_vm,
                                                 a.out, a.ld_out, a.dev_info);
  k_fused_info_finish<<<1, 64, 0, st>>>(a.dev_info);
  return hipGetLastError();
}

}  // namespace loca
