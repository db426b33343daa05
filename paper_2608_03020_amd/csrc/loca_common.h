// loca_common.h -- device types and helpers shared by the libloca kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/loca.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef double f64x4_t __attribute__((ext_vector_type(4)));

#define LOCA_LDS __attribute__((address_space(3)))
#define LOCA_DEV __device__ __forceinline__

namespace loca {

constexpr int kWave = 64;

// ------------------------------------------------------------------ bf16 <-> f32

LOCA_DEV float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// round to nearest even (inputs here are finite)
LOCA_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> LOCA_DEV float load_as_f32(const T* p);
template <> LOCA_DEV float load_as_f32<float>(const float* p) { return *p; }
template <> LOCA_DEV float load_as_f32<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// ------------------------------------------------------------------ branch-free guarded loads
// The load always reads an in-bounds address (the base when `ok` is false) and the
// value is selected afterwards, so loops of guarded loads issue back to back instead
// of waiting on each other behind branches.
template <typename T>
LOCA_DEV T ld_or_zero(const T* base, int64_t idx, bool ok) {
  const T v = base[ok ? idx : 0];
  return ok ? v : (T)0;
}

// Copy a ROWS x COLS block (row stride ldg) from global memory into LDS (row stride
// lds_ld) with NT threads, zero outside rows < rows_ok, cols < cols_ok.  Loads are
// issued in batches of BATCH before any LDS store.  g must point at a valid element.
template <typename T, int ROWS, int COLS, int NT, int BATCH = 16>
LOCA_DEV void g2s_block(T* s, int lds_ld, const T* __restrict__ g, int64_t ldg, int64_t rows_ok, int64_t cols_ok) {
  constexpr int PER = (ROWS * COLS) / NT;
  static_assert((ROWS * COLS) % NT == 0, "block must split evenly over the threads");
#pragma unroll
  for (int q0 = 0; q0 < PER; q0 += BATCH) {
    T v[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int e = threadIdx.x + (q0 + u) * NT;
      const int r = e / COLS, c = e % COLS;
      v[u] = (q0 + u < PER) ? ld_or_zero(g, (int64_t)r * ldg + c, r < rows_ok && c < cols_ok) : (T)0;
    }
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      if (q0 + u < PER) {
        const int e = threadIdx.x + (q0 + u) * NT;
        s[(e / COLS) * lds_ld + (e % COLS)] = v[u];
      }
    }
  }
}

// ------------------------------------------------------------------ reductions

LOCA_DEV double wave_sum(double v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  return v;  // valid in lane 0
}
LOCA_DEV float wave_sum(float v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  return v;
}
LOCA_DEV float wave_max(float v) {
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;  // valid in all lanes
}

// Deterministic block sum (fixed tree).  `scratch` has blockDim.x/64 entries.
template <typename T>
LOCA_DEV T block_sum(T v, T* scratch) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) scratch[wid] = v;
  __syncthreads();
  T r = 0;
  if (threadIdx.x == 0)
    for (int i = 0; i < nw; ++i) r += scratch[i];
  return r;  // valid in thread 0
}

// ------------------------------------------------------------------ LDS transpose read (gfx950)
// ds_read_b64_tr_b16: within each 16-lane group the four 8-byte chunks given by
// lanes 4r..4r+3 form row r of a 4 x 16 block of 16-bit values; lane c of the
// group receives column c (rows 0..3).
LOCA_DEV s16x4_t lds_read_tr16(const uint16_t* lds_ptr) {
  typedef LOCA_LDS s16x4_t lds_v4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(LOCA_LDS void*)lds_ptr);
}

// MFMA operand of v_mfma_f32_32x32x16_bf16 from a K-major LDS tile
// tile[k][col] (row stride ld elements, ld % 4 == 0): the operand of lane l is
// the 8 values tile[ks + 8*(l/32) + e][c0 + l%32], e = 0..7.
LOCA_DEV bf16x8_t frag32_tr(const uint16_t* tile, int ld, int c0, int ks, int lane) {
  const int g = lane >> 4, w = lane & 15;
  const int col = c0 + 16 * (g & 1) + 4 * (w & 3);
  const int row = ks + 8 * (g >> 1) + (w >> 2);
  s16x4_t lo = lds_read_tr16(tile + row * ld + col);
  s16x4_t hi = lds_read_tr16(tile + (row + 4) * ld + col);
  typedef short s16x8_t __attribute__((ext_vector_type(8)));
  s16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

LOCA_DEV f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Result element r of lane l of a 32x32 MFMA block: row, col within the block.
LOCA_DEV int mfma32_row(int lane, int r) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
LOCA_DEV int mfma32_col(int lane) { return lane & 31; }

// f64 16x16x4: A lane l = A[l%16][l/16], B lane l = B[l/16][l%16];
// result r of lane l = D[l/16 + 4r][l%16].
LOCA_DEV f64x4_t mfma_f64(double a, double b, f64x4_t c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
// f32 32x32x2: A lane l = A[l%32][l/32], B lane l = B[l/32][l%32]; result as mfma32_row/col.
LOCA_DEV f32x16_t mfma_f32x2(float a, float b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------ direct-to-LDS staging (gfx950)
// Building blocks of the pipelined kernels that copy 32-row x 256-column bf16 stages
// straight from global memory into LDS (global_load_lds_dwordx4 / buffer_load ... lds).
// A stage is stored with rows of 512 bytes whose 16-byte chunks are XOR-swizzled,
// chunk c of row r at c ^ 4(r & 3), so that the transpose reads of a half wave are
// conflict-free.

LOCA_DEV int dl_swz(int row) { return 4 * (row & 3); }

// operand of v_mfma_f32_32x32x16_bf16 from a swizzled 32 x 256 stage (see frag32_tr)
LOCA_DEV bf16x8_t frag32_tr_swz(const uint16_t* tile, int c0, int ks, int lane) {
  const int g = lane >> 4, w = lane & 15;
  const int col = c0 + 16 * (g & 1) + 4 * (w & 3);
  const int row = ks + 8 * (g >> 1) + (w >> 2);
  const int lc = col >> 3, within = col & 7;
  const uint16_t* p0 = tile + row * 256 + 8 * (lc ^ dl_swz(row)) + within;
  const uint16_t* p1 = tile + (row + 4) * 256 + 8 * (lc ^ dl_swz(row + 4)) + within;
  s16x4_t lo = lds_read_tr16(p0);
  s16x4_t hi = lds_read_tr16(p1);
  typedef short s16x8_t __attribute__((ext_vector_type(8)));
  s16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8_t, v);
}

// s_waitcnt immediate that waits until at most n vector-memory operations are outstanding
constexpr int vmcnt_imm(int n) { return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8); }

// 16-byte global -> LDS copy for every lane: lane l's chunk lands at lds_base + 16 l.
// Issued as inline assembly so that the compiler does not treat it as a store to the
// ring slot being read and drain it before every LDS read; completion is tracked by
// the explicit vmcnt waits of the pipeline.
LOCA_DEV void lds_dma16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(lds_base) : "m0", "memory");
}
// The same copy through the buffer path: `voff` is a byte offset into the buffer of the
// resource `rsrc` (base, byte range, raw format); offsets at or past the range return zeros.
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
LOCA_DEV void lds_dma16_buf(uint32_t voff, i32x4_t rsrc, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds" ::"v"(voff), "s"(lds_base),
               "s"(rsrc) : "m0", "memory");
}
LOCA_DEV i32x4_t buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r[0] = (int32_t)(uint32_t)(a & 0xffffffffu);
  r[1] = (int32_t)(uint32_t)((a >> 32) & 0xffffu);  // stride 0
  r[2] = (int32_t)bytes;
  r[3] = 0x00020000;  // raw 32-bit data format
#pragma unroll
  for (int u = 0; u < 4; ++u) r[u] = __builtin_amdgcn_readfirstlane(r[u]);  // wave-uniform: scalar registers
  return r;
}
constexpr uint32_t kBufOutside = 0x80000000u;  // past every range used here (< 2^31 bytes)

// Workgroup barrier without a memory fence (the pipeline waits for its own loads explicitly).
LOCA_DEV void barrier_nofence() { asm volatile("s_barrier" ::: "memory"); }
// this wave's LDS operations complete and visible to its own lanes (no workgroup barrier)
LOCA_DEV void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), the other counters left alone
  __builtin_amdgcn_wave_barrier();
}

// Upper tile u (I <= J, T tiles per side) in an order that keeps consecutive tiles
// compact: bands of kBand tile rows, each band column by column (rows top to bottom).
// A window of 32 consecutive tiles then spans about 4 rows x 8 columns of tiles, so the
// tiles an XCD runs at the same time share more of their panels than in row order.
constexpr int kBand = 4;
LOCA_DEV void upper_tile_banded(int u, int T, int& I, int& J) {
  int r0 = 0;
  for (;;) {  // skip whole bands
    const int h = T - r0 < kBand ? T - r0 : kBand;
    const int cnt = h * (T - r0) - h * (h - 1) / 2;  // tiles of rows r0 .. r0 + h - 1 with J >= I
    if (u < cnt) break;
    u -= cnt;
    r0 += h;
  }
  int j = r0;
  for (;;) {  // columns of the band: column j holds rows r0 .. min(j, r0 + kBand - 1)
    const int hc = (j - r0 + 1) < kBand ? (j - r0 + 1) : kBand;
    if (u < hc) break;
    u -= hc;
    ++j;
  }
  I = r0 + u;
  J = j;
}

// The hardware hands consecutive workgroups to the eight XCDs in turn, and each XCD
// has its own L2.  Workgroup L is therefore given logical tile x * per + idx, with
// x = L % 8 and idx = L / 8, so that the tiles one XCD runs at the same time are
// neighbours in the upper triangle of one block and share their column panels in L2.
LOCA_DEV int xcd_logical(int L, int total) {
  const int per = total / 8, rem = total % 8;
  const int x = L % 8, idx = L / 8;
  return x * per + (x < rem ? x : rem) + idx;
}

}  // namespace loca
