// Internal helpers shared by the library's translation units (not part of
// the C ABI).  gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dr_api.h"

namespace dr {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// 16x16x32 bf16 MFMA, fp32 accumulate.  Lane l supplies A[l%16][8*(l/16)..+8]
// and B[8*(l/16)..+8][l%16]; C[4*(l/16)+j][l%16] lands in register j.
__device__ __forceinline__ f32x4 mma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// 16x16x4 fp32 MFMA.  Lane l supplies A[l%16][l/16] and B[l/16][l%16]; the
// C layout is the same as for mma_bf16.
__device__ __forceinline__ f32x4 mma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---- buffer -> LDS DMA (gfx950): lane l of a wave writes 16 bytes at the
// wave-uniform LDS address + 16 l; an offset outside the descriptor reads 0.

#define DR_WAIT_VM(n) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory")
#define DR_LDS_SYNC() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr unsigned kOobOffset = 0xFFFFFFF0u;   // outside every descriptor: reads as zeros

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// aux: cache policy of the load (2 = non-temporal on gfx950)
template <int AUX>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, unsigned char* lds_block, unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds_block, 16, voff, 0, 0, AUX);
}
constexpr int kAuxStream = 2;
constexpr int kAuxCached = 0;

// LDS layout of an operand tile for the bf16 MFMA: 16-row blocks of 2 KB
// (rows of 128 bytes = 8 segments of 16 bytes), segment seg of row r stored
// in slot seg ^ ((r >> 1) & 7).  The 16-byte reads of one MFMA operand (16
// rows, one segment per group of 16 lanes) then fall on distinct banks, and
// one wave's DMA fills one 8-row half block (1 KB) with lane l holding row
// l / 8, slot l % 8.  (The LDS serves 32 lanes of a 16-byte read at a time:
// rows with equal r mod 4 must get distinct slots across two segments, and
// measured bank-conflict counts are zero for this layout.)
__device__ __forceinline__ u32x4 swz_read(const unsigned char* blk, int r, int seg) {
  return *reinterpret_cast<const u32x4*>(blk + r * 128 + ((seg ^ ((r >> 1) & 7)) * 16));
}
// the segment that lane l loads when its wave fills half block h (0 or 1)
__device__ __forceinline__ int swz_seg_of_lane(int l, int h) { return (l & 7) ^ (4 * h + (l >> 4)); }

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

// gfx950 transposing LDS read: within each 16-lane group, source lane
// 4q + r addresses 4 consecutive 16-bit columns c..c+3 of row q; lane j of
// the group receives column c_0 + j of the four rows (its four values are
// rows 0..3 in order).
__device__ __forceinline__ v4s lds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
}

// swizzle of the 32-byte slots of a token row: rows that one transposing
// read touches (q = r & 3 and bit 3 of r) land in distinct bank groups
__device__ __forceinline__ int slot_xor(int r) { return (r & 3) | (((r >> 3) & 1) << 2); }

// fixed-order wave sum by DPP moves (no LDS round trips); the total is
// exact in lane 63 only: pairs, quads (quad_perm), halves of a row
// (row_half_mirror), rows (row_mirror), then row_bcast15 / row_bcast31
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_d(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROWS, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROWS, 0xF, false);
  return __hiloint2double(hi, lo);
}
__device__ __forceinline__ double wave_sum_l63(double v) {
  v += dpp_d<0xB1, 0xF>(v);    // quad_perm [1, 0, 3, 2]
  v += dpp_d<0x4E, 0xF>(v);    // quad_perm [2, 3, 0, 1]
  v += dpp_d<0x141, 0xF>(v);   // row_half_mirror
  v += dpp_d<0x140, 0xF>(v);   // row_mirror
  v += dpp_d<0x142, 0xA>(v);   // row_bcast15 into rows 1 and 3
  v += dpp_d<0x143, 0xC>(v);   // row_bcast31 into rows 2 and 3
  return v;
}

// the same fixed-order DPP wave sum for fp32 (total in lane 63 only)
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xF, false));
}
__device__ __forceinline__ float wave_sum_l63f(float v) {
  v += dpp_f<0xB1, 0xF>(v);
  v += dpp_f<0x4E, 0xF>(v);
  v += dpp_f<0x141, 0xF>(v);
  v += dpp_f<0x140, 0xF>(v);
  v += dpp_f<0x142, 0xA>(v);
  v += dpp_f<0x143, 0xC>(v);
  return v;
}

// Mixed-precision iterative refinement (fp32 factor, fp64 residuals) of a
// span solve: a = max|dx| of the next-to-last correction, b = max|dx| of
// the last one, X = max|x| after it.  The corrections shrink geometrically
// with rate about b / a, so b * b / a estimates the error left in x.  The
// solve counts as converged when the last correction is negligible, or
// when the corrections contract and that estimate is below 1e-6 of |x|
// (ten times under the 1e-5 relative accuracy the span solve promises).
__device__ __forceinline__ bool refine_converged(double a, double b, double X) {
  if (!(b <= 1e300) || !(X <= 1e300)) return false;   // NaN or inf
  if (b <= 1e-9 * X) return true;
  return b <= 0.5 * a && b * b <= 1e-6 * X * a;
}

// ---- one-wave Cholesky factor and inverse of a 16 x 16 tile (the diagonal
// tiles of the blocked factorisations).  Lane l holds row r = l % 16 of the
// tile in a[0..15]; each 16-lane row of the wave holds the whole tile
// (entries right of the diagonal are ignored).  On return a is row r of L
// (zeros right of the diagonal) and x row r of L^-1.  Column j: the pivot
// d = a_j[j]; L[r][j] = a_r[j] / sqrt(d); the later columns take
// a_r[c] -= L[r][j] L[c][j].  Values cross lanes only inside a 16-lane row,
// by the DPP row_newbcast source modifier (lane n of the row to every lane
// of it), fused into the fma that uses them: one instruction per update and
// no trip through a scalar register.  Lane j + 1 forms its next pivot from
// its own L[j+1][j] (the value the broadcast would bring it), so the chain
// from one pivot to the next is a broadcast, a reciprocal square root (the
// hardware estimate, 1 ulp: the factor is refined in fp64 by its users), a
// product and an fma.  The inverse is a forward elimination of [D | I] run
// alongside: y starts as row r of I, and at step j rows below j take
// -(L[r][j] / L[j][j]) times row j (its columns <= j, the only ones it has
// yet), so row r of L^-1 is y / L[r][r] at the end; these updates fill the
// latency of the pivot chain.  A DPP source must not have been written by
// the two instructions before it: the first update of a column carries two
// wait states after the write of L[.][j]; an inverse update reads y[c],
// last written by the inverse updates of the previous column, at least
// fourteen of these (ordered) instructions back.  All 64 lanes must be
// active.  Returns the 1-based index of the first pivot that is not
// positive, else 0 (the tile's values are then meaningless).
template <int N>
__device__ __forceinline__ float row_bcast16(float v) {   // lane N of this lane's 16-lane row
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + N, 0xF, 0xF, false));
}
// acc += (src of lane N of this lane's 16-lane row) * mul, one instruction;
// NOP: two wait states first (a VALU write of src must be that far back)
template <int N, bool NOP>
__device__ __forceinline__ void fmac_row(float& acc, float src, float mul) {
  if (NOP)
    asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
                 : "+v"(acc) : "v"(src), "v"(mul), "n"(N));
  else
    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
                 : "+v"(acc) : "v"(src), "v"(mul), "n"(N));
}
#define DR_ROW_CASES(F) F(0) F(1) F(2) F(3) F(4) F(5) F(6) F(7) F(8) F(9) F(10) F(11) F(12) F(13) F(14) F(15)
__device__ __forceinline__ float row_bcast(float v, int n) {   // n a constant after unrolling
  switch (n) {
#define DR_CASE(K) case K: return row_bcast16<K>(v);
    DR_ROW_CASES(DR_CASE)
#undef DR_CASE
  }
  return v;
}
template <bool NOP>
__device__ __forceinline__ void fmac_rown(float& acc, float src, float mul, int n) {
  switch (n) {
#define DR_CASE(K) case K: fmac_row<K, NOP>(acc, src, mul); break;
    DR_ROW_CASES(DR_CASE)
#undef DR_CASE
  }
}
__device__ __forceinline__ int tile16_chol_inv(float (&a)[16], float (&x)[16], int r) {
  auto gt = [r](int j) { return (float)((unsigned)(j - r) >> 31); };   // 1 if r > j
  auto eq = [&](int j) { return gt(j - 1) - gt(j); };                 // 1 if r == j
  float y[16], dv[16], dg[16];
#pragma unroll
  for (int m = 0; m < 16; ++m) {
    a[m] *= gt(m - 1);
    y[m] = eq(m);
  }
  int bad = 0;
  float p = a[0];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const float d = row_bcast(p, j);
    if (bad == 0 && !(d > 0.f)) bad = j + 1;
    const float rs = __builtin_amdgcn_rsqf(d);
    dv[j] = rs;
    dg[j] = d * rs;
    const float u = a[j] * rs;
    if (j + 1 < 16) p = fmaf(-u, u, a[j + 1]);
    const float f = gt(j) * u;
    a[j] = f;
    const float nf = -f, ng = -(f * rs);
#pragma unroll
    for (int c = j + 1; c < 16; ++c) {
      if (c == j + 1) fmac_rown<true>(a[c], f, nf, c);
      else fmac_rown<false>(a[c], f, nf, c);
    }
#pragma unroll
    for (int c = 0; c <= j; ++c) fmac_rown<false>(y[c], y[c], ng, j);
  }
  float ld = 0.f, li = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    ld = fmaf(eq(j), dg[j], ld);
    li = fmaf(eq(j), dv[j], li);
  }
#pragma unroll
  for (int m = 0; m < 16; ++m) {
    a[m] = fmaf(a[m], gt(m), eq(m) * ld);
    x[m] = y[m] * li;
  }
  return __builtin_amdgcn_readfirstlane(bad);
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline dr_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? DR_OK : DR_ERR_HIP;
}

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// blocked Cholesky ridge solve for large groups (chol.hip)
constexpr int64_t kSpanLargeMaxN = 65536;
size_t span_large_workspace(int64_t n);
dr_status span_large(const float* K, const float* s, const float* t2, int64_t n, int P, float lambda, int mode,
                     float* w, float* lam_eff, float* resid2, int32_t* info, void* ws, size_t ws_bytes,
                     hipStream_t hs);

// Direct scorer over the update-assembly kernel (update.hip): s[l][i] =
// <gstar_l, G_i^(l)> for bf16 layers, gstar_l = gstar + g_off[l]
size_t direct_workspace(const dr_layer* layers, int num_layers, int64_t n);
dr_status direct_scores(const dr_layer* layers, int num_layers, int64_t n, int64_t T, const int32_t* len,
                        const float* gstar, const int64_t* g_off, float* s, void* workspace, hipStream_t hs);

}  // namespace dr
