// Ridge projection onto the span for large groups (dr_project_span with
// n > 256, e.g. the Gram-dominated workload's n = 16384): the ridge form of
// Eq. (proj), Sec. 3.3.1, (K + lam_eff I) w = s, solved by a blocked
// right-looking Cholesky factorisation in fp32 followed by iterative
// refinement with fp64 residuals of the exact fp32 K.
//
// Workspace (one group at a time; groups run one after another):
//   L     fp32 [n][ldL]   the factor (lower triangle; the rest is never read)
//   inv   fp32 [nblk][128][128]: the inverse of every 128x128 diagonal
//         block of L (used by the panel solve)
//   sinv  fp32 [nsb][1024][1024]: the inverse of every 1024x1024 diagonal
//         super-block of L, lower blocks only (used by the L solve; 64 MiB
//         at n = 16384)
//   sinvt fp32 [nsb][1024][1024]: the same inverses transposed, upper
//         blocks only (used by the L^T solve, so that both solves apply
//         their super-block inverse row by row)
//   x, dx, r, z  fp64 [npad] solution, correction, residual, work
//   ctl   status shared by the kernels of one group (skip / info / lam_eff)
//
// Per 128-column panel k:
//   lg_potrf_kernel  one workgroup factors and inverts the diagonal block
//                    in 16-column steps on packed 16x16 LDS tiles: one wave
//                    factors and inverts each 16x16 diagonal tile in
//                    registers (tile16_chol_inv), one step ahead of the
//                    others; the panel solve, the trailing update and the
//                    tiles of the inverse are fp32 MFMA products.
//   lg_trsm_kernel   L21 = A21 L11^-T as an fp32 MFMA product with the
//                    inverse, 64 rows per workgroup.
// Both keep their LDS under 96 KiB, so either fits on a CU beside one
// trailing-update workgroup while the update runs.
// Trailing updates: steps of four panels (rank 512) while the bulk of the
// update fills the CUs on bf16 MFMA, then pairs (rank 256).  Per step, two
// launches on the caller's stream: the head (lg_syrk_kernel, fp32 MFMA on
// 128x128 or 64x64 tiles: the next step's panel columns) and the bulk
// (lg_split_kernel + lg_syrk6_kernel on bf16 planes, or lg_syrk_kernel);
// meanwhile a second stream factors the next step's panels in turn (block
// factor, panel solve, rank-128 update of the step's other panel columns),
// so those latency-bound steps run under the bulk.
// Solve: the inverses of the 1024x1024 diagonal super-blocks are built a
// block row at a time from the 128x128 ones (lg_sinv_kernel) on a third
// stream as the factorisation finalises each block, with the first
// solve's forward sweep; then L y = r and L^T dx = y go super-block by
// super-block, two wide launches each (the super-block's share of the
// solution as a product with its inverse, then its update of the rest of
// the right-hand side), x += dx; the first solve and up to kRefine
// refinement steps, each preceded by r = s - (K + lam_eff I) x in fp64
// read straight from K, until the corrections pass the convergence test.
// The extra streams and their events are created once per device and kept.
// Every kernel first reads ctl->skip: once a group's result is decided (a
// non-finite input, an empty span, a non-positive pivot) the remaining
// launches of that group return at once.

#include <mutex>
#include <type_traits>

#include "common.h"

namespace dr {
namespace {

constexpr int NB = 128;        // panel width
constexpr int SB = 8;          // 128-blocks per super-block of the triangular solves
constexpr int SBN = SB * NB;   // rows of a super-block (leading dimension of its inverse)
constexpr int LDP = NB + 4;    // LDS row stride (floats) of staged slices: b128 reads are conflict-free
constexpr int kRefine = 2;

struct LgCtl {
  int skip;        // the group's result is decided; later kernels return at once
  int nonfinite;   // some entry of K or s is not finite
  int info;        // reported info (1-based pivot, or DR_INFO_NONFINITE)
  float lam;       // lam_eff
  int done;        // refinement converged before its last step; its remaining kernels return at once
  double dxn[kRefine + 1];   // max |dx| of each solve (the first solve's dx is x itself)
};

struct LgLayout {
  long long n, ldL, nblk, npad;
  size_t off_L, off_inv, off_sinv, off_sinvt, off_pl, off_x, off_dx, off_r, off_z, off_ctl, total;
};

LgLayout lg_layout(long long n) {
  LgLayout l;
  l.n = n;
  l.ldL = (long long)align_up((size_t)n, 4);
  l.nblk = (n + NB - 1) / NB;
  l.npad = l.nblk * NB;
  size_t o = 0;
  l.off_L = o;    o = align_up(o + (size_t)n * l.ldL * 4, 256);
  l.off_inv = o;  o = align_up(o + (size_t)l.nblk * NB * NB * 4, 256);
  l.off_sinv = o; o = align_up(o + (size_t)((l.nblk + SB - 1) / SB) * SBN * SBN * 4, 256);
  l.off_sinvt = o; o = align_up(o + (size_t)((l.nblk + SB - 1) / SB) * SBN * SBN * 4, 256);
  l.off_pl = o;   o = align_up(o + (size_t)3 * n * 4 * NB * 2, 256);   // three bf16 planes of four panels
  l.off_x = o;    o = align_up(o + (size_t)l.npad * 8, 256);
  l.off_dx = o;   o = align_up(o + (size_t)l.npad * 8, 256);
  l.off_r = o;    o = align_up(o + (size_t)l.npad * 8, 256);
  l.off_z = o;    o = align_up(o + (size_t)l.npad * 8, 256);
  l.off_ctl = o;  o = align_up(o + sizeof(LgCtl), 256);
  l.total = o;
  return l;
}

__device__ __forceinline__ bool finite_f(float v) { return (__float_as_uint(v) & 0x7f800000u) != 0x7f800000u; }


template <int NT>
__device__ double block_sum_d(double v, double* sh) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r += sh[i];   // same order in every thread
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------- set-up

__global__ void lg_init_kernel(LgCtl* ctl, const float* s, int n, int npad, double* x, double* dx, double* r,
                               double* z) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) {
    ctl->skip = 0;
    ctl->nonfinite = 0;
    ctl->info = 0;
    ctl->lam = 0.f;
    ctl->done = 0;
    for (int k = 0; k <= kRefine; ++k) ctl->dxn[k] = 0.0;
  }
  if (i < npad) {
    x[i] = 0.0;
    dx[i] = 0.0;
    z[i] = 0.0;
    r[i] = i < n ? (double)s[i] : 0.0;
  }
}

// non-finite check over all n*n entries of K (float4 when 16-byte aligned)
// trace, lam_eff and the early outcomes of s (non-finite entries) and of
// the trace (empty span); non-finite entries of K are found by lg_load_kernel
__global__ __launch_bounds__(1024) void lg_setup_kernel(const float* K, const float* s, int n, float lambda, int mode,
                                                        LgCtl* ctl, float* lam_eff_out) {
  __shared__ double sh[16];
  __shared__ int sbad;
  if (threadIdx.x == 0) sbad = 0;
  __syncthreads();
  double tr = 0.0;
  bool bad = false;
  for (int i = threadIdx.x; i < n; i += 1024) {
    tr += (double)K[(long long)i * n + i];
    bad |= !finite_f(s[i]);
  }
  if (bad) sbad = 1;
  tr = block_sum_d<1024>(tr, sh);   // contains a barrier: sbad is visible after it
  if (threadIdx.x == 0) {
    const bool nonfinite = sbad != 0;
    const float lam = mode == DR_RIDGE_REL_TRACE ? (float)((double)lambda * tr / (double)n) : lambda;
    ctl->lam = lam;
    if (nonfinite) {
      ctl->skip = 1;
      ctl->nonfinite = 1;
      ctl->info = DR_INFO_NONFINITE;
      *lam_eff_out = 0.f;
    } else {
      if (mode == DR_RIDGE_REL_TRACE && tr == 0.0) ctl->skip = 1;
      *lam_eff_out = lam;
    }
  }
}

// L = lower triangle of K + lam_eff I, and the finiteness scan of all of K
// in the same pass (the upper triangle is read only for the scan), columns
// c0 .. c1 - 1 (c0 a multiple of 4): row i, 4096 columns per workgroup, a
// float4 per thread and step (scalar loads when n is not a multiple of 4
// or K is not 16-byte aligned).  L is written
// only when the group is still open; a non-finite entry closes it with
// DR_INFO_NONFINITE, over the empty-span outcome of a zero trace.
constexpr int kLoadCols = 4096;
__global__ __launch_bounds__(256) void lg_load_kernel(const float* K, int n, int vec, int c0, int c1, float* L,
                                                      long long ldL, LgCtl* ctl, float* lam_eff_out) {
  __shared__ int any;
  const int i = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) any = 0;
  const bool write = ctl->skip == 0;
  const float lam = ctl->lam;
  const float* kr = K + (long long)i * n;
  __syncthreads();
  bool bad = false;
#pragma unroll
  for (int u = 0; u < kLoadCols / 1024; ++u) {
    const int c = c0 + blockIdx.y * kLoadCols + 1024 * u + 4 * tid;
    if (c >= c1) break;
    float4 v;
    if (vec) {
      v = *reinterpret_cast<const float4*>(kr + c);
    } else {
      v.x = kr[c];
      v.y = c + 1 < n ? kr[c + 1] : 0.f;
      v.z = c + 2 < n ? kr[c + 2] : 0.f;
      v.w = c + 3 < n ? kr[c + 3] : 0.f;
    }
    bad |= !(finite_f(v.x) && finite_f(v.y) && finite_f(v.z) && finite_f(v.w));
    if (write && c <= i) {
      if (c == i) v.x += lam;
      if (c + 1 == i) v.y += lam;
      if (c + 2 == i) v.z += lam;
      if (c + 3 == i) v.w += lam;
      // columns past the diagonal (and past n, up to ldL) are never read
      *reinterpret_cast<float4*>(L + (long long)i * ldL + c) = v;
    }
  }
  if (bad) any = 1;
  __syncthreads();
  if (tid == 0 && any) {   // every workgroup that finds one stores the same outcome
    ctl->nonfinite = 1;
    ctl->skip = 1;
    ctl->info = DR_INFO_NONFINITE;
    *lam_eff_out = 0.f;
  }
}

// ---------------------------------------------------------------- panel

__device__ __forceinline__ void tile_pair(int q, int& I, int& J) {
  int i = (int)((sqrtf(8.f * q + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= q) ++i;
  while (i * (i + 1) / 2 > q) --i;
  I = i;
  J = q - i * (i + 1) / 2;
}

constexpr int LDA = NB + 4;   // LDS row stride (floats) of staged 128-wide blocks

// C[row][col] += sum_{m < len} A[ra + row][ca + m] B[rb + col][cb + m] on one
// 16x16 tile (both operands read along their rows, a float4 per lane)
__device__ __forceinline__ f32x4 tile_nt(const float* A, int ra, int ca, const float* B, int rb, int cb, int len,
                                         int lr, int lq, f32x4 acc) {
  for (int m = 0; m < len; m += 16) {
    const float4 av = *reinterpret_cast<const float4*>(&A[(ra + lr) * LDA + ca + m + 4 * lq]);
    const float4 bv = *reinterpret_cast<const float4*>(&B[(rb + lr) * LDA + cb + m + 4 * lq]);
    acc = mma_f32(av.x, bv.x, acc);
    acc = mma_f32(av.y, bv.y, acc);
    acc = mma_f32(av.z, bv.z, acc);
    acc = mma_f32(av.w, bv.w, acc);
  }
  return acc;
}

// C[row][col] += sum_{m < len} A[ra + row][ca + m] B[rb + m][cb + col]
__device__ __forceinline__ f32x4 tile_nn(const float* A, int ra, int ca, const float* B, int rb, int cb, int len,
                                         int lr, int lq, f32x4 acc) {
  for (int m = 0; m < len; m += 16) {
    const float4 av = *reinterpret_cast<const float4*>(&A[(ra + lr) * LDA + ca + m + 4 * lq]);
    const float* bp = &B[(rb + m + 4 * lq) * LDA + cb + lr];
    acc = mma_f32(av.x, bp[0], acc);
    acc = mma_f32(av.y, bp[LDA], acc);
    acc = mma_f32(av.z, bp[2 * LDA], acc);
    acc = mma_f32(av.w, bp[3 * LDA], acc);
  }
  return acc;
}

// Factor and invert the kb x kb diagonal block at (k, k) (kb <= 128; the
// block is padded to 128 with the identity) in one workgroup, in LDS as
// packed lower-triangle 16x16 tiles (72 KiB in all, so the workgroup fits
// on a CU beside a trailing-update workgroup):
//   eight waves; the diagonal tile D_J is factored and inverted in
//   registers by wave 0 (tile16_chol_inv), one step ahead: while six
//   waves take the trailing tiles of step J, wave 0 updates tile
//   (J+1, J+1) first and factors it (wave 4, which shares wave 0's SIMD,
//   stays out of that phase); tile (0, 0) is loaded and factored by wave 0
//   while the others load the rest of the block;
//   panel tiles L_IJ = A_IJ D_J^-T and trailing tiles A_IK -= L_IJ L_KJ^T
//   are 16x16x16 fp32 MFMA products (two barriers per step);
//   row J of the inverse, X_Jm = -X_JJ sum_{i=m}^{J-1} L_Ji X_im (m < J),
//   needs only rows < J of it, the final tiles L_Ji and D_J^-1, so the six
//   waves form it in step J after their trailing tiles, while wave 0
//   factors tile J+1.
// Row r of every tile is stored at row position prm(r), so the rows
// 4q + j (q = 0..3) that one MFMA result register covers fall in four
// different LDS bank groups.
__device__ __forceinline__ int prm(int r) { return 4 * (r & 3) + (r >> 2); }
__device__ __forceinline__ int ptile(int I, int J) { return (I * (I + 1) / 2 + J) * 256; }   // J <= I
__device__ __forceinline__ int otile(int I, int J) { return (I * (I - 1) / 2 + J) * 256; }   // J < I

constexpr int kPotrfWaves = 8;   // wave 0 factors the diagonal tiles, the others the rest
template <int PB>
__global__ __launch_bounds__(64 * kPotrfWaves) void lg_potrf_kernel(float* L, long long ldL, int k, int kb,
                                                                    float* inv, LgCtl* ctl) {
  static_assert(PB == 16, "16x16 tiles");
  constexpr int NW = kPotrfWaves;
  if (ctl->skip) return;
  constexpr int NT = NB / 16;
  __shared__ __attribute__((aligned(16))) float Lt[NT * (NT + 1) / 2 * 256];   // the block, then its factor
  __shared__ __attribute__((aligned(16))) float Xd[NT * 256];                  // inverses of the diagonal tiles
  __shared__ __attribute__((aligned(16))) float Xo[NT * (NT - 1) / 2 * 256];   // off-diagonal tiles of the inverse
  __shared__ int bad_s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;

  // the block into the tiles: rows past kb are identity rows; a float4
  // chunk is read only if it starts on or left of the diagonal (it then
  // ends inside the row), and entries right of the diagonal are cleared.
  // Wave 0 loads tile (0, 0) alone and factors it (below) while the other
  // waves load the rest.
  const int lrow = lane >> 2, lc4 = 4 * (lane & 3);
  auto load_tile = [&](int q) {
    int I, J;
    tile_pair(q, I, J);
    const int i = 16 * I + lrow, j = 16 * J + lc4;
    return (i < kb && j <= i) ? *reinterpret_cast<const float4*>(L + (long long)(k + i) * ldL + k + j)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  auto store_tile = [&](int q, float4 a) {
    int I, J;
    tile_pair(q, I, J);
    const int i = 16 * I + lrow, j = 16 * J + lc4;
    if (i < kb) {
      if (j + 1 > i) a.y = 0.f;
      if (j + 2 > i) a.z = 0.f;
      if (j + 3 > i) a.w = 0.f;
    } else {
      a.x = j == i ? 1.f : 0.f;
      a.y = j + 1 == i ? 1.f : 0.f;
      a.z = j + 2 == i ? 1.f : 0.f;
      a.w = j + 3 == i ? 1.f : 0.f;
    }
    *reinterpret_cast<float4*>(&Lt[q * 256 + prm(lrow) * 16 + lc4]) = a;
  };
  constexpr int NQ = NT * (NT + 1) / 2;
  if (w == 0) {
    if (tid == 0) bad_s = 0;
    store_tile(0, load_tile(0));
  } else {
    constexpr int UQ = (NQ - 1 + NW - 2) / (NW - 1);
    float4 v[UQ];
#pragma unroll
    for (int u = 0; u < UQ; ++u) {
      const int q = w + (NW - 1) * u;   // 1 .. NQ - 1
      v[u] = q < NQ ? load_tile(q) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < UQ; ++u) {
      const int q = w + (NW - 1) * u;
      if (q < NQ) store_tile(q, v[u]);
    }
  }

  // wave 0: factor and invert diagonal tile J (block-relative pivot on failure)
  auto factor_diag = [&](int J) __attribute__((always_inline)) {
    float* D = Lt + ptile(J, J) + prm(lr) * 16;
    float a[16], xr[16];
#pragma unroll
    for (int m = 0; m < 16; m += 4) {
      const float4 t = *reinterpret_cast<const float4*>(D + m);
      a[m] = t.x;
      a[m + 1] = t.y;
      a[m + 2] = t.z;
      a[m + 3] = t.w;
    }
    const int bad_j = tile16_chol_inv(a, xr, lr);
    if (lane < 16) {
#pragma unroll
      for (int m = 0; m < 16; m += 4) {
        *reinterpret_cast<float4*>(D + m) = make_float4(a[m], a[m + 1], a[m + 2], a[m + 3]);
        *reinterpret_cast<float4*>(&Xd[J * 256 + prm(lr) * 16 + m]) = make_float4(xr[m], xr[m + 1], xr[m + 2], xr[m + 3]);
      }
    }
    if (lane == 0 && bad_j && bad_s == 0) bad_s = 16 * J + bad_j;
  };
  // C = A B^T on one tile pair (both read along their rows)
  auto nt16 = [&](const float* A, const float* B) {
    const float4 av = *reinterpret_cast<const float4*>(A + prm(lr) * 16 + 4 * lq);
    const float4 bv = *reinterpret_cast<const float4*>(B + prm(lr) * 16 + 4 * lq);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = mma_f32(av.x, bv.x, acc);
    acc = mma_f32(av.y, bv.y, acc);
    acc = mma_f32(av.z, bv.z, acc);
    acc = mma_f32(av.w, bv.w, acc);
    return acc;
  };

  // tile (I, J), J < I, of the inverse: T = sum_{m=J}^{I-1} L_Im X_mJ
  // (inv_sum over a range of m, X_mJ read as the MFMA B operand, k = row),
  // then X_IJ = -X_II T (inv_store)
  auto inv_sum = [&](int I, int J, int m0, int m1, f32x4 t) {
    for (int m = m0; m < m1; ++m) {
      const float4 av = *reinterpret_cast<const float4*>(Lt + ptile(I, m) + prm(lr) * 16 + 4 * lq);
      const float* X = m == J ? Xd + J * 256 : Xo + otile(m, J);
      t = mma_f32(av.x, X[prm(4 * lq + 0) * 16 + lr], t);
      t = mma_f32(av.y, X[prm(4 * lq + 1) * 16 + lr], t);
      t = mma_f32(av.z, X[prm(4 * lq + 2) * 16 + lr], t);
      t = mma_f32(av.w, X[prm(4 * lq + 3) * 16 + lr], t);
    }
    return t;
  };
  auto inv_store = [&](int I, int J, f32x4 t) {
    // X_IJ = -X_II T: T's result layout (row 4 lq + j, column lr in
    // register j) is the B operand of reduction index 4 lq + j
    const float4 xv = *reinterpret_cast<const float4*>(Xd + I * 256 + prm(lr) * 16 + 4 * lq);
    f32x4 x = {0.f, 0.f, 0.f, 0.f};
    x = mma_f32(xv.x, t[0], x);
    x = mma_f32(xv.y, t[1], x);
    x = mma_f32(xv.z, t[2], x);
    x = mma_f32(xv.w, t[3], x);
#pragma unroll
    for (int j = 0; j < 4; ++j) Xo[otile(I, J) + prm(4 * lq + j) * 16 + lr] = -x[j];
  };
  auto inv_tile = [&](int I, int J) { inv_store(I, J, inv_sum(I, J, J, I, f32x4{0.f, 0.f, 0.f, 0.f})); };
  // results out while the steps run: column J of the factor (tiles (I, J),
  // the chunk rule of the load: entries right of the diagonal inside a
  // chunk are never read) and block row I of the inverse (zero right of
  // its diagonal tile), one wave each
  auto write_lcol = [&](int J) {
    const int r = lane >> 2, c4 = 4 * (lane & 3);
    for (int I = J; I < NT; ++I) {
      const int i = 16 * I + r, j = 16 * J + c4;
      if (i < kb && j <= i)
        *reinterpret_cast<float4*>(L + (long long)(k + i) * ldL + k + j) =
            *reinterpret_cast<const float4*>(&Lt[ptile(I, J) + prm(r) * 16 + c4]);
    }
  };
  auto write_inv_row = [&](int I, int t0, int nt) {
    for (int e = t0; e < 16 * (NB / 4); e += nt) {
      const int r = e / (NB / 4), c = 4 * (e % (NB / 4)), J = c >> 4;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (J == I) v = *reinterpret_cast<const float4*>(&Xd[I * 256 + prm(r) * 16 + (c & 15)]);
      else if (J < I) v = *reinterpret_cast<const float4*>(&Xo[otile(I, J) + prm(r) * 16 + (c & 15)]);
      *reinterpret_cast<float4*>(inv + (long long)(16 * I + r) * NB + c) = v;
    }
  };
  static_assert(NT == NW, "one partial sum of the last inverse row per inverse wave");
  f32x4 tlast = {0.f, 0.f, 0.f, 0.f};   // wave v: row NT - 1, column v, over m < NT - 2

  if (w == 0) factor_diag(0);
  __syncthreads();
  for (int J = 0; J < NT; ++J) {
    if (bad_s) break;
    for (int I = J + 1 + w; I < NT; I += NW) {
      float* A = Lt + ptile(I, J);
      const f32x4 acc = nt16(A, Xd + J * 256);
#pragma unroll
      for (int j = 0; j < 4; ++j) A[prm(4 * lq + j) * 16 + lr] = acc[j];
    }
    __syncthreads();
    const int rest = NT - 1 - J, nrest = rest * (rest + 1) / 2;
    auto trail = [&](int q) {
      int I, K2;
      tile_pair(q, I, K2);
      I += J + 1;
      K2 += J + 1;
      const f32x4 p = nt16(Lt + ptile(I, J), Lt + ptile(K2, J));
      float* C = Lt + ptile(I, K2);
#pragma unroll
      for (int j = 0; j < 4; ++j) C[prm(4 * lq + j) * 16 + lr] -= p[j];
    };
    if (w == 0) {
      if (rest > 0) {   // tile (J+1, J+1) is trailing tile 0
        trail(0);
        factor_diag(J + 1);
      }
    } else if (w == 4) {
      // wave 4 shares wave 0's SIMD: it only writes out what is final
      write_lcol(J);
      if (J > 0) write_inv_row(J - 1, lane, 64);
    } else {
      // waves 1..3 and 5..7: the other trailing tiles, then row J of the
      // inverse; in step NT - 2 also the sums of row NT - 1 that need
      // only rows < NT - 2, so that step NT - 1 adds one term to each
      const int v = w < 4 ? w - 1 : w - 2;   // 0 .. 5
      for (int q = 1 + v; q < nrest; q += NW - 2) trail(q);
      if (J == NT - 1) {
        for (int m = v; m < J; m += NW - 2)
          inv_store(J, m, m < NT - 2 ? inv_sum(J, m, NT - 2, NT - 1, tlast) : inv_sum(J, m, m, J, f32x4{0.f, 0.f, 0.f, 0.f}));
      } else {
        for (int m = v; m < J; m += NW - 2) inv_tile(J, m);
        if (J == NT - 2) tlast = inv_sum(NT - 1, v, v, NT - 2, tlast);
      }
    }
    __syncthreads();
  }
  if (bad_s) {
    // padded pivots are exactly 1: a failure is always inside the block
    if (tid == 0) {
      ctl->info = k + bad_s;
      ctl->skip = 1;
    }
    return;
  }
  // the factor's columns and the inverse's rows above the last went out
  // during the steps
  write_inv_row(NT - 1, tid, 64 * NW);
}
constexpr int kPotrfPB = 16;

// L21 = A21 L11^-T: rows k+128+64b .. +64, X[r][c] = sum_m A[r][m] Inv[c][m].
// 16x16x4 fp32 MFMA; each lane reads a float4 along the reduction of both
// operands, so the four MFMAs of one 16-wide step take the reduction indices
// {t, 4+t, 8+t, 12+t} -- the same set for A and B, which is all that matters.
__global__ __launch_bounds__(256) void lg_trsm_kernel(float* L, long long ldL, int n, int k, const float* inv,
                                                      const LgCtl* ctl) {
  if (ctl->skip) return;
  // only the inverse goes through LDS (68 KiB, so the workgroup fits on a CU
  // beside a trailing-update workgroup); each wave reads its 16 rows of A21
  // straight into the MFMA operand layout
  __shared__ __attribute__((aligned(16))) float Bs[NB][LDP];
  const int tid = threadIdx.x;
  const int r0 = k + NB + 64 * blockIdx.x;
  const int w = tid >> 6, lane = tid & 63, lr = lane & 15, lq = lane >> 4;
  float4 av[NB / 16];
  {
    const int row = r0 + 16 * w + lr;
#pragma unroll
    for (int kk = 0; kk < NB / 16; ++kk)
      av[kk] = row < n ? *reinterpret_cast<const float4*>(L + (long long)row * ldL + k + 16 * kk + 4 * lq)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
    // every load of the thread in flight before the LDS writes
    constexpr int UB = NB * (NB / 4) / 256;
    float4 vb[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int t = tid + 256 * u, rr = t / (NB / 4), cq = t % (NB / 4);
      vb[u] = *reinterpret_cast<const float4*>(inv + (long long)rr * NB + 4 * cq);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int t = tid + 256 * u;
      *reinterpret_cast<float4*>(&Bs[t / (NB / 4)][4 * (t % (NB / 4))]) = vb[u];
    }
  }
  __syncthreads();
  f32x4 acc[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < NB / 16; ++kk) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const float4 bv = *reinterpret_cast<const float4*>(&Bs[16 * cb + lr][16 * kk + 4 * lq]);
      acc[cb] = mma_f32(av[kk].x, bv.x, acc[cb]);
      acc[cb] = mma_f32(av[kk].y, bv.y, acc[cb]);
      acc[cb] = mma_f32(av[kk].z, bv.z, acc[cb]);
      acc[cb] = mma_f32(av[kk].w, bv.w, acc[cb]);
    }
  }
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = r0 + 16 * w + 4 * lq + j;
      if (row < n) L[(long long)row * ldL + k + 16 * cb + lr] = acc[cb][j];
    }
  }
}


// A22 -= L21 L21^T on the lower-triangle 128x128 tiles of the trailing
// matrix (rows and columns from k1 = k + W).  The W-column panel slices
// of both tile rows stream through LDS in 32-column chunks (buffer ->
// LDS DMA, double buffered, 32 KiB per chunk, so two workgroups share a
// CU), in the conflict-free operand layout of the bf16 kernels (a 32-float
// row is 8 segments of 4 floats).  The tile of A22 is read into registers
// before the products and updated at the end.  Wave (wr, wc) computes the
// 64x64 sub-tile (wr, wc) with fp32 16x16x4 MFMA; each lane's 4-float
// segment feeds 4 MFMAs (reduction indices {t, 4 + t, 8 + t, 12 + t}, the
// same set for both operands).  On a diagonal tile the strictly upper
// sub-tile is skipped and only entries on or below the diagonal are written.
constexpr int SY_CH = 32;                 // panel columns per chunk

// W: panel width (the update has rank W: 128 for one panel, 256 for two).
// TS: tile edge, 128 (waves of 64 x 64) or 64 (waves of 32 x 32: a quarter
// of the products per workgroup, for launches with fewer 128-tiles than
// CUs, where the products of one tile are the latency).
// head = true: the tiles of the first h panels' columns (h NB / TS tile
// columns, column by column: they hold the next panels); head = false:
// every tile with I >= J >= h NB / TS.
// A workgroup takes tiles blockIdx.x, blockIdx.x + gridDim.x, ... < ntiles:
// a grid smaller than the chip leaves CUs free for the factorisation chain
// running on the other stream.
template <int W, int TS>
__global__ __launch_bounds__(256, 2) void lg_syrk_kernel(float* L, long long ldL, int n, int k, int h, int head,
                                                         int ntiles, const LgCtl* ctl) {
  static_assert(TS == 128 || TS == 64, "tile edge");
  constexpr int PANEL = TS * SY_CH * 4;   // bytes of one tile row's chunk
  constexpr int RB = TS / 32;             // 16-row blocks per wave
  constexpr int HB = TS / 32;             // DMA half blocks (8 rows) per wave and panel
  if (ctl->skip) return;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * 2 * PANEL];
  constexpr int NCH = W / SY_CH;
  static_assert(NCH % 2 == 0, "the next tile's first chunk goes to stage 0");
  const int k1 = k + W;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w & 1, wc = w >> 1;
  const int lr = lane & 15, lg = lane >> 4;
  // a tile's coordinates and this lane's DMA row offsets
  struct Tile {
    int ri, rj;
    bool diag;
    unsigned offi[HB], offj[HB];
  };
  int segs[HB];
#pragma unroll
  for (int u = 0; u < HB; ++u) segs[u] = swz_seg_of_lane(lane, (w + 4 * u) & 1);
  const int hc = h * (NB / TS);   // tile columns of the head
  auto tile_of = [&](int qt) {
    int I, J;
    if (head) {
      const int T = (n - k1 + TS - 1) / TS;
      J = 0;
      while (qt >= T - J) {
        qt -= T - J;
        ++J;
      }
      I = J + qt;
    } else {
      tile_pair(qt, I, J);
      I += hc;
      J += hc;
    }
    Tile t;
    t.ri = k1 + TS * I;
    t.rj = k1 + TS * J;
    t.diag = I == J;
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const int r = 8 * (w + 4 * u) + (lane >> 3);
      t.offi[u] = t.ri + r < n ? (unsigned)((long long)r * ldL * 4) : kOobOffset;
      t.offj[u] = t.rj + r < n ? (unsigned)((long long)r * ldL * 4) : kOobOffset;
    }
    return t;
  };
  // DMA of one chunk: wave w fills half blocks w, w + 4, ... of each panel
  auto issue = [&](const Tile& t, int ch, int st) {
    const __amdgpu_buffer_rsrc_t rsi = make_rsrc(L + (long long)t.ri * ldL, kOobOffset);
    const __amdgpu_buffer_rsrc_t rsj = make_rsrc(L + (long long)t.rj * ldL, kOobOffset);
    unsigned char* sb = lds + st * 2 * PANEL;
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const unsigned cofs = (unsigned)((k + SY_CH * ch + 4 * segs[u]) * 4);
      dma16<kAuxCached>(rsi, sb + (w + 4 * u) * 1024, t.offi[u] == kOobOffset ? kOobOffset : t.offi[u] + cofs);
      dma16<kAuxCached>(rsj, sb + PANEL + (w + 4 * u) * 1024,
                        t.offj[u] == kOobOffset ? kOobOffset : t.offj[u] + cofs);
    }
  };
  int qt = blockIdx.x;
  if (qt >= ntiles) return;
  Tile cur = tile_of(qt);
  issue(cur, 0, 0);
  for (; qt < ntiles; qt += gridDim.x) {
    const int qn = qt + gridDim.x;
    const Tile nxt = tile_of(qn < ntiles ? qn : qt);
    const bool active = !(cur.diag && wc > wr);
    // this lane's C entries (rows 4 lg + q of each 16-row block, column lr),
    // loaded under the first chunk's products
    f32x4 c[RB][RB];
    f32x4 acc[RB][RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cb = 0; cb < RB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      DR_WAIT_VM(0);
      DR_LDS_SYNC();
      // the last chunk brings in the next tile's first one (stage 0 was
      // last read by chunk NCH - 2, before this barrier)
      if (ch + 1 < NCH)
        issue(cur, ch + 1, (ch + 1) & 1);
      else if (qn < ntiles)
        issue(nxt, 0, 0);
      if (ch == 0 && active) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int cb = 0; cb < RB; ++cb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int row = cur.ri + (TS / 2) * wr + 16 * rb + 4 * lg + q;
              const int col = cur.rj + (TS / 2) * wc + 16 * cb + lr;
              c[rb][cb][q] = (row < n && col < n) ? L[(long long)row * ldL + col] : 0.f;
            }
      }
      if (active) {
        const unsigned char* sa = lds + (ch & 1) * 2 * PANEL;
        const unsigned char* sbp = sa + PANEL;
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          const int seg = 4 * sub + lg;
          f32x4 fa[RB], fb[RB];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) fa[rb] = __builtin_bit_cast(f32x4, swz_read(sa + (RB * wr + rb) * 2048, lr, seg));
#pragma unroll
          for (int cb = 0; cb < RB; ++cb) fb[cb] = __builtin_bit_cast(f32x4, swz_read(sbp + (RB * wc + cb) * 2048, lr, seg));
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cb = 0; cb < RB; ++cb)
#pragma unroll
              for (int t = 0; t < 4; ++t) acc[rb][cb] = mma_f32(fa[rb][t], fb[cb][t], acc[rb][cb]);
        }
      }
    }
    if (active) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < RB; ++cb)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = cur.ri + (TS / 2) * wr + 16 * rb + 4 * lg + q;
            const int col = cur.rj + (TS / 2) * wc + 16 * cb + lr;
            if (row < n && col < n && (!cur.diag || col <= row))
              L[(long long)row * ldL + col] = c[rb][cb][q] - acc[rb][cb][q];
          }
    }
    cur = nxt;
  }
}

// ------------------------------------------- bulk update on bf16 MFMA
//
// The bulk of the rank-256 trailing update, A22 -= L21 L21^T, with the fp32
// products taken on bf16 MFMA (16 times the fp32 MFMA rate):
//   lg_split_kernel  writes the step's panel rows below it (L21, W = 512 or
//                    256 columns) as three bf16 planes, x = x1 + x2 + x3 with
//                    x1 = bf16(x), x2 = bf16(x - x1), x3 = bf16(x - x1 - x2)
//                    (round to nearest even; each difference is exact in
//                    fp32), so x1 + x2 + x3 holds x to about 2^-24.
//   lg_syrk6_kernel  C -= sum over the six plane pairs (a, b) with
//                    a + b <= 2 (0-based: 00, 01, 10, 02, 11, 20) of
//                    P_a P_b^T: every product of bf16 values is exact in
//                    fp32 and the accumulation is fp32, and the dropped
//                    pairs (12, 21, 22) weigh 2^-24 and less, so each
//                    element's error is about 3 * 2^-24 of |x||y|: fp32
//                    products, at a sixth of the bf16 MFMA rate (2.6 times
//                    the fp32 MFMA rate).  The six products are run as one
//                    bf16 contraction over 6 W virtual columns, 64 per
//                    step: step s reads plane a of the tile's row panel and
//                    plane b of its column panel, columns 64 (s mod W/64)
//                    ..., for the pair s / (W/64).
// The tile machinery is that of the large-n Gram kernel: 256 x 256 tiles
// of the trailing matrix right of the head's tile columns (tiles
// I >= J >= skip in units of 256 from the trailing matrix's first row), four
// waves of 128 x 128 fp32 accumulators, a two-stage buffer -> LDS DMA ring
// of 64-column steps in the conflict-free operand layout.  At the end C is
// read, reduced and written as float4 straight from registers (on a
// diagonal tile only entries on or below the diagonal).

constexpr int S6_T = 256;                      // tile edge
constexpr int S6_K = 64;                       // virtual columns per step
constexpr int S6_PANEL = S6_T * S6_K * 2;      // bytes of one operand panel per step (32 KiB)
constexpr int S6_STAGE = 2 * S6_PANEL;
#ifndef DR_S6_MIN_ROUNDS
#define DR_S6_MIN_ROUNDS 1
#endif
constexpr int kS6MinRounds = DR_S6_MIN_ROUNDS;   // rounds of tiles below which the fp32 kernel takes the bulk

__device__ __forceinline__ unsigned bf16_rne_bits(float x) {
  const unsigned u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// rows k1 .. n-1, columns k .. k+W-1 of L -> planes [3][n][W] bf16 (row r of
// a plane is row k1 + r); one thread per 8 columns of a row
template <int W>
__global__ __launch_bounds__(256) void lg_split_kernel(const float* L, long long ldL, int n, int k, int k1,
                                                       unsigned short* pl, const LgCtl* ctl) {
  if (ctl->skip) return;
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  const int r = (int)(t / (W / 8)), c = (int)(t % (W / 8)) * 8;
  if (k1 + r >= n) return;
  const float* src = L + (long long)(k1 + r) * ldL + k + c;
  const float4 v0 = *reinterpret_cast<const float4*>(src);
  const float4 v1 = *reinterpret_cast<const float4*>(src + 4);
  const float x[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
  unsigned p0[4], p1[4], p2[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    unsigned h[2], m[2], l[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float v = x[2 * q + e];
      h[e] = bf16_rne_bits(v);
      const float r1 = v - __uint_as_float(h[e] << 16);
      m[e] = bf16_rne_bits(r1);
      const float r2 = r1 - __uint_as_float(m[e] << 16);
      l[e] = bf16_rne_bits(r2);
    }
    p0[q] = h[0] | (h[1] << 16);
    p1[q] = m[0] | (m[1] << 16);
    p2[q] = l[0] | (l[1] << 16);
  }
  const long long plane = (long long)n * W;
  unsigned short* d = pl + (long long)r * W + c;
  *reinterpret_cast<u32x4*>(d) = u32x4{p0[0], p0[1], p0[2], p0[3]};
  *reinterpret_cast<u32x4*>(d + plane) = u32x4{p1[0], p1[1], p1[2], p1[3]};
  *reinterpret_cast<u32x4*>(d + 2 * plane) = u32x4{p2[0], p2[1], p2[2], p2[3]};
}

// W: the width of the panels (the rank of the update): 256 (a pair) or 512
// (four panels); skip: the tile columns left to the head update (the next
// step's panels).  Four waves of 128 x 128 (one per SIMD) with the
// accumulators pinned in AGPRs by in-place asm MFMAs; per 64-column step
// the first half's products run with the second half's fragment reads
// between them, then one barrier, then the second half's products with the
// DMA of step s + 2 and the reads of step s + 1's first half between them.
// At the end each 16 x 16 block goes through a 4 x 4 transpose inside each
// quad of lanes (DPP), so lane 4 m + c holds four consecutive columns of one
// row: C is read, reduced and written as float4 straight from registers.
template <int W>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void lg_syrk6_kernel(const unsigned char* pl, float* L, long long ldL, int n, int k1, int skip, int ntiles,
                     const LgCtl* ctl) {
  constexpr int SPP = W / S6_K;         // steps per plane pair
  constexpr int S6_STEPS = 6 * SPP;     // 24 or 48
  if (ctl->skip) return;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * S6_STAGE];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w >> 1, wc = w & 1;   // 128-row half of the tile's rows, of its columns
  const int lr = lane & 15, lg = lane >> 4, qc = lane & 3, qm = lr >> 2;
  const int rows = n - k1;             // rows of the planes
  const long long planeB = (long long)n * W * 2;
  int segs[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) segs[u] = swz_seg_of_lane(lane, (w + 4 * u) & 1);
  for (int qt = blockIdx.x; qt < ntiles; qt += gridDim.x) {
    int I, J;
    tile_pair(qt, I, J);
    const int rowA0 = S6_T * (I + skip), rowB0 = S6_T * (J + skip);   // plane rows (trailing rows from k1)
    const bool diag = I == J;
    unsigned offA[8], offB[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = 8 * (w + 4 * u) + (lane >> 3);
      offA[u] = rowA0 + r < rows ? (unsigned)(r * W * 2) : kOobOffset;
      offB[u] = rowB0 + r < rows ? (unsigned)(r * W * 2) : kOobOffset;
    }
    // DMA q (0..15) of step s into stage st (q even: row panel, odd: column
    // panel; half block w + 4 (q / 2)); steps past the last load zeros
    auto dma1 = [&](int s, int st, int q) {
      const int t = s / SPP, c0 = S6_K * (s % SPP);
      const int pa = t == 2 || t == 4 ? 1 : (t == 5 ? 2 : 0);   // plane pairs 00 01 10 02 11 20
      const int pb = t == 1 || t == 4 ? 1 : (t == 3 ? 2 : 0);
      const int u = q >> 1;
      const unsigned cb = (unsigned)((c0 + segs[u] * 8) * 2);
      unsigned char* sb = lds + st * S6_STAGE;
      if (q & 1) {
        const __amdgpu_buffer_rsrc_t rb = make_rsrc(pl + pb * planeB + (long long)rowB0 * W * 2, kOobOffset);
        dma16<kAuxCached>(rb, sb + S6_PANEL + (w + 4 * u) * 1024,
                          offB[u] == kOobOffset || s >= S6_STEPS ? kOobOffset : offB[u] + cb);
      } else {
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(pl + pa * planeB + (long long)rowA0 * W * 2, kOobOffset);
        dma16<kAuxCached>(ra, sb + (w + 4 * u) * 1024,
                          offA[u] == kOobOffset || s >= S6_STEPS ? kOobOffset : offA[u] + cb);
      }
    };
    auto rd1 = [&](u32x4* fa, u32x4* fb, const unsigned char* sa, int kh, int q) {
      const int seg = 4 * kh + lg;
      if (q & 1) fb[q >> 1] = swz_read(sa + S6_PANEL + (wc * 8 + (q >> 1)) * 2048, lr, seg);
      else fa[q >> 1] = swz_read(sa + (wr * 8 + (q >> 1)) * 2048, lr, seg);
    };
    f32x4 acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // the zeros are in place before the prologue: the compiler does not
        // see the MFMAs inside the asm, so it would not space a register
        // write and the product that reads it apart
        asm volatile("" : "+a"(acc[i][j]));
      }
    auto mma = [&](int i, int j, const u32x4* fa, const u32x4* fb) {
      asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc[i][j]) : "v"(fa[i]), "v"(fb[j]));
    };
    u32x4 fa0[8], fb0[8], fa1[8], fb1[8];
    __syncthreads();   // every wave is done with the ring (previous tile)
#pragma unroll
    for (int q = 0; q < 16; ++q) dma1(0, 0, q);
    DR_WAIT_VM(0);
    DR_LDS_SYNC();
#pragma unroll
    for (int q = 0; q < 16; ++q) dma1(1, 1, q);
#pragma unroll
    for (int q = 0; q < 16; ++q) rd1(fa0, fb0, lds, 0, q);
    for (int s = 0; s < S6_STEPS; ++s) {
      const unsigned char* sa = lds + (s & 1) * S6_STAGE;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        rd1(fa1, fb1, sa, 1, q);
#pragma unroll
        for (int m = 4 * q; m < 4 * q + 4; ++m) mma(m & 7, m >> 3, fa0, fb0);
      }
      DR_WAIT_VM(0);
      DR_LDS_SYNC();
      const unsigned char* sn = lds + ((s + 1) & 1) * S6_STAGE;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        dma1(s + 2, s & 1, q);
        rd1(fa0, fb0, sn, 0, q);
#pragma unroll
        for (int m = 4 * q; m < 4 * q + 4; ++m) mma(m & 7, m >> 3, fa1, fb1);
      }
    }
    // the last products' results are read below: wait states after an MFMA
    // that the compiler does not see inside the asm
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");

    // C -= acc.  Block (i, j) after the quad transpose: lane 4 m + c holds
    // row 16 i + 4 (l / 16) + c, columns 16 j + 4 m .. + 3 of the wave's
    // quarter.  Rows past n are skipped; a column start past n reads column 0
    // instead (k1 and the tile origin are multiples of 4 and the row stride
    // is n rounded up to 4, so a float4 that starts below n lies in its row)
    // and writes nothing; on a diagonal tile only entries on or below the
    // diagonal are written.  Two block rows at a time, software-pipelined:
    // the next pair's sixteen float4 of C are requested before the current
    // pair is reduced and written.
    const int rq = k1 + rowA0 + wr * 128 + 4 * lg + qc;   // + 16 i
    const int cq = k1 + rowB0 + wc * 128 + 4 * qm;        // + 16 j
    const bool fast_tile_now = !diag && k1 + rowA0 + S6_T <= n && k1 + rowB0 + S6_T <= n;
    auto load_c = [&](f32x4 (&cv)[2][8], int ib) {
#pragma unroll
      for (int di = 0; di < 2; ++di)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int row = rq + 16 * (ib + di), col = cq + 16 * j;
          // (a row past n reads row n - 1 instead and writes nothing: the
          // loads stay unconditional, so their waits stay counted)
          cv[di][j] = *reinterpret_cast<const f32x4*>(L + (long long)(row < n ? row : n - 1) * ldL + (col < n ? col : 0));
        }
    };
    auto reduce_c = [&](const f32x4 (&cv)[2][8], int ib, auto fast_tile) {
      constexpr bool fast = decltype(fast_tile)::value;
#pragma unroll
      for (int di = 0; di < 2; ++di)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const f32x4 v = acc[ib + di][j];
          float x0 = v[0], x1 = v[1], x2 = v[2], x3 = v[3];
          {  // exchange across bit 0 of the quad lane
            const float s01 = (qc & 1) ? x0 : x1, s23 = (qc & 1) ? x2 : x3;
            const float r01 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s01), 0xB1, 0xF, 0xF, false));
            const float r23 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s23), 0xB1, 0xF, 0xF, false));
            if (qc & 1) { x0 = r01; x2 = r23; } else { x1 = r01; x3 = r23; }
          }
          {  // exchange across bit 1
            const float s02 = (qc & 2) ? x0 : x2, s13 = (qc & 2) ? x1 : x3;
            const float r02 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s02), 0x4E, 0xF, 0xF, false));
            const float r13 = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(s13), 0x4E, 0xF, 0xF, false));
            if (qc & 2) { x0 = r02; x1 = r13; } else { x2 = r02; x3 = r13; }
          }
          const int row = rq + 16 * (ib + di), col = cq + 16 * j;
          const f32x4 r = cv[di][j] - f32x4{x0, x1, x2, x3};
          float* dst = L + (long long)row * ldL + col;
          if (fast) {
            *reinterpret_cast<f32x4*>(dst) = r;
          } else if (row < n) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (col + e < n && (!diag || col + e <= row)) dst[e] = r[e];
          }
        }
    };
    // (the empty asm statements keep the compiler from regrouping the loads
    // and stores of different pairs)
    auto pipeline = [&](auto fast_tile) {
      f32x4 cva[2][8], cvb[2][8];
      load_c(cva, 0);
      load_c(cvb, 2);
      asm volatile("" ::: "memory");
      reduce_c(cva, 0, fast_tile);
      asm volatile("" ::: "memory");
      load_c(cva, 4);
      asm volatile("" ::: "memory");
      reduce_c(cvb, 2, fast_tile);
      asm volatile("" ::: "memory");
      load_c(cvb, 6);
      asm volatile("" ::: "memory");
      reduce_c(cva, 4, fast_tile);
      asm volatile("" ::: "memory");
      reduce_c(cvb, 6, fast_tile);
    };
    if (fast_tile_now)
      pipeline(std::true_type{});
    else
      pipeline(std::false_type{});
  }
}

// ---------------------------------------------------------------- solves

// Triangular solves by super-blocks of SB diagonal blocks (1024 rows).
// After the factorisation, the inverse of every 1024 x 1024 diagonal
// super-block of L is formed (lower triangle, from the 128 x 128 block
// inverses), and its transpose; a solve then takes two wide launches per
// super-block: the super-block's part of the solution as one product with
// its inverse (or the transpose, for L^T), and its contribution to the rest
// of the right-hand side.

// Block row ii of the inverse X of super-block S: block (ii, jj), jj < ii,
//   X_ij = -X_ii sum_{m=j}^{i-1} L_im X_mj,
// needs only the factor's block row ii (final once block ii is factored),
// the rows of X above it and X_ii, the inverse of the 128 x 128 diagonal
// block (read where the block factor left it); jj = ii copies X_ii onto the
// diagonal; the same row of several super-blocks in one launch (grid y).
// Each block is split over SV_CQ workgroups by column quarters
// (the chain of products of a block is the latency that counts); the
// 128 x 128 L_im and the quarter of X_mj are staged in LDS and wave w
// computes rows 32 w .. 32 w + 31 of the quarter with fp32 MFMA.  The block
// also goes, transposed, into block (jj, ii) of the transpose.
constexpr int SV_CQ = 4, SV_CW = NB / SV_CQ, SV_LDB = SV_CW + 4;

// C[row][col] += sum_{m < len} A[ra + row][ca + m] B[rb + m][cb + col], B
// with row stride SV_LDB
__device__ __forceinline__ f32x4 tile_nn_q(const float* A, int ra, const float* B, int cb, int lr, int lq, f32x4 acc) {
  for (int m = 0; m < NB; m += 16) {
    const float4 av = *reinterpret_cast<const float4*>(&A[(ra + lr) * LDA + m + 4 * lq]);
    const float* bp = &B[(m + 4 * lq) * SV_LDB + cb + lr];
    acc = mma_f32(av.x, bp[0], acc);
    acc = mma_f32(av.y, bp[SV_LDB], acc);
    acc = mma_f32(av.z, bp[2 * SV_LDB], acc);
    acc = mma_f32(av.w, bp[3 * SV_LDB], acc);
  }
  return acc;
}

__global__ __launch_bounds__(256) void lg_sinv_kernel(const float* L, long long ldL, int n, int nblk,
                                                      const float* inv, float* sinv, float* sinvt, int S0, int ii,
                                                      const LgCtl* ctl) {
  if (ctl->skip) return;
  const int S = S0 + blockIdx.y;   // row ii of super-blocks S0, S0 + 1, ...
  const int jj = blockIdx.x / SV_CQ, cq = blockIdx.x % SV_CQ, d = ii - jj;
  const int bj = SB * S + jj, bi = bj + d;
  if (d < 0 || bi >= nblk) return;
  float* X = sinv + (long long)S * SBN * SBN;     // [SBN][SBN]
  float* XT = sinvt + (long long)S * SBN * SBN;   // [SBN][SBN], X transposed
  const int tid = threadIdx.x, c0 = SV_CW * cq;
  if (d == 0) {
    const float* ib = inv + (long long)bi * NB * NB;
    for (int e = tid; e < NB * SV_CW / 4; e += 256) {
      // columns c0.. of all rows of X_ii, and rows c0.. of its transpose
      const int r = e / (SV_CW / 4), c = c0 + 4 * (e % (SV_CW / 4));
      *reinterpret_cast<float4*>(X + (long long)(NB * ii + r) * SBN + NB * ii + c) =
          *reinterpret_cast<const float4*>(ib + r * NB + c);
      const int t = c0 + e / (NB / 4), cc = 4 * (e % (NB / 4));
      *reinterpret_cast<float4*>(XT + (long long)(NB * ii + t) * SBN + NB * ii + cc) =
          make_float4(ib[cc * NB + t], ib[(cc + 1) * NB + t], ib[(cc + 2) * NB + t], ib[(cc + 3) * NB + t]);
    }
    return;
  }
  __shared__ __attribute__((aligned(16))) float As[NB * LDA];
  __shared__ __attribute__((aligned(16))) float Bs[NB * SV_LDB];
  const int lane = tid & 63, w = tid >> 6, lr = lane & 15, lq = lane >> 4;
  // stage a 128 x 128 block into As (row stride ld, rows >= rows_valid read as 0)
  auto stage_a = [&](const float* src, long long ld, int rows_valid) {
    float4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = tid + 256 * u, r = e / (NB / 4), c = 4 * (e % (NB / 4));
      v[u] = r < rows_valid ? *reinterpret_cast<const float4*>(src + (long long)r * ld + c)
                            : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = tid + 256 * u, r = e / (NB / 4), c = 4 * (e % (NB / 4));
      *reinterpret_cast<float4*>(&As[r * LDA + c]) = v[u];
    }
  };
  // columns c0 .. c0 + SV_CW of a 128-row block of X into Bs
  auto stage_b = [&](const float* src) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, r = e / (SV_CW / 4), c = 4 * (e % (SV_CW / 4));
      v[u] = *reinterpret_cast<const float4*>(src + (long long)r * SBN + c0 + c);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, r = e / (SV_CW / 4), c = 4 * (e % (SV_CW / 4));
      *reinterpret_cast<float4*>(&Bs[r * SV_LDB + c]) = v[u];
    }
  };
  constexpr int CT = SV_CW / 16;   // 16-column tiles of the quarter
  f32x4 acc[2][CT];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[a][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int rows_i = n - NB * bi < NB ? n - NB * bi : NB;   // rows of L that exist in block row bi
  for (int m = bj; m < bi; ++m) {
    stage_a(L + (long long)NB * bi * ldL + NB * m, ldL, rows_i);        // L_im
    stage_b(X + (long long)(NB * (m - SB * S)) * SBN + NB * jj);        // X_mj, the quarter
    __syncthreads();
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int c = 0; c < CT; ++c) acc[a][c] = tile_nn_q(As, 32 * w + 16 * a, Bs, 16 * c, lr, lq, acc[a][c]);
    __syncthreads();
  }
  // T into Bs, X_ii into As, then X_ij = -X_ii T
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q) Bs[(32 * w + 16 * a + 4 * lq + q) * SV_LDB + 16 * c + lr] = acc[a][c][q];
  stage_a(inv + (long long)bi * NB * NB, NB, NB);
  __syncthreads();
  f32x4 xo[2][CT];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < CT; ++c) xo[a][c] = tile_nn_q(As, 32 * w + 16 * a, Bs, 16 * c, lr, lq, f32x4{0.f, 0.f, 0.f, 0.f});
  __syncthreads();   // every wave is done reading As and Bs
  // the quarter of X_ij = -X_ii T through LDS, then out row by row and,
  // transposed, into rows c0.. of block (jj, ii) of XT (coalesced both ways)
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q) Bs[(32 * w + 16 * a + 4 * lq + q) * SV_LDB + 16 * c + lr] = -xo[a][c][q];
  __syncthreads();
  for (int e = tid; e < NB * SV_CW / 4; e += 256) {
    const int r = e / (SV_CW / 4), c = 4 * (e % (SV_CW / 4));
    *reinterpret_cast<float4*>(X + (long long)(NB * ii + r) * SBN + NB * jj + c0 + c) =
        *reinterpret_cast<const float4*>(&Bs[r * SV_LDB + c]);
    const int t = e / (NB / 4), cc = 4 * (e % (NB / 4));
    *reinterpret_cast<float4*>(XT + (long long)(NB * jj + c0 + t) * SBN + NB * ii + cc) =
        make_float4(Bs[cc * SV_LDB + t], Bs[(cc + 1) * SV_LDB + t], Bs[(cc + 2) * SV_LDB + t],
                    Bs[(cc + 3) * SV_LDB + t]);
  }
}

// out[i] = (or -=) sum_c M[i][c] v_c for rows i < rows, columns c < width
// (<= SBN); mode 1 limits row i to the 128-blocks on or left of its own (a
// lower-triangular block matrix), mode 2 to those on or right of it (an
// upper one); the other blocks are never read.  RW rows per wave, 4 waves
// per workgroup, all their loads in flight; lane l takes columns
// 4 l + 256 t; each row's sum is a fixed-order DPP reduction.
template <int RW>
__global__ __launch_bounds__(256) void lg_rowdot_kernel(const float* M, long long ldM, int rows, int width, int mode,
                                                        const double* v, double* out, int sub, const LgCtl* ctl) {
  if (ctl->skip || ctl->done) return;
  constexpr int CT = SBN / 256;   // float4 columns per lane
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row0 = 4 * RW * blockIdx.x + RW * w;
  float4 mv[RW][CT];
#pragma unroll
  for (int u = 0; u < RW; ++u) {
    const int row = row0 + u;
    const int lo = mode == 2 ? NB * (row / NB) : 0;
    const int hi = mode == 1 ? min(width, NB * (row / NB + 1)) : width;
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = 4 * lane + 256 * t;
      mv[u][t] = (row < rows && c >= lo && c < hi) ? *reinterpret_cast<const float4*>(M + (long long)row * ldM + c)
                                                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  double vv[CT][4];
#pragma unroll
  for (int t = 0; t < CT; ++t) {
    const int c = 4 * lane + 256 * t;
#pragma unroll
    for (int q = 0; q < 4; ++q) vv[t][q] = c < width ? v[c + q] : 0.0;
  }
#pragma unroll
  for (int u = 0; u < RW; ++u) {
    double acc = 0.0;
#pragma unroll
    for (int t = 0; t < CT; ++t)
      acc += (double)mv[u][t].x * vv[t][0] + (double)mv[u][t].y * vv[t][1] + (double)mv[u][t].z * vv[t][2] +
             (double)mv[u][t].w * vv[t][3];
    acc = wave_sum_l63(acc);
    const int row = row0 + u;
    if (lane == 63 && row < rows) out[row] = sub ? out[row] - acc : acc;
  }
}

// out[c] -= sum_i M[i][c] v_i for columns c < 64 * gridDim.x and rows
// i < rows (<= SBN).  64 columns per workgroup of 1024 threads: lane l of
// wave w reads a float4 of columns 4 (l % 16) in row stream 4 w + l / 16;
// the 64 streams take every 64th row, so all 1024 rows of a super-block are
// in flight at once (a wave load covers 4 rows x 256 bytes); the stream sums
// of a column are added in a fixed order.
constexpr int kColThreads = 1024;
__global__ __launch_bounds__(kColThreads) void lg_coldot_kernel(const float* M, long long ldM, int rows,
                                                                const double* v, double* out, const LgCtl* ctl) {
  if (ctl->skip || ctl->done) return;
  constexpr int NS = kColThreads / 16, CU = SBN / NS;   // row streams, rows of a stream
  __shared__ double vs[SBN], part[NS][64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int i = tid; i < rows; i += kColThreads) vs[i] = v[i];
  const int m0 = 64 * blockIdx.x, c4 = lane & 15, st = 4 * w + (lane >> 4);
  const float* col = M + m0 + 4 * c4;
  __syncthreads();   // vs
  // the stream's rows in two rounds of CH loads in flight (registers)
  constexpr int CH = CU / 2;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    float4 mv[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int i = st + NS * (h * CH + u);
      mv[u] = i < rows ? *reinterpret_cast<const float4*>(col + (long long)i * ldM) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int i = st + NS * (h * CH + u);
      const double vi = i < rows ? vs[i] : 0.0;
      a0 = fma((double)mv[u].x, vi, a0);
      a1 = fma((double)mv[u].y, vi, a1);
      a2 = fma((double)mv[u].z, vi, a2);
      a3 = fma((double)mv[u].w, vi, a3);
    }
  }
  part[st][4 * c4] = a0;
  part[st][4 * c4 + 1] = a1;
  part[st][4 * c4 + 2] = a2;
  part[st][4 * c4 + 3] = a3;
  __syncthreads();
  if (tid < 64) {
    double t = 0.0;
    for (int q = 0; q < NS; ++q) t += part[q][tid];
    out[m0 + tid] -= t;
  }
}

// x += dx, and the solve's max |dx| into ctl->dxn[it] (one workgroup).
// After the first refinement step (it = 1) the corrections so far are the
// first solution x0 and dx1: if they already pass the convergence test
// (the geometric estimate |dx1|^2 / |x0| of the error left), the second
// step's kernels return at once.
__global__ __launch_bounds__(1024) void lg_axpy_kernel(double* x, const double* dx, int npad, int it, LgCtl* ctl) {
  __shared__ double sh[16], shx[16];
  if (ctl->skip || ctl->done) return;
  double m = 0.0, mx = 0.0;
  for (int i = threadIdx.x; i < npad; i += 1024) {
    const double xi = x[i] + dx[i];
    x[i] = xi;
    m = fmax(m, fabs(dx[i]));
    mx = fmax(mx, fabs(xi));
  }
  for (int off = 32; off > 0; off >>= 1) {
    m = fmax(m, __shfl_xor(m, off, 64));
    mx = fmax(mx, __shfl_xor(mx, off, 64));
  }
  if ((threadIdx.x & 63) == 0) {
    sh[threadIdx.x >> 6] = m;
    shx[threadIdx.x >> 6] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double r = 0.0, X = 0.0;
    for (int q = 0; q < 16; ++q) {
      r = fmax(r, sh[q]);
      X = fmax(X, shx[q]);
    }
    ctl->dxn[it] = r;
    if (it >= 1 && it < kRefine && refine_converged(ctl->dxn[it - 1], r, X)) ctl->done = 1;
  }
}

// r = s - (K + lam I) x and kx = K x in fp64, one wave per row of K
__global__ __launch_bounds__(256) void lg_resid_kernel(const float* K, int n, const float* s, const double* x,
                                                       double* r, double* kx, const LgCtl* ctl) {
  if (ctl->skip || (!kx && ctl->done)) return;   // the final pass (kx != nullptr) always runs
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const float* kr = K + (long long)row * n;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  int j = lane;
  for (; j + 192 < n; j += 256) {
    a0 += (double)kr[j] * x[j];
    a1 += (double)kr[j + 64] * x[j + 64];
    a2 += (double)kr[j + 128] * x[j + 128];
    a3 += (double)kr[j + 192] * x[j + 192];
  }
  for (; j < n; j += 64) a0 += (double)kr[j] * x[j];
  double acc = (a0 + a1) + (a2 + a3);
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) {
    r[row] = (double)s[row] - acc - (double)ctl->lam * x[row];
    if (kx) kx[row] = acc;
  }
}

// The same with four rows per wave (n a multiple of 4, K 16-byte aligned):
// each load of x (fp64) serves four rows of K, where one row per wave
// fetched x from L2 once per row, twice the bytes of K itself.  Lane l takes
// columns 4 l + 256 t as a float4 of each row; rows past n reread row n - 1
// and their sums are dropped.
__global__ __launch_bounds__(256) void lg_resid4_kernel(const float* K, int n, const float* s, const double* x,
                                                        double* r, double* kx, const LgCtl* ctl) {
  if (ctl->skip || (!kx && ctl->done)) return;   // the final pass (kx != nullptr) always runs
  const int lane = threadIdx.x & 63;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 4;
  if (row0 >= n) return;
  const float* kr[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) kr[u] = K + (long long)min(row0 + u, n - 1) * n;
  double acc[4][2] = {{0.0, 0.0}, {0.0, 0.0}, {0.0, 0.0}, {0.0, 0.0}};
#pragma unroll 2
  for (int j = 4 * lane; j < n; j += 256) {
    const double2 x01 = *reinterpret_cast<const double2*>(x + j);
    const double2 x23 = *reinterpret_cast<const double2*>(x + j + 2);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 kv = *reinterpret_cast<const float4*>(kr[u] + j);
      acc[u][0] = fma((double)kv.x, x01.x, acc[u][0]);
      acc[u][1] = fma((double)kv.y, x01.y, acc[u][1]);
      acc[u][0] = fma((double)kv.z, x23.x, acc[u][0]);
      acc[u][1] = fma((double)kv.w, x23.y, acc[u][1]);
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const double t = wave_sum_l63(acc[u][0] + acc[u][1]);
    const int row = row0 + u;
    if (lane == 63 && row < n) {
      r[row] = (double)s[row] - t - (double)ctl->lam * x[row];
      if (kx) kx[row] = t;
    }
  }
}

__global__ __launch_bounds__(1024) void lg_final_kernel(const float* s, const float* t2, int n, const double* x,
                                                        const double* kx, const LgCtl* ctl, float* w, float* resid2,
                                                        int* info) {
  __shared__ double sh[16];
  __shared__ double shm[16];
  const bool skip = ctl->skip != 0;
  double q = 0.0, xm = 0.0;
  for (int i = threadIdx.x; i < n; i += 1024) {
    if (skip) {
      w[i] = 0.f;
    } else {
      w[i] = (float)x[i];
      q += x[i] * kx[i] - 2.0 * (double)s[i] * x[i];
      xm = fmax(xm, fabs(x[i]));
    }
  }
  for (int off = 32; off > 0; off >>= 1) xm = fmax(xm, __shfl_xor(xm, off, 64));
  if ((threadIdx.x & 63) == 0) shm[threadIdx.x >> 6] = xm;
  q = block_sum_d<1024>(q, sh);   // its barriers also publish shm
  if (threadIdx.x == 0) {
    double X = 0.0;
    for (int k = 0; k < 16; ++k) X = fmax(X, shm[k]);
    const bool converged = ctl->done || refine_converged(ctl->dxn[kRefine - 1], ctl->dxn[kRefine], X);
    resid2[0] = skip ? t2[0] : (float)((double)t2[0] + q);
    // a non-finite input outranks a pivot failure (the factorisation of the
    // first panels starts before the whole of K is scanned)
    info[0] = skip ? (ctl->nonfinite ? DR_INFO_NONFINITE : ctl->info) : (converged ? 0 : DR_INFO_NOT_CONVERGED);
  }
}

}  // namespace

size_t span_large_workspace(int64_t n) { return lg_layout(n).total; }

// the blocked solver's own streams and events (default priority), besides
// the caller's stream: aux runs the diagonal-block chain one pair ahead;
// sol forms the inverses of the diagonal super-blocks and the first forward
// solve while the factorisation is still running
struct LgStreams {
  hipStream_t aux = nullptr, sol = nullptr;
  hipEvent_t ev_col = nullptr, ev_next = nullptr, ev_blk = nullptr, ev_bulk = nullptr, ev_sol = nullptr;
};
static dr_status span_large_groups(const float* K, const float* s, const float* t2, int n, int P, float lambda,
                                   int mode, float* w, float* lam_eff, float* resid2, int32_t* info,
                                   const LgLayout& lay, unsigned char* base, hipStream_t hs, const LgStreams& st);

// The solver's two extra streams (default priority) and their events: one
// set per device, created by the first blocked solve on that device and
// kept until the process ends, so a call creates and destroys nothing.  A
// call holds its device's lock while it enqueues, so that the records of
// the events and the waits on them pair up when several host threads call
// at once (their work then shares the extra streams in call order).
namespace {
constexpr int kMaxDevices = 64;
struct AuxSet {
  std::mutex mu;
  bool ready = false;
  LgStreams st;
};
AuxSet g_aux[kMaxDevices];

void destroy_streams(LgStreams& st) {
  if (st.ev_col) (void)hipEventDestroy(st.ev_col);
  if (st.ev_next) (void)hipEventDestroy(st.ev_next);
  if (st.ev_blk) (void)hipEventDestroy(st.ev_blk);
  if (st.ev_bulk) (void)hipEventDestroy(st.ev_bulk);
  if (st.ev_sol) (void)hipEventDestroy(st.ev_sol);
  if (st.aux) (void)hipStreamDestroy(st.aux);
  if (st.sol) (void)hipStreamDestroy(st.sol);
  st = LgStreams{};
}
}  // namespace

dr_status span_large(const float* K, const float* s, const float* t2, int64_t n64, int P, float lambda, int mode,
                     float* w, float* lam_eff, float* resid2, int32_t* info, void* ws, size_t ws_bytes,
                     hipStream_t hs) {
  const LgLayout lay = lg_layout(n64);
  if (!ws || ws_bytes < lay.total) return DR_ERR_WORKSPACE;
  if (!aligned16(ws)) return DR_ERR_ARG;
  const int n = (int)n64;
  unsigned char* base = static_cast<unsigned char*>(ws);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return DR_ERR_HIP;
  AuxSet& a = g_aux[dev];
  std::lock_guard<std::mutex> lock(a.mu);
  if (!a.ready) {
    LgStreams& st = a.st;
    if (hipStreamCreateWithFlags(&st.aux, hipStreamNonBlocking) != hipSuccess ||
        hipStreamCreateWithFlags(&st.sol, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&st.ev_col, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&st.ev_next, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&st.ev_blk, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&st.ev_bulk, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&st.ev_sol, hipEventDisableTiming) != hipSuccess) {
      destroy_streams(st);
      return DR_ERR_HIP;
    }
    a.ready = true;
  }
  return span_large_groups(K, s, t2, n, P, lambda, mode, w, lam_eff, resid2, info, lay, base, hs, a.st);
}

static dr_status span_large_groups(const float* K, const float* s, const float* t2, int n, int P, float lambda,
                                   int mode, float* w, float* lam_eff, float* resid2, int32_t* info,
                                   const LgLayout& lay, unsigned char* base, hipStream_t hs, const LgStreams& st) {
  hipStream_t aux = st.aux, sol = st.sol;
  hipEvent_t ev_col = st.ev_col, ev_next = st.ev_next, ev_blk = st.ev_blk, ev_bulk = st.ev_bulk, ev_sol = st.ev_sol;
  // the bulk trailing update runs persistent on 7/8 of the two-per-CU
  // workgroup slots: one CU in four keeps room (LDS and waves) for one more
  // workgroup, where the diagonal-block chain of the next pair (factor,
  // panel solve, rank-128 update, each under 96 KiB of LDS) runs beside the
  // update instead of queueing behind it
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus < 32)
    cus = 256;
  const int rest_slots = 2 * cus - cus / 4;
  float* L = reinterpret_cast<float*>(base + lay.off_L);
  float* inv = reinterpret_cast<float*>(base + lay.off_inv);
  float* sinv = reinterpret_cast<float*>(base + lay.off_sinv);
  float* sinvt = reinterpret_cast<float*>(base + lay.off_sinvt);
  double* x = reinterpret_cast<double*>(base + lay.off_x);
  double* dx = reinterpret_cast<double*>(base + lay.off_dx);
  double* r = reinterpret_cast<double*>(base + lay.off_r);
  double* z = reinterpret_cast<double*>(base + lay.off_z);
  LgCtl* ctl = reinterpret_cast<LgCtl*>(base + lay.off_ctl);
  unsigned short* pl = reinterpret_cast<unsigned short*>(base + lay.off_pl);
  const long long ldL = lay.ldL;
  const int nblk = (int)lay.nblk, npad = (int)lay.npad;
  const long long nn = (long long)n * n;
  for (int p = 0; p < P; ++p) {
    const float* Kp = K + (long long)p * nn;
    const float* sp = s + (long long)p * n;
    hipLaunchKernelGGL(lg_init_kernel, dim3((npad + 255) / 256), dim3(256), 0, hs, ctl, sp, n, npad, x, dx, r, z);
    const int vec = aligned16(Kp) && n % 4 == 0;
    hipLaunchKernelGGL(lg_setup_kernel, dim3(1), dim3(1024), 0, hs, Kp, sp, n, lambda, mode, ctl, lam_eff + p);

    // Right-looking blocked factorisation by steps of four or two panels,
    // with look-ahead.  The trailing matrix takes one rank-512 update per
    // step of four panels while that update fills the CUs on bf16 MFMA
    // (a quarter of the passes over it of rank-128 updates), then one
    // rank-256 update per pair.  For the step of panels b .. b + m - 1 the
    // aux stream factors panel b, applies it to the step's other panel
    // columns (rank 128), factors panel b + 1, and so on, then updates the
    // next step's panel columns with the step's panels (head) and goes on
    // to factor them; the main stream meanwhile updates the rest (bulk).
    // The head and the bulk touch disjoint tiles and run side by side; the
    // head follows the previous step's bulk, whose columns include its own.
    // the head update of rank W (the first h panels' columns right of
    // k + W), on 64-tiles when 128-tiles would not give every CU one
    auto head_update_w = [&](auto wtag, int k, int h, hipStream_t strm) {
      constexpr int W = decltype(wtag)::value;
      const int rows = n - k - W;
      const int T = (rows + NB - 1) / NB;
      const int n128 = h * T - h * (h - 1) / 2;
      if (n128 >= cus) {
        hipLaunchKernelGGL((lg_syrk_kernel<W, 128>), dim3(n128), dim3(256), 0, strm, L, ldL, n, k, h, 1, n128, ctl);
      } else {
        const int T64 = (rows + 63) / 64;
        int n64 = 0;
        for (int J = 0; J < 2 * h; ++J) n64 += T64 - J > 0 ? T64 - J : 0;
        hipLaunchKernelGGL((lg_syrk_kernel<W, 64>), dim3(n64), dim3(256), 0, strm, L, ldL, n, k, h, 1, n64, ctl);
      }
    };
    auto head_update = [&](int W, int k, int h, hipStream_t strm) {
      if (W == NB)
        head_update_w(std::integral_constant<int, NB>{}, k, h, strm);
      else if (W == 2 * NB)
        head_update_w(std::integral_constant<int, 2 * NB>{}, k, h, strm);
      else
        head_update_w(std::integral_constant<int, 4 * NB>{}, k, h, strm);
    };
    auto factor_panel = [&](int b, hipStream_t strm) {
      const int k = NB * b;
      const int kb = n - k < NB ? n - k : NB;
      float* ib = inv + (long long)b * NB * NB;
      hipLaunchKernelGGL(lg_potrf_kernel<kPotrfPB>, dim3(1), dim3(64 * kPotrfWaves), 0, strm, L, ldL, k, kb, ib, ctl);
      const int rest = n - k - NB;
      if (rest > 0)
        hipLaunchKernelGGL(lg_trsm_kernel, dim3((rest + 63) / 64), dim3(256), 0, strm, L, ldL, n, k, ib, ctl);
    };
    // Triangular solves by super-blocks of SB diagonal blocks (lg_sinv_kernel
    // forms the inverses).  L z = r for super-block S (r is consumed): its
    // share of z as one product with the inverse, then its update of the
    // right-hand side below it.
    const int nsb = (nblk + SB - 1) / SB;
    auto fwd_step = [&](int S, hipStream_t strm) {
      const int o0 = SBN * S, nb = nblk - SB * S < SB ? nblk - SB * S : SB, width = NB * nb;
      const float* Xs = sinv + (long long)S * SBN * SBN;
      hipLaunchKernelGGL(lg_rowdot_kernel<1>, dim3((width + 3) / 4), dim3(256), 0, strm, Xs, (long long)SBN, width,
                         width, 1, r + o0, z + o0, 0, ctl);
      const int below = n - o0 - width;
      if (below > 0)
        hipLaunchKernelGGL(lg_rowdot_kernel<4>, dim3((below + 15) / 16), dim3(256), 0, strm,
                           L + (long long)(o0 + width) * ldL + o0, ldL, below, width, 0, z + o0, r + o0 + width, 1,
                           ctl);
    };
    // Block bb of the factor is final (factored, and its column below
    // solved): on the sol stream, row bb % SB of its super-block's inverse,
    // and the first solve's forward step of the super-block once its last
    // row is in.  So the inverses and the first forward solve run beside the
    // factorisation, and only the last block's row and forward step follow
    // it.  While the bulk updates run on bf16 MFMA the GPU is full and work
    // beside them only slows them down; from the first pair whose bulk does
    // not (the last pairs leave most CUs idle), the blocks factored so far
    // are queued at once, then each block as soon as it is final.
    auto after_block = [&](int bb) {
      const int S = bb / SB, ii = bb % SB;
      hipLaunchKernelGGL(lg_sinv_kernel, dim3((ii + 1) * SV_CQ), dim3(256), 0, sol, L, ldL, n, nblk, inv, sinv, sinvt,
                         S, ii, ctl);
      if (ii == SB - 1 || bb == nblk - 1) fwd_step(S, sol);
    };
    const int slots6 = cus - cus / 8;
    // panels in the step starting at block b: four while the rank-512 bulk
    // after them has a round of 256 x 256 tiles for the CUs it runs on
    auto width_at = [&](int b) -> int {
      if (b >= nblk) return 0;
      const int restq = n - NB * b - 4 * NB;
      if (b + 4 <= nblk && restq > 0) {
        const int T2 = (restq + S6_T - 1) / S6_T;
        if (T2 > 2 && (T2 - 2) * (T2 - 1) / 2 >= kS6MinRounds * slots6) return 4;
      }
      return b + 1 < nblk ? 2 : 1;
    };
    int queued = 0;      // blocks whose inverse rows are queued on sol
    bool late = false;   // the bulk updates have left bf16 MFMA
    // K into L in two parts: the first step's panel columns, which its
    // chain needs, then the rest, which the first head and bulk need
    int b = 0, m = width_at(0);
    auto load = [&](int c0, int c1) {
      if (c1 > c0)
        hipLaunchKernelGGL(lg_load_kernel, dim3(n, (c1 - c0 + kLoadCols - 1) / kLoadCols), dim3(256), 0, hs, Kp, n, vec,
                           c0, c1, L, ldL, ctl, lam_eff + p);
    };
    load(0, NB * m < n ? NB * m : n);
    if (hipEventRecord(ev_col, hs) != hipSuccess) return DR_ERR_HIP;
    if (hipStreamWaitEvent(aux, ev_col, 0) != hipSuccess) return DR_ERR_HIP;
    load(NB * m, n);
    if (hipEventRecord(ev_bulk, hs) != hipSuccess) return DR_ERR_HIP;   // no bulk yet
    while (b < nblk) {
      const int k = NB * b, W = NB * m;
      for (int i = 0; i < m; ++i) {
        factor_panel(b + i, aux);
        if (late) {
          if (hipEventRecord(ev_blk, aux) != hipSuccess || hipStreamWaitEvent(sol, ev_blk, 0) != hipSuccess)
            return DR_ERR_HIP;
          after_block(b + i);
          queued = b + i + 1;
        }
        if (i + 1 < m) head_update(NB, k + NB * i, m - 1 - i, aux);
      }
      if (hipEventRecord(ev_next, aux) != hipSuccess || hipStreamWaitEvent(hs, ev_next, 0) != hipSuccess)
        return DR_ERR_HIP;
      const int b2 = b + m, m2 = width_at(b2);
      const int rest = n - k - W;
      // the bulk on bf16 MFMA (split planes) while it has enough 256 x 256
      // tiles for the 7/8 of the CUs it runs on (one workgroup each); the
      // head takes the next step's m2 panel columns, skip tile columns
      const int skip = NB * m2 / S6_T;
      const int T2 = rest > 0 ? (rest + S6_T - 1) / S6_T : 0;
      const int n6 = T2 > skip ? (T2 - skip) * (T2 - skip + 1) / 2 : 0;
      const bool bulk6 = m >= 2 && m2 >= 2 && rest > 0 && n6 >= kS6MinRounds * slots6;
      late = late || !bulk6;
      if (late && queued < b2) {
        if (hipStreamWaitEvent(sol, ev_next, 0) != hipSuccess) return DR_ERR_HIP;
        // whole super-blocks of the backlog: each row of all of them in one
        // launch, then their forward steps; the rest block by block
        while (queued < b2 && queued % SB != 0) after_block(queued++);
        const int S_lo = queued / SB, S_hi = b2 / SB;
        if (S_hi > S_lo) {
          for (int ii = 0; ii < SB; ++ii)
            hipLaunchKernelGGL(lg_sinv_kernel, dim3((ii + 1) * SV_CQ, S_hi - S_lo), dim3(256), 0, sol, L, ldL, n, nblk,
                               inv, sinv, sinvt, S_lo, ii, ctl);
          for (int S = S_lo; S < S_hi; ++S) fwd_step(S, sol);
          queued = SB * S_hi;
        }
        while (queued < b2) after_block(queued++);
      }
      if (m2 == 0 || rest <= 0) break;
      if (hipStreamWaitEvent(aux, ev_bulk, 0) != hipSuccess) return DR_ERR_HIP;
      head_update(W, k, m2, aux);
      const int k1 = k + W;
      if (bulk6) {
        if (W == 4 * NB) {
          hipLaunchKernelGGL(lg_split_kernel<4 * NB>, dim3((rest * 64 + 255) / 256), dim3(256), 0, hs, L, ldL, n, k, k1,
                             pl, ctl);
          hipLaunchKernelGGL(lg_syrk6_kernel<4 * NB>, dim3(n6 < slots6 ? n6 : slots6), dim3(256), 0, hs,
                             reinterpret_cast<const unsigned char*>(pl), L, ldL, n, k1, skip, n6, ctl);
        } else {
          hipLaunchKernelGGL(lg_split_kernel<2 * NB>, dim3((rest * 32 + 255) / 256), dim3(256), 0, hs, L, ldL, n, k, k1,
                             pl, ctl);
          hipLaunchKernelGGL(lg_syrk6_kernel<2 * NB>, dim3(n6 < slots6 ? n6 : slots6), dim3(256), 0, hs,
                             reinterpret_cast<const unsigned char*>(pl), L, ldL, n, k1, skip, n6, ctl);
        }
      } else {
        const int T = (rest + NB - 1) / NB;
        const int nrest = T > m2 ? (T - m2) * (T - m2 + 1) / 2 : 0;
        if (nrest > 0) {
          // many rounds of tiles: the chain has slack, 15/16 of the slots;
          // under two rounds: the chain is the longer path, 3/4 of them
          const int slots =
              nrest >= 8 * cus ? 2 * cus - cus / 8 : (nrest < 4 * cus ? 2 * cus - cus / 2 : rest_slots);
          const int grid = nrest < slots ? nrest : slots;
          // (a step of one panel is the last: it has no bulk)
          if (W == 4 * NB)
            hipLaunchKernelGGL((lg_syrk_kernel<4 * NB, 128>), dim3(grid), dim3(256), 0, hs, L, ldL, n, k, m2, 0, nrest,
                               ctl);
          else
            hipLaunchKernelGGL((lg_syrk_kernel<2 * NB, 128>), dim3(grid), dim3(256), 0, hs, L, ldL, n, k, m2, 0, nrest,
                               ctl);
        }
      }
      if (hipEventRecord(ev_bulk, hs) != hipSuccess) return DR_ERR_HIP;
      b = b2;
      m = m2;
    }
    // r = s - (K + lam I) x, and K x into kx when kx != nullptr
    const bool rows4 = n % 4 == 0 && aligned16(Kp);
    auto resid = [&](double* kx) {
      if (rows4)
        hipLaunchKernelGGL(lg_resid4_kernel, dim3((n + 15) / 16), dim3(256), 0, hs, Kp, n, sp, x, r, kx, ctl);
      else
        hipLaunchKernelGGL(lg_resid_kernel, dim3((n + 3) / 4), dim3(256), 0, hs, Kp, n, sp, x, r, kx, ctl);
    };
    // the inverses and the first forward solve are in
    if (hipEventRecord(ev_sol, sol) != hipSuccess || hipStreamWaitEvent(hs, ev_sol, 0) != hipSuccess)
      return DR_ERR_HIP;
    for (int it = 0; it <= kRefine; ++it) {
      // L z = r (r is consumed; the first solve's was done beside the
      // factorisation), then L^T dx = z (z is consumed), by super-blocks
      if (it > 0) {
        resid(nullptr);
        for (int S = 0; S < nsb; ++S) fwd_step(S, hs);
      }
      for (int S = nsb - 1; S >= 0; --S) {
        const int o0 = SBN * S, nb = nblk - SB * S < SB ? nblk - SB * S : SB, width = NB * nb;
        const float* XTs = sinvt + (long long)S * SBN * SBN;
        hipLaunchKernelGGL(lg_rowdot_kernel<1>, dim3((width + 3) / 4), dim3(256), 0, hs, XTs, (long long)SBN, width,
                           width, 2, z + o0, dx + o0, 0, ctl);
        const int rows = n - o0 < width ? n - o0 : width;
        if (o0 > 0)
          hipLaunchKernelGGL(lg_coldot_kernel, dim3(o0 / 64), dim3(kColThreads), 0, hs, L + (long long)o0 * ldL, ldL,
                             rows, dx + o0, z, ctl);
      }
      hipLaunchKernelGGL(lg_axpy_kernel, dim3(1), dim3(1024), 0, hs, x, dx, npad, it, ctl);
    }
    resid(z);
    hipLaunchKernelGGL(lg_final_kernel, dim3(1), dim3(1024), 0, hs, sp, t2 + p, n, x, z, ctl, w + (long long)p * n,
                       resid2 + p, info + p);
    const dr_status rc = launch_status();
    if (rc != DR_OK) return rc;
  }
  return DR_OK;
}

}  // namespace dr
