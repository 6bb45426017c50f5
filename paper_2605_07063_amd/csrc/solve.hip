// Projection of the mean target gradient onto the feasible set spanned by
// the general-data gradients, in Gram form (Eq. (proj), Sec. 3.3.1):
//   span:  (K + lam_eff I) w = s                 (dr_project_span)
//   cone:  min_{w >= 0} 1/2 w^T K w - s^T w      (dr_project_cone)
// One workgroup per group p.  Both report resid2 = ||gbar - G^T w||^2 =
// t2 - 2 s.w + w.K.w without touching G.
//
// span_small_kernel (n <= 256): the lower triangle of K + lam_eff I is held
// in LDS as 16 x 16 fp32 tiles (at most 136 KiB) and factored right-looking
// in 16-column steps by the whole workgroup (a one-wave register factor of
// the diagonal tile, then fp32 MFMA tile products); forward / back substitution
// run in fp32 on vectors held in the registers of one wave, 16 rows at a time
// through the stored inverses of the diagonal tiles (v_readlane broadcasts,
// no block barrier); two steps of iterative
// refinement recompute s - (K + lam_eff I) w in fp64 from the fp32 K read
// from global memory (one wave per row), which brings the solution to
// fp64-level accuracy whenever cond(K + lam_eff I) * 2^-24 < 1.
//
// n <= 64 (the tiny, small-block and long-context workloads) is latency
// bound, and everything runs in fp64 on the exact fp32 inputs (no refinement
// needed):
//   n <= 16       span_wave_kernel / cone_wave_kernel, one 64-lane wave,
//                 lane i owns row i, no block barriers;
//   16 < n <= 64  span_cols_kernel (rows across lanes, 16-column slices
//                 across waves, one barrier per pivot) and cone_quad_kernel
//                 (four lanes per row, one barrier per step).
//
// cone_pg_kernel (n <= 256): projected gradient on the Jacobi-scaled
// problem, written on the unscaled variable: with r_i = K_ii^-1/2,
//   w_i <- max(0, w_i - r_i^2 (K w - s)_i / Lhat),  Lhat = max_i sum_j r_i |K_ij| r_j,
// which is exactly w~ <- max(0, w~ - (K~ w~ - s~)/Lhat) for w~ = w / r.
// K stays in registers as the exact fp32 input (rows split over a
// power-of-two group of lanes within one wave); w and all sums are fp64.
//
// simplex_pg_kernel (n <= 256, dr_project_simplex): soft weighting over the
// probability simplex, min_{w in simplex} w^T K w - 2 s^T w, by accelerated
// projected gradient (FISTA) with step 1/L, L = 2 max_i sum_j |K_ij|, and
// the exact Euclidean projection onto the simplex (Michelot's iteration:
// theta = (sum_{v_i > theta} v_i - 1) / #{v_i > theta} until the set stops
// shrinking, a handful of block reductions).  Same K layout as the cone.
// simplex_wave_kernel (n <= 64): the same iteration on one wave, every
// reduction a wave reduction (no block barrier per step).

#include "common.h"

namespace dr {
namespace {

constexpr int kSpanThreads = 1024;
constexpr int kSpanMaxN = 256;
constexpr int kConeThreads = 1024;
constexpr int kConeMaxN = 256;

__device__ __forceinline__ int tri(int i, int j) { return i * (i + 1) / 2 + j; }   // j <= i

// block-wide fp64 sum over kSpanThreads / kConeThreads threads (fixed order)
template <int NT>
__device__ double block_sum(double v, double* scratch) {
  const int tid = threadIdx.x;
  for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
  if ((tid & 63) == 0) scratch[tid >> 6] = v;
  __syncthreads();
  double r = 0.0;
  if (tid == 0) {
    for (int w = 0; w < NT / 64; ++w) r += scratch[w];
    scratch[NT / 64] = r;
  }
  __syncthreads();
  r = scratch[NT / 64];
  __syncthreads();
  return r;
}

// block-wide maximum of |v| over NT threads
template <int NT>
__device__ double block_absmax(double v, double* scratch) {
  const int tid = threadIdx.x;
  v = fabs(v);
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_down(v, off, 64));
  if ((tid & 63) == 0) scratch[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) {
    double r = 0.0;
    for (int w = 0; w < NT / 64; ++w) r = fmax(r, scratch[w]);
    scratch[NT / 64] = r;
  }
  __syncthreads();
  const double r = scratch[NT / 64];
  __syncthreads();
  return r;
}

constexpr int kWaveN = 64;

__device__ __forceinline__ double wave_sum(double v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ double wave_max(double v) {
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  return v;
}
// value of lane src (src uniform) as a scalar broadcast
__device__ __forceinline__ double readlane_d(double v, int src) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), src);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), src);
  return __hiloint2double(hi, lo);
}

// The lower triangle of the (padded) matrix as 16 x 16 tiles: tile (I, J),
// J <= I, starts at float (I (I + 1) / 2 + J) * 256, and row r of a tile is
// stored at row position rperm(r), so that the rows 4q + j (q = 0..3) that
// one MFMA result register covers fall in four different LDS bank groups
// while a tile row stays 16 contiguous floats.
constexpr int kSpanTiles = kSpanMaxN / 16;
__device__ __forceinline__ int rperm(int r) { return 4 * (r & 3) + (r >> 2); }
__device__ __forceinline__ int tile_at(int I, int J) { return (I * (I + 1) / 2 + J) * 256; }
// offset of column i inside the tile row that holds it
__device__ __forceinline__ int col_off(int i) { return (i >> 4) * 256 + (i & 15); }
// start of row k of the matrix (tile column 0)
__device__ __forceinline__ int row_at(int k) { return tile_at(k >> 4, 0) + rperm(k & 15) * 16; }

__device__ __forceinline__ float readlane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
// q -> (I, J) with q = I (I + 1) / 2 + J, 0 <= J <= I
__device__ __forceinline__ void tri_pair(int q, int& I, int& J) {
  int i = (int)((sqrtf(8.f * q + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= q) ++i;
  while (i * (i + 1) / 2 > q) --i;
  I = i;
  J = q - i * (i + 1) / 2;
}

__global__ __launch_bounds__(kSpanThreads) void span_small_kernel(const float* K, const float* s, const float* t2,
                                                                  int n, float lambda, int mode, float* w,
                                                                  float* lam_eff_out, float* resid2, int* info) {
  __shared__ __attribute__((aligned(16))) float Lt[kSpanTiles * (kSpanTiles + 1) / 2 * 256];
  __shared__ __attribute__((aligned(16))) float Xt[kSpanTiles * 256];   // inverses of the diagonal tiles
  __shared__ double x[kSpanMaxN], y[kSpanMaxN], sd[kSpanMaxN];   // sd: s, staged once
  __shared__ double scratch[kSpanThreads / 64 + 1];
  __shared__ int flag;
  // q -> (I, J) of the lower block triangle, q = I (I + 1) / 2 + J, as a
  // table (the trailing update would otherwise take a square root and two
  // correction loops per tile)
  constexpr int kTriQ = kSpanTiles * (kSpanTiles + 1) / 2;
  __shared__ unsigned char tri_tab[2][kTriQ];
  const int p = blockIdx.x, tid = threadIdx.x;
  const int wid = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lq = lane >> 4;
  constexpr int NW = kSpanThreads / 64;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const int nt = (n + 15) >> 4;

  // K into the tiles: wave w reads rows w, w + 16, ... of K whole (lanes
  // across the row, coalesced, 32 loads in flight per lane), checks every
  // entry for finiteness, adds the diagonal to the trace and stores the
  // entries of the lower block triangle (block column <= block row, so the
  // diagonal tiles hold both of their triangles); rows and columns from n up
  // to 16 nt are padded with the identity
  if (tid == 0) flag = 0;
  if (tid < kTriQ) {
    int I, J;
    tri_pair(tid, I, J);
    tri_tab[0][tid] = (unsigned char)I;
    tri_tab[1][tid] = (unsigned char)J;
  }
  double tr = 0.0;
  bool bad = false;
  for (int i = tid; i < n; i += kSpanThreads) bad |= !isfinite(sp[i]);
  {
    constexpr int RB = 8, C4 = kSpanMaxN / 64;
    for (int r0 = wid; r0 < n; r0 += RB * NW) {
      float v[RB][C4];
#pragma unroll
      for (int t = 0; t < RB; ++t) {
        const int i = min(r0 + NW * t, n - 1);
#pragma unroll
        for (int c = 0; c < C4; ++c) v[t][c] = Kp[(long long)i * n + min(lane + 64 * c, n - 1)];
      }
#pragma unroll
      for (int t = 0; t < RB; ++t) {
        const int i = r0 + NW * t;
        if (i >= n) break;
#pragma unroll
        for (int c = 0; c < C4; ++c) {
          const int j = lane + 64 * c;
          if (j >= n) continue;
          bad |= !isfinite(v[t][c]);
          if (i == j) tr += (double)v[t][c];
          if ((j >> 4) <= (i >> 4)) Lt[row_at(i) + col_off(j)] = v[t][c];
        }
      }
    }
    if (n & 15) {
      const int I = nt - 1;
      for (int e = tid; e < 16 * 16 * nt; e += kSpanThreads) {
        const int i = 16 * I + (e >> 4) / nt, j = 16 * ((e >> 4) % nt) + (e & 15);
        if (i >= n || j >= n) Lt[row_at(i) + col_off(j)] = i == j ? 1.f : 0.f;
      }
    }
  }
  __syncthreads();
  if (bad) flag = 1;
  tr = block_sum<kSpanThreads>(tr, scratch);
  const bool nonfinite = flag != 0;
  __syncthreads();

  const float lam = mode == DR_RIDGE_REL_TRACE ? (float)((double)lambda * tr / (double)n) : lambda;
  if (nonfinite || (mode == DR_RIDGE_REL_TRACE && tr == 0.0)) {
    for (int i = tid; i < n; i += kSpanThreads) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      lam_eff_out[p] = nonfinite ? 0.f : lam;
      resid2[p] = t2[p];
      info[p] = nonfinite ? DR_INFO_NONFINITE : 0;
    }
    return;
  }
  for (int i = tid; i < n; i += kSpanThreads) Lt[row_at(i) + col_off(i)] += lam;
  if (tid == 0) flag = 0;
  __syncthreads();

  // right-looking blocked Cholesky, 16 columns per step.  The diagonal tile
  // D_J is factored and inverted in registers by wave 0 alone (lane r holds
  // row r; the pivot and the column reach the other lanes by v_readlane),
  // one step ahead: while waves 1.. take the trailing tiles of step J, wave 0
  // updates tile (J+1, J+1) first and factors it.  Per step, two barriers:
  // panel tiles L_IJ = A_IJ D_J^-T, then trailing tiles A_IK -= L_IJ L_KJ^T,
  // each one 16x16x16 fp32 MFMA product.
  auto factor_diag = [&](int J) __attribute__((always_inline)) {
    float* D = Lt + tile_at(J, J) + rperm(lr) * 16;
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
        *reinterpret_cast<float4*>(&Xt[J * 256 + lr * 16 + m]) = make_float4(xr[m], xr[m + 1], xr[m + 2], xr[m + 3]);
      }
    }
    if (lane == 0 && bad_j) flag = 16 * J + bad_j;
  };
  auto trail_tile = [&](int J, int I, int Kt) {
    const float4 av = *reinterpret_cast<const float4*>(&Lt[tile_at(I, J) + rperm(lr) * 16 + 4 * lq]);
    const float4 bv = *reinterpret_cast<const float4*>(&Lt[tile_at(Kt, J) + rperm(lr) * 16 + 4 * lq]);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = mma_f32(av.x, bv.x, acc);
    acc = mma_f32(av.y, bv.y, acc);
    acc = mma_f32(av.z, bv.z, acc);
    acc = mma_f32(av.w, bv.w, acc);
    float* C = Lt + tile_at(I, Kt);
#pragma unroll
    for (int j = 0; j < 4; ++j) C[rperm(4 * lq + j) * 16 + lr] -= acc[j];
  };
  if (wid == 0) factor_diag(0);
  __syncthreads();
  for (int J = 0; J < nt; ++J) {
    if (flag) break;
    for (int I = J + 1 + wid; I < nt; I += NW) {
      float* A = Lt + tile_at(I, J);
      const float4 av = *reinterpret_cast<const float4*>(&A[rperm(lr) * 16 + 4 * lq]);
      const float4 bv = *reinterpret_cast<const float4*>(&Xt[J * 256 + lr * 16 + 4 * lq]);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = mma_f32(av.x, bv.x, acc);
      acc = mma_f32(av.y, bv.y, acc);
      acc = mma_f32(av.z, bv.z, acc);
      acc = mma_f32(av.w, bv.w, acc);
#pragma unroll
      for (int j = 0; j < 4; ++j) A[rperm(4 * lq + j) * 16 + lr] = acc[j];
    }
    __syncthreads();
    const int rest = nt - 1 - J, nrest = rest * (rest + 1) / 2;
    if (wid == 0) {
      if (rest > 0) {   // tile (J+1, J+1) is trailing tile 0
        trail_tile(J, J + 1, J + 1);
        factor_diag(J + 1);
      }
    } else {
      // the other trailing tiles over waves 1.., two per wave at a time
      // (distinct tiles, so the loads of both are issued before either
      // result is written)
      for (int q0 = wid; q0 < nrest; q0 += 2 * (NW - 1)) {
        float4 av[2], bv[2];
        int C[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int qq = min(q0 + h * (NW - 1), nrest - 1);   // nrest <= kTriQ
          const int I = tri_tab[0][qq] + J + 1, Kt = tri_tab[1][qq] + J + 1;
          av[h] = *reinterpret_cast<const float4*>(&Lt[tile_at(I, J) + rperm(lr) * 16 + 4 * lq]);
          bv[h] = *reinterpret_cast<const float4*>(&Lt[tile_at(Kt, J) + rperm(lr) * 16 + 4 * lq]);
          C[h] = tile_at(I, Kt);
        }
        f32x4 acc[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          acc[h] = f32x4{0.f, 0.f, 0.f, 0.f};
          acc[h] = mma_f32(av[h].x, bv[h].x, acc[h]);
          acc[h] = mma_f32(av[h].y, bv[h].y, acc[h]);
          acc[h] = mma_f32(av[h].z, bv[h].z, acc[h]);
          acc[h] = mma_f32(av[h].w, bv[h].w, acc[h]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (q0 + h * (NW - 1) >= nrest) break;
#pragma unroll
          for (int j = 0; j < 4; ++j) Lt[C[h] + rperm(4 * lq + j) * 16 + lr] -= acc[h][j];
        }
      }
    }
    __syncthreads();
  }
  if (flag) {
    for (int i = tid; i < n; i += kSpanThreads) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      lam_eff_out[p] = lam;
      resid2[p] = t2[p];
      info[p] = flag;
    }
    return;
  }

  // solve (L L^T) z = rhs in place (rhs in y on entry, z in y on exit) on
  // wave 0 alone, in fp32 (the factor's precision; the refinement recovers
  // the rest), by 16-row blocks: lane l keeps rows l, l + 64, ... of the
  // right-hand side in registers.  Block J takes its 16 entries from their
  // lanes by v_readlane, applies the stored inverse of the diagonal tile
  // (X_J forward, X_J^T backward) on the 16 lanes that own the block, and
  // broadcasts the result the same way; every lane then subtracts its rows'
  // share of block column J of L (forward: rows below the block) or block
  // row J (backward: rows above it).  Rows past n hold values that are never
  // broadcast or stored (the identity padding keeps those of the last block
  // at exactly 0).
  auto chol_solve = [&]() {
    if (wid == 0) {
      constexpr int R = kSpanMaxN / 64;
      const int kb = lane >> 4, kc = lane & 15;   // lane's 16-row group and row within it
      float v[R];
#pragma unroll
      for (int m = 0; m < R; ++m) v[m] = lane + 64 * m < n ? (float)y[lane + 64 * m] : 0.f;
#pragma unroll
      for (int mb = 0; mb < R; ++mb) {
#pragma unroll 1
        for (int jj = 0; jj < 4; ++jj) {
          const int J = 4 * mb + jj;
          if (J >= nt) break;
          // The LDS reads of the block depend on J only: X_J's row and the
          // first register's row of block column J go out before the
          // broadcasts, and each later register's row while the previous
          // one is applied.  Registers mb + 1.. always hold rows below the
          // block; register mb does unless jj = 3.
          const int m0 = jj < 3 ? mb : mb + 1;
          auto lrow_at = [&](int m) { return Lt + row_at(lane + 64 * m) + J * 256; };   // row k of tile (k / 16, J)
          auto ld16 = [](const float* p, float (&o)[16]) {
#pragma unroll
            for (int c = 0; c < 16; c += 4) {
              const float4 t4 = *reinterpret_cast<const float4*>(p + c);
              o[c] = t4.x;
              o[c + 1] = t4.y;
              o[c + 2] = t4.z;
              o[c + 3] = t4.w;
            }
          };
          float xrow[16], lcur[16], lnext[16];   // row kc of X_J; rows of block column J
          ld16(&Xt[J * 256 + kc * 16], xrow);
          if (m0 < R) ld16(lrow_at(m0), lcur);
          float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < 16; ++c) acc[c & 3] = fmaf(xrow[c], readlane_f(v[mb], 16 * jj + c), acc[c & 3]);
          v[mb] = kb == jj ? (acc[0] + acc[1]) + (acc[2] + acc[3]) : v[mb];
          float yb[16];
#pragma unroll
          for (int c = 0; c < 16; ++c) yb[c] = readlane_f(v[mb], 16 * jj + c);
#pragma unroll
          for (int m = mb; m < R; ++m) {
            if (m < m0) continue;
            if (m + 1 < R) ld16(lrow_at(m + 1), lnext);
            const int k = lane + 64 * m;
            float d[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < 16; ++c) d[c & 3] = fmaf(lcur[c], yb[c], d[c & 3]);
            v[m] = (k >> 4) > J ? v[m] - ((d[0] + d[1]) + (d[2] + d[3])) : v[m];
            if (m + 1 < R) {
#pragma unroll
              for (int c = 0; c < 16; ++c) lcur[c] = lnext[c];
            }
          }
        }
      }
#pragma unroll
      for (int mb = R - 1; mb >= 0; --mb) {
#pragma unroll 1
        for (int jj = 3; jj >= 0; --jj) {
          const int J = 4 * mb + jj;
          if (J >= nt) continue;
          // As in the forward sweep: X_J's column and the first register's
          // column of block row J before the broadcasts, each later one
          // while the previous is applied.  Registers 0..mb - 1 always hold
          // rows above the block; register mb does unless jj = 0.
          const int m1 = jj > 0 ? mb : mb - 1;   // last register with rows above the block
          auto lcol_at = [&](int m, float (&o)[16]) {
            const int k = lane + 64 * m;
            const float* Lc = Lt + tile_at(J, min(k >> 4, J)) + (k & 15);   // column k of block row J
#pragma unroll
            for (int c = 0; c < 16; ++c) o[c] = Lc[rperm(c) * 16];
          };
          float xcol[16], lcur[16], lnext[16];   // column kc of X_J; columns of block row J
#pragma unroll
          for (int c = 0; c < 16; ++c) xcol[c] = Xt[J * 256 + c * 16 + kc];
          if (m1 >= 0) lcol_at(0, lcur);
          float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < 16; ++c) acc[c & 3] = fmaf(xcol[c], readlane_f(v[mb], 16 * jj + c), acc[c & 3]);
          v[mb] = kb == jj ? (acc[0] + acc[1]) + (acc[2] + acc[3]) : v[mb];
          float zb[16];
#pragma unroll
          for (int c = 0; c < 16; ++c) zb[c] = readlane_f(v[mb], 16 * jj + c);
#pragma unroll
          for (int m = 0; m <= mb; ++m) {
            if (m > m1) continue;
            if (m + 1 <= m1) lcol_at(m + 1, lnext);
            const int k = lane + 64 * m;
            float d[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < 16; ++c) d[c & 3] = fmaf(lcur[c], zb[c], d[c & 3]);
            v[m] = (k >> 4) < J ? v[m] - ((d[0] + d[1]) + (d[2] + d[3])) : v[m];
            if (m + 1 <= m1) {
#pragma unroll
              for (int c = 0; c < 16; ++c) lcur[c] = lnext[c];
            }
          }
        }
      }
#pragma unroll
      for (int m = 0; m < R; ++m)
        if (lane + 64 * m < n) y[lane + 64 * m] = (double)v[m];
    }
    __syncthreads();
  };

  // (K x)_i in fp64 from the fp32 K for every row: one wave per row, the
  // lanes across the row (coalesced), all of a wave's rows loaded before
  // the fixed-order wave reductions; f(i, (K x)_i) on lane 63
  auto kx_rows = [&](auto&& f) {
    constexpr int RB = 8, C4 = kSpanMaxN / 64;
    double xv[C4];
#pragma unroll
    for (int c = 0; c < C4; ++c) xv[c] = lane + 64 * c < n ? x[lane + 64 * c] : 0.0;
    for (int t0 = 0; wid + NW * t0 < n; t0 += RB) {
      float kv[RB][C4];
#pragma unroll
      for (int t = 0; t < RB; ++t) {
        const int i = min(wid + NW * (t0 + t), n - 1);
#pragma unroll
        for (int c = 0; c < C4; ++c) kv[t][c] = Kp[(long long)i * n + min(lane + 64 * c, n - 1)];
      }
#pragma unroll
      for (int t = 0; t < RB; ++t) {
        const int i = wid + NW * (t0 + t);
        if (i >= n) break;
        double acc = 0.0;
#pragma unroll
        for (int c = 0; c < C4; ++c) acc += (double)kv[t][c] * xv[c];
        acc = wave_sum_l63(acc);
        if (lane == 63) f(i, acc);
      }
    }
  };

  for (int i = tid; i < n; i += kSpanThreads) y[i] = sd[i] = (double)sp[i];
  __syncthreads();
  chol_solve();
  double x0m = 0.0;
  for (int i = tid; i < n; i += kSpanThreads) {
    x[i] = y[i];
    x0m = fmax(x0m, fabs(y[i]));
  }
  // (block_absmax's barriers also publish x)
  double dprev = block_absmax<kSpanThreads>(x0m, scratch);

  // at most two steps of iterative refinement: y = s - (K + lam I) x in
  // fp64 from the fp32 K, solve, x += y; the sizes of the last two
  // corrections (the first solution counts as the first) decide whether
  // the refinement converged, and it stops as soon as they do
  bool converged = false;
  for (int it = 0; it < 2 && !converged; ++it) {
    kx_rows([&](int i, double kx) { y[i] = sd[i] - (double)lam * x[i] - kx; });
    __syncthreads();
    chol_solve();
    double dm = 0.0, xm = 0.0;
    for (int i = tid; i < n; i += kSpanThreads) {
      x[i] += y[i];
      dm = fmax(dm, fabs(y[i]));
      xm = fmax(xm, fabs(x[i]));
    }
    const double dcur = block_absmax<kSpanThreads>(dm, scratch);
    converged = refine_converged(dprev, dcur, block_absmax<kSpanThreads>(xm, scratch));
    dprev = dcur;
  }

  // resid2 = t2 - 2 s.x + x.K.x
  double part = 0.0;
  kx_rows([&](int i, double kx) { part += x[i] * kx - 2.0 * sd[i] * x[i]; });
  const double q = block_sum<kSpanThreads>(part, scratch);
  for (int i = tid; i < n; i += kSpanThreads) w[(long long)p * n + i] = (float)x[i];
  if (tid == 0) {
    lam_eff_out[p] = lam;
    resid2[p] = (float)((double)t2[p] + q);
    info[p] = converged ? 0 : DR_INFO_NOT_CONVERGED;
  }
}

// MAXC: K entries held per thread (columns part, part + tpr, ...)
template <int MAXC>
__global__ __launch_bounds__(kConeThreads) void cone_pg_kernel(const float* K, const float* s, const float* t2, int n,
                                                               int max_iter, float kkt_tol, float* w, float* resid2,
                                                               int* iters, float* kkt, int* info) {
  __shared__ double wbuf[2][kConeMaxN];
  __shared__ double rsc[kConeMaxN];
  __shared__ double scratch[kConeThreads / 64 + 1];
  __shared__ int flag;
  const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;

  // lanes per row: a power of two <= 64 with rows * tpr <= kConeThreads
  int npad = 1;
  while (npad < n) npad <<= 1;
  int tpr = kConeThreads / npad;
  if (tpr > 64) tpr = 64;
  const int row = tid / tpr, part = tid % tpr;
  const bool has_row = row < n;

  if (tid == 0) flag = 0;
  __syncthreads();
  int bad = 0;
  for (int e = tid; e < n * n; e += kConeThreads)
    if (!isfinite(Kp[e])) bad = 1;
  for (int i = tid; i < n; i += kConeThreads)
    if (!isfinite(sp[i])) bad = 1;
  if (bad) flag = 1;
  for (int i = tid; i < n; i += kConeThreads) {
    const float d = Kp[(long long)i * n + i];
    rsc[i] = d > 0.f ? 1.0 / sqrt((double)d) : 0.0;
    wbuf[0][i] = 0.0;
  }
  __syncthreads();
  if (flag) {
    for (int i = tid; i < n; i += kConeThreads) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      resid2[p] = t2[p];
      iters[p] = 0;
      kkt[p] = 0.f;
      info[p] = DR_INFO_NONFINITE;
    }
    return;
  }

  // this thread's slice of row `row`: columns part, part + tpr, ...
  // MAXC > 0: the slice lives in registers; MAXC == 0: it is re-read from
  // global memory (L2-resident) every iteration (n > 128)
  constexpr int KREG = MAXC > 0 ? MAXC : 1;
  float kr[KREG];
  double lrow = 0.0;
  if constexpr (MAXC > 0) {
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int j = part + c * tpr;
      kr[c] = (has_row && j < n) ? Kp[(long long)row * n + j] : 0.f;
      if (has_row && j < n) lrow += fabs((double)kr[c]) * rsc[j];
    }
  } else {
    kr[0] = 0.f;
    if (has_row)
      for (int j = part; j < n; j += tpr) lrow += fabs((double)Kp[(long long)row * n + j]) * rsc[j];
  }
  for (int off = tpr / 2; off > 0; off >>= 1) lrow += __shfl_xor(lrow, off, 64);
  double lmax = has_row ? lrow * rsc[row] : 0.0;
  for (int off = 32; off > 0; off >>= 1) lmax = fmax(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) scratch[tid >> 6] = lmax;
  double sabs = 0.0;
  for (int i = 0; i < n; ++i) sabs = fmax(sabs, fabs(rsc[i] * (double)sp[i]));
  __syncthreads();
  double Lhat = 0.0;
  for (int q = 0; q < kConeThreads / 64; ++q) Lhat = fmax(Lhat, scratch[q]);
  __syncthreads();
  const double den = sabs > 0.0 ? sabs : 2.2250738585072014e-308;
  const double ri = has_row ? rsc[row] : 0.0;
  const double si = has_row ? (double)sp[row] : 0.0;

  int it = 0, cur = 0;
  double rho = 0.0, gi = 0.0;
  while (true) {
    const double* wc = wbuf[cur];
    double acc = 0.0;
    if constexpr (MAXC > 0) {
#pragma unroll
      for (int c = 0; c < MAXC; ++c) {
        const int j = part + c * tpr;
        if (j < n) acc += (double)kr[c] * wc[j];
      }
    } else {
      if (has_row)
        for (int j = part; j < n; j += tpr) acc += (double)Kp[(long long)row * n + j] * wc[j];
    }
    for (int off = tpr / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    gi = acc - si;                        // (K w - s)_row
    const double wi = has_row ? wc[row] : 0.0;
    // scaled KKT residual |min(w~_i, g~_i)|
    double v = 0.0;
    if (has_row && ri > 0.0) v = fabs(fmin(wi / ri, ri * gi));
    for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
    if (lane == 0) scratch[tid >> 6] = v;
    __syncthreads();
    double vmax = 0.0;
    for (int q = 0; q < kConeThreads / 64; ++q) vmax = fmax(vmax, scratch[q]);
    rho = vmax / den;
    if ((kkt_tol > 0.f && rho <= (double)kkt_tol) || it >= max_iter || Lhat == 0.0) break;
    if (has_row && part == 0) {
      const double nw = wi - ri * ri * gi / Lhat;
      wbuf[cur ^ 1][row] = nw > 0.0 ? nw : 0.0;
    }
    __syncthreads();
    cur ^= 1;
    ++it;
  }

  // resid2 = t2 - s.w + w.(K w - s)
  __syncthreads();   // every wave has read the last residual maxima
  double contrib = 0.0;
  if (has_row && part == 0) {
    const double wi = wbuf[cur][row];
    contrib = wi * gi - si * wi;
    w[(long long)p * n + row] = (float)wi;
  }
  const double q = block_sum<kConeThreads>(contrib, scratch);
  if (tid == 0) {
    resid2[p] = (float)((double)t2[p] + q);
    iters[p] = it;
    kkt[p] = (float)rho;
    info[p] = (kkt_tol > 0.f && rho > (double)kkt_tol) ? DR_INFO_NOT_CONVERGED : 0;
  }
}


// ---------------------------------------------------------------------------
// Single-wave solvers for n <= 64 (one 64-lane wave per group, lane i owns
// row i, everything in fp64 on the exact fp32 inputs; no block barriers).


typedef __attribute__((ext_vector_type(2))) double f64x2;

// sum over the 4 lanes of a quad with DPP quad permutes (xor 1, xor 2)
__device__ __forceinline__ double quad_sum(double v) {
  int lo = __double2loint(v), hi = __double2hiint(v);
  double o = __hiloint2double(__builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false),
                              __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false));
  v += o;
  lo = __double2loint(v);
  hi = __double2hiint(v);
  o = __hiloint2double(__builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false),
                       __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false));
  return v + o;
}

// Cholesky of K + lam I in fp64: lane i keeps row i of the factor in
// registers.  Every broadcast (the pivot, the column L_kj, the solution
// components) is a v_readlane from the owning lane -- no LDS and no waits in
// the factorisation.  The back substitution needs column i of L in lane i:
// the rows go through LDS once and each lane reads its column in one batch.
// NM is the padded size (16, 32 or 64); lanes >= n hold zero rows.
template <int NM>
__global__ __launch_bounds__(kWaveN) void span_wave_kernel(const float* K, const float* s, const float* t2, int n,
                                                           float lambda, int mode, float* w, float* lam_eff_out,
                                                           float* resid2, int* info) {
  __shared__ double Lr[NM][NM + 1];
  const int p = blockIdx.x, i = threadIdx.x;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const bool own = i < n;
  double a[NM];
  bool bad = own && !isfinite(sp[i]);
#pragma unroll
  for (int k = 0; k < NM; ++k) {
    const float v = (own && k < n) ? Kp[(long long)i * n + k] : 0.f;
    bad |= !isfinite(v);
    a[k] = (double)v;
  }
  double kii = 0.0;
#pragma unroll
  for (int k = 0; k < NM; ++k)
    if (k == i) kii = a[k];
  const double tr = wave_sum(own ? kii : 0.0);
  const bool nonfinite = __any(bad);
  const float lam = mode == DR_RIDGE_REL_TRACE ? (float)((double)lambda * tr / (double)n) : lambda;
  if (nonfinite || (mode == DR_RIDGE_REL_TRACE && tr == 0.0)) {
    if (own) w[(long long)p * n + i] = 0.f;
    if (i == 0) {
      lam_eff_out[p] = nonfinite ? 0.f : lam;
      resid2[p] = t2[p];
      info[p] = nonfinite ? DR_INFO_NONFINITE : 0;
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < NM; ++k)
    if (k == i && own) a[k] += (double)lam;

  int bad_pivot = 0;
  double dinv = 0.0;   // 1 / L_ii of this lane's row
#pragma unroll
  for (int j = 0; j < NM; ++j) {
    if (j < n && bad_pivot == 0) {
      const double d = readlane_d(a[j], j);        // the pivot, from lane j
      if (!(d > 0.0)) {
        bad_pivot = j + 1;
      } else {
        const double ljj = sqrt(d);
        const double inv = 1.0 / ljj;
        if (i == j) dinv = inv;
        const double lij = i > j ? a[j] * inv : (i == j ? ljj : 0.0);
        a[j] = i >= j ? lij : a[j];
        // a[k] -= L_ij L_kj for k > j, L_kj from lane k (entries above the
        // diagonal are never read)
#pragma unroll
        for (int k = j + 1; k < NM; ++k)
          if (k < n) a[k] -= lij * readlane_d(a[j], k);
      }
    }
  }
  if (bad_pivot) {
    if (own) w[(long long)p * n + i] = 0.f;
    if (i == 0) {
      lam_eff_out[p] = lam;
      resid2[p] = t2[p];
      info[p] = bad_pivot;
    }
    return;
  }
  // L y = s (lane i holds y_i and row i of L)
  double y = own ? (double)sp[i] : 0.0;
#pragma unroll
  for (int j = 0; j < NM; ++j) {
    if (j < n) {
      if (i == j) y *= dinv;
      const double yj = readlane_d(y, j);
      if (i > j && own) y -= a[j] * yj;
    }
  }
  // column i of L into lane i, through LDS
#pragma unroll
  for (int k = 0; k < NM; ++k) Lr[i][k] = a[k];
  __syncthreads();
  double lc[NM];
#pragma unroll
  for (int j = 0; j < NM; ++j) lc[j] = Lr[j][i];
  // L^T x = y
#pragma unroll
  for (int j = NM - 1; j >= 0; --j) {
    if (j < n) {
      if (i == j) y *= dinv;
      const double xj = readlane_d(y, j);
      if (i < j) y -= lc[j] * xj;
    }
  }
  const double x = own ? y : 0.0;
  // resid2 = t2 - 2 s.x + x.K.x with the fp32 K (no ridge)
  double kx = 0.0;
#pragma unroll
  for (int k = 0; k < NM; ++k) {
    const float kik = (own && k < n) ? Kp[(long long)i * n + k] : 0.f;
    kx += (double)kik * readlane_d(x, k);
  }
  const double q = wave_sum(own ? x * kx - 2.0 * (double)sp[i] * x : 0.0);
  if (own) w[(long long)p * n + i] = (float)x;
  if (i == 0) {
    lam_eff_out[p] = lam;
    resid2[p] = (float)((double)t2[p] + q);
    info[p] = 0;
  }
}

// Jacobi-preconditioned projected gradient, one wave: lane i keeps row i of
// the fp32 K in registers and w_i in fp64; each step publishes w through
// LDS (double buffered) and reads it back as broadcast pairs.
template <int NM>
__global__ __launch_bounds__(kWaveN) void cone_wave_kernel(const float* K, const float* s, const float* t2, int n,
                                                           int max_iter, float kkt_tol, float* w, float* resid2,
                                                           int* iters, float* kkt, int* info) {
  __shared__ __attribute__((aligned(16))) double wb[2][kWaveN];
  __shared__ __attribute__((aligned(16))) double rs[kWaveN];
  const int p = blockIdx.x, i = threadIdx.x;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const bool own = i < n;
  float kr[NM];
  bool bad = own && !isfinite(sp[i]);
  double kii = 0.0;
#pragma unroll
  for (int j = 0; j < NM; ++j) {
    kr[j] = (own && j < n) ? Kp[(long long)i * n + j] : 0.f;
    bad |= !isfinite(kr[j]);
    if (j == i) kii = (double)kr[j];
  }
  const double si = own ? (double)sp[i] : 0.0;
  const double ri = kii > 0.0 ? 1.0 / sqrt(kii) : 0.0;
  rs[i] = ri;
  wb[0][i] = 0.0;
  __syncthreads();
  if (__any(bad)) {
    if (own) w[(long long)p * n + i] = 0.f;
    if (i == 0) {
      resid2[p] = t2[p];
      iters[p] = 0;
      kkt[p] = 0.f;
      info[p] = DR_INFO_NONFINITE;
    }
    return;
  }
  double lrow = 0.0;
#pragma unroll
  for (int j = 0; j < NM; ++j) lrow += fabs((double)kr[j]) * rs[j];
  const double Lhat = wave_max(own ? lrow * ri : 0.0);
  const double den0 = wave_max(own ? fabs(ri * si) : 0.0);
  const double den = den0 > 0.0 ? den0 : 2.2250738585072014e-308;
  const double step = ri * ri / (Lhat > 0.0 ? Lhat : 1.0);
  const bool check_each = kkt_tol > 0.f;

  int it = 0, cur = 0;
  double rho = 0.0, g = 0.0, wi = 0.0;
  while (true) {
    double wv[NM];
#pragma unroll
    for (int j = 0; j < NM; j += 2) {
      const f64x2 v = *reinterpret_cast<const f64x2*>(&wb[cur][j]);
      wv[j] = v.x;
      wv[j + 1] = v.y;
    }
    double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
    for (int j = 0; j < NM; j += 2) {
      acc0 += (double)kr[j] * wv[j];
      acc1 += (double)kr[j + 1] * wv[j + 1];
    }
    g = (acc0 + acc1) - si;
    const bool last = it >= max_iter || Lhat == 0.0;
    if (check_each || last) {
      const double v = (own && ri > 0.0) ? fabs(fmin(wi / ri, ri * g)) : 0.0;
      rho = wave_max(v) / den;
      if ((check_each && rho <= (double)kkt_tol) || last) break;
    }
    const double nw = wi - step * g;
    wi = nw > 0.0 ? nw : 0.0;
    wb[cur ^ 1][i] = own ? wi : 0.0;
    __syncthreads();
    cur ^= 1;
    ++it;
  }
  const double q = wave_sum(own ? wi * g - si * wi : 0.0);
  if (own) w[(long long)p * n + i] = (float)wi;
  if (i == 0) {
    resid2[p] = (float)((double)t2[p] + q);
    iters[p] = it;
    kkt[p] = (float)rho;
    info[p] = (kkt_tol > 0.f && rho > (double)kkt_tol) ? DR_INFO_NOT_CONVERGED : 0;
  }
}


// Jacobi-preconditioned projected gradient for n <= 64 on four waves: wave v
// owns rows 16v..16v+15, four lanes per row each hold a quarter of the row
// of K in fp64 registers; partial dot products meet through quad shuffles,
// and w is exchanged through LDS (double buffered) with one barrier per step.
template <int NM>
__global__ __launch_bounds__(256) void cone_quad_kernel(const float* K, const float* s, const float* t2, int n,
                                                        int max_iter, float kkt_tol, float* w, float* resid2,
                                                        int* iters, float* kkt, int* info) {
  constexpr int Q = NM / 4;   // columns per lane
  __shared__ __attribute__((aligned(16))) double wb[2][NM];
  __shared__ double rs[NM];
  __shared__ double red[4];
  __shared__ int flag;
  const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = wave * 16 + (lane >> 2), q = lane & 3;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const bool own = row < n;
  if (tid == 0) flag = 0;
  if (tid < NM) {
    const float d = tid < n ? Kp[(long long)tid * n + tid] : 0.f;
    rs[tid] = d > 0.f ? 1.0 / sqrt((double)d) : 0.0;
    wb[0][tid] = 0.0;
  }
  __syncthreads();
  double kr[Q];
  bool bad = own && q == 0 && !isfinite(sp[row]);
  double lrow = 0.0;
#pragma unroll
  for (int c = 0; c < Q; ++c) {
    const int j = q * Q + c;
    const float v = (own && j < n) ? Kp[(long long)row * n + j] : 0.f;
    bad |= !isfinite(v);
    kr[c] = (double)v;
    lrow += fabs(kr[c]) * rs[j];
  }
  if (bad) flag = 1;
  lrow = quad_sum(lrow);
  const double ri = own ? rs[row] : 0.0;
  const double si = own ? (double)sp[row] : 0.0;
  double lmax = own ? lrow * ri : 0.0, smax = own ? fabs(ri * si) : 0.0;
  for (int off = 32; off > 0; off >>= 1) {
    lmax = fmax(lmax, __shfl_xor(lmax, off, 64));
    smax = fmax(smax, __shfl_xor(smax, off, 64));
  }
  __shared__ double wl[4], wsx[4];
  if (lane == 0) {
    wl[wave] = lmax;
    wsx[wave] = smax;
  }
  __syncthreads();
  if (flag) {
    if (own && q == 0) w[(long long)p * n + row] = 0.f;
    if (tid == 0) {
      resid2[p] = t2[p];
      iters[p] = 0;
      kkt[p] = 0.f;
      info[p] = DR_INFO_NONFINITE;
    }
    return;
  }
  const double Lhat = fmax(fmax(wl[0], wl[1]), fmax(wl[2], wl[3]));
  const double den0 = fmax(fmax(wsx[0], wsx[1]), fmax(wsx[2], wsx[3]));
  const double den = den0 > 0.0 ? den0 : 2.2250738585072014e-308;
  const double step = ri * ri / (Lhat > 0.0 ? Lhat : 1.0);
  const bool check_each = kkt_tol > 0.f;

  int it = 0, cur = 0;
  double rho = 0.0, g = 0.0, wi = 0.0;
  while (true) {
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < Q; c += 2) {
      const f64x2 v = *reinterpret_cast<const f64x2*>(&wb[cur][q * Q + c]);
      acc += kr[c] * v.x;
      acc += kr[c + 1] * v.y;
    }
    acc = quad_sum(acc);
    g = acc - si;
    const bool last = it >= max_iter || Lhat == 0.0;
    if (check_each || last) {
      double v = (own && q == 0 && ri > 0.0) ? fabs(fmin(wi / ri, ri * g)) : 0.0;
      for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
      if (lane == 0) red[wave] = v;
      __syncthreads();
      rho = fmax(fmax(red[0], red[1]), fmax(red[2], red[3])) / den;
      __syncthreads();
      if ((check_each && rho <= (double)kkt_tol) || last) break;
    }
    const double nw = wi - step * g;
    wi = nw > 0.0 ? nw : 0.0;
    if (q == 0 && row < NM) wb[cur ^ 1][row] = own ? wi : 0.0;
    __syncthreads();
    cur ^= 1;
    ++it;
  }
  double contrib = (own && q == 0) ? wi * g - si * wi : 0.0;
  for (int off = 32; off > 0; off >>= 1) contrib += __shfl_xor(contrib, off, 64);
  if (lane == 0) red[wave] = contrib;
  __syncthreads();
  if (own && q == 0) w[(long long)p * n + row] = (float)wi;
  if (tid == 0) {
    resid2[p] = (float)((double)t2[p] + ((red[0] + red[1]) + (red[2] + red[3])));
    iters[p] = it;
    kkt[p] = (float)rho;
    info[p] = (kkt_tol > 0.f && rho > (double)kkt_tol) ? DR_INFO_NOT_CONVERGED : 0;
  }
}


// 1 / sqrt(d) for d > 0 (normal range): the hardware estimate and two
// Newton steps r <- r + r/2 (1 - d r^2), a few ulp in fp64, about a third of
// the dependent steps of a correctly rounded sqrt followed by a divide.
__device__ __forceinline__ double rsqrt_newton(double d) {
  double r = __builtin_amdgcn_rsq(d);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const double e = fma(-d * r, r, 1.0);
    r = fma(0.5 * r, e, r);
  }
  return r;
}

// Cholesky of K + lam I in fp64 for 16 < n <= 64 on NM/16 waves.  Lane i of
// wave c holds A[i][16c .. 16c + 16) in registers.  The matrix is padded to
// NM with identity rows and columns (the padded part of the factor is the
// identity and the padded solution is zero), so the pivot loop has a fixed
// trip count: column j = 16 jb + jc with jc unrolled, the register holding
// column j (or j + 1) is known at compile time, and which waves still have
// columns to update is a scalar branch.  Before pivot j the owner of column j
// has published A[.][j] to an LDS column buffer (double buffered), so each
// pivot costs one barrier.  The factor then goes to LDS and wave 0 does the
// two triangular solves (the L^T solve reads column i of L into lane i once).
template <int NM>
__global__ __launch_bounds__(NM * 4) void span_cols_kernel(const float* K, const float* s, const float* t2, int n,
                                                           float lambda, int mode, float* w, float* lam_eff_out,
                                                           float* resid2, int* info) {
  constexpr int CW = 16, NW = NM / CW;
  __shared__ __attribute__((aligned(16))) double colb[2][NM];
  __shared__ double Lr[NM][NM + 1];
  __shared__ __attribute__((aligned(16))) double xs[NM];
  __shared__ double kxp[NW][NM];
  __shared__ double red[NW];
  __shared__ int flag;
  const int p = blockIdx.x, tid = threadIdx.x, i = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, known uniform
  const int c0 = wv * CW;                                     // first column held by this wave
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const bool own = i < n;    // a row of K
  const bool inm = i < NM;   // a row of the padded matrix
  if (tid == 0) flag = 0;
  __syncthreads();
  double a[CW];
  float kq[CW];   // this lane's slice of the fp32 K row, kept for the residual
  bool bad = own && wv == 0 && !isfinite(sp[i]);
  double kii = 0.0;
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    const int k = c0 + c;
    const float v = (own && k < n) ? Kp[(long long)i * n + k] : 0.f;
    bad |= !isfinite(v);
    kq[c] = v;
    a[c] = (double)v;
    if (k == i) kii = a[c];
  }
  if (bad) flag = 1;
  const double trw = wave_sum(kii);
  if (i == 0) red[wv] = trw;
  __syncthreads();
  double tr = 0.0;
#pragma unroll
  for (int v = 0; v < NW; ++v) tr += red[v];
  const bool nonfinite = flag != 0;
  const float lam = mode == DR_RIDGE_REL_TRACE ? (float)((double)lambda * tr / (double)n) : lambda;
  if (nonfinite || (mode == DR_RIDGE_REL_TRACE && tr == 0.0)) {
    if (own && wv == 0) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      lam_eff_out[p] = nonfinite ? 0.f : lam;
      resid2[p] = t2[p];
      info[p] = nonfinite ? DR_INFO_NONFINITE : 0;
    }
    return;
  }
#pragma unroll
  for (int c = 0; c < CW; ++c)
    if (c0 + c == i) a[c] = own ? a[c] + (double)lam : (inm ? 1.0 : 0.0);
  if (wv == 0 && inm) colb[0][i] = a[0];
  __syncthreads();

  int bad_pivot = 0;   // first j with a non-positive pivot (then the rest is discarded)
  for (int jb = 0; jb < NW; ++jb) {
#pragma unroll
    for (int jc = 0; jc < CW; ++jc) {
      const int j = jb * CW + jc;
      const double* cb = colb[jc & 1];
      double d = cb[j];
      if (!(d > 0.0)) {
        if (bad_pivot == 0) bad_pivot = j + 1;
        d = 1.0;
      }
      const double r = rsqrt_newton(d);
      const double lij = (inm && i > j) ? cb[i] * r : 0.0;
      const double f = lij * r;   // L_ij / L_jj
      if (wv == jb) {
        // column j becomes L_:j (entries above the diagonal are never read)
        a[jc] = i > j ? lij : (i == j ? d * r : 0.0);
#pragma unroll
        for (int c = jc + 1; c < CW; ++c) a[c] = fma(-f, cb[c0 + c], a[c]);
        if (jc + 1 < CW && inm) colb[(jc + 1) & 1][i] = a[jc + 1];
      } else if (wv > jb) {
        // A_ik -= L_ij L_kj = f A_kj for all of this wave's columns
#pragma unroll
        for (int c = 0; c < CW; c += 2) {
          const f64x2 lk = *reinterpret_cast<const f64x2*>(&cb[c0 + c]);
          a[c] = fma(-f, lk.x, a[c]);
          a[c + 1] = fma(-f, lk.y, a[c + 1]);
        }
        if (jc + 1 == CW && wv == jb + 1 && inm) colb[0][i] = a[0];
      }
      __syncthreads();
    }
  }
  if (bad_pivot) {
    if (own && wv == 0) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      lam_eff_out[p] = lam;
      resid2[p] = t2[p];
      info[p] = bad_pivot;
    }
    return;
  }
  // the factor to LDS (lower triangle; the rest is never read)
  if (inm) {
#pragma unroll
    for (int c = 0; c < CW; ++c) Lr[i][c0 + c] = a[c];
  }
  __syncthreads();
  if (wv == 0) {
    double lrow[NM], lcol[NM];
#pragma unroll
    for (int k = 0; k < NM; ++k) {
      lrow[k] = inm ? Lr[i][k] : 0.0;
      lcol[k] = inm ? Lr[k][i] : 0.0;
    }
    const double di = inm ? 1.0 / Lr[i][i] : 0.0;
    double y = own ? (double)sp[i] : 0.0;
#pragma unroll
    for (int j = 0; j < NM; ++j) {
      if (i == j) y *= di;
      const double yj = readlane_d(y, j);
      if (i > j) y = fma(-lrow[j], yj, y);
    }
#pragma unroll
    for (int j = NM - 1; j >= 0; --j) {
      if (i == j) y *= di;
      const double xj = readlane_d(y, j);
      if (i < j) y = fma(-lcol[j], xj, y);
    }
    if (inm) xs[i] = own ? y : 0.0;
  }
  __syncthreads();
  // resid2 = t2 - 2 s.x + x.K.x with the fp32 K (no ridge), K from registers
  double kx = 0.0;
#pragma unroll
  for (int c = 0; c < CW; c += 2) {
    const f64x2 xv = *reinterpret_cast<const f64x2*>(&xs[c0 + c]);
    kx += (double)kq[c] * xv.x + (double)kq[c + 1] * xv.y;
  }
  if (inm) kxp[wv][i] = kx;
  __syncthreads();
  if (wv == 0) {
    double kxi = 0.0;
#pragma unroll
    for (int v = 0; v < NW; ++v) kxi += inm ? kxp[v][i] : 0.0;
    const double x = own ? xs[i] : 0.0;
    const double q = wave_sum(own ? x * kxi - 2.0 * (double)sp[i] * x : 0.0);
    if (own) w[(long long)p * n + i] = (float)x;
    if (i == 0) {
      lam_eff_out[p] = lam;
      resid2[p] = (float)((double)t2[p] + q);
      info[p] = 0;
    }
  }
}


// ---------------------------------------------------------------------------
// Soft weighting over the simplex.

template <int MAXC>
__global__ __launch_bounds__(kConeThreads) void simplex_pg_kernel(const float* K, const float* s, const float* t2, int n,
                                                                  int max_iter, float tol, float* w, float* resid2,
                                                                  int* iters, float* res_out, int* info) {
  __shared__ double ybuf[kConeMaxN];       // the point the gradient is taken at
  __shared__ double wprev[kConeMaxN];
  __shared__ double vbuf[kConeMaxN];       // y - grad / L, projected next
  __shared__ double scratch[kConeThreads / 64 + 1];
  __shared__ double red_d[kConeThreads / 64];
  __shared__ int red_i[kConeThreads / 64];
  __shared__ int flag;
  const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  int npad = 1;
  while (npad < n) npad <<= 1;
  int tpr = kConeThreads / npad;
  if (tpr > 64) tpr = 64;
  const int row = tid / tpr, part = tid % tpr;
  const bool has_row = row < n;

  if (tid == 0) flag = 0;
  __syncthreads();
  int bad = 0;
  for (int e = tid; e < n * n; e += kConeThreads)
    if (!isfinite(Kp[e])) bad = 1;
  for (int i = tid; i < n; i += kConeThreads)
    if (!isfinite(sp[i])) bad = 1;
  if (bad) flag = 1;
  __syncthreads();
  if (flag) {
    for (int i = tid; i < n; i += kConeThreads) w[(long long)p * n + i] = 0.f;
    if (tid == 0) {
      resid2[p] = t2[p];
      iters[p] = 0;
      res_out[p] = 0.f;
      info[p] = DR_INFO_NONFINITE;
    }
    return;
  }

  // block-wide (sum, count) of v_i over v_i > theta: one Michelot pass
  auto pass = [&](double theta, double& sum, int& cnt) {
    double ls = 0.0;
    int lc = 0;
    for (int i = tid; i < n; i += kConeThreads)
      if (vbuf[i] > theta) {
        ls += vbuf[i];
        ++lc;
      }
    for (int off = 32; off > 0; off >>= 1) {
      ls += __shfl_xor(ls, off, 64);
      lc += __shfl_xor(lc, off, 64);
    }
    if (lane == 0) {
      red_d[wave] = ls;
      red_i[wave] = lc;
    }
    __syncthreads();
    sum = 0.0;
    cnt = 0;
    for (int q = 0; q < kConeThreads / 64; ++q) {
      sum += red_d[q];
      cnt += red_i[q];
    }
    __syncthreads();
  };

  constexpr int KREG = MAXC > 0 ? MAXC : 1;
  float kr[KREG];
  double lrow = 0.0;
  if constexpr (MAXC > 0) {
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int j = part + c * tpr;
      kr[c] = (has_row && j < n) ? Kp[(long long)row * n + j] : 0.f;
      lrow += fabs((double)kr[c]);
    }
  } else {
    kr[0] = 0.f;
    if (has_row)
      for (int j = part; j < n; j += tpr) lrow += fabs((double)Kp[(long long)row * n + j]);
  }
  for (int off = tpr / 2; off > 0; off >>= 1) lrow += __shfl_xor(lrow, off, 64);
  double lmax = has_row ? lrow : 0.0;
  for (int off = 32; off > 0; off >>= 1) lmax = fmax(lmax, __shfl_xor(lmax, off, 64));
  if (lane == 0) scratch[wave] = lmax;
  // start: the best single vertex, argmin_i K_ii - 2 s_i (lowest index on ties)
  double fbest = 0.0;
  int ibest = -1;
  for (int i = tid; i < n; i += kConeThreads) {
    const double f = (double)Kp[(long long)i * n + i] - 2.0 * (double)sp[i];
    if (ibest < 0 || f < fbest) {
      fbest = f;
      ibest = i;
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    const double fo = __shfl_xor(fbest, off, 64);
    const int io = __shfl_xor(ibest, off, 64);
    if (io >= 0 && (ibest < 0 || fo < fbest || (fo == fbest && io < ibest))) {
      fbest = fo;
      ibest = io;
    }
  }
  if (lane == 0) {
    red_d[wave] = fbest;
    red_i[wave] = ibest;
  }
  __syncthreads();
  double L = 0.0;
  for (int q = 0; q < kConeThreads / 64; ++q) L = fmax(L, scratch[q]);
  L *= 2.0;
  int i0 = -1;
  double f0 = 0.0;
  for (int q = 0; q < kConeThreads / 64; ++q) {
    const int io = red_i[q];
    if (io >= 0 && (i0 < 0 || red_d[q] < f0 || (red_d[q] == f0 && io < i0))) {
      f0 = red_d[q];
      i0 = io;
    }
  }
  __syncthreads();
  for (int i = tid; i < n; i += kConeThreads) {
    ybuf[i] = i == i0 ? 1.0 : 0.0;
    wprev[i] = ybuf[i];
  }
  __syncthreads();
  const double si = has_row ? (double)sp[row] : 0.0;

  int it = 0;
  double res = 0.0, tk = 1.0;
  while (L > 0.0 && it < max_iter) {
    // v = y - 2 (K y - s) / L
    double acc = 0.0;
    if constexpr (MAXC > 0) {
#pragma unroll
      for (int c = 0; c < MAXC; ++c) {
        const int j = part + c * tpr;
        if (j < n) acc += (double)kr[c] * ybuf[j];
      }
    } else {
      if (has_row)
        for (int j = part; j < n; j += tpr) acc += (double)Kp[(long long)row * n + j] * ybuf[j];
    }
    for (int off = tpr / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (has_row && part == 0) vbuf[row] = ybuf[row] - 2.0 * (acc - si) / L;
    __syncthreads();
    // theta with sum_i max(v_i - theta, 0) = 1
    double sum;
    int cnt, prev = n + 1;
    double theta = -1.0e308;
    while (true) {
      pass(theta, sum, cnt);
      if (cnt == prev || cnt == 0) break;
      prev = cnt;
      theta = (sum - 1.0) / (double)cnt;
    }
    // w = max(v - theta, 0); residual = max |w - y|; momentum step
    const double tn = 0.5 * (1.0 + sqrt(1.0 + 4.0 * tk * tk));
    const double beta = (tk - 1.0) / tn;
    double r = 0.0;
    for (int i = tid; i < n; i += kConeThreads) {
      const double wi = fmax(vbuf[i] - theta, 0.0);
      r = fmax(r, fabs(wi - ybuf[i]));
      const double yn = wi + beta * (wi - wprev[i]);
      wprev[i] = wi;
      ybuf[i] = yn;
    }
    for (int off = 32; off > 0; off >>= 1) r = fmax(r, __shfl_xor(r, off, 64));
    if (lane == 0) scratch[wave] = r;
    __syncthreads();
    res = 0.0;
    for (int q = 0; q < kConeThreads / 64; ++q) res = fmax(res, scratch[q]);
    __syncthreads();
    tk = tn;
    ++it;
    if (tol > 0.f && res <= (double)tol) break;
  }

  // w = the last projected point; resid2 = t2 + w.K.w - 2 s.w
  double acc = 0.0;
  if constexpr (MAXC > 0) {
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int j = part + c * tpr;
      if (j < n) acc += (double)kr[c] * wprev[j];
    }
  } else {
    if (has_row)
      for (int j = part; j < n; j += tpr) acc += (double)Kp[(long long)row * n + j] * wprev[j];
  }
  for (int off = tpr / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  double contrib = 0.0;
  if (has_row && part == 0) {
    const double wi = wprev[row];
    contrib = wi * acc - 2.0 * si * wi;
    w[(long long)p * n + row] = (float)wi;
  }
  const double q = block_sum<kConeThreads>(contrib, scratch);
  if (tid == 0) {
    resid2[p] = (float)((double)t2[p] + q);
    iters[p] = it;
    res_out[p] = (float)res;
    info[p] = (tol > 0.f && res > (double)tol) ? DR_INFO_NOT_CONVERGED : 0;
  }
}

// simplex_pg_kernel for n <= 64 on one wave: lane i keeps row i of K in
// registers and its own y_i, v_i, w_i; y is published through LDS for the
// product and every block reduction of the block version (Michelot's
// passes, the residual, the start vertex) is a wave reduction, so a step
// has no block barrier.  Same iteration as simplex_pg_kernel.
__global__ __launch_bounds__(kWaveN) void simplex_wave_kernel(const float* K, const float* s, const float* t2, int n,
                                                              int max_iter, float tol, float* w, float* resid2,
                                                              int* iters, float* res_out, int* info) {
  __shared__ __attribute__((aligned(16))) double yb[kWaveN];
  const int p = blockIdx.x, i = threadIdx.x;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const bool own = i < n;
  float kr[kWaveN];
  bool bad = own && !isfinite(sp[i]);
  double lrow = 0.0;
#pragma unroll
  for (int j = 0; j < kWaveN; ++j) {
    kr[j] = (own && j < n) ? Kp[(long long)i * n + j] : 0.f;
    bad |= !isfinite(kr[j]);
    lrow += fabs((double)kr[j]);
  }
  if (__any(bad)) {
    if (own) w[(long long)p * n + i] = 0.f;
    if (i == 0) {
      resid2[p] = t2[p];
      iters[p] = 0;
      res_out[p] = 0.f;
      info[p] = DR_INFO_NONFINITE;
    }
    return;
  }
  const double L = 2.0 * wave_max(own ? lrow : 0.0);
  const double si = own ? (double)sp[i] : 0.0;
  // start: the best single vertex, argmin_i K_ii - 2 s_i (lowest index on ties)
  double fbest = own ? (double)Kp[(long long)i * n + i] - 2.0 * si : 0.0;
  int ibest = own ? i : -1;
  for (int off = 32; off > 0; off >>= 1) {
    const double fo = __shfl_xor(fbest, off, 64);
    const int io = __shfl_xor(ibest, off, 64);
    if (io >= 0 && (ibest < 0 || fo < fbest || (fo == fbest && io < ibest))) {
      fbest = fo;
      ibest = io;
    }
  }
  double y = i == ibest ? 1.0 : 0.0, wp = y;
  auto product = [&](double x) {   // (K x)_i with x_j held by lane j
    yb[i] = x;
    __syncthreads();   // (one wave) the LDS writes are visible
    double a0 = 0.0, a1 = 0.0;
#pragma unroll
    for (int j = 0; j < kWaveN; j += 2) {
      const f64x2 v = *reinterpret_cast<const f64x2*>(&yb[j]);
      a0 += (double)kr[j] * v.x;
      a1 += (double)kr[j + 1] * v.y;
    }
    __syncthreads();   // every lane has read yb before the next write
    return a0 + a1;
  };

  int it = 0;
  double res = 0.0, tk = 1.0;
  while (L > 0.0 && it < max_iter) {
    // v = y - 2 (K y - s) / L
    const double acc = product(own ? y : 0.0);
    const double v = own ? y - 2.0 * (acc - si) / L : 0.0;
    // theta with sum_i max(v_i - theta, 0) = 1
    int prev = n + 1;
    double theta = -1.0e308;
    while (true) {
      const bool in = own && v > theta;
      double sum = in ? v : 0.0;
      int cnt = in ? 1 : 0;
      for (int off = 32; off > 0; off >>= 1) {
        sum += __shfl_xor(sum, off, 64);
        cnt += __shfl_xor(cnt, off, 64);
      }
      if (cnt == prev || cnt == 0) break;
      prev = cnt;
      theta = (sum - 1.0) / (double)cnt;
    }
    // w = max(v - theta, 0); residual = max |w - y|; momentum step
    const double tn = 0.5 * (1.0 + sqrt(1.0 + 4.0 * tk * tk));
    const double beta = (tk - 1.0) / tn;
    const double wi = own ? fmax(v - theta, 0.0) : 0.0;
    res = wave_max(own ? fabs(wi - y) : 0.0);
    y = wi + beta * (wi - wp);
    wp = wi;
    tk = tn;
    ++it;
    if (tol > 0.f && res <= (double)tol) break;
  }

  // w = the last projected point; resid2 = t2 + w.K.w - 2 s.w
  const double acc = product(own ? wp : 0.0);
  const double q = wave_sum(own ? wp * acc - 2.0 * si * wp : 0.0);
  if (own) w[(long long)p * n + i] = (float)wp;
  if (i == 0) {
    resid2[p] = (float)((double)t2[p] + q);
    iters[p] = it;
    res_out[p] = (float)res;
    info[p] = (tol > 0.f && res > (double)tol) ? DR_INFO_NOT_CONVERGED : 0;
  }
}

__global__ void empty_group_kernel(const float* t2, int P, float* lam_eff, float* resid2, int32_t* iters, float* kkt,
                                   int32_t* info) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  if (lam_eff) lam_eff[p] = 0.f;
  resid2[p] = t2[p];
  if (iters) iters[p] = 0;
  if (kkt) kkt[p] = 0.f;
  info[p] = 0;
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_span_workspace_size(int64_t n, int P) {
  (void)P;   // groups above kSpanMaxN are solved one after another in one workspace
  if (n <= dr::kSpanMaxN || n > dr::kSpanLargeMaxN) return 0;
  return dr::span_large_workspace(n);
}

extern "C" size_t dr_cone_workspace_size(int64_t n, int P) {
  (void)n;
  (void)P;
  return 0;
}

extern "C" dr_status dr_project_span(const float* K, const float* s, const float* t2, int64_t n, int P, float lambda,
                                     dr_ridge_mode mode, float* w, float* lam_eff, float* resid2, int32_t* info,
                                     void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  if (n < 0 || P < 0) return DR_ERR_ARG;
  if (mode != DR_RIDGE_ABS && mode != DR_RIDGE_REL_TRACE) return DR_ERR_ARG;
  if (!(lambda >= 0.f) || !(lambda <= 3.4e38f)) return DR_ERR_ARG;
  if (P == 0) return DR_OK;
  if (!t2 || !lam_eff || !resid2 || !info) return DR_ERR_ARG;
  if (n > 0 && (!K || !s || !w)) return DR_ERR_ARG;
  if (n > kSpanLargeMaxN) return DR_ERR_UNSUPPORTED;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (n > kSpanMaxN)
    return span_large(K, s, t2, n, P, lambda, (int)mode, w, lam_eff, resid2, info, workspace, ws_bytes, hs);
  if (n == 0) {
    hipLaunchKernelGGL(empty_group_kernel, dim3((P + 255) / 256), dim3(256), 0, hs, t2, P, lam_eff, resid2,
                       (int32_t*)nullptr, (float*)nullptr, info);
    return launch_status();
  }
  if (n <= 16)
    hipLaunchKernelGGL(span_wave_kernel<16>, dim3(P), dim3(kWaveN), 0, hs, K, s, t2, (int)n, lambda, (int)mode, w,
                       lam_eff, resid2, info);
  else if (n <= 32)
    hipLaunchKernelGGL(span_cols_kernel<32>, dim3(P), dim3(128), 0, hs, K, s, t2, (int)n, lambda, (int)mode, w,
                       lam_eff, resid2, info);
  else if (n <= kWaveN)
    hipLaunchKernelGGL(span_cols_kernel<64>, dim3(P), dim3(256), 0, hs, K, s, t2, (int)n, lambda, (int)mode, w,
                       lam_eff, resid2, info);
  else
    hipLaunchKernelGGL(span_small_kernel, dim3(P), dim3(kSpanThreads), 0, hs, K, s, t2, (int)n, lambda, (int)mode,
                       w, lam_eff, resid2, info);
  return launch_status();
}

extern "C" dr_status dr_project_cone(const float* K, const float* s, const float* t2, int64_t n, int P, int max_iter,
                                     float kkt_tol, float* w, float* resid2, int32_t* iters, float* kkt, int32_t* info,
                                     void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  (void)workspace;
  (void)ws_bytes;
  if (n < 0 || P < 0 || max_iter < 0 || !(kkt_tol == kkt_tol)) return DR_ERR_ARG;
  if (P == 0) return DR_OK;
  if (!t2 || !resid2 || !iters || !kkt || !info) return DR_ERR_ARG;
  if (n > 0 && (!K || !s || !w)) return DR_ERR_ARG;
  if (n > kConeMaxN) return DR_ERR_UNSUPPORTED;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (n == 0) {
    hipLaunchKernelGGL(empty_group_kernel, dim3((P + 255) / 256), dim3(256), 0, hs, t2, P, (float*)nullptr, resid2,
                       iters, kkt, info);
    return launch_status();
  }
  if (n <= kWaveN) {
    if (n <= 16)
      hipLaunchKernelGGL(cone_wave_kernel<16>, dim3(P), dim3(kWaveN), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                         resid2, iters, kkt, info);
    else if (n <= 32)
      hipLaunchKernelGGL(cone_quad_kernel<32>, dim3(P), dim3(256), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                         resid2, iters, kkt, info);
    else
      hipLaunchKernelGGL(cone_quad_kernel<64>, dim3(P), dim3(256), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                         resid2, iters, kkt, info);
    return launch_status();
  }
  int npad = 1;
  while (npad < n) npad <<= 1;
  int tpr = kConeThreads / npad;
  if (tpr > 64) tpr = 64;
  const int cols = (npad + tpr - 1) / tpr;
  if (cols <= 4)
    hipLaunchKernelGGL(cone_pg_kernel<4>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                       resid2, iters, kkt, info);
  else if (cols <= 16)
    hipLaunchKernelGGL(cone_pg_kernel<16>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                       resid2, iters, kkt, info);
  else
    hipLaunchKernelGGL(cone_pg_kernel<0>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, kkt_tol, w,
                       resid2, iters, kkt, info);
  return launch_status();
}

extern "C" dr_status dr_project_simplex(const float* K, const float* s, const float* t2, int64_t n, int P, int max_iter,
                                        float tol, float* w, float* resid2, int32_t* iters, float* res, int32_t* info,
                                        void* stream) {
  using namespace dr;
  if (n < 0 || P < 0 || max_iter < 0 || !(tol == tol)) return DR_ERR_ARG;
  if (P == 0) return DR_OK;
  if (!t2 || !resid2 || !iters || !res || !info) return DR_ERR_ARG;
  if (n > 0 && (!K || !s || !w)) return DR_ERR_ARG;
  if (n > kConeMaxN) return DR_ERR_UNSUPPORTED;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (n == 0) {   // the simplex of zero examples is empty: nothing to project onto
    hipLaunchKernelGGL(empty_group_kernel, dim3((P + 255) / 256), dim3(256), 0, hs, t2, P, (float*)nullptr, resid2,
                       iters, res, info);
    return launch_status();
  }
  if (n <= kWaveN) {
    hipLaunchKernelGGL(simplex_wave_kernel, dim3(P), dim3(kWaveN), 0, hs, K, s, t2, (int)n, max_iter, tol, w, resid2,
                       iters, res, info);
    return launch_status();
  }
  int npad = 1;
  while (npad < n) npad <<= 1;
  int tpr = kConeThreads / npad;
  if (tpr > 64) tpr = 64;
  const int cols = (npad + tpr - 1) / tpr;
  if (cols <= 4)
    hipLaunchKernelGGL(simplex_pg_kernel<4>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, tol, w,
                       resid2, iters, res, info);
  else if (cols <= 16)
    hipLaunchKernelGGL(simplex_pg_kernel<16>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, tol, w,
                       resid2, iters, res, info);
  else
    hipLaunchKernelGGL(simplex_pg_kernel<0>, dim3(P), dim3(kConeThreads), 0, hs, K, s, t2, (int)n, max_iter, tol, w,
                       resid2, iters, res, info);
  return launch_status();
}
