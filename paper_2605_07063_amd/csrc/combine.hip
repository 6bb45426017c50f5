// Update direction in sketch space (dr_combine): u[cols_p] = G[:, cols_p]^T w_p
// per group p -- the assembled update of Eq. (proj) for span / cone weights,
// or the subset mean g_S of the top-k rule when w = 1/k on the subset
// (Sec. 3.3.2).
//
// n <= 256 (the per-step batches): combine_small_kernel, one pass.  A
// workgroup takes 64 columns; its four waves take the rows i = q mod 4
// (q = wave), fp64 accumulation in row order, and the four partial sums
// are added in a fixed order through LDS.
// Larger n: combine_partial_kernel, one thread per column, a chunk of rows
// per workgroup, fp64 accumulation in row order (rows are coalesced across
// the workgroup's threads); combine_reduce_kernel sums the row-chunk
// partials in chunk order.  Deterministic.

#include "common.h"

namespace dr {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxGroups = 128;
constexpr int kTargetWGs = 2048;
constexpr int kSmallN = 256;

struct CombineArgs {
  const unsigned char* G;
  long long ldG;
  int n;
  long long goff[kMaxGroups + 1];
  int P;
  int rows_per_chunk, nchunks, colblocks;
  const float* w;     // [P_total][n], offset to this launch's first group
  double* partial;    // [nchunks][cols] indexed by absolute column - goff[0] of the call
  long long col_base; // goff[0] of the call
};

template <bool BF16>
__global__ __launch_bounds__(kThreads) void combine_partial_kernel(CombineArgs a) {
  const int cb = blockIdx.x, ch = blockIdx.y, p = blockIdx.z;
  const long long c = a.goff[p] + (long long)cb * kThreads + threadIdx.x;
  if (c >= a.goff[p + 1]) return;
  const int r0 = ch * a.rows_per_chunk;
  int r1 = r0 + a.rows_per_chunk;
  r1 = r1 < a.n ? r1 : a.n;
  const float* wp = a.w + (long long)p * a.n;
  double acc = 0.0;
  for (int i = r0; i < r1; ++i) {
    float g;
    if constexpr (BF16)
      g = __uint_as_float((unsigned)reinterpret_cast<const unsigned short*>(a.G)[(long long)i * a.ldG + c] << 16);
    else
      g = reinterpret_cast<const float*>(a.G)[(long long)i * a.ldG + c];
    acc += (double)wp[i] * (double)g;
  }
  a.partial[(long long)ch * (a.goff[a.P] - a.col_base) + (c - a.col_base)] = acc;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void combine_small_kernel(CombineArgs a, float* u) {
  __shared__ double part[4][64];
  const int p = blockIdx.y;
  const int cl = threadIdx.x & 63, q = threadIdx.x >> 6;
  const long long c = a.goff[p] + (long long)blockIdx.x * 64 + cl;
  const bool ok = c < a.goff[p + 1];
  const float* wp = a.w + (long long)p * a.n;
  double acc = 0.0;
  if (ok) {
    int i = q;
    for (; i + 12 < a.n; i += 16) {   // four rows in flight
      float g[4];
#pragma unroll
      for (int u4 = 0; u4 < 4; ++u4) {
        const long long e = (long long)(i + 4 * u4) * a.ldG + c;
        if constexpr (BF16)
          g[u4] = __uint_as_float((unsigned)reinterpret_cast<const unsigned short*>(a.G)[e] << 16);
        else
          g[u4] = reinterpret_cast<const float*>(a.G)[e];
      }
#pragma unroll
      for (int u4 = 0; u4 < 4; ++u4) acc += (double)wp[i + 4 * u4] * (double)g[u4];
    }
    for (; i < a.n; i += 4) {
      float g;
      if constexpr (BF16)
        g = __uint_as_float((unsigned)reinterpret_cast<const unsigned short*>(a.G)[(long long)i * a.ldG + c] << 16);
      else
        g = reinterpret_cast<const float*>(a.G)[(long long)i * a.ldG + c];
      acc += (double)wp[i] * (double)g;
    }
  }
  part[q][cl] = acc;
  __syncthreads();
  if (q == 0 && ok) u[c] = (float)((part[0][cl] + part[1][cl]) + (part[2][cl] + part[3][cl]));
}

__global__ __launch_bounds__(kThreads) void combine_reduce_kernel(CombineArgs a, float* u) {
  const long long width = a.goff[a.P] - a.col_base;
  const long long c = (long long)blockIdx.x * kThreads + threadIdx.x;
  if (c >= width) return;
  double acc = 0.0;
  for (int ch = 0; ch < a.nchunks; ++ch) acc += a.partial[(long long)ch * width + c];
  u[a.col_base + c] = (float)acc;
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_combine_workspace_size(int64_t n, const int64_t* goff, int P) {
  if (!goff || P < 1 || n < 0 || n <= dr::kSmallN) return 0;
  const int64_t width = goff[P] - goff[0];
  int64_t maxw = 0;
  for (int p = 0; p < P; ++p) maxw = goff[p + 1] - goff[p] > maxw ? goff[p + 1] - goff[p] : maxw;
  const int gp = P < dr::kMaxGroups ? P : dr::kMaxGroups;
  const int64_t colblocks = (maxw + dr::kThreads - 1) / dr::kThreads;
  int64_t nch = colblocks * gp > 0 ? (dr::kTargetWGs + colblocks * gp - 1) / (colblocks * gp) : 1;
  const int64_t maxch = (n + 63) / 64;
  if (nch > maxch) nch = maxch;
  if (nch < 1) nch = 1;
  return (size_t)nch * (size_t)(width > 0 ? width : 0) * sizeof(double);
}

extern "C" dr_status dr_combine(const void* G, int64_t n, int64_t ldG, dr_dtype dtype, const int64_t* goff, int P,
                                const float* w, float* u, void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!goff || P < 1 || n < 0 || n > (1 << 30) || goff[0] < 0) return DR_ERR_ARG;
  for (int p = 0; p < P; ++p)
    if (goff[p + 1] < goff[p]) return DR_ERR_ARG;
  if (goff[P] > goff[0] && !u) return DR_ERR_ARG;
  if (n > 0 && (!G || !w || ldG < goff[P])) return DR_ERR_ARG;
  const size_t need = dr_combine_workspace_size(n, goff, P);
  if (need > 0 && (!workspace || ws_bytes < need)) return DR_ERR_WORKSPACE;
  const int64_t width = goff[P] - goff[0];
  if (width == 0) return DR_OK;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  int64_t maxw = 0;
  for (int p = 0; p < P; ++p) maxw = goff[p + 1] - goff[p] > maxw ? goff[p + 1] - goff[p] : maxw;
  const int gp_all = P < kMaxGroups ? P : kMaxGroups;
  const int64_t colblocks = (maxw + kThreads - 1) / kThreads;
  int64_t nch = (kTargetWGs + colblocks * gp_all - 1) / (colblocks * gp_all);
  const int64_t maxch = (n + 63) / 64;
  if (nch > maxch) nch = maxch;
  if (nch < 1) nch = 1;
  const int rows_per_chunk = (int)((n + nch - 1) / nch);
  for (int p0 = 0; p0 < P; p0 += kMaxGroups) {
    const int gp = P - p0 < kMaxGroups ? P - p0 : kMaxGroups;
    CombineArgs a = {};
    a.G = static_cast<const unsigned char*>(G);
    a.ldG = ldG;
    a.n = (int)n;
    for (int p = 0; p <= gp; ++p) a.goff[p] = goff[p0 + p];
    a.P = gp;
    a.rows_per_chunk = rows_per_chunk > 0 ? rows_per_chunk : 1;
    a.nchunks = (int)nch;
    a.colblocks = (int)colblocks;
    a.w = w + (long long)p0 * n;
    a.partial = static_cast<double*>(workspace);
    a.col_base = goff[p0];
    if (a.goff[gp] == a.col_base) continue;
    if (n <= kSmallN) {
      dim3 grid((unsigned)((maxw + 63) / 64), (unsigned)gp);
      if (dtype == DR_BF16)
        hipLaunchKernelGGL(combine_small_kernel<true>, grid, dim3(kThreads), 0, hs, a, u);
      else
        hipLaunchKernelGGL(combine_small_kernel<false>, grid, dim3(kThreads), 0, hs, a, u);
      dr_status st = launch_status();
      if (st != DR_OK) return st;
      continue;
    }
    if (n > 0) {
      dim3 grid((unsigned)colblocks, (unsigned)nch, (unsigned)gp);
      if (dtype == DR_BF16)
        hipLaunchKernelGGL(combine_partial_kernel<true>, grid, dim3(kThreads), 0, hs, a);
      else
        hipLaunchKernelGGL(combine_partial_kernel<false>, grid, dim3(kThreads), 0, hs, a);
      dr_status st = launch_status();
      if (st != DR_OK) return st;
    } else {
      a.nchunks = 0;
    }
    const long long wdt = a.goff[gp] - a.col_base;
    hipLaunchKernelGGL(combine_reduce_kernel, dim3((unsigned)((wdt + kThreads - 1) / kThreads)), dim3(kThreads), 0, hs,
                       a, u);
    dr_status st = launch_status();
    if (st != DR_OK) return st;
  }
  return DR_OK;
}
