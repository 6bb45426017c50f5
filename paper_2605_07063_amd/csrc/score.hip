// Exact per-sample scores of one linear layer (dr_score_exact), the three
// contraction orders of Sec. 4.3 for s_i = <gbar*, g_i> with the mean target
// gradient gbar* = (1/m) sum_j G*_j:
//   DIRECT  materialise each G_i (tile by tile, never stored) and take its
//           inner product with gbar* (update-assembly kernel in score mode,
//           update.hip);
//   PIP     sum_t dy_{i,t}^T gbar* x_{i,t}: a GEMM of the example's token
//           rows with gbar* followed by a dot with the dy rows (pip_kernel);
//   GIP     (1/m) sum_j <D_i D*_j^T, X_i X*_j^T>: the two T x T token
//           cross-correlations of every (example, target) pair, multiplied
//           elementwise and summed (gip_kernel).
// gbar* is assembled first from the target rows with weights 1/m (the
// update-assembly kernel); PIP multiplies by it in bf16 as a hi + lo pair
// (two MFMAs, relative rounding ~2^-17 instead of bf16's 2^-9).
//
// pip_kernel / gip_kernel: 128 x 128 output tiles per workgroup, 4 waves of
// 64 x 64, operands are row panels whose reduction index is contiguous in
// memory (token rows of x / dy, rows of gbar*), staged by buffer->LDS DMA
// in 64-wide steps through a 2-stage ring in the swizzled 128-byte-row
// layout of the Gram kernel.  Rows past a length and columns past a width
// load as zeros (out-of-range buffer offsets), so padding is never read.
// Partial sums go to fp64 workspace slots and are reduced in a fixed order.

#include "common.h"

namespace dr {
namespace {

constexpr int kSThreads = 256;
constexpr int kST = 128;                  // tile rows / columns
constexpr int kSK = 64;                   // reduction step (one 128-byte row)
constexpr int kSPanel = kST * kSK * 2;    // 16 KB

__device__ __forceinline__ int clamp_len(const int* len, int i, int T) {
  int L = len ? len[i] : T;
  return L < 0 ? 0 : (L > T ? T : L);
}

// Row panel of one operand: this lane's four rows (half blocks w, w+4,
// w+8, w+12 of the 128-row panel) as byte offsets, or kOobOffset.
struct PanelRows {
  unsigned off[4];
  int seg[4];
};

__device__ __forceinline__ PanelRows panel_rows(int w, int lane, int rows_valid, long long row_bytes) {
  PanelRows p;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int hb = w + 4 * u;
    const int r = 8 * hb + (lane >> 3);
    p.seg[u] = swz_seg_of_lane(lane, hb & 1);
    p.off[u] = r < rows_valid ? (unsigned)((long long)r * row_bytes) : kOobOffset;
  }
  return p;
}

__device__ __forceinline__ void issue_panel(__amdgpu_buffer_rsrc_t rs, const PanelRows& pr, unsigned char* dst, int w,
                                            int k0, int K) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int col = k0 + 8 * pr.seg[u];
    const unsigned o = (pr.off[u] == kOobOffset || col >= K) ? kOobOffset : pr.off[u] + (unsigned)(col * 2);
    dma16<kAuxCached>(rs, dst + (w + 4 * u) * 1024, o);
  }
}

// acc[i][j] += A[64 wr + 16 i + .][k] B[64 wc + 16 j + .][k] over k < K for
// NB B panels (summed), A and B given as row panels
template <int NB>
__device__ __forceinline__ void panel_gemm(unsigned char* lds, __amdgpu_buffer_rsrc_t ra, const PanelRows& pa,
                                           const __amdgpu_buffer_rsrc_t* rb, const PanelRows& pb, int K,
                                           f32x4 (&acc)[4][4]) {
  constexpr int kStage = (1 + NB) * kSPanel;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w >> 1, wc = w & 1, lr = lane & 15, lg = lane >> 4;
  const int nk = (K + kSK - 1) / kSK;
  auto issue = [&](int t, int st) {
    unsigned char* sb = lds + st * kStage;
    issue_panel(ra, pa, sb, w, t * kSK, K);
#pragma unroll
    for (int b = 0; b < NB; ++b) issue_panel(rb[b], pb, sb + (1 + b) * kSPanel, w, t * kSK, K);
  };
  issue(0, 0);
  for (int t = 0; t < nk; ++t) {
    DR_WAIT_VM(0);
    DR_LDS_SYNC();
    if (t + 1 < nk) issue(t + 1, (t + 1) & 1);
    const unsigned char* sa = lds + (t & 1) * kStage;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      const int seg = 4 * kh + lg;
      u32x4 fa[4], fb[NB][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[i] = swz_read(sa + (4 * wr + i) * 2048, lr, seg);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) fb[b][j] = swz_read(sa + (1 + b) * kSPanel + (4 * wc + j) * 2048, lr, seg);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mma_bf16(fa[i], fb[b][j], acc[i][j]);
    }
  }
  DR_LDS_SYNC();   // the ring is free for the next use
}

__device__ double block_sum_256(double v, double* red) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = 0.0;
  for (int q = 0; q < kSThreads / 64; ++q) t += red[q];
  return t;
}

struct ScoreLayer {
  const unsigned char* x;
  const unsigned char* dy;
  long long ldx, lddy;       // elements per token
  long long exx, exdy;       // bytes per example
  int d_in, d_out, T, n, m;
  const int* len;            // [n + m] or null
};

// ---------------------------------------------------------------- PIP

// workgroup (i, token block tb, output block ob):
// part[(i TB + tb) OB + ob] = sum_{t in block, t < len_i} sum_{o in block} dy_{i,t,o} (gbar* x_{i,t})_o
__global__ __launch_bounds__(kSThreads) void pip_kernel(ScoreLayer a, const unsigned char* ghi,
                                                        const unsigned char* glo, int TB, int OB, double* part) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * 3 * kSPanel];
  __shared__ double red[kSThreads / 64];
  const int i = blockIdx.x / TB, tb = blockIdx.x % TB, ob = blockIdx.y;
  const int L = clamp_len(a.len, i, a.T);
  const int t0 = tb * kST, o0 = ob * kST;
  if (t0 >= L) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w >> 1, wc = w & 1, lc = lane & 15, g = lane >> 4;
  const unsigned char* xb = a.x + (long long)i * a.exx + (long long)t0 * a.ldx * 2;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(xb, kOobOffset);
  __amdgpu_buffer_rsrc_t rb[2] = {make_rsrc(ghi + (long long)o0 * a.d_in * 2, kOobOffset),
                                  make_rsrc(glo + (long long)o0 * a.d_in * 2, kOobOffset)};
  const PanelRows pa = panel_rows(w, lane, L - t0, a.ldx * 2);
  const PanelRows pb = panel_rows(w, lane, a.d_out - o0, (long long)a.d_in * 2);
  f32x4 acc[4][4];
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[p][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  panel_gemm<2>(lds, ra, pa, rb, pb, a.d_in, acc);
  // dot with the dy rows of the block (valid tokens and outputs only)
  const __bf16* dyb = reinterpret_cast<const __bf16*>(a.dy + (long long)i * a.exdy);
  float d = 0.f;
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + 64 * wr + 16 * p + 4 * g + r;
      if (t >= L) continue;
      const __bf16* row = dyb + (long long)t * a.lddy;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = o0 + 64 * wc + 16 * q + lc;
        if (o < a.d_out) d = fmaf(acc[p][q][r], (float)row[o], d);
      }
    }
  const double tot = block_sum_256((double)d, red);
  if (tid == 0) part[((long long)i * TB + tb) * OB + ob] = tot;
}

__global__ void pip_reduce_kernel(const double* part, int n, int T, const int* len, int TB, int OB, float* s) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int L = clamp_len(len, i, T);
  const int nb = (L + kST - 1) / kST;
  double t = 0.0;
  for (int tb = 0; tb < nb; ++tb)
    for (int ob = 0; ob < OB; ++ob) t += part[((long long)i * TB + tb) * OB + ob];
  s[i] = (float)t;
}

// gbar* (fp32) -> bf16 hi + lo (hi = RNE(g), lo = RNE(g - hi))
__global__ void split_kernel(const float* g, long long count, __bf16* hi, __bf16* lo) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= count) return;
  const float v = g[e];
  const __bf16 h = (__bf16)v;
  hi[e] = h;
  lo[e] = (__bf16)(v - (float)h);
}

// ---------------------------------------------------------------- GIP

// workgroup (i, tb) x (j, sb): part = sum over the 128 x 128 block of
// (D_i D*_j^T) .* (X_i X*_j^T)
__global__ __launch_bounds__(kSThreads) void gip_kernel(ScoreLayer a, int TB, double* part) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * 2 * kSPanel];
  __shared__ double red[kSThreads / 64];
  const int i = blockIdx.x / TB, tb = blockIdx.x % TB;
  const int j = blockIdx.y / TB, sb = blockIdx.y % TB;
  const int L = clamp_len(a.len, i, a.T), Lj = clamp_len(a.len, a.n + j, a.T);
  const int t0 = tb * kST, s0 = sb * kST;
  if (t0 >= L || s0 >= Lj) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  f32x4 dd[4][4], xx[4][4];
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      dd[p][q] = f32x4{0.f, 0.f, 0.f, 0.f};
      xx[p][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  {
    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(a.dy + (long long)i * a.exdy + (long long)t0 * a.lddy * 2, kOobOffset);
    const __amdgpu_buffer_rsrc_t rb[1] = {
        make_rsrc(a.dy + (long long)(a.n + j) * a.exdy + (long long)s0 * a.lddy * 2, kOobOffset)};
    panel_gemm<1>(lds, ra, panel_rows(w, lane, L - t0, a.lddy * 2), rb, panel_rows(w, lane, Lj - s0, a.lddy * 2),
                  a.d_out, dd);
  }
  {
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.x + (long long)i * a.exx + (long long)t0 * a.ldx * 2, kOobOffset);
    const __amdgpu_buffer_rsrc_t rb[1] = {
        make_rsrc(a.x + (long long)(a.n + j) * a.exx + (long long)s0 * a.ldx * 2, kOobOffset)};
    panel_gemm<1>(lds, ra, panel_rows(w, lane, L - t0, a.ldx * 2), rb, panel_rows(w, lane, Lj - s0, a.ldx * 2),
                  a.d_in, xx);
  }
  // rows past a length are zero in both products: no masking needed
  float d = 0.f;
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) d = fmaf(dd[p][q][r], xx[p][q][r], d);
  const double tot = block_sum_256((double)d, red);
  if (tid == 0) part[((long long)i * TB + tb) * ((long long)a.m * TB) + (long long)j * TB + sb] = tot;
}

__global__ void gip_reduce_kernel(const double* part, int n, int m, int T, const int* len, int TB, float* s) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int nb = (clamp_len(len, i, T) + kST - 1) / kST;
  double t = 0.0;
  for (int tb = 0; tb < nb; ++tb)
    for (int j = 0; j < m; ++j) {
      const int nsb = (clamp_len(len, n + j, T) + kST - 1) / kST;
      for (int sb = 0; sb < nsb; ++sb) t += part[((long long)i * TB + tb) * ((long long)m * TB) + (long long)j * TB + sb];
    }
  s[i] = (float)(t / (double)m);
}

__global__ void fill_kernel(float* p, long long count, float v) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < count) p[e] = v;
}

// ---------------------------------------------------------------- host

struct ScorePlan {
  size_t off_wm, off_g, off_upd, off_hi, off_lo, off_part, off_direct, bytes;
};

dr_layer target_layer(const dr_layer& L, int64_t n, int64_t T) {
  dr_layer t = L;
  t.x = static_cast<const unsigned char*>(L.x) + n * T * L.ldx * 2;
  t.dy = static_cast<const unsigned char*>(L.dy) + n * T * L.lddy * 2;
  return t;
}

ScorePlan score_plan(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T, int method) {
  int64_t gmax = 1, partmax = 1;
  size_t updmax = 0, dirmax = 0;
  const int64_t TB = (T + kST - 1) / kST;
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    const int64_t g = L.d_out * L.d_in;
    gmax = g > gmax ? g : gmax;
    const dr_layer t = target_layer(L, n, T);
    const size_t u = dr_update_workspace_size(&t, 1, m, T, DR_BF16);
    updmax = u > updmax ? u : updmax;
    if (method == DR_SCORE_PIP) {
      const int64_t OB = (L.d_out + kST - 1) / kST;
      partmax = n * TB * OB > partmax ? n * TB * OB : partmax;
    }
    if (method == DR_SCORE_DIRECT) {
      const size_t d = direct_workspace(&L, 1, n);
      dirmax = d > dirmax ? d : dirmax;
    }
  }
  if (method == DR_SCORE_GIP) partmax = n * TB * m * TB > 1 ? n * TB * m * TB : 1;
  ScorePlan p;
  size_t o = 0;
  p.off_wm = o;     o = align_up(o + (size_t)(m > 0 ? m : 1) * 4, 256);
  p.off_g = o;      if (method != DR_SCORE_GIP) o = align_up(o + (size_t)gmax * 4, 256);
  p.off_upd = o;    if (method != DR_SCORE_GIP) o = align_up(o + updmax, 256);
  p.off_hi = o;     if (method == DR_SCORE_PIP) o = align_up(o + (size_t)gmax * 2, 256);
  p.off_lo = o;     if (method == DR_SCORE_PIP) o = align_up(o + (size_t)gmax * 2, 256);
  p.off_part = o;   if (method != DR_SCORE_DIRECT) o = align_up(o + (size_t)partmax * 8, 256);
  p.off_direct = o; if (method == DR_SCORE_DIRECT) o = align_up(o + dirmax, 256);
  p.bytes = o;
  return p;
}

dr_status validate_score(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T, dr_dtype dtype,
                         int method, const float* s) {
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (dtype != DR_BF16) return DR_ERR_UNSUPPORTED;
  if (method != DR_SCORE_DIRECT && method != DR_SCORE_GIP && method != DR_SCORE_PIP) return DR_ERR_ARG;
  if (!layers || num_layers < 1 || n < 0 || m < 1 || T < 0) return DR_ERR_ARG;
  if (n + m > (1 << 24) || T > (1 << 20)) return DR_ERR_ARG;
  if (n > 0 && !s) return DR_ERR_ARG;
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    if (L.d_in < 1 || L.d_out < 1 || L.d_in % 8 || L.d_out % 8) return DR_ERR_ARG;
    if (L.d_in > (1 << 28) || L.d_out > (1 << 28)) return DR_ERR_ARG;
    if (L.ldx < L.d_in || L.lddy < L.d_out || L.ldx % 8 || L.lddy % 8) return DR_ERR_ARG;
    if (T > 0 && (!L.x || !L.dy || !aligned16(L.x) || !aligned16(L.dy))) return DR_ERR_ARG;
    if (T * L.ldx * 2 >= (int64_t)kOobOffset - 64 || T * L.lddy * 2 >= (int64_t)kOobOffset - 64)
      return DR_ERR_UNSUPPORTED;
    if (L.d_out * L.d_in * 2 >= (int64_t)kOobOffset - 64) return DR_ERR_UNSUPPORTED;
  }
  return DR_OK;
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_score_workspace_size(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T,
                                          dr_dtype dtype, dr_score_method method) {
  if (!layers || num_layers < 1 || n < 0 || m < 1 || T < 0 || dtype != DR_BF16) return 0;
  for (int l = 0; l < num_layers; ++l)
    if (layers[l].d_in < 1 || layers[l].d_out < 1) return 0;
  return dr::score_plan(layers, num_layers, n, m, T, (int)method).bytes;
}

extern "C" dr_status dr_score_exact(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T,
                                    const int32_t* len, dr_dtype dtype, dr_score_method method, float* s,
                                    void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  dr_status st = validate_score(layers, num_layers, n, m, T, dtype, (int)method, s);
  if (st != DR_OK) return st;
  const ScorePlan pl = score_plan(layers, num_layers, n, m, T, (int)method);
  if (!workspace || ws_bytes < pl.bytes) return DR_ERR_WORKSPACE;
  if (n == 0) return DR_OK;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  float* wm = reinterpret_cast<float*>(ws + pl.off_wm);
  float* gstar = reinterpret_cast<float*>(ws + pl.off_g);
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, hs, wm, (long long)m,
                     1.0f / (float)m);
  if ((st = launch_status()) != DR_OK) return st;
  const int TB = (int)((T + kST - 1) / kST);
  for (int l = 0; l < num_layers && st == DR_OK; ++l) {
    const dr_layer& L = layers[l];
    float* sl = s + (int64_t)l * n;
    if (method != DR_SCORE_GIP) {
      // gbar* = (1/m) sum_j G*_j from the target rows
      const dr_layer t = target_layer(L, n, T);
      const int64_t zero = 0;
      st = dr_assemble_update(&t, 1, m, T, len ? len + n : nullptr, DR_BF16, wm, 1, m, nullptr, gstar, &zero,
                              ws + pl.off_upd, pl.off_hi - pl.off_upd, stream);
      if (st != DR_OK) break;
    }
    ScoreLayer a;
    a.x = static_cast<const unsigned char*>(L.x);
    a.dy = static_cast<const unsigned char*>(L.dy);
    a.ldx = L.ldx;
    a.lddy = L.lddy;
    a.exx = T * L.ldx * 2;
    a.exdy = T * L.lddy * 2;
    a.d_in = (int)L.d_in;
    a.d_out = (int)L.d_out;
    a.T = (int)T;
    a.n = (int)n;
    a.m = (int)m;
    a.len = len;
    double* part = reinterpret_cast<double*>(ws + pl.off_part);
    if (method == DR_SCORE_DIRECT) {
      const int64_t zero = 0;
      st = direct_scores(&L, 1, n, T, len, gstar, &zero, sl, ws + pl.off_direct, hs);
    } else if (method == DR_SCORE_PIP) {
      const long long cnt = L.d_out * L.d_in;
      __bf16* hi = reinterpret_cast<__bf16*>(ws + pl.off_hi);
      __bf16* lo = reinterpret_cast<__bf16*>(ws + pl.off_lo);
      hipLaunchKernelGGL(split_kernel, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, hs, (const float*)gstar, cnt,
                         hi, lo);
      const int OB = (int)((L.d_out + kST - 1) / kST);
      hipLaunchKernelGGL(pip_kernel, dim3((unsigned)(n * TB), OB), dim3(kSThreads), 0, hs, a,
                         reinterpret_cast<const unsigned char*>(hi), reinterpret_cast<const unsigned char*>(lo), TB,
                         OB, part);
      hipLaunchKernelGGL(pip_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, hs, (const double*)part,
                         (int)n, (int)T, len, TB, OB, sl);
      st = launch_status();
    } else {
      hipLaunchKernelGGL(gip_kernel, dim3((unsigned)(n * TB), (unsigned)(m * TB)), dim3(kSThreads), 0, hs, a, TB,
                         part);
      hipLaunchKernelGGL(gip_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, hs, (const double*)part,
                         (int)n, (int)m, (int)T, len, TB, sl);
      st = launch_status();
    }
  }
  return st;
}
