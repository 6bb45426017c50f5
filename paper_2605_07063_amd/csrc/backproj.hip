// Back-projection of a sketch-space vector to parameter space
// (dr_back_project): for every layer with first-stage projectors P_in,
// P_out (second stage the identity), the transpose of the factorised
// compressor maps the layer's block x~ of a sketch-space vector to
//   U_l = P_out^T X' P_in,  X' = x~ as [k_out][k_in]     (d_out x d_in)
// (App. C.1, "Backward projection"), never forming Pi^T.  Applied to the
// sketch-space update u~ = G~^T w it gives the parameter-space update of the
// MeSO variant of the layer-wise algorithm.
//
// Up to 16 layers go in one launch (blockIdx.z = layer), so that the small
// per-layer grids fill the chip together.
//   bp_left_kernel   T = X' P_in   [k_out][d_in] fp32 (small, workspace),
//                    one 64-column slice of T per workgroup, fp32 MFMA
//                    (16x16x4) with both operands staged in LDS
//   bp_right_kernel  U = P_out^T T, one 64 (d_out) x 256 (d_in) tile per
//                    workgroup: each thread owns 16 rows x 4 columns, so a
//                    float4 of T read from L2 feeds 64 FMAs; the P_out columns
//                    of the tile sit in LDS.  The d_out x d_in fp32 write is
//                    the HBM bound.  (fp32 MFMA has the same peak as fp32
//                    FMA on this chip; staged or not, it measured slower here.)

#include "common.h"

namespace dr {
namespace {

constexpr int kBpLayers = 16;  // layers per launch (blockIdx.z)
constexpr int kBpTile = 64;    // columns of T per workgroup of bp_left_kernel
constexpr int kBpRows = 16;    // bp_right_kernel: rows per wave (4 waves: 64 rows per tile)
constexpr int kBpCols = 256;   // bp_right_kernel: columns per tile (4 per lane)
constexpr int kBpMaxK = 64;
constexpr int kBpLd = 132;     // LDS row stride (floats)

template <typename TP>
__device__ __forceinline__ float ld(const TP* p, long long i) {
  return (float)p[i];
}

struct BpArgs {
  const void* p_in[kBpLayers];
  const void* p_out[kBpLayers];
  const float* x[kBpLayers];   // the layer's block of the sketch-space vector
  float* T[kBpLayers];         // [k_out][d_in] workspace
  float* U[kBpLayers];         // [d_out][d_in] output
  int k_in[kBpLayers], k_out[kBpLayers], d_in[kBpLayers], d_out[kBpLayers];
};

// T[a][c] = sum_b X'[a][b] P_in[b][c] for c in this workgroup's 64 columns;
// a < k_out <= 64 (4 row tiles), 4 column tiles: wave w takes column tile w
// of every row tile.  Rows and columns past k_in / k_out /
// d_in are zero in LDS.
template <typename TP>
__global__ __launch_bounds__(256) void bp_left_kernel(BpArgs g) {
  __shared__ __attribute__((aligned(16))) float xs[kBpMaxK * 68];   // X'[a][b], stride 68
  __shared__ __attribute__((aligned(16))) float ps[kBpMaxK * kBpLd];   // P_in[b][c - c0]
  const int l = blockIdx.z;
  const int k_in = g.k_in[l], k_out = g.k_out[l], d_in = g.d_in[l];
  const int c0 = blockIdx.x * kBpTile;
  if (c0 >= d_in) return;
  const float* x = g.x[l];
  const TP* p_in = static_cast<const TP*>(g.p_in[l]);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, lr = lane & 15, lq = lane >> 4;
  {
    // every load of the thread in flight before the LDS writes
    float xv[kBpMaxK * kBpMaxK / 256], pv[kBpMaxK * kBpTile / 256];
#pragma unroll
    for (int u = 0; u < kBpMaxK * kBpMaxK / 256; ++u) {
      const int e = tid + 256 * u, a = e >> 6, b = e & 63;
      xv[u] = (a < k_out && b < k_in) ? x[a * k_in + b] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBpMaxK * kBpTile / 256; ++u) {
      const int e = tid + 256 * u, b = e / kBpTile, c = e % kBpTile;
      pv[u] = (b < k_in && c0 + c < d_in) ? ld(p_in, (long long)b * d_in + c0 + c) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBpMaxK * kBpMaxK / 256; ++u) {
      const int e = tid + 256 * u;
      xs[(e >> 6) * 68 + (e & 63)] = xv[u];
    }
#pragma unroll
    for (int u = 0; u < kBpMaxK * kBpTile / 256; ++u) {
      const int e = tid + 256 * u;
      ps[(e / kBpTile) * kBpLd + e % kBpTile] = pv[u];
    }
  }
  __syncthreads();
  f32x4 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int kq = (k_in + 3) & ~3;
  for (int b0 = 0; b0 < kq; b0 += 4) {
    const float bv = ps[(b0 + lq) * kBpLd + 16 * w + lr];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = mma_f32(xs[(16 * i + lr) * 68 + b0 + lq], bv, acc[i]);
  }
  float* T = g.T[l];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int a = 16 * i + 4 * lq + q, c = c0 + 16 * w + lr;
      if (a < k_out && c < d_in) T[(long long)a * d_in + c] = acc[i][q];
    }
}

// U[o][c] = sum_a P_out[a][o] T[a][c] for a 64 (d_out) x 256 (d_in) tile:
// wave v owns rows 16 v .. 16 v + 15, lane l columns 4 l .. 4 l + 3; the
// tile's P_out columns sit in LDS (every lane of a wave reads the same four
// 16-byte words per a: broadcasts), T comes from L2 as float4.
template <typename TP>
__global__ __launch_bounds__(256) void bp_right_kernel(BpArgs g) {
  __shared__ __attribute__((aligned(16))) float po[kBpMaxK][kBpRows * 4];
  const int l = blockIdx.z;
  const int k_out = g.k_out[l], d_out = g.d_out[l], d_in = g.d_in[l];
  const TP* p_out = static_cast<const TP*>(g.p_out[l]);
  const float* T = g.T[l];
  float* U = g.U[l];
  const int o0 = blockIdx.y * (kBpRows * 4);
  if (o0 >= d_out || blockIdx.x * kBpCols >= d_in) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int v = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = blockIdx.x * kBpCols + 4 * lane;
  for (int e = tid; e < k_out * kBpRows * 4; e += 256) {
    const int a = e / (kBpRows * 4), r = e % (kBpRows * 4);
    po[a][r] = o0 + r < d_out ? ld(p_out, (long long)a * d_out + o0 + r) : 0.f;
  }
  __syncthreads();
  if (c >= d_in) return;
  float4 acc[kBpRows];
#pragma unroll
  for (int r = 0; r < kBpRows; ++r) acc[r] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int a0 = 0; a0 < k_out; a0 += 8) {   // eight rows of T in flight before the FMAs
    float4 tv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      tv[e] = a0 + e < k_out ? *reinterpret_cast<const float4*>(T + (long long)(a0 + e) * d_in + c)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (a0 + e >= k_out) break;
      const float4 t = tv[e];
      const float4* pr = reinterpret_cast<const float4*>(&po[a0 + e][kBpRows * v]);
#pragma unroll
      for (int q = 0; q < kBpRows / 4; ++q) {
        const float4 pq = pr[q];
        const float pv[4] = {pq.x, pq.y, pq.z, pq.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float4& A = acc[4 * q + u];
          A.x = fmaf(pv[u], t.x, A.x);
          A.y = fmaf(pv[u], t.y, A.y);
          A.z = fmaf(pv[u], t.z, A.z);
          A.w = fmaf(pv[u], t.w, A.w);
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kBpRows; ++r) {
    const int o = o0 + kBpRows * v + r;
    if (o < d_out) *reinterpret_cast<float4*>(U + (long long)o * d_in + c) = acc[r];
  }
}

}  // namespace
}  // namespace dr

extern "C" size_t dr_backproject_workspace_size(const dr_layer* layers, int num_layers) {
  if (!layers || num_layers < 1) return 0;
  // one launch holds up to 16 layers: room for the largest such run of T blocks
  size_t best = 256;
  for (int f = 0; f < num_layers; f += dr::kBpLayers) {
    size_t o = 0;
    for (int l = f; l < num_layers && l < f + dr::kBpLayers; ++l)
      o = dr::align_up(o + (size_t)(layers[l].k_out > 0 ? layers[l].k_out : 0) *
                               (size_t)(layers[l].d_in > 0 ? layers[l].d_in : 0) * 4, 256);
    best = o > best ? o : best;
  }
  return best;
}

extern "C" dr_status dr_back_project(const dr_layer* layers, int num_layers, dr_dtype dtype, const float* u, float* U,
                                     const int64_t* u_offset, void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  if (dtype != DR_BF16 && dtype != DR_F32) return DR_ERR_DTYPE;
  if (!layers || num_layers < 1 || !u || !U || !u_offset) return DR_ERR_ARG;
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    if (L.k_in < 1 || L.k_out < 1 || L.k_in > kBpMaxK || L.k_out > kBpMaxK) return DR_ERR_ARG;
    if (L.d_in < 1 || L.d_out < 1 || L.d_in > (1 << 28) || L.d_out > (1 << 28)) return DR_ERR_ARG;
    if (!L.p_in || !L.p_out || L.col_offset < 0 || u_offset[l] < 0) return DR_ERR_ARG;
    if ((L.d_out + 4 * kBpRows - 1) / (4 * kBpRows) > 65535) return DR_ERR_UNSUPPORTED;   // grid rows
    if (L.d_in % 4 || !aligned16(U + u_offset[l])) return DR_ERR_ARG;   // float4 columns and stores
  }
  if (!workspace || ws_bytes < dr_backproject_workspace_size(layers, num_layers)) return DR_ERR_WORKSPACE;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  for (int f = 0; f < num_layers; f += kBpLayers) {
    const int count = num_layers - f < kBpLayers ? num_layers - f : kBpLayers;
    BpArgs g = {};
    int dimax = 1, domax = 1;
    size_t o = 0;
    for (int j = 0; j < count; ++j) {
      const dr_layer& L = layers[f + j];
      g.p_in[j] = L.p_in;
      g.p_out[j] = L.p_out;
      g.x[j] = u + L.col_offset;
      g.T[j] = reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) + o);
      o = align_up(o + (size_t)L.k_out * (size_t)L.d_in * 4, 256);
      g.U[j] = U + u_offset[f + j];
      g.k_in[j] = (int)L.k_in;
      g.k_out[j] = (int)L.k_out;
      g.d_in[j] = (int)L.d_in;
      g.d_out[j] = (int)L.d_out;
      dimax = g.d_in[j] > dimax ? g.d_in[j] : dimax;
      domax = g.d_out[j] > domax ? g.d_out[j] : domax;
    }
    const dim3 gl((dimax + kBpTile - 1) / kBpTile, 1, count);
    const dim3 gr((dimax + kBpCols - 1) / kBpCols, (domax + 4 * kBpRows - 1) / (4 * kBpRows), count);
    if (dtype == DR_BF16) {
      hipLaunchKernelGGL(bp_left_kernel<__bf16>, gl, dim3(256), 0, hs, g);
      hipLaunchKernelGGL(bp_right_kernel<__bf16>, gr, dim3(256), 0, hs, g);
    } else {
      hipLaunchKernelGGL(bp_left_kernel<float>, gl, dim3(256), 0, hs, g);
      hipLaunchKernelGGL(bp_right_kernel<float>, gr, dim3(256), 0, hs, g);
    }
    const dr_status st = launch_status();
    if (st != DR_OK) return st;
  }
  return DR_OK;
}
