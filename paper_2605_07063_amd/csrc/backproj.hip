// Back-projection of a sketch-space vector to parameter space
// (dr_back_project): for every layer with first-stage projectors P_in,
// P_out (second stage the identity), the transpose of the factorised
// compressor maps the layer's block x~ of a sketch-space vector to
//   U_l = P_out^T X' P_in,  X' = x~ as [k_out][k_in]     (d_out x d_in)
// (App. C.1, "Backward projection"), never forming Pi^T.  Applied to the
// sketch-space update u~ = G~^T w it gives the parameter-space update of the
// MeSO variant of the layer-wise algorithm.
//
//   bp_left_kernel   T = X' P_in   [k_out][d_in] fp32 (small, workspace)
//   bp_right_kernel  U = P_out^T T, one 64 (d_out) x 256 (d_in) tile per
//                    workgroup: each thread owns 16 rows x 4 columns, so a
//                    float4 of T read from L2 feeds 64 FMAs; the P_out columns
//                    of the tile sit in LDS.  The d_out x d_in fp32 write is
//                    the HBM bound.

#include "common.h"

namespace dr {
namespace {

constexpr int kBpRows = 16;    // rows per wave (4 waves: 64 rows per tile)
constexpr int kBpCols = 256;   // columns per tile (4 per lane)
constexpr int kBpMaxK = 64;

template <typename TP>
__device__ __forceinline__ float ld(const TP* p, long long i) {
  return (float)p[i];
}

// T[a][c] = sum_b X'[a][b] P_in[b][c]
template <typename TP>
__global__ __launch_bounds__(256) void bp_left_kernel(const float* x, const TP* p_in, int k_in, int d_in, float* T) {
  const int a = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= d_in) return;
  float acc = 0.f;
  for (int b = 0; b < k_in; ++b) acc = fmaf(x[a * k_in + b], ld(p_in, (long long)b * d_in + c), acc);
  T[(long long)a * d_in + c] = acc;
}

// U[o][c] = sum_a P_out[a][o] T[a][c] for a 64 (d_out) x 256 (d_in) tile:
// wave v owns rows 16 v .. 16 v + 15, lane l columns 4 l .. 4 l + 3; the
// tile's P_out columns sit in LDS (every lane of a wave reads the same four
// 16-byte words per a: broadcasts), T comes from L2 as float4.
template <typename TP>
__global__ __launch_bounds__(256) void bp_right_kernel(const TP* p_out, const float* T, int k_out, int d_out, int d_in,
                                                       float* U) {
  __shared__ __attribute__((aligned(16))) float po[kBpMaxK][kBpRows * 4];
  const int o0 = blockIdx.y * (kBpRows * 4);
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
  for (int a = 0; a < k_out; ++a) {
    const float4 t = *reinterpret_cast<const float4*>(T + (long long)a * d_in + c);
    const float4* pr = reinterpret_cast<const float4*>(&po[a][kBpRows * v]);
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
  int64_t mx = 1;
  for (int l = 0; l < num_layers; ++l) {
    const int64_t t = layers[l].k_out * layers[l].d_in;
    mx = t > mx ? t : mx;
  }
  return dr::align_up((size_t)mx * 4, 256);
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
  float* T = static_cast<float*>(workspace);
  for (int l = 0; l < num_layers; ++l) {
    const dr_layer& L = layers[l];
    const int k_in = (int)L.k_in, k_out = (int)L.k_out, d_in = (int)L.d_in, d_out = (int)L.d_out;
    const float* x = u + L.col_offset;
    float* Ul = U + u_offset[l];
    const dim3 gl((d_in + 255) / 256, k_out), gr((d_in + kBpCols - 1) / kBpCols, (d_out + 4 * kBpRows - 1) / (4 * kBpRows));
    if (dtype == DR_BF16) {
      hipLaunchKernelGGL(bp_left_kernel<__bf16>, gl, dim3(256), 0, hs, x, static_cast<const __bf16*>(L.p_in), k_in,
                         d_in, T);
      hipLaunchKernelGGL(bp_right_kernel<__bf16>, gr, dim3(256), 0, hs, static_cast<const __bf16*>(L.p_out),
                         (const float*)T, k_out, d_out, d_in, Ul);
    } else {
      hipLaunchKernelGGL(bp_left_kernel<float>, gl, dim3(256), 0, hs, x, static_cast<const float*>(L.p_in), k_in,
                         d_in, T);
      hipLaunchKernelGGL(bp_right_kernel<float>, gr, dim3(256), 0, hs, static_cast<const float*>(L.p_out),
                         (const float*)T, k_out, d_out, d_in, Ul);
    }
    const dr_status st = launch_status();
    if (st != DR_OK) return st;
  }
  return DR_OK;
}
