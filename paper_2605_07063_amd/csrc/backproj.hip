// Back-projection of a sketch-space vector to parameter space
// (dr_back_project): for every layer with first-stage projectors P_in,
// P_out (second stage the identity), the transpose of the factorised
// compressor maps the layer's block x~ of a sketch-space vector to
//   U_l = P_out^T X' P_in,  X' = x~ as [k_out][k_in]     (d_out x d_in)
// (App. C.3, "Backward projection"), never forming Pi^T.  Applied to the
// sketch-space update u~ = G~^T w it gives the parameter-space update of the
// MeSO variant of the layer-wise algorithm.
//
// Up to 16 layers go in one launch (blockIdx.z = layer), so that the small
// per-layer grids fill the chip together.
//   bp_left_kernel   T = X' P_in   [k_out][d_in] (small, workspace), one
//                    64-column slice of T per workgroup, fp32 MFMA (16x16x4)
//                    with both operands staged in LDS; written as fp32, or
//                    as three bf16 planes for bp_mfma_kernel
//   bp_mfma_kernel   bf16 projectors: U = P_out^T (T1 + T2 + T3) on bf16 MFMA
//                    (see the kernel)
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
// bf16 round to nearest even of a finite fp32 value
__device__ __forceinline__ unsigned short bf16_rne(float x) {
  const unsigned u = __float_as_uint(x);
  return (unsigned short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_val(unsigned short h) { return __uint_as_float((unsigned)h << 16); }

template <typename TP, bool PLANES>
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
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int a = 16 * i + 4 * lq + q, c = c0 + 16 * w + lr;
      if (a >= k_out || c >= d_in) continue;
      const float t = acc[i][q];
      if constexpr (PLANES) {
        // T = T1 + T2 + T3 in bf16 planes [3][k_out][d_in] (each the nearest
        // bf16 to what the previous ones leave; the sum is T to about 2^-24)
        unsigned short* Tp = reinterpret_cast<unsigned short*>(g.T[l]);
        const unsigned short h1 = bf16_rne(t);
        const float r1 = t - bf16_val(h1);
        const unsigned short h2 = bf16_rne(r1);
        const unsigned short h3 = bf16_rne(r1 - bf16_val(h2));
        const long long plane = (long long)k_out * d_in;
        Tp[(long long)a * d_in + c] = h1;
        Tp[plane + (long long)a * d_in + c] = h2;
        Tp[2 * plane + (long long)a * d_in + c] = h3;
      } else {
        g.T[l][(long long)a * d_in + c] = t;
      }
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

// bf16 P_out (16-byte aligned, d_in and d_out multiples of 8): U = P_out^T T
// with T given as three bf16 planes, i.e. sum_{p < 3} P_out^T T_p, as one
// bf16 MFMA contraction over 3 * k_out rows (each product exact in fp32,
// fp32 accumulation).  One 128 (d_out) x 128 (d_in) tile per workgroup:
// P_out[:, o-tile] and the three T[:, c-tile] planes (64 rows of 256 bytes
// each, 32-byte slots XOR-swizzled per row) are staged in LDS and read as
// MFMA operands by the gfx950 transposing read (8 consecutive rows a per
// lane); wave (wr, wc) holds a 64 x 64 quarter.  The finished tile goes back
// through LDS so that U is written in whole 512-byte rows.
constexpr int kBmTile = 128;
constexpr int kBmRow = kBmTile * 2;          // bytes of one staged row
constexpr int kBmSlab = kBpMaxK * kBmRow;    // 16 KB: one operand slab
constexpr int kBmOutLd = kBmTile + 4;        // output staging stride (floats)
constexpr int kBmLds = 4 * kBmSlab > kBmTile * kBmOutLd * 4 ? 4 * kBmSlab : kBmTile * kBmOutLd * 4;

__global__ __launch_bounds__(256, 2) void bp_mfma_kernel(BpArgs g) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kBmLds];
  const int l = blockIdx.z;
  const int k_out = g.k_out[l], d_out = g.d_out[l], d_in = g.d_in[l];
  const int o0 = blockIdx.y * kBmTile, c0 = blockIdx.x * kBmTile;
  if (o0 >= d_out || c0 >= d_in) return;
  const unsigned short* pg = static_cast<const unsigned short*>(g.p_out[l]);
  const unsigned short* tg = reinterpret_cast<const unsigned short*>(g.T[l]);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  {
    // slab 0 = P_out[a][o0 ..], slabs 1..3 = plane p[a][c0 ..]; 16-byte chunks,
    // every load of the thread in flight before the LDS writes
    u32x4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = tid + 256 * u, slab = e >> 10, r = (e >> 4) & 63, col = 8 * (e & 15);
      const bool ok = r < k_out && (slab == 0 ? o0 + col < d_out : c0 + col < d_in);
      const unsigned short* src = slab == 0 ? pg + (long long)r * d_out + o0 + col
                                            : tg + ((long long)(slab - 1) * k_out + r) * d_in + c0 + col;
      v[u] = ok ? *reinterpret_cast<const u32x4*>(src) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int e = tid + 256 * u, slab = e >> 10, r = (e >> 4) & 63, ch = e & 15;
      *reinterpret_cast<u32x4*>(lds + slab * kBmSlab + r * kBmRow + (((ch >> 1) ^ slot_xor(r)) * 32) + (ch & 1) * 16) =
          v[u];
    }
  }
  __syncthreads();
  // fragment reads: lane (g4, q, rr) of the transposing read addresses row
  // 8 g4 + q (+4 for the second half) and 8-byte piece rr of a 16-column
  // block; the block's logical slot is XOR-ed with the row's swizzle
  const int g4 = lane >> 4, q = (lane >> 2) & 3, rr = lane & 3;
  const int fx = q | ((g4 & 1) << 2);
  const int wr = w >> 1, wc = w & 1;
  const unsigned rbase = (unsigned)((8 * g4 + q) * kBmRow + rr * 8);
  unsigned offa[4], offb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) offa[i] = rbase + (unsigned)(((4 * wr + i) ^ fx) * 32);
#pragma unroll
  for (int j = 0; j < 4; ++j) offb[j] = rbase + (unsigned)(((4 * wc + j) ^ fx) * 32);
  auto frag = [&](const unsigned char* base) {
    const v4s lo = lds_read_tr16(base);
    const v4s hi = lds_read_tr16(base + 4 * kBmRow);
    return u32x4{__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y, __builtin_bit_cast(uint2, hi).x,
                 __builtin_bit_cast(uint2, hi).y};
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nh = k_out > 32 ? 2 : 1;   // 32-row slices of the sketch index a (rows >= k_out are zero)
  for (int h = 0; h < nh; ++h) {
    u32x4 fa[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = frag(lds + h * 32 * kBmRow + offa[i]);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      u32x4 fb[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) fb[j] = frag(lds + (1 + p) * kBmSlab + h * 32 * kBmRow + offb[j]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma_bf16(fa[i], fb[j], acc[i][j]);
    }
  }
  __syncthreads();
  float* outs = reinterpret_cast<float*>(lds);   // [128][kBmOutLd]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        outs[(64 * wr + 16 * i + 4 * g4 + qq) * kBmOutLd + 64 * wc + 16 * j + (lane & 15)] = acc[i][j][qq];
  __syncthreads();
  float* U = g.U[l];
#pragma unroll
  for (int u = 0; u < kBmTile * kBmTile / 4 / 256; ++u) {
    const int e = tid + 256 * u, r = e >> 5, c = 4 * (e & 31);
    if (o0 + r < d_out && c0 + c < d_in)
      *reinterpret_cast<float4*>(U + (long long)(o0 + r) * d_in + c0 + c) =
          *reinterpret_cast<const float4*>(&outs[r * kBmOutLd + c]);
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
                               (size_t)(layers[l].d_in > 0 ? layers[l].d_in : 0) * 6, 256);
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
    bool mfma = dtype == DR_BF16;
    size_t o = 0;
    for (int j = 0; j < count; ++j) {
      const dr_layer& L = layers[f + j];
      g.p_in[j] = L.p_in;
      g.p_out[j] = L.p_out;
      g.x[j] = u + L.col_offset;
      g.T[j] = reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) + o);
      o = align_up(o + (size_t)L.k_out * (size_t)L.d_in * 6, 256);   // fp32 T or three bf16 planes
      mfma = mfma && L.d_in % 8 == 0 && L.d_out % 8 == 0 && aligned16(L.p_out);
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
    if (mfma) {
      const dim3 gm((dimax + kBmTile - 1) / kBmTile, (domax + kBmTile - 1) / kBmTile, count);
      hipLaunchKernelGGL((bp_left_kernel<__bf16, true>), gl, dim3(256), 0, hs, g);
      hipLaunchKernelGGL(bp_mfma_kernel, gm, dim3(256), 0, hs, g);
    } else if (dtype == DR_BF16) {
      hipLaunchKernelGGL((bp_left_kernel<__bf16, false>), gl, dim3(256), 0, hs, g);
      hipLaunchKernelGGL(bp_right_kernel<__bf16>, gr, dim3(256), 0, hs, g);
    } else {
      hipLaunchKernelGGL((bp_left_kernel<float, false>), gl, dim3(256), 0, hs, g);
      hipLaunchKernelGGL(bp_right_kernel<float>, gr, dim3(256), 0, hs, g);
    }
    const dr_status st = launch_status();
    if (st != DR_OK) return st;
  }
  return DR_OK;
}
