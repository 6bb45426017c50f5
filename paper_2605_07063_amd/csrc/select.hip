// Top-k selection by alignment score (dr_select_topk): the top-k rule of
// Sec. 3.3.2, applied per group as in the group-wise decomposition of
// Sec. 3.3.3 (Select-S of the one-pass algorithms, Sec. 4.2).
//
// One 1024-thread workgroup per group.  Scores map to order-preserving
// 32-bit keys (sign-magnitude flip; -0.0 folded onto +0.0).  Four passes of
// an 8-bit radix select (LDS histogram with integer atomics, digit found
// by one wave with a shuffle scan over the 256 bins in descending order)
// give the k-th largest key t and the number `need` of keys equal to t that
// belong to the top k.  A final pass keeps every key > t and the `need`
// lowest-index keys equal to t: each thread owns a contiguous index range,
// two block-wide exclusive scans give its rank among equal keys and its
// output position, so the indices come out in ascending order.
// Everything is integer: the result is exact and deterministic.

#include "common.h"

namespace dr {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ unsigned score_key(float f) {
  unsigned u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;   // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ bool is_nan_bits(float f) { return (__float_as_uint(f) & 0x7fffffffu) > 0x7f800000u; }

// exclusive scan of one unsigned per thread over the block; returns the
// exclusive prefix, total in *tot
__device__ unsigned block_excl_scan(unsigned v, unsigned* wsum, unsigned* tot) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  unsigned inc = v;
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned t = __shfl_up(inc, off, 64);
    if (lane >= off) inc += t;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    unsigned x = lane < kWaves ? wsum[lane] : 0u;
    unsigned xi = x;
    for (int off = 1; off < 64; off <<= 1) {
      const unsigned t = __shfl_up(xi, off, 64);
      if (lane >= off) xi += t;
    }
    if (lane < kWaves) wsum[lane] = xi - x;   // exclusive wave offsets
    if (lane == kWaves - 1) wsum[kWaves] = xi;
  }
  __syncthreads();
  const unsigned r = wsum[wave] + inc - v;
  *tot = wsum[kWaves];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void topk_kernel(const float* s, long long n, long long k, int* idx, float* w,
                                                        int* info) {
  __shared__ unsigned hist[256];
  __shared__ unsigned wsum[kWaves + 1];
  __shared__ unsigned sh_digit, sh_need;
  __shared__ int nanflag;
  const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* sp = s + (long long)p * n;
  int* ip = idx + (long long)p * k;
  float* wp = w ? w + (long long)p * n : nullptr;

  if (tid == 0) nanflag = 0;
  __syncthreads();
  bool nan_seen = false;
  for (long long i = tid; i < n; i += kThreads) nan_seen |= is_nan_bits(sp[i]);
  if (nan_seen) nanflag = 1;
  __syncthreads();
  if (nanflag) {
    for (long long i = tid; i < k; i += kThreads) ip[i] = -1;
    if (wp)
      for (long long i = tid; i < n; i += kThreads) wp[i] = 0.f;
    if (tid == 0) info[p] = DR_INFO_NONFINITE;
    return;
  }
  if (k == 0) {
    if (wp)
      for (long long i = tid; i < n; i += kThreads) wp[i] = 0.f;
    if (tid == 0) info[p] = 0;
    return;
  }

  unsigned prefix = 0u, mask = 0u, need = (unsigned)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    for (long long i = tid; i < n; i += kThreads) {
      const unsigned key = score_key(sp[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      unsigned c[4], loc = 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        c[t] = hist[255 - 4 * lane - t];
        loc += c[t];
      }
      unsigned inc = loc;
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned t = __shfl_up(inc, off, 64);
        if (lane >= off) inc += t;
      }
      unsigned before = inc - loc;
      if (before < need && need <= inc) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (before + c[t] >= need) {
            sh_digit = 255u - 4u * lane - t;
            sh_need = need - before;
            break;
          }
          before += c[t];
        }
      }
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    need = sh_need;
    __syncthreads();
  }
  const unsigned thr = prefix;

  // selection over contiguous per-thread index ranges
  const long long per = (n + kThreads - 1) / kThreads;
  const long long i0 = (long long)tid * per;
  const long long i1 = i0 + per < n ? i0 + per : n;
  unsigned gt = 0u, eq = 0u;
  for (long long i = i0; i < i1; ++i) {
    const unsigned key = score_key(sp[i]);
    gt += key > thr;
    eq += key == thr;
  }
  unsigned tot;
  const unsigned eq_base = block_excl_scan(eq, wsum, &tot);
  unsigned take = need > eq_base ? need - eq_base : 0u;
  take = take < eq ? take : eq;
  const unsigned out_base = block_excl_scan(gt + take, wsum, &tot);
  unsigned pos = out_base, taken = 0u;
  const float wk = 1.0f / (float)k;
  for (long long i = i0; i < i1; ++i) {
    const unsigned key = score_key(sp[i]);
    bool sel = key > thr;
    if (key == thr && taken < take) {
      sel = true;
      ++taken;
    }
    if (sel && pos < (unsigned)k) ip[pos++] = (int)i;
    if (wp) wp[i] = sel ? wk : 0.f;
  }
  if (tid == 0) info[p] = 0;
}

}  // namespace
}  // namespace dr

extern "C" dr_status dr_select_topk(const float* s, int64_t n, int P, int64_t k, int32_t* idx, float* w,
                                    int32_t* info, void* stream) {
  using namespace dr;
  if (n < 0 || P < 0 || k < 0 || k > n) return DR_ERR_ARG;
  if (n > (1LL << 30)) return DR_ERR_UNSUPPORTED;
  if (P == 0) return DR_OK;
  if (!info || (n > 0 && !s) || (k > 0 && !idx)) return DR_ERR_ARG;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(topk_kernel, dim3(P), dim3(kThreads), 0, hs, s, (long long)n, (long long)k, idx, w, info);
  return launch_status();
}
