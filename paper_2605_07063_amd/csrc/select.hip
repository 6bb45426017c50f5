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

// The other two subset rules of Sec. 3.3.2 live here as well:
//   threshold_kernel  (dr_select_threshold) one workgroup per group: keep
//                     s_i > tau (or >= tau; negative score filtering is
//                     tau = 0 inclusive), indices in ascending order by two
//                     passes over contiguous per-thread ranges and a block
//                     scan, weights 1 / |S| on the kept set.
//   greedy_kernel     (dr_select_greedy) one workgroup per group, k steps;
//                     r_c = sum_{i in S} K_ic of every candidate is kept in
//                     fp64 in LDS (n <= 16384).  A step
//                     evaluates f(S + c) = (A + 2 r_c + K_cc) / t^2 -
//                     2 (B + s_c) / t in fp64 for every candidate, takes the
//                     block-wide minimum (ties to the lowest index), then
//                     adds row c* of K to every r.  The fp64 operations are
//                     written in one fixed order without contraction, so the
//                     choice does not depend on the compiler.
//   nan_scan_kernel   flags a NaN anywhere in K or s per group before the
//                     greedy steps (grid-stride over all entries).

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


// ------------------------------------------------------------ thresholding

__global__ __launch_bounds__(kThreads) void threshold_kernel(const float* s, long long n, float tau, int inclusive,
                                                             int* idx, int* count, float* w, int* info) {
  __shared__ unsigned wsum[kWaves + 1];
  __shared__ int nanflag;
  const int p = blockIdx.x, tid = threadIdx.x;
  const float* sp = s + (long long)p * n;
  int* ip = idx ? idx + (long long)p * n : nullptr;
  float* wp = w ? w + (long long)p * n : nullptr;
  if (tid == 0) nanflag = 0;
  __syncthreads();
  bool nan_seen = false;
  for (long long i = tid; i < n; i += kThreads) nan_seen |= is_nan_bits(sp[i]);
  if (nan_seen) nanflag = 1;
  __syncthreads();
  const bool bad = nanflag != 0;
  const long long per = (n + kThreads - 1) / kThreads;
  const long long i0 = (long long)tid * per;
  const long long i1 = i0 + per < n ? i0 + per : n;
  unsigned c = 0u;
  if (!bad)
    for (long long i = i0; i < i1; ++i) {
      const float v = sp[i];
      c += inclusive ? (v >= tau) : (v > tau);
    }
  unsigned tot;
  unsigned pos = block_excl_scan(c, wsum, &tot);
  const float wk = tot > 0u ? 1.0f / (float)tot : 0.f;
  for (long long i = i0; i < i1; ++i) {
    const float v = sp[i];
    const bool keep = !bad && (inclusive ? (v >= tau) : (v > tau));
    if (keep && ip) ip[pos++] = (int)i;
    if (wp) wp[i] = keep ? wk : 0.f;
  }
  if (ip)
    for (long long i = (long long)tot + tid; i < n; i += kThreads) ip[i] = -1;
  if (tid == 0) {
    count[p] = (int)tot;
    info[p] = bad ? DR_INFO_NONFINITE : 0;
  }
}

// ------------------------------------------------------------ greedy

constexpr int kGThreads = 512;                       // 2 waves per SIMD: 256 VGPRs for the candidates
constexpr int kGWaves = kGThreads / 64;
constexpr int kGreedyPer = 32;                       // candidates per thread
constexpr long long kGreedyMaxN = (long long)kGThreads * kGreedyPer;

// NaN anywhere in K_p or s_p -> flag[p] = 1 (flag cleared by the host-side
// launch of nan_clear first)
__global__ void nan_clear_kernel(int* flag, int P) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < P) flag[p] = 0;
}

__global__ __launch_bounds__(256) void nan_scan_kernel(const float* K, const float* s, long long n, int* flag) {
  __shared__ int any;
  const int p = blockIdx.y;
  if (threadIdx.x == 0) any = 0;
  __syncthreads();
  const float* Kp = K + (long long)p * n * n;
  bool bad = false;
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x; q < n * n; q += stride)
    bad |= is_nan_bits(Kp[q]);
  if (blockIdx.x == 0)
    for (long long i = threadIdx.x; i < n; i += blockDim.x) bad |= is_nan_bits(s[(long long)p * n + i]);
  if (bad) any = 1;
  __syncthreads();
  if (threadIdx.x == 0 && any) atomicOr(&flag[p], 1);
}

// exclusive scan over the 512-thread greedy workgroup
__device__ unsigned block_excl_scan_g(unsigned v, unsigned* wsum, unsigned* tot) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  unsigned inc = v;
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned t = __shfl_up(inc, off, 64);
    if (lane >= off) inc += t;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  if (tid == 0) {
    unsigned run = 0u;
    for (int v2 = 0; v2 < kGWaves; ++v2) {
      const unsigned x = wsum[v2];
      wsum[v2] = run;
      run += x;
    }
    wsum[kGWaves] = run;
  }
  __syncthreads();
  const unsigned r = wsum[wave] + inc - v;
  *tot = wsum[kGWaves];
  __syncthreads();
  return r;
}

#pragma clang fp contract(off)
__device__ __forceinline__ double greedy_f(double A, double B, double r, double kcc, double sc, double t) {
  return ((A + 2.0 * r) + kcc) / (t * t) - (2.0 * (B + sc)) / t;
}
#pragma clang fp contract(on)

// diag[p][i] = K_p[i][i] (contiguous, so the greedy steps read it coalesced)
__global__ __launch_bounds__(256) void diag_kernel(const float* K, long long n, float* diag) {
  const int p = blockIdx.y;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) diag[(long long)p * n + i] = K[(long long)p * n * n + i * n + i];
}

__global__ __launch_bounds__(kGThreads) void greedy_kernel(const float* K, const float* s, long long n, long long k,
                                                           const int* nanflag, const float* diag, int* idx, float* w,
                                                           int* info) {
  __shared__ double r[kGreedyMaxN];            // r_c = sum_{i in S} K_ic
  __shared__ unsigned char taken[kGreedyMaxN];
  __shared__ double bf[kGWaves];
  __shared__ int bi[kGWaves];
  __shared__ unsigned wsum[kGWaves + 1];
  const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* Kp = K + (long long)p * n * n;
  const float* sp = s + (long long)p * n;
  const float* dp = diag + (long long)p * n;
  int* ip = idx + (long long)p * k;
  float* wp = w ? w + (long long)p * n : nullptr;
  if (nanflag[p]) {
    for (long long i = tid; i < k; i += kGThreads) ip[i] = -1;
    if (wp)
      for (long long i = tid; i < n; i += kGThreads) wp[i] = 0.f;
    if (tid == 0) info[p] = DR_INFO_NONFINITE;
    return;
  }
  for (long long i = tid; i < n; i += kGThreads) {
    r[i] = 0.0;
    taken[i] = 0;
  }
  __syncthreads();
  double A = 0.0, B = 0.0;
  for (long long step = 0; step < k; ++step) {
    const double t = (double)(step + 1);
    double fbest = 0.0;
    int ibest = -1;
    for (long long i = tid; i < n; i += kGThreads) {   // ascending within the thread: ties keep the first
      if (taken[i]) continue;
      const double f = greedy_f(A, B, r[i], (double)dp[i], (double)sp[i], t);
      if (ibest < 0 || f < fbest) {
        fbest = f;
        ibest = (int)i;
      }
    }
    // wave then block minimum of (f, index); -1 = no candidate
    for (int off = 32; off > 0; off >>= 1) {
      const double fo = __shfl_xor(fbest, off, 64);
      const int io = __shfl_xor(ibest, off, 64);
      if (io >= 0 && (ibest < 0 || fo < fbest || (fo == fbest && io < ibest))) {
        fbest = fo;
        ibest = io;
      }
    }
    if (lane == 0) {
      bf[wave] = fbest;
      bi[wave] = ibest;
    }
    __syncthreads();
    double F = 0.0;
    int I = -1;
    for (int v = 0; v < kGWaves; ++v) {
      const int io = bi[v];
      if (io >= 0 && (I < 0 || bf[v] < F || (bf[v] == F && io < I))) {
        F = bf[v];
        I = io;
      }
    }
    // add the winner: A += 2 r_c + K_cc, B += s_c, r += K[c]
    {
#pragma clang fp contract(off)
      A = (A + 2.0 * r[I]) + (double)dp[I];
      B = B + (double)sp[I];
    }
    __syncthreads();   // every thread has read r[I] before it changes
    const float* row = Kp + (long long)I * n;
    for (long long i = tid; i < n; i += kGThreads) r[i] = r[i] + (double)row[i];
    if (tid == 0) taken[I] = 1;
    __syncthreads();
  }
  // ascending indices of the chosen set, kGThreads indices at a time
  const float wk = k > 0 ? 1.0f / (float)k : 0.f;
  unsigned base = 0u;
  for (long long i0 = 0; i0 < n; i0 += kGThreads) {
    const long long i = i0 + tid;
    const bool chosen = i < n && taken[i];
    unsigned tot;
    const unsigned pos = block_excl_scan_g(chosen ? 1u : 0u, wsum, &tot);
    if (chosen) ip[base + pos] = (int)i;
    if (wp && i < n) wp[i] = chosen ? wk : 0.f;
    base += tot;
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

extern "C" dr_status dr_select_threshold(const float* s, int64_t n, int P, float tau, int inclusive, int32_t* idx,
                                         int32_t* count, float* w, int32_t* info, void* stream) {
  using namespace dr;
  if (n < 0 || P < 0) return DR_ERR_ARG;
  if (n > (1LL << 30)) return DR_ERR_UNSUPPORTED;
  if (tau != tau) return DR_ERR_ARG;
  if (P == 0) return DR_OK;
  if (!info || !count || (n > 0 && !s)) return DR_ERR_ARG;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(threshold_kernel, dim3(P), dim3(kThreads), 0, hs, s, (long long)n, tau, inclusive ? 1 : 0, idx,
                     count, w, info);
  return launch_status();
}

extern "C" size_t dr_greedy_workspace_size(int64_t n, int P) {
  if (n < 0 || P <= 0) return 0;
  return dr::align_up((size_t)P * 4, 256) + dr::align_up((size_t)P * (size_t)n * 4, 256);
}

extern "C" dr_status dr_select_greedy(const float* K, const float* s, int64_t n, int P, int64_t k, int32_t* idx,
                                      float* w, int32_t* info, void* workspace, size_t ws_bytes, void* stream) {
  using namespace dr;
  if (n < 0 || P < 0 || k < 0 || k > n) return DR_ERR_ARG;
  if (n > kGreedyMaxN) return DR_ERR_UNSUPPORTED;
  if (P == 0) return DR_OK;
  if (!info || (n > 0 && (!K || !s)) || (k > 0 && !idx)) return DR_ERR_ARG;
  if (!workspace || ws_bytes < dr_greedy_workspace_size(n, P)) return DR_ERR_WORKSPACE;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  int* flag = static_cast<int*>(workspace);
  float* diag = reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) + align_up((size_t)P * 4, 256));
  hipLaunchKernelGGL(nan_clear_kernel, dim3((P + 255) / 256), dim3(256), 0, hs, flag, P);
  if (n > 0) {
    hipLaunchKernelGGL(diag_kernel, dim3((unsigned)((n + 255) / 256), P), dim3(256), 0, hs, K, (long long)n, diag);
    const long long nn = (long long)n * n;
    long long blocks = (nn + 256 * 16 - 1) / (256 * 16);
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(nan_scan_kernel, dim3((unsigned)blocks, P), dim3(256), 0, hs, K, s, (long long)n, flag);
  }
  hipLaunchKernelGGL(greedy_kernel, dim3(P), dim3(kGThreads), 0, hs, K, s, (long long)n, (long long)k, flag, diag,
                     idx, w, info);
  return launch_status();
}
