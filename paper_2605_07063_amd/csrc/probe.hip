// Measurement probes (libdrprobe.so, include/dr_probe.h): the ceilings the
// benchmark reports beside the datasheet peaks.  Not part of the method.
//   stream read : every byte of a buffer read once, a non-temporal
//                 16-byte load per lane per step, grid-stride over the
//                 whole buffer; one value per workgroup is stored so that
//                 the loads cannot be dropped.
//   MFMA loops  : each wave issues back-to-back matrix instructions on
//                 eight independent accumulators whose operands stay in
//                 registers (no memory traffic); bf16 16x16x32 and fp32
//                 16x16x4, the shapes the library's kernels use.

#include "common.h"
#include "dr_probe.h"

namespace dr {
namespace {

constexpr int kReadThreads = 256;
constexpr int kMfmaThreads = 256;

__global__ __launch_bounds__(kReadThreads) void probe_read_kernel(const u32x4* buf, long long n16, float* sink) {
  __shared__ unsigned int red[kReadThreads / 64];
  const long long stride = (long long)gridDim.x * kReadThreads;
  unsigned int acc = 0u;
  for (long long i = (long long)blockIdx.x * kReadThreads + threadIdx.x; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(buf + i);
    acc ^= (v.x ^ v.y) ^ (v.z ^ v.w);
  }
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = (float)(red[0] ^ red[1] ^ red[2] ^ red[3]);
}

// eight independent accumulators, each updated in place by inline assembly
// (left to the compiler, the loop-carried accumulators get copied between
// register tuples every iteration, which chains the products)
#define DR_PROBE_LOOP(INSTR, A, B)                                                                \
  f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0; \
  for (int it = 0; it < iters; ++it) {                                                            \
    asm volatile(INSTR " %0, %8, %9, %0\n\t" INSTR " %1, %8, %9, %1\n\t"                          \
                 INSTR " %2, %8, %9, %2\n\t" INSTR " %3, %8, %9, %3\n\t"                          \
                 INSTR " %4, %8, %9, %4\n\t" INSTR " %5, %8, %9, %5\n\t"                          \
                 INSTR " %6, %8, %9, %6\n\t" INSTR " %7, %8, %9, %7"                                \
                 : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7)   \
                 : "v"(A), "v"(B));                                                              \
  }                                                                                               \
  asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");                                                \
  const f32x4 t = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));                             \
  sink[(long long)blockIdx.x * kMfmaThreads + threadIdx.x] = (t[0] + t[1]) + (t[2] + t[3]);

__global__ __launch_bounds__(kMfmaThreads) void probe_mfma_bf16_kernel(int iters, float* sink) {
  // bf16 pairs of 1, 0.5, 0.25 and -1 (finite values only)
  const u32x4 a = {0x3f803f80u, 0x3f003f00u, 0x3e803e80u, 0xbf803f80u};
  const u32x4 b = {0x3f003f80u, 0x3e803f00u, 0x3f80bf80u, 0x3f803e80u};
  DR_PROBE_LOOP("v_mfma_f32_16x16x32_bf16", a, b)
}

__global__ __launch_bounds__(kMfmaThreads) void probe_mfma_f32_kernel(int iters, float* sink) {
  const float a = 1.0f + 1e-3f * (float)threadIdx.x, b = 0.5f - 1e-3f * (float)threadIdx.x;
  DR_PROBE_LOOP("v_mfma_f32_16x16x4_f32", a, b)
}

}  // namespace
}  // namespace dr

extern "C" int dr_probe_read(const void* buf, size_t bytes, float* sink, int blocks, void* stream) {
  if (!buf || !sink || blocks < 1 || blocks > DR_PROBE_MAX_BLOCKS || bytes < 16 || (bytes & 15) ||
      !dr::aligned16(buf))
    return 1;
  hipLaunchKernelGGL(dr::probe_read_kernel, dim3(blocks), dim3(dr::kReadThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), static_cast<const dr::u32x4*>(buf),
                     (long long)(bytes / 16), sink);
  return hipGetLastError() == hipSuccess ? 0 : 7;
}

extern "C" int dr_probe_mfma(int bf16, int iters, float* sink, int blocks, void* stream) {
  if (!sink || blocks < 1 || blocks > DR_PROBE_MAX_BLOCKS || iters < 1) return 1;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (bf16)
    hipLaunchKernelGGL(dr::probe_mfma_bf16_kernel, dim3(blocks), dim3(dr::kMfmaThreads), 0, hs, iters, sink);
  else
    hipLaunchKernelGGL(dr::probe_mfma_f32_kernel, dim3(blocks), dim3(dr::kMfmaThreads), 0, hs, iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : 7;
}
