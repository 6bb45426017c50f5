/*
 * dr_probe.h -- measurement probes of libdrprobe.so (not part of the
 * method): the HBM and MFMA ceilings that roofline fractions are also
 * reported against, next to the datasheet peaks.  Device pointers; the
 * caller owns every buffer; calls only enqueue work on `stream`
 * (a hipStream_t, NULL = the default stream).  Return 0 on success, 1 for
 * an invalid argument (checked before any HIP call), 7 for a launch error.
 */
#ifndef DR_PROBE_H
#define DR_PROBE_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DR_PROBE_MAX_BLOCKS 65536

/* Read every byte of buf[0, bytes) once (bytes a multiple of 16, buf
 * 16-byte aligned) with `blocks` workgroups of 256 threads; one float per
 * workgroup goes to sink[blocks]. */
int dr_probe_read(const void* buf, size_t bytes, float* sink, int blocks, void* stream);

/* `blocks` workgroups of 256 threads (4 waves); every wave issues
 * 8 * iters matrix instructions on register operands: bf16 != 0 ->
 * 16x16x32 bf16 (16384 flops each), else 16x16x4 fp32 (2048 flops each).
 * One float per thread goes to sink[blocks * 256]. */
int dr_probe_mfma(int bf16, int iters, float* sink, int blocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif
