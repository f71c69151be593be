/*
 * ws_ceilings.h -- C ABI of libwsceil.so: two gfx950 microbenchmarks that
 * measure the practical ceilings the attention kernels are compared with
 * (the benchmark reports fractions of both beside the fractions of the
 * published peaks).  They compute nothing of the attention method.
 *
 * Conventions: device pointers are HIP device memory of the current device;
 * `stream` is a hipStream_t passed as void* (NULL = default stream); the
 * calls only enqueue (stream-ordered) and return 0 or a HIP error code.
 */
#ifndef WS_CEILINGS_H
#define WS_CEILINGS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * wsc_mfma_loop -- dense bf16 matrix-core ceiling.  num_groups work-groups
 * of 8 waves (two per SIMD); each wave issues iters x 4 x chains
 * v_mfma_f32_32x32x16_bf16 (32 x 32 x 16 multiply-adds each) on register
 * operands, into `chains` (1..4) independent accumulators, no memory
 * traffic in the loop.  Work: num_groups * 8 * iters * 4 * chains * 32768
 * flops.  out: device f32 [num_groups] (one checksum per work-group, so the
 * loop is not removed).  num_groups >= 1, iters >= 1, 1 <= chains <= 4.
 */
int wsc_mfma_loop(float *out, int32_t num_groups, int32_t iters, int32_t chains, void *stream);

/*
 * wsc_stream_read -- streaming HBM read ceiling.  Reads `bytes` bytes of
 * src (16-byte aligned, bytes a multiple of 16) once with 16-byte loads
 * (four in flight per lane), num_groups work-groups of 256 threads striding
 * over it, and writes one XOR checksum per work-group to out (device
 * uint32 [num_groups]).
 */
int wsc_stream_read(const void *src, size_t bytes, uint32_t *out, int32_t num_groups, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* WS_CEILINGS_H */
