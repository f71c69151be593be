// gfx950 microbenchmarks of the two ceilings the attention kernels run
// against: the dense bf16 MFMA rate and the streaming HBM read rate
// (declared in include/ws_ceilings.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ws_ceilings.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Two waves per SIMD, C independent dependency chains per wave: dependent
// accumulation is cheap on this matrix core, and the rate of the loop
// depends a little on the chain count, so the benchmark takes the best of
// several.
template <int C>
__global__ __launch_bounds__(512) void mfma_loop_kernel(float *out, int iters) {
    const int lane = threadIdx.x & 63;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)((lane * 8 + e) % 17));
        b[e] = (__bf16)(0.001f * (float)((lane * 5 + e) % 13));
    }
    f32x16 acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int c = 0; c < C; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) s += acc[c][v];
    __shared__ float red[512];
    red[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int k = 0; k < 512; ++k) t += red[k];
        out[blockIdx.x] = t;
    }
}

// Grid-stride 16-byte non-temporal loads, four per lane in flight.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4 *src, uint64_t n16, uint32_t *out) {
    const uint64_t stride = (uint64_t)gridDim.x * 256;
    uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 x0 = __builtin_nontemporal_load(src + i);
        const u32x4 x1 = __builtin_nontemporal_load(src + i + stride);
        const u32x4 x2 = __builtin_nontemporal_load(src + i + 2 * stride);
        const u32x4 x3 = __builtin_nontemporal_load(src + i + 3 * stride);
        acc ^= x0 ^ x1 ^ x2 ^ x3;
    }
    for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(src + i);
    uint32_t s = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    __shared__ uint32_t red[256];
    red[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int k = 0; k < 256; ++k) t ^= red[k];
        out[blockIdx.x] = t;
    }
}

}  // namespace

extern "C" {

int wsc_mfma_loop(float *out, int32_t num_groups, int32_t iters, int32_t chains, void *stream) {
    if (!out || num_groups < 1 || iters < 1 || chains < 1 || chains > 4) return (int)hipErrorInvalidValue;
    void (*k)(float *, int) = chains == 1 ? mfma_loop_kernel<1>
                            : chains == 2 ? mfma_loop_kernel<2>
                            : chains == 3 ? mfma_loop_kernel<3> : mfma_loop_kernel<4>;
    hipLaunchKernelGGL(k, dim3((unsigned)num_groups), dim3(512), 0, (hipStream_t)stream, out, (int)iters);
    return (int)hipGetLastError();
}

int wsc_stream_read(const void *src, size_t bytes, uint32_t *out, int32_t num_groups, void *stream) {
    if (!src || !out || num_groups < 1 || (bytes & 15) || ((uintptr_t)src & 15)) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)num_groups), dim3(256), 0, (hipStream_t)stream,
                       (const u32x4 *)src, (uint64_t)(bytes / 16), out);
    return (int)hipGetLastError();
}

}  // extern "C"
