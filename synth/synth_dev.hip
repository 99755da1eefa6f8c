/*
 * GPU side of the synthetic-input generator (see philox.h): fills device
 * buffers with the same bf16 / byte streams as synth_host.c, so multi-GB
 * weight sets are generated in place instead of crossing the host link.
 * Built with hipcc into libsynth_dev.so; C entry points, plain pointers.
 */
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SYNTH_FN static __device__ inline
#include "philox.h"

/* Each thread produces 8 consecutive bf16 (one 16-byte store when aligned). */
__global__ void __launch_bounds__(256)
k_fill_bf16(uint16_t *__restrict__ out, uint64_t n, uint64_t seed, uint64_t tensor, uint64_t first)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * 8;
    for (uint64_t i = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8; i < n; i += stride) {
        uint16_t v[8];
        uint64_t e = first + i;
        if (((e & 1) == 0) && i + 8 <= n) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                synth_u32x4 r = synth_draw(seed, tensor, (e >> 1) + q);
                v[2 * q] = synth_bf16_from_u32x2(r.v[0], r.v[1]);
                v[2 * q + 1] = synth_bf16_from_u32x2(r.v[2], r.v[3]);
            }
            if ((((uintptr_t)(out + i)) & 15) == 0) {
                uint4 w;
                w.x = v[0] | ((uint32_t)v[1] << 16);
                w.y = v[2] | ((uint32_t)v[3] << 16);
                w.z = v[4] | ((uint32_t)v[5] << 16);
                w.w = v[6] | ((uint32_t)v[7] << 16);
                *(uint4 *)(out + i) = w;
            } else {
                for (int q = 0; q < 8; ++q) out[i + q] = v[q];
            }
        } else {
            for (uint64_t q = 0; q < 8 && i + q < n; ++q)
                out[i + q] = synth_bf16(seed, tensor, e + q);
        }
    }
}

__global__ void __launch_bounds__(256)
k_fill_bytes(uint8_t *__restrict__ out, uint64_t n, uint64_t seed, uint64_t stream, uint64_t first)
{
    const uint64_t gstride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;; t += gstride) {
        /* thread t covers stream bytes [16*(first/16 + t), +16) */
        uint64_t k0 = ((first >> 4) + t) << 4;
        if (k0 >= first + n) break;
        synth_u32x4 r = synth_draw(seed, stream, k0 >> 4);
        const uint8_t *b = (const uint8_t *)r.v;
        for (int q = 0; q < 16; ++q) {
            uint64_t k = k0 + q;
            if (k >= first && k < first + n) out[k - first] = b[q];
        }
    }
}

static int grid_for(uint64_t items)
{
    uint64_t g = (items + 255) / 256;
    if (g > 65536) g = 65536;
    if (g == 0) g = 1;
    return (int)g;
}

extern "C" int synth_dev_fill_bf16(void *out, uint64_t n, uint64_t seed, uint64_t tensor,
                                   uint64_t first, void *stream)
{
    if (n == 0) return 0;
    if (!out) return -1;
    hipLaunchKernelGGL(k_fill_bf16, dim3(grid_for((n + 7) / 8)), dim3(256), 0, (hipStream_t)stream,
                       (uint16_t *)out, n, seed, tensor, first);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" int synth_dev_fill_bytes(void *out, uint64_t n, uint64_t seed, uint64_t stream_id,
                                    uint64_t first, void *stream)
{
    if (n == 0) return 0;
    if (!out) return -1;
    hipLaunchKernelGGL(k_fill_bytes, dim3(grid_for((n + 15) / 16 + 1)), dim3(256), 0, (hipStream_t)stream,
                       (uint8_t *)out, n, seed, stream_id, first);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}
