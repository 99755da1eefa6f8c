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

/* One piece of a batched fill: elements first..first+n-1 of tensor `tensor`, written at out. */
typedef struct {
    uint64_t out, n, tensor, first;
} synth_piece;

/* Workgroup g fills pieces g, g + grid, ...: a whole weight set in one launch. */
__global__ void __launch_bounds__(256)
k_fill_bf16_pieces(const synth_piece *__restrict__ pieces, uint64_t count, uint64_t seed)
{
    for (uint64_t p = blockIdx.x; p < count; p += gridDim.x) {
        const synth_piece pc = pieces[p];
        uint16_t *const out = (uint16_t *)pc.out;
        for (uint64_t i = (uint64_t)threadIdx.x * 8; i < pc.n; i += (uint64_t)blockDim.x * 8) {
            const uint64_t e = pc.first + i;
            if (((e & 1) == 0) && i + 8 <= pc.n && (((uintptr_t)(out + i)) & 15) == 0) {
                uint16_t v[8];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    synth_u32x4 r = synth_draw(seed, pc.tensor, (e >> 1) + q);
                    v[2 * q] = synth_bf16_from_u32x2(r.v[0], r.v[1]);
                    v[2 * q + 1] = synth_bf16_from_u32x2(r.v[2], r.v[3]);
                }
                uint4 w;
                w.x = v[0] | ((uint32_t)v[1] << 16);
                w.y = v[2] | ((uint32_t)v[3] << 16);
                w.z = v[4] | ((uint32_t)v[5] << 16);
                w.w = v[6] | ((uint32_t)v[7] << 16);
                *(uint4 *)(out + i) = w;
            } else {
                for (uint64_t q = 0; q < 8 && i + q < pc.n; ++q) out[i + q] = synth_bf16(seed, pc.tensor, e + q);
            }
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

/* Fills many bf16 ranges under one seed with a single launch: `pieces` is a host array of
 * `count` {device address, elements, tensor id, first element} records.  The table is
 * uploaded to a temporary device buffer; the call returns once the fill has finished. */
extern "C" int synth_dev_fill_bf16_pieces(const void *pieces, uint64_t count, uint64_t seed, void *stream)
{
    if (count == 0) return 0;
    if (!pieces) return -1;
    synth_piece *d = NULL;
    const size_t bytes = count * sizeof(synth_piece);
    if (hipMalloc((void **)&d, bytes) != hipSuccess) return -5;
    hipStream_t s = (hipStream_t)stream;
    int rc = 0;
    if (hipMemcpyAsync(d, pieces, bytes, hipMemcpyHostToDevice, s) != hipSuccess) rc = -4;
    if (rc == 0) {
        const uint64_t grid = count < 16384 ? count : 16384;
        hipLaunchKernelGGL(k_fill_bf16_pieces, dim3((uint32_t)grid), dim3(256), 0, s, d, count, seed);
        if (hipGetLastError() != hipSuccess) rc = -4;
    }
    if (hipStreamSynchronize(s) != hipSuccess) rc = -4;
    (void)hipFree(d);
    return rc;
}
