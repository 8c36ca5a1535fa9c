// bench_stream.hip -- STREAM-style reference kernels for bench.py (not part of the library).
//
// They measure what a plain HIP kernel reaches on this device for the access patterns a
// collective is made of: a contiguous copy (read once, write once), a read-only and a write-only
// sweep, a read-only sweep of many regions at the same offset, and a bf16 sum of S regions into
// one (the reduce-scatter's pattern). bench.py reports the collectives' effective bandwidth
// against these figures beside the 8 TB/s datasheet peak.
//
// Every wavefront of a grid of `blocks` workgroups (4 wavefronts each) handles chunks of
// `chunk_bytes` in turn (chunk c goes to wavefront c mod W; a grid of one wavefront per chunk
// gives each wavefront one), U x 16 bytes per lane per step, with non-temporal loads and stores
// (the reduction's stores are ordinary ones, as in the library's reductions).
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int U>
__global__ void __launch_bounds__(256) stream_copy(const u32x4* a, u32x4* b, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    for (uint64_t c = wave; c < n16 / c16; c += nw) {
        const u32x4* s = a + c * c16;
        u32x4* d = b + c * c16;
        for (uint64_t i = 0; i < c16; i += 64 * U) {
            u32x4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
            for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u], d + i + u * 64 + lane);
        }
    }
}

template <int U>
__global__ void __launch_bounds__(256) stream_read(const u32x4* a, uint32_t* sink, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    uint32_t acc = 0;
    for (uint64_t c = wave; c < n16 / c16; c += nw) {
        const u32x4* s = a + c * c16;
        for (uint64_t i = 0; i < c16; i += 64 * U) {
            u32x4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
            for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;  // keeps the loads; practically never stores
}

template <int U>
__global__ void __launch_bounds__(256) stream_write(u32x4* b, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    u32x4 v = {lane, 1u, 2u, 3u};
    for (uint64_t c = wave; c < n16 / c16; c += nw)
        for (uint64_t i = 0; i < c16; i += 64 * U)
#pragma unroll
            for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v, b + c * c16 + i + u * 64 + lane);
}

// Read-only sweep of `streams` regions at once, the access pattern of an N-source reduction:
// `a` holds the regions back to back; wavefront w reads chunk c = w, w + W, ... of every region
// in turn (the same offset in each), 4 x 16 bytes per lane per step.
__global__ void __launch_bounds__(256) stream_read_multi(const u32x4* a, uint32_t* sink, uint64_t region16,
                                                         uint32_t streams, uint64_t c16) {
    constexpr int U = 4;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    uint32_t acc = 0;
    for (uint64_t c = wave; c < region16 / c16; c += nw) {
        for (uint32_t r = 0; r < streams; ++r) {
            const u32x4* s = a + r * region16 + c * c16;
            for (uint64_t i = 0; i < c16; i += 64 * U) {
                u32x4 v[U];
#pragma unroll
                for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
                for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
            }
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

// bf16 sum of `streams` regions (back to back in `a`, a multiple of 4 of them) into `b`: chunk c
// of every region is read 4 regions x 4 vectors per lane at a time, summed in fp32 in region
// order, rounded to nearest even once and stored.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__global__ void __launch_bounds__(256) stream_reduce_bf16(const u32x4* a, u32x4* b, uint64_t region16,
                                                          uint32_t streams, uint64_t c16) {
    constexpr int U = 4, SB = 4;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    for (uint64_t c = wave; c < region16 / c16; c += nw) {
        for (uint64_t i = 0; i < c16; i += 64 * U) {
            float acc[U][8];
            for (uint32_t r0 = 0; r0 < streams; r0 += SB) {
                u32x4 v[SB][U];
#pragma unroll
                for (int j = 0; j < SB; ++j)
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        v[j][u] = __builtin_nontemporal_load(a + (uint64_t)(r0 + j) * region16 + c * c16 + i + u * 64 + lane);
#pragma unroll
                for (int j = 0; j < SB; ++j)
#pragma unroll
                    for (int u = 0; u < U; ++u)
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const float lo = __uint_as_float(v[j][u][k] << 16);
                            const float hi = __uint_as_float(v[j][u][k] & 0xFFFF0000u);
                            acc[u][2 * k] = (r0 + j == 0) ? lo : acc[u][2 * k] + lo;
                            acc[u][2 * k + 1] = (r0 + j == 0) ? hi : acc[u][2 * k + 1] + hi;
                        }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                u32x4 w;
#pragma unroll
                for (int k = 0; k < 4; ++k) w[k] = bf16_rne(acc[u][2 * k]) | (bf16_rne(acc[u][2 * k + 1]) << 16);
                b[c * c16 + i + u * 64 + lane] = w;
            }
        }
    }
}

template <int U>
void launch_stream(int kind, const void* a, void* b, uint64_t n16, uint64_t c16, int blocks, hipStream_t s) {
    if (kind == 0) hipLaunchKernelGGL(stream_copy<U>, dim3(blocks), dim3(256), 0, s, (const u32x4*)a, (u32x4*)b, n16, c16);
    else if (kind == 1) hipLaunchKernelGGL(stream_read<U>, dim3(blocks), dim3(256), 0, s, (const u32x4*)a, (uint32_t*)b, n16, c16);
    else hipLaunchKernelGGL(stream_write<U>, dim3(blocks), dim3(256), 0, s, (u32x4*)b, n16, c16);
}

}  // namespace

// kind 0 copy (a -> b), 1 read-only (a; b receives at most one word), 2 write-only (b); unroll
// 4 or 8 vectors per lane per step. bytes must be a multiple of chunk_bytes, and chunk_bytes of
// 1 KiB x unroll. Returns a hipError_t, or -1 for arguments the kernels cannot take.
extern "C" int bench_stream(int kind, int unroll, const void* a, void* b, uint64_t bytes, uint64_t chunk_bytes,
                            int blocks, void* stream) {
    if ((unroll != 4 && unroll != 8) || chunk_bytes == 0 || chunk_bytes % (16 * 64 * (uint64_t)unroll) ||
        bytes % chunk_bytes || blocks <= 0 || kind < 0 || kind > 2)
        return -1;
    const uint64_t n16 = bytes / 16, c16 = chunk_bytes / 16;
    hipStream_t s = (hipStream_t)stream;
    if (unroll == 4) launch_stream<4>(kind, a, b, n16, c16, blocks, s);
    else launch_stream<8>(kind, a, b, n16, c16, blocks, s);
    return (int)hipGetLastError();
}

// Read-only sweep of `streams` regions of bytes / streams each (see stream_read_multi); b receives
// at most one word. bytes must be a multiple of streams * chunk_bytes, and chunk_bytes of 4 KiB.
extern "C" int bench_stream_multi(const void* a, void* b, uint64_t bytes, uint32_t streams, uint64_t chunk_bytes,
                                  int blocks, void* stream) {
    if (streams == 0 || chunk_bytes == 0 || chunk_bytes % (16 * 64 * 4) || bytes % (streams * chunk_bytes) ||
        blocks <= 0)
        return -1;
    hipLaunchKernelGGL(stream_read_multi, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)a,
                       (uint32_t*)b, bytes / streams / 16, streams, chunk_bytes / 16);
    return (int)hipGetLastError();
}

// bf16 sum of `streams` regions of region_bytes each (back to back in a) into b (region_bytes);
// streams a multiple of 4, region_bytes a multiple of chunk_bytes, chunk_bytes of 4 KiB.
extern "C" int bench_stream_reduce(const void* a, void* b, uint64_t region_bytes, uint32_t streams,
                                   uint64_t chunk_bytes, int blocks, void* stream) {
    if (streams == 0 || streams % 4 || chunk_bytes == 0 || chunk_bytes % (16 * 64 * 4) || region_bytes % chunk_bytes ||
        blocks <= 0)
        return -1;
    hipLaunchKernelGGL(stream_reduce_bf16, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)a,
                       (u32x4*)b, region_bytes / 16, streams, chunk_bytes / 16);
    return (int)hipGetLastError();
}
