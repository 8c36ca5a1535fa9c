// bench_stream.hip -- STREAM-style reference kernels for bench.py (not part of the library).
//
// They measure what a plain HIP kernel reaches on this device for the three access patterns a
// collective is made of: a contiguous copy (read once, write once), a read-only sweep and a
// write-only sweep. bench.py reports the collectives' effective bandwidth against the copy
// figure as "% of the measured copy ceiling", beside the 8 TB/s datasheet peak.
//
// Every wavefront of a grid of `blocks` workgroups (4 wavefronts each) copies chunks of
// `chunk_bytes` in turn (chunk c goes to wavefront c mod W), 4 x 16 bytes per lane per step,
// with non-temporal loads and stores.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kU = 4;

__global__ void __launch_bounds__(256) stream_copy(const u32x4* a, u32x4* b, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    for (uint64_t c = wave; c < n16 / c16; c += nw) {
        const u32x4* s = a + c * c16;
        u32x4* d = b + c * c16;
        for (uint64_t i = 0; i < c16; i += 64 * kU) {
            u32x4 v[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
            for (int u = 0; u < kU; ++u) __builtin_nontemporal_store(v[u], d + i + u * 64 + lane);
        }
    }
}

__global__ void __launch_bounds__(256) stream_read(const u32x4* a, uint32_t* sink, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    uint32_t acc = 0;
    for (uint64_t c = wave; c < n16 / c16; c += nw) {
        const u32x4* s = a + c * c16;
        for (uint64_t i = 0; i < c16; i += 64 * kU) {
            u32x4 v[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
            for (int u = 0; u < kU; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;  // keeps the loads; practically never stores
}

__global__ void __launch_bounds__(256) stream_write(u32x4* b, uint64_t n16, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    u32x4 v = {lane, 1u, 2u, 3u};
    for (uint64_t c = wave; c < n16 / c16; c += nw)
        for (uint64_t i = 0; i < c16; i += 64 * kU)
#pragma unroll
            for (int u = 0; u < kU; ++u) __builtin_nontemporal_store(v, b + c * c16 + i + u * 64 + lane);
}

// Read-only sweep of `streams` regions at once, the access pattern of an N-source reduction:
// `a` holds the regions back to back; wavefront w reads chunk c = w, w + W, ... of every region
// in turn (the same offset in each), 4 x 16 bytes per lane per step.
__global__ void __launch_bounds__(256) stream_read_multi(const u32x4* a, uint32_t* sink, uint64_t region16,
                                                         uint32_t streams, uint64_t c16) {
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t wave = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6), nw = (uint64_t)gridDim.x * 4;
    uint32_t acc = 0;
    for (uint64_t c = wave; c < region16 / c16; c += nw) {
        for (uint32_t r = 0; r < streams; ++r) {
            const u32x4* s = a + r * region16 + c * c16;
            for (uint64_t i = 0; i < c16; i += 64 * kU) {
                u32x4 v[kU];
#pragma unroll
                for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(s + i + u * 64 + lane);
#pragma unroll
                for (int u = 0; u < kU; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
            }
        }
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

}  // namespace

// kind 0 copy (a -> b), 1 read-only (a; b receives at most one word), 2 write-only (b).
// bytes must be a multiple of chunk_bytes, and chunk_bytes of 4 KiB. Returns a hipError_t, or
// -1 for arguments the kernels cannot take.
extern "C" int bench_stream(int kind, const void* a, void* b, uint64_t bytes, uint64_t chunk_bytes, int blocks,
                            void* stream) {
    if (chunk_bytes == 0 || chunk_bytes % (16 * 64 * kU) || bytes % chunk_bytes || blocks <= 0 || kind < 0 || kind > 2)
        return -1;
    const uint64_t n16 = bytes / 16, c16 = chunk_bytes / 16;
    hipStream_t s = (hipStream_t)stream;
    if (kind == 0) hipLaunchKernelGGL(stream_copy, dim3(blocks), dim3(256), 0, s, (const u32x4*)a, (u32x4*)b, n16, c16);
    else if (kind == 1) hipLaunchKernelGGL(stream_read, dim3(blocks), dim3(256), 0, s, (const u32x4*)a, (uint32_t*)b, n16, c16);
    else hipLaunchKernelGGL(stream_write, dim3(blocks), dim3(256), 0, s, (u32x4*)b, n16, c16);
    return (int)hipGetLastError();
}

// Read-only sweep of `streams` regions of bytes / streams each (see stream_read_multi); b receives
// at most one word. bytes must be a multiple of streams * chunk_bytes, and chunk_bytes of 4 KiB.
extern "C" int bench_stream_multi(const void* a, void* b, uint64_t bytes, uint32_t streams, uint64_t chunk_bytes,
                                  int blocks, void* stream) {
    if (streams == 0 || chunk_bytes == 0 || chunk_bytes % (16 * 64 * kU) || bytes % (streams * chunk_bytes) ||
        blocks <= 0)
        return -1;
    hipLaunchKernelGGL(stream_read_multi, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)a,
                       (uint32_t*)b, bytes / streams / 16, streams, chunk_bytes / 16);
    return (int)hipGetLastError();
}
