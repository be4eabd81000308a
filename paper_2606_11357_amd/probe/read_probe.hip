// Streaming-read ceiling probe (measurement context for the decode GEMV, not
// part of the matmul library): every byte of a device buffer is read exactly
// once, 16 bytes per lane per load, and nothing is written but one word per
// launch that is stored only if the running XOR of all data equals a fixed
// constant (so the loads cannot be removed).  Workgroup b reads the b-th
// contiguous share of the buffer, as a GEMV workgroup streams its panel;
// each thread keeps UNROLL loads in flight.  Built as its own shared
// library, used only by the benchmark's context figures.
//
//   int tf_probe_read(const void* buf, int64_t bytes, int grid, int block,
//                     int unroll, uint32_t* sink, void* stream)
// buf: device pointer, 16-byte aligned; bytes: a multiple of 16; grid: 1 to
// 65536 workgroups; block: 64, 128, 256, 512 or 1024 threads; unroll: 1, 2,
// 4, 8 or 16; sink: one device word.  Returns 0, -1 on a bad argument (nothing
// launched) or -2 if the launch failed.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int UNROLL>
__global__ void read_kernel(const u32x4* __restrict__ p, int64_t n16, int64_t per_block,
                            uint32_t* __restrict__ sink) {
    const int64_t b0 = (int64_t)blockIdx.x * per_block;
    const int64_t b1 = b0 + per_block < n16 ? b0 + per_block : n16;
    if (b0 >= b1) return;
    const int64_t step = (int64_t)blockDim.x * UNROLL;
    uint32_t acc = 0;
    // every iteration keeps UNROLL loads in flight; a chunk past the share
    // re-reads the share's last chunk (in bounds, a cache hit) and is not
    // counted
    for (int64_t i = b0 + threadIdx.x; i < b1; i += step) {
        u32x4 v[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t j = i + u * (int64_t)blockDim.x;
            v[u] = __builtin_nontemporal_load(p + (j < b1 ? j : b1 - 1));
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
            if (i + u * (int64_t)blockDim.x < b1) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    if (acc == 0x9E3779B9u) sink[0] = acc;
}

}  // namespace

extern "C" int tf_probe_read(const void* buf, int64_t bytes, int grid, int block, int unroll,
                             uint32_t* sink, void* stream) {
    if (!buf || !sink || bytes <= 0 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(buf) & 15) != 0)
        return -1;
    if (grid < 1 || grid > 65536 || (block != 64 && block != 128 && block != 256 && block != 512 && block != 1024))
        return -1;
    const int64_t n16 = bytes / 16;
    const int64_t per = (n16 + grid - 1) / grid;
    const u32x4* p = static_cast<const u32x4*>(buf);
    hipStream_t s = static_cast<hipStream_t>(stream);
    switch (unroll) {
        case 1: read_kernel<1><<<grid, block, 0, s>>>(p, n16, per, sink); break;
        case 2: read_kernel<2><<<grid, block, 0, s>>>(p, n16, per, sink); break;
        case 4: read_kernel<4><<<grid, block, 0, s>>>(p, n16, per, sink); break;
        case 8: read_kernel<8><<<grid, block, 0, s>>>(p, n16, per, sink); break;
        case 16: read_kernel<16><<<grid, block, 0, s>>>(p, n16, per, sink); break;
        default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -2;
}
