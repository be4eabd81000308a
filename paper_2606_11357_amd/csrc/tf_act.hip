// Gated activation between the two GEMMs of a transformer MLP (the
// layer-level composite around the fused matmul; not part of the paper's
// method): H = silu(G) * U with G, U the two halves of one [M, 2N] fp16 or
// bfloat16 matrix, the output of a GEMM whose weight concatenates the gate
// and up projections along N.  HBM-bound: 6 bytes moved per output.
#include "tf_internal.h"

namespace tf {
namespace {

typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// One thread per 8 consecutive outputs of a row: two 16-byte loads, one
// 16-byte store.  silu(g) = g / (1 + e^-g) in fp32; the product is rounded
// to the element type once (nearest even).
template <bool BF>
__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t* __restrict__ gu,
                                                       uint16_t* __restrict__ h, int64_t M,
                                                       int64_t N) {
    const int64_t per_row = N / 8;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= M * per_row) return;
    const int64_t m = i / per_row, c = (i - m * per_row) * 8;
    const u16x8 g = *reinterpret_cast<const u16x8*>(gu + m * 2 * N + c);
    const u16x8 u = *reinterpret_cast<const u16x8*>(gu + m * 2 * N + N + c);
    u16x8 out;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float gf = scale_f32<BF>(g[j]);     // the 16-bit pattern as fp32, exact
        const float uf = scale_f32<BF>(u[j]);
        const float silu = gf / (1.0f + expf(-gf));
        out[j] = round_out<BF>(silu * uf);
    }
    *reinterpret_cast<u16x8*>(h + m * N + c) = out;
}

}  // namespace

int launch_silu_mul(const uint16_t* gu, int64_t M, int64_t N, uint16_t* h, hipStream_t s, bool bf) {
    const int64_t threads = M * (N / 8);
    const int64_t blocks = (threads + 255) / 256;
    if (bf) return launch(silu_mul_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, s, gu, h, M, N);
    return launch(silu_mul_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, s, gu, h, M, N);
}

}  // namespace tf
