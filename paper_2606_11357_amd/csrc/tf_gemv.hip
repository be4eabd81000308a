// Decode GEMV (Section 2.1: batch-1 generation makes linear layers
// matrix-vector products; Section 4.3 "GEMV microkernel"; Section 4.4).
//
// y[m, n] = sum_k x[m, k] * s[g, n] * (q[k, n] - z[g, n]),  1 <= M <= 8.
//
// Mapping (the GPU form of the principle of Section 4.4: every compute unit
// streams its own weight slice, activations are shared, each workgroup owns
// distinct outputs and no partial sums leave it):
//  - one workgroup per panel of PW columns, all of K;
//  - each wave streams whole 1 KiB atoms (one 16-byte load per lane);
//  - a lane owns T columns x 8 rows of an atom, so one 16-byte slice of x per
//    activation row is reused across its T columns (the widening idea of
//    Section 4.3: one activation fragment feeds many outputs);
//  - per group the lane accumulates sum_k x * (q - z) with v_dot2_f32_f16 on
//    exact fp16 integer pairs, then applies s once per group (Eq. 2 factored
//    over the group: s is constant on it);
//  - the four lanes sharing a column combine with cross-lane shuffles, the
//    waves through LDS, in a fixed order (bitwise reproducible).
#include "tf_internal.h"

namespace tf {
namespace {

constexpr int kGemvThreads = 256;
constexpr int kGemvWaves = kGemvThreads / 64;

template <int BITS, int M>
__global__ __launch_bounds__(kGemvThreads) void gemv_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int K, int N, int group, int64_t s_off, int64_t z_off, int na, int ng) {
    constexpr int T = BITS == 4 ? 4 : 2;         // columns per lane
    constexpr int PW = BITS == 4 ? 64 : 32;      // panel width
    const int p = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int c = lane & 15, kg = lane >> 4;

    float acc[M][T];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int t = 0; t < T; ++t) acc[m][t] = 0.f;

    const uint4* wbase = reinterpret_cast<const uint4*>(packed) + (int64_t)p * na * 64 + lane;
    const uint16_t* sbase = reinterpret_cast<const uint16_t*>(packed + s_off) + (int64_t)p * ng * PW + c * T;
    const uint8_t* zbase = packed + z_off + (int64_t)p * ng * PW + c * T;
    const int atoms_per_group = group / kAtomK;

    // Each wave takes whole groups; inside a group it walks the group's atoms.
    for (int g = wave; g < ng; g += kGemvWaves) {
        float part[M][T];
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < T; ++t) part[m][t] = 0.f;

        uint32_t negz[T];
        _Float16 sc[T];
        {
            const uint16_t* sp = sbase + (int64_t)g * PW;
            const uint8_t* zp = zbase + (int64_t)g * PW;
#pragma unroll
            for (int t = 0; t < T; ++t) {
                sc[t] = __builtin_bit_cast(_Float16, sp[t]);
                negz[t] = neg_zero_pair(zp[t]);
            }
        }
        for (int ai = 0; ai < atoms_per_group; ++ai) {
            const int a = g * atoms_per_group + ai;
            const uint4 wv = wbase[(int64_t)a * 64];
            const int k0 = a * kAtomK + 8 * kg;
            uint4 xv[M];
#pragma unroll
            for (int m = 0; m < M; ++m)
                xv[m] = *reinterpret_cast<const uint4*>(A + (int64_t)m * K + k0);
            const uint32_t wd[4] = {wv.x, wv.y, wv.z, wv.w};
            if constexpr (BITS == 4) {
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    uint32_t cp[4];
                    w4_code_pairs(wd[t], cp);
                    half2_t d[4];
#pragma unroll
                    for (int pr = 0; pr < 4; ++pr) d[pr] = as_h2(cp[pr]) + as_h2(negz[t]);
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        const uint32_t xd[4] = {xv[m].x, xv[m].y, xv[m].z, xv[m].w};
                        float v = part[m][t];
#pragma unroll
                        for (int pr = 0; pr < 4; ++pr)
                            v = __builtin_amdgcn_fdot2(d[pr], as_h2(xd[pr]), v, false);
                        part[m][t] = v;
                    }
                }
            } else {
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    uint32_t cp[4];
                    w8_code_pairs(wd[2 * t], cp);
                    w8_code_pairs(wd[2 * t + 1], cp + 2);
                    half2_t d[4];
#pragma unroll
                    for (int pr = 0; pr < 4; ++pr) d[pr] = as_h2(cp[pr]) + as_h2(negz[t]);
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        const uint32_t xd[4] = {xv[m].x, xv[m].y, xv[m].z, xv[m].w};
                        float v = part[m][t];
#pragma unroll
                        for (int pr = 0; pr < 4; ++pr)
                            v = __builtin_amdgcn_fdot2(d[pr], as_h2(xd[pr]), v, false);
                        part[m][t] = v;
                    }
                }
            }
        }
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < T; ++t) acc[m][t] = fmaf((float)sc[t], part[m][t], acc[m][t]);
    }

    // Lanes c, c+16, c+32, c+48 hold the same columns: combine over kg.
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int t = 0; t < T; ++t) {
            float v = acc[m][t];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            acc[m][t] = v;
        }

    __shared__ float red[kGemvWaves][M][PW];
    if (kg == 0) {
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < T; ++t) red[wave][m][c + 16 * t] = acc[m][t];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < M * PW; i += kGemvThreads) {
        const int m = i / PW, col = i % PW;
        const int n = p * PW + col;
        if (n < N) {
            float v = 0.f;
#pragma unroll
            for (int w = 0; w < kGemvWaves; ++w) v += red[w][m][col];
            C[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
        }
    }
}

template <int BITS>
int launch_bits(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                hipStream_t s) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    dim3 grid((unsigned)L.np), block(kGemvThreads);
    int K = (int)L.K, N = (int)L.N, G = L.group, na = (int)L.na, ng = (int)L.ng;
    switch (M) {
#define TF_GEMV_CASE(MM)                                                                        \
    case MM:                                                                                    \
        return launch(gemv_kernel<BITS, MM>, grid, block, 0, s, A, pk, C, K, N, G, L.s_off,     \
                      L.z_off, na, ng);
        TF_GEMV_CASE(1)
        TF_GEMV_CASE(2)
        TF_GEMV_CASE(3)
        TF_GEMV_CASE(4)
        TF_GEMV_CASE(5)
        TF_GEMV_CASE(6)
        TF_GEMV_CASE(7)
        TF_GEMV_CASE(8)
#undef TF_GEMV_CASE
    }
    return TF_ERR_ARG;
}

}  // namespace

int launch_gemv(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                hipStream_t s) {
    return L.bits == 4 ? launch_bits<4>(L, A, packed, C, M, s) : launch_bits<8>(L, A, packed, C, M, s);
}

}  // namespace tf
