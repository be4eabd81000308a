// Prefill GEMM (Section 2.1; Section 4.3 "GEMM microkernel"):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 MFMA, fp32 accumulate.
//
// Each workgroup owns a BM x BN tile of C and walks K in 32-row steps (one
// packed atom per panel).  Per step the A tile goes through LDS; every wave
// loads the packed atom of its own panel straight into registers (one 16-byte
// load per lane), unpacks and dequantizes it (Eq. 2, one rounding) into the
// exact register layout of the v_mfma_f32_16x16x32_f16 B operand, and reuses
// each dequantized operand across all of its M sub-tiles (Section 4.1.1 /
// 4.3: dequantize a weight tile once, reuse it for every activation row).
#include "tf_internal.h"

namespace tf {
namespace {

constexpr int kBM = 128, kBN = 128, kBK = 32;
constexpr int kGemmThreads = 256;

__device__ __forceinline__ int a_swz(int row, int chunk) { return row * 4 + (chunk ^ ((row >> 2) & 3)); }

template <int BITS>
__global__ __launch_bounds__(kGemmThreads) void gemm_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int group, int64_t s_off, int64_t z_off, int na, int ng, int np) {
    constexpr int PW = BITS == 4 ? 64 : 32;
    constexpr int T = PW / 16;
    __shared__ uint4 As[kBM * kBK / 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int c = lane & 15, kg = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.y * kBM;
    const int64_t col0 = (int64_t)blockIdx.x * kBN;

    float4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[i][t] = float4_t{0.f, 0.f, 0.f, 0.f};

    constexpr int kPanels = 64 / PW;    // panels per wave (1 for 4-bit, 2 for 8-bit)
    const uint16_t* sreg = reinterpret_cast<const uint16_t*>(packed + s_off);
    const uint8_t* zreg = packed + z_off;

    for (int a = 0; a < na; ++a) {
        // ---- A tile (BM x 32 halves) global -> registers
        uint4 av[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int idx = tid + kGemmThreads * r;
            const int row = idx >> 2, ch = idx & 3;
            const int64_t grow = row0 + row;
            av[r] = grow < M ? *reinterpret_cast<const uint4*>(A + grow * K + (int64_t)a * kBK + ch * 8)
                             : uint4{0, 0, 0, 0};
        }
        // ---- B: packed atoms of this wave's panels -> dequantized operands
        half8_t b[4];
        const int g = (a * kBK) / group;
#pragma unroll
        for (int pp = 0; pp < kPanels; ++pp) {
            const int64_t panel = col0 / PW + wn * kPanels + pp;
            uint4 wv = uint4{0, 0, 0, 0};
            uint16_t sb[T];
            uint8_t zb[T];
            if (panel < np) {
                wv = reinterpret_cast<const uint4*>(packed)[(panel * na + a) * 64 + lane];
                const int64_t meta = (panel * ng + g) * PW + c * T;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    sb[t] = sreg[meta + t];
                    zb[t] = zreg[meta + t];
                }
            } else {
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    sb[t] = 0;
                    zb[t] = 0;
                }
            }
            const uint32_t wd[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const half2_t s2 = as_h2((uint32_t)sb[t] | ((uint32_t)sb[t] << 16));
                if constexpr (BITS == 4)
                    b[t] = dq_w4_dword(wd[t], neg_zero_pair(zb[t]), s2);
                else
                    b[pp * T + t] = dq_w8_dwords(wd[2 * t], wd[2 * t + 1], neg_zero_pair(zb[t]), s2);
            }
        }
        __syncthreads();   // previous step's LDS reads are done
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int idx = tid + kGemmThreads * r;
            As[a_swz(idx >> 2, idx & 3)] = av[r];
        }
        __syncthreads();
        // ---- MFMA over the wave's 64 x 64 tile
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int lrow = wm * 64 + 16 * i + c;
            const half8_t af = __builtin_bit_cast(half8_t, As[a_swz(lrow, kg)]);
#pragma unroll
            for (int t = 0; t < 4; ++t)
                acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, b[t], acc[i][t], 0, 0, 0);
        }
    }

    // ---- epilogue: lane holds column c of each 16x16 block, rows 4 kg + r
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int64_t col = col0 + wn * 64 + 16 * t + c;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = row0 + wm * 64 + 16 * i + 4 * kg + r;
                if (row < M && col < N)
                    C[row * N + col] = __builtin_bit_cast(uint16_t, (_Float16)acc[i][t][r]);
            }
        }
}

}  // namespace

int64_t gemm_workspace_bytes(const Layout&, int64_t) { return 0; }

int launch_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void*, size_t, hipStream_t s) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    dim3 grid((unsigned)((L.N + kBN - 1) / kBN), (unsigned)((M + kBM - 1) / kBM));
    dim3 block(kGemmThreads);
    if (L.bits == 4)
        return launch(gemm_kernel<4>, grid, block, 0, s, A, pk, C, (int)M, (int)L.K, (int)L.N,
                      L.group, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np);
    return launch(gemm_kernel<8>, grid, block, 0, s, A, pk, C, (int)M, (int)L.K, (int)L.N,
                  L.group, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np);
}

}  // namespace tf
