// Prefill GEMM (Section 2.1; Section 4.3 "GEMM microkernel"):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 MFMA, fp32 accumulate.
//
// Workgroup tile BM x BN = 128 x 256, four waves side by side along N; each
// wave owns 128 rows x 64 columns.  K is walked in steps of BK = 32 rows.
//  - A (fp16) goes global -> registers -> LDS, double buffered and XOR
//    swizzled so the MFMA operand reads are bank-conflict free; the next
//    step's A is in flight while the current one is multiplied, and there is
//    one barrier per step.
//  - B never exists as fp16 in memory: each wave loads the packed atoms of
//    its own 64 columns (one 16-byte load per lane per 32 rows), unpacks and
//    dequantizes them (Eq. 2, rounded once) straight into the register layout
//    of the v_mfma_f32_16x16x32_f16 B operand, and reuses every dequantized
//    operand across its 8 row sub-tiles (Sections 4.1.1 and 4.3: dequantize a
//    weight tile once, reuse it for every activation row).
//  - Tiles are numbered so that each XCD (workgroups are dealt round-robin
//    over the 8 XCDs) works on a contiguous band of tiles sharing rows of A,
//    which then stay in that XCD's L2.
#include "tf_internal.h"

namespace tf {
namespace {

constexpr int kBM = 128, kBN = 256, kBK = 32;
constexpr int kSub = kBK / kAtomK;     // 32-row sub-steps per step
constexpr int kGemmThreads = 256;
constexpr int kXcds = 8;

// LDS position (in 16-byte chunks) of chunk `ch` of A row `row` (kBK halves
// = kChunks chunks per row).  The XOR with row bits spreads the 16 lanes of
// one ds_read_b128 (16 rows, same chunk) over distinct bank groups of the
// 64-bank LDS: rows 4 apart are 64 chunks (one bank cycle) apart.
constexpr int kChunks = kBK / 8;
__device__ __forceinline__ int a_slot(int row, int ch) {
    return kChunks == 8 ? row * 8 + (ch ^ ((row >> 1) & 7)) : row * 4 + (ch ^ ((row >> 2) & 3));
}

template <int BITS>
struct GemmCfg {
    static constexpr int PW = BITS == 4 ? 64 : 32;
    static constexpr int T = PW / 16;                 // columns per lane per atom
    static constexpr int PANELS = 64 / PW;            // panels per wave (64 columns)
    static constexpr int ATOMS = PANELS * (kBK / kAtomK);   // atom loads per wave per step
};

template <int BITS>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int group, int gshift, int64_t s_off, int64_t z_off, int na, int ng,
    int np, int tiles_m, int tiles_n) {
    using Cfg = GemmCfg<BITS>;
    constexpr int PW = Cfg::PW, T = Cfg::T, PANELS = Cfg::PANELS;
    __shared__ __align__(16) u32x4 As[2][kBM * kBK / 8];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 15, kg = lane >> 4;
    const uint32_t magic = magic_reg();

    // XCD-aware tile order: block b runs on XCD b % 8; give XCD x the x-th
    // contiguous band of the row-major tile list.
    const int total = tiles_m * tiles_n;
    const int b = blockIdx.x;
    int tile;
    {
        const int per = total / kXcds, rem = total % kXcds;
        const int x = b % kXcds, i = b / kXcds;
        tile = x * per + min(x, rem) + i;
    }
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int64_t row0 = (int64_t)tm * kBM;
    const int64_t col0 = (int64_t)tn * kBN + wave * 64;      // this wave's 64 columns

    float4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[i][t] = float4_t{0.f, 0.f, 0.f, 0.f};

    // ---- A staging: 128 rows x kBK halves, kAR 16-byte chunks per thread.
    // Rows past M read row M-1 instead (in bounds; those rows are never stored).
    constexpr int kAR = kBM * kChunks / kGemmThreads;
    const uint16_t* arow[kAR];
#pragma unroll
    for (int r = 0; r < kAR; ++r) {
        const int idx = tid + kGemmThreads * r;
        const int64_t grow = min<int64_t>(row0 + idx / kChunks, (int64_t)M - 1);
        arow[r] = A + grow * K + (idx % kChunks) * 8;
    }
    u32x4 av[kAR];
    auto load_a = [&](int step) {
#pragma unroll
        for (int r = 0; r < kAR; ++r) av[r] = *reinterpret_cast<const u32x4*>(arow[r] + step * kBK);
    };
    auto store_a = [&](int buf) {
#pragma unroll
        for (int r = 0; r < kAR; ++r) {
            const int idx = tid + kGemmThreads * r;
            As[buf][a_slot(idx / kChunks, idx % kChunks)] = av[r];
        }
    };

    // ---- B: this wave's packed atoms and its columns' metadata.  Panels past
    // N read the last panel instead (in bounds; their columns are never stored).
    const u32x4* wp[PANELS];
    const uint8_t* sp[PANELS];
    const uint8_t* zp[PANELS];
    bool pvalid[PANELS];
#pragma unroll
    for (int pp = 0; pp < PANELS; ++pp) {
        int64_t panel = col0 / PW + pp;
        pvalid[pp] = panel < np;
        panel = min<int64_t>(panel, np - 1);
        wp[pp] = reinterpret_cast<const u32x4*>(packed) + panel * na * 64 + lane;
        sp[pp] = packed + s_off + (panel * ng * PW + c * T) * 2;
        zp[pp] = packed + z_off + panel * ng * PW + c * T;
    }
    // One step's packed weights and raw metadata: [k sub-step][panel].
    struct BStep {
        u32x4 w[kSub][PANELS];
        uint32_t s[kSub][PANELS][(T + 1) / 2];   // T fp16 scales
        uint32_t z[kSub][PANELS];                // T zero-point bytes (low T bytes)
    };
    auto load_b = [&](int step, BStep& bs) {
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            const int a = step * kSub + j;
            const int g = (a * kAtomK) >> gshift;     // group size is a power of two here
#pragma unroll
            for (int pp = 0; pp < PANELS; ++pp) {
                bs.w[j][pp] = wp[pp][a * 64];
                if constexpr (BITS == 4) {
                    const uint2 sv = *reinterpret_cast<const uint2*>(sp[pp] + g * PW * 2);
                    bs.s[j][pp][0] = sv.x;
                    bs.s[j][pp][1] = sv.y;
                    bs.z[j][pp] = *reinterpret_cast<const uint32_t*>(zp[pp] + g * PW);
                } else {
                    bs.s[j][pp][0] = *reinterpret_cast<const uint32_t*>(sp[pp] + g * PW * 2);
                    bs.z[j][pp] = *reinterpret_cast<const uint16_t*>(zp[pp] + g * PW);
                }
            }
        }
    };

    // One step per trip.  The next step's A is loaded into registers at the top
    // and written to the other LDS buffer after the multiply; the packed B of
    // the next step was loaded one step earlier and moves into place at the
    // bottom, while the loads for the step after it go out.  Prefetch indices
    // are clamped instead of branched on (a clamped load repeats a valid step
    // whose data is never used).
    const int steps = na / kSub;     // the launcher requires K % kBK == 0
    BStep bcur, bnext;
    load_a(0);
    load_b(0, bcur);
    store_a(0);
    load_b(min(1, steps - 1), bnext);
    for (int step = 0; step < steps; ++step) {
        const int buf = step & 1;
        load_a(min(step + 1, steps - 1));
        __syncthreads();               // As[buf] complete; As[buf ^ 1] no longer read
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            half8_t bop[4];
#pragma unroll
            for (int pp = 0; pp < PANELS; ++pp) {
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const uint32_t sh = (bcur.s[j][pp][t / 2] >> (16 * (t & 1))) & 0xFFFFu;
                    const uint32_t sb = pvalid[pp] ? sh : 0u;
                    const uint32_t zb = pvalid[pp] ? (bcur.z[j][pp] >> (8 * t)) & 0xFFu : 0u;
                    const half2_t s2 = as_h2(sb | (sb << 16));
                    if constexpr (BITS == 4)
                        bop[t] = dq_w4_dword(bcur.w[j][pp][t], magic, neg_zero_pair(zb), s2);
                    else
                        bop[pp * T + t] = dq_w8_dwords(bcur.w[j][pp][2 * t], bcur.w[j][pp][2 * t + 1],
                                                       neg_zero_pair(zb), s2);
                }
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const half8_t af = __builtin_bit_cast(half8_t, As[buf][a_slot(16 * i + c, kChunks / kSub * j + kg)]);
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bop[t], acc[i][t], 0, 0, 0);
            }
        }
        store_a(buf ^ 1);
        bcur = bnext;
        load_b(min(step + 2, steps - 1), bnext);
    }

    // ---- epilogue: lane holds column c of each 16x16 block, rows 4 kg + r
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int64_t col = col0 + 16 * t + c;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = row0 + 16 * i + 4 * kg + r;
                if (row < M && col < N)
                    C[row * N + col] = __builtin_bit_cast(uint16_t, (_Float16)acc[i][t][r]);
            }
        }
}

// Generic kernel for the cases the main one leaves out (group size not a
// power of two): 128 x 128 tiles, 32-row steps, single-buffered.
constexpr int kBM1 = 128, kBN1 = 128, kBK1 = 32;

__device__ __forceinline__ int a_swz1(int row, int chunk) { return row * 4 + (chunk ^ ((row >> 2) & 3)); }

template <int BITS>
__global__ __launch_bounds__(kGemmThreads) void gemm_kernel_k32(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int group, int64_t s_off, int64_t z_off, int na, int ng, int np) {
    constexpr int PW = BITS == 4 ? 64 : 32;
    constexpr int T = PW / 16;
    __shared__ u32x4 As[kBM1 * kBK1 / 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int c = lane & 15, kg = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.y * kBM1;
    const int64_t col0 = (int64_t)blockIdx.x * kBN1;

    float4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[i][t] = float4_t{0.f, 0.f, 0.f, 0.f};

    constexpr int kPanels = 64 / PW;
    const uint16_t* sreg = reinterpret_cast<const uint16_t*>(packed + s_off);
    const uint8_t* zreg = packed + z_off;

    for (int a = 0; a < na; ++a) {
        u32x4 av[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int idx = tid + kGemmThreads * r;
            const int row = idx >> 2, ch = idx & 3;
            const int64_t grow = row0 + row;
            av[r] = grow < M ? *reinterpret_cast<const u32x4*>(A + grow * K + (int64_t)a * kBK1 + ch * 8)
                             : u32x4{0u, 0u, 0u, 0u};
        }
        half8_t b[4];
        const int g = (a * kBK1) / group;
#pragma unroll
        for (int pp = 0; pp < kPanels; ++pp) {
            const int64_t panel = col0 / PW + wn * kPanels + pp;
            u32x4 wv = u32x4{0u, 0u, 0u, 0u};
            uint16_t sb[T];
            uint8_t zb[T];
#pragma unroll
            for (int t = 0; t < T; ++t) {
                sb[t] = 0;
                zb[t] = 0;
            }
            if (panel < np) {
                wv = reinterpret_cast<const u32x4*>(packed)[(panel * na + a) * 64 + lane];
                const int64_t meta = (panel * ng + g) * PW + c * T;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    sb[t] = sreg[meta + t];
                    zb[t] = zreg[meta + t];
                }
            }
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const half2_t s2 = as_h2((uint32_t)sb[t] | ((uint32_t)sb[t] << 16));
                if constexpr (BITS == 4)
                    b[t] = dq_w4_dword(wv[t], magic_reg(), neg_zero_pair(zb[t]), s2);
                else
                    b[pp * T + t] = dq_w8_dwords(wv[2 * t], wv[2 * t + 1], neg_zero_pair(zb[t]), s2);
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int idx = tid + kGemmThreads * r;
            As[a_swz1(idx >> 2, idx & 3)] = av[r];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const half8_t af = __builtin_bit_cast(half8_t, As[a_swz1(wm * 64 + 16 * i + c, kg)]);
#pragma unroll
            for (int t = 0; t < 4; ++t)
                acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, b[t], acc[i][t], 0, 0, 0);
        }
    }

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

template <int BITS>
int launch_bits(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                hipStream_t s) {
    const bool pow2_group = (L.group & (L.group - 1)) == 0;
    if (L.K % kBK == 0 && pow2_group) {
        const int tiles_m = (int)((M + kBM - 1) / kBM);
        const int tiles_n = (int)((L.N + kBN - 1) / kBN);
        const int gshift = __builtin_ctz((unsigned)L.group);
        return launch(gemm_kernel<BITS>, dim3((unsigned)(tiles_m * tiles_n)), dim3(kGemmThreads), 0, s,
                      A, pk, C, (int)M, (int)L.K, (int)L.N, L.group, gshift, L.s_off, L.z_off,
                      (int)L.na, (int)L.ng, (int)L.np, tiles_m, tiles_n);
    }
    dim3 grid((unsigned)((L.N + kBN1 - 1) / kBN1), (unsigned)((M + kBM1 - 1) / kBM1));
    return launch(gemm_kernel_k32<BITS>, grid, dim3(kGemmThreads), 0, s, A, pk, C, (int)M, (int)L.K,
                  (int)L.N, L.group, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np);
}

}  // namespace

int64_t gemm_workspace_bytes(const Layout&, int64_t) { return 0; }

int launch_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void*, size_t, hipStream_t s) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    return L.bits == 4 ? launch_bits<4>(L, A, pk, C, M, s) : launch_bits<8>(L, A, pk, C, M, s);
}

}  // namespace tf
