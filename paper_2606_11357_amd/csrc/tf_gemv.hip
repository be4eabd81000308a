// Decode GEMV (Section 2.1: batch-1 generation makes linear layers
// matrix-vector products; Section 4.3 "GEMV microkernel"; Section 4.4).
//
// y[m, n] = sum_k x[m, k] * s[g, n] * (q[k, n] - z[g, n]),  1 <= M <= 8; the
// same kernel with 16 row slots also serves the GEMM entry points for
// 9 <= M <= 16 (skinny prefill), where the weights, not the matrix cores,
// bound the time.
//
// Mapping (the GPU form of the principle of Section 4.4: every compute unit
// streams its own weight slice, the activations are shared, each workgroup
// owns distinct outputs and no partial sum leaves it):
//  - a workgroup owns a panel of PW output columns and all of K, or, when the
//    panels alone are too few to fill the chip and a workspace is given, one
//    slice of K;
//  - every wave first loads its slice of x and its groups' metadata, then all
//    of its U weight atoms (one 16-byte load per lane per atom), and consumes
//    the atoms in arrival order; x and metadata sit in wave-private LDS;
//  - a lane owns T columns x 8 rows of an atom: one 16-byte activation slice
//    per row of A feeds its T columns (the widening idea of Section 4.3: one
//    activation fragment reused across many outputs).
// Arithmetic (Eq. 2 summed over a group, where s and z are constant):
//    sum_k x (s (q - z)) = s * (sum_k x q - z * sum_k x).
//  - M < 4: codes are read as exact fp16 integers 1024 + q (or 1024 + 16 q,
//    which needs no shift) and dotted with x by v_dot2_f32_f16; the offsets
//    and z are removed per group with the per-lane sums of x.
//  - M >= 4: each weight is dequantized once to fp16 with the GEMM's code,
//    RNE(s (q - z)), and dotted with all M rows of x.
// All sums are fp32.  Lanes sharing a column combine by cross-lane shuffles,
// the waves through LDS; K-slices through a workspace, added by the last
// slice to finish in slice order.  Every order is fixed, so results are
// bitwise reproducible.
#include "tf_internal.h"

#include <algorithm>

namespace tf {
namespace {

template <int BITS, int M, int WAVES, int U>
struct GemvCfg {
    static constexpr int T = BITS == 4 ? 4 : 2;      // columns per lane
    static constexpr int PW = BITS == 4 ? 64 : 32;   // panel width
    static constexpr int ROUND_ATOMS = WAVES * U;    // atoms of one round of the workgroup
    static constexpr int XB = U * kAtomK * 2;        // bytes of one row of x per wave-round
    static constexpr int SB = U * PW * 2;            // scale bytes of up to U groups
    static constexpr int ZB = U * PW;                // zero-point bytes of up to U groups
    static constexpr bool FACT = M < 4;
    static_assert(XB == 512 && SB <= 1024 && ZB <= 512, "one cooperative load per lane each");
};

// One wave's staging area in LDS (private to the wave: no barrier needed).
template <int M, int U, int PW>
struct WaveStage {
    uint64_t x[M][U * kAtomK / 4];     // M rows x U*32 halves
    u32x4 s[U * PW * 2 / 16];
    uint64_t z[U * PW / 8];
};

// APG: atoms per group when known at compile time (4 for G = 128), else 0.
template <int BITS, int M, int WAVES, int U, int APG>
__global__ __launch_bounds__(WAVES * 64) void gemv_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int K, int N, int group, int64_t s_off, int64_t z_off, int na, int ng, int S, int AS,
    float* __restrict__ ws_part, uint32_t* __restrict__ ws_cnt, int mr) {
    // mr <= M rows of A and C exist; row slots past them re-read row mr - 1
    // (in bounds) and are never stored.
    using Cfg = GemvCfg<BITS, M, WAVES, U>;
    static_assert(APG == 0 || U % APG == 0, "a wave's run must hold whole groups");
    constexpr int T = Cfg::T, PW = Cfg::PW, RA = Cfg::ROUND_ATOMS;
    constexpr bool FACT = Cfg::FACT;
    constexpr int NT = WAVES * 64;
    using Stage = WaveStage<M, U, PW>;
    union Smem {
        Stage st[WAVES];
        float red[WAVES][M][PW];
    };
    __shared__ __align__(16) Smem sm;

    const int p = blockIdx.x;
    const int split = blockIdx.y;                       // K-slice of this workgroup
    const int a_begin = split * AS;
    const int a_end = min(na, a_begin + AS);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar) index math
    const int c = lane & 15, kg = lane >> 4;
    const int apg = APG > 0 ? APG : group / kAtomK;
    const uint32_t magic = magic_reg();
    const u32x4* wpanel = reinterpret_cast<const u32x4*>(packed) + (int64_t)p * na * 64 + lane;
    const uint8_t* spanel = packed + s_off + (int64_t)p * ng * PW * 2;
    const uint8_t* zpanel = packed + z_off + (int64_t)p * ng * PW;
    const int64_t s_last = ((int64_t)ng * PW * 2 - 16);     // last 16-byte slot of the panel's scales
    const int64_t z_last = ((int64_t)ng * PW - 8);
    const int rounds = (a_end - a_begin + RA - 1) / RA;
    Stage& st = sm.st[wave];

    float y[M][T];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int t = 0; t < T; ++t) y[m][t] = 0.f;

    // Loads of one round: first the wave's slice of x and its groups'
    // metadata (small), then its U weight atoms.  Addresses are clamped into
    // the panel so every load is in bounds and the code stays branch-free;
    // atoms past K are skipped at use.
    struct Buf {
        uint64_t xr[M];
        u32x4 sr;
        uint64_t zr;
        u32x4 w[U];
    };
    auto issue = [&](int r, Buf& b) {
        const int a0 = a_begin + r * RA + wave * U;
        const int k0 = min(a0, na - 1) * kAtomK;
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const int k = min(k0 + 4 * lane, K - 4);
            b.xr[m] = *reinterpret_cast<const uint64_t*>(A + (int64_t)min(m, mr - 1) * K + k);
        }
        const int g0 = min(a0, na - 1) / apg;
        b.sr = *reinterpret_cast<const u32x4*>(spanel + min((int64_t)g0 * PW * 2 + 16 * lane, s_last));
        b.zr = *reinterpret_cast<const uint64_t*>(zpanel + min((int64_t)g0 * PW + 8 * lane, z_last));
#pragma unroll
        for (int i = 0; i < U; ++i)
            b.w[i] = __builtin_nontemporal_load(wpanel + (int64_t)min(a0 + i, na - 1) * 64);
    };

    auto consume = [&](int r, Buf& b) {
        const int a0 = a_begin + r * RA + wave * U;
        if (a0 >= a_end) return;
        const int g0 = a0 / apg;
        int pos = a0 - g0 * apg;      // atom a0's place inside its group
        int gl = 0;                   // current group, relative to g0
        // stage this wave's x slice and metadata (wave-private LDS)
#pragma unroll
        for (int m = 0; m < M; ++m) st.x[m][lane] = b.xr[m];
        if (16 * lane < Cfg::SB) st.s[lane] = b.sr;
        if (8 * lane < Cfg::ZB) st.z[lane] = b.zr;

        float alo[M][T], ahi[M][T], sxlo[M], sxhi[M];
        auto reset = [&]() {
#pragma unroll
            for (int m = 0; m < M; ++m) {
                sxlo[m] = 0.f;
                sxhi[m] = 0.f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    alo[m][t] = 0.f;
                    ahi[m][t] = 0.f;
                }
            }
        };
        reset();
        const half2_t ones = {(_Float16)1.0f, (_Float16)1.0f};
        const uint8_t* sbytes = reinterpret_cast<const uint8_t*>(st.s);
        const uint8_t* zbytes = reinterpret_cast<const uint8_t*>(st.z);

#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int a = a0 + i;
            if (a >= a_end) break;
            u32x4 xv[M];
#pragma unroll
            for (int m = 0; m < M; ++m)
                xv[m] = *reinterpret_cast<const u32x4*>(&st.x[m][(i * kAtomK + 8 * kg) / 4]);
            const uint32_t wd[4] = {b.w[i][0], b.w[i][1], b.w[i][2], b.w[i][3]};
            if constexpr (!FACT) {
                // dequantize once per weight (the GEMM's code: RNE(s (q - z))) and
                // let every row of A reuse it
                const uint8_t* zp = zbytes + gl * PW + c * T;
                const uint16_t* sp = reinterpret_cast<const uint16_t*>(sbytes + (gl * PW + c * T) * 2);
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const uint32_t sb = sp[t];
                    const half2_t s2 = as_h2(sb | (sb << 16));
                    half8_t w8;
                    const uint32_t nz = neg_zero_pair(zp[t]);
                    if constexpr (BITS == 4)
                        w8 = dq_w4_dword(wd[t], magic, nz, neg_zero64_pair(nz), s2);
                    else
                        w8 = dq_w8_dwords(wd[2 * t], wd[2 * t + 1], nz, s2);
                    const half2_t w2[4] = {{w8[0], w8[1]}, {w8[2], w8[3]}, {w8[4], w8[5]}, {w8[6], w8[7]}};
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        float v = y[m][t];
#pragma unroll
                        for (int pr = 0; pr < 4; ++pr)
                            v = __builtin_amdgcn_fdot2(w2[pr], as_h2(xv[m][pr]), v, false);
                        y[m][t] = v;
                    }
                }
                if (APG > 0 ? (i + 1) % (APG > 0 ? APG : 1) == 0 : ++pos == apg) {
                    pos = 0;
                    ++gl;
                }
                continue;
            }
#pragma unroll
            for (int t = 0; t < T; ++t) {
                uint32_t P[4];
                if constexpr (BITS == 4) {
                    w4_code_pairs_x16(wd[t], magic, P);
                } else {
                    w8_code_pairs(wd[2 * t], P);
                    w8_code_pairs(wd[2 * t + 1], P + 2);
                }
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const uint32_t xd[4] = {xv[m][0], xv[m][1], xv[m][2], xv[m][3]};
                    float lo = alo[m][t], hi = ahi[m][t];
                    lo = __builtin_amdgcn_fdot2(as_h2(P[0]), as_h2(xd[0]), lo, false);
                    lo = __builtin_amdgcn_fdot2(as_h2(P[2]), as_h2(xd[2]), lo, false);
                    if constexpr (BITS == 4) {
                        hi = __builtin_amdgcn_fdot2(as_h2(P[1]), as_h2(xd[1]), hi, false);
                        hi = __builtin_amdgcn_fdot2(as_h2(P[3]), as_h2(xd[3]), hi, false);
                    } else {
                        lo = __builtin_amdgcn_fdot2(as_h2(P[1]), as_h2(xd[1]), lo, false);
                        lo = __builtin_amdgcn_fdot2(as_h2(P[3]), as_h2(xd[3]), lo, false);
                    }
                    alo[m][t] = lo;
                    ahi[m][t] = hi;
                }
            }
            if constexpr (FACT) {
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const uint32_t xd[4] = {xv[m][0], xv[m][1], xv[m][2], xv[m][3]};
                    float lo = sxlo[m], hi = sxhi[m];
                    lo = __builtin_amdgcn_fdot2(as_h2(xd[0]), ones, lo, false);
                    lo = __builtin_amdgcn_fdot2(as_h2(xd[2]), ones, lo, false);
                    if constexpr (BITS == 4) {
                        hi = __builtin_amdgcn_fdot2(as_h2(xd[1]), ones, hi, false);
                        hi = __builtin_amdgcn_fdot2(as_h2(xd[3]), ones, hi, false);
                    } else {
                        lo = __builtin_amdgcn_fdot2(as_h2(xd[1]), ones, lo, false);
                        lo = __builtin_amdgcn_fdot2(as_h2(xd[3]), ones, lo, false);
                    }
                    sxlo[m] = lo;
                    sxhi[m] = hi;
                }
            }
            // close the group at its last atom or at the end of this wave's run
            // (with APG known, runs start on group boundaries: see plan_gemv)
            const bool group_end = APG > 0 ? (i + 1) % (APG > 0 ? APG : 1) == 0 : ++pos == apg;
            const bool run_end = APG > 0 ? false : (i == U - 1 || a + 1 == a_end);
            if (group_end || run_end || (APG > 0 && a + 1 == a_end)) {
                const uint16_t* sp = reinterpret_cast<const uint16_t*>(sbytes + (gl * PW + c * T) * 2);
                const uint8_t* zp = zbytes + gl * PW + c * T;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const float s = (float)__builtin_bit_cast(_Float16, sp[t]);
                    if constexpr (FACT) {
                        const float zf = (float)zp[t];
#pragma unroll
                        for (int m = 0; m < M; ++m) {
                            float v;
                            if constexpr (BITS == 4) {
                                v = fmaf(ahi[m][t], 0.0625f, alo[m][t]);
                                v = fmaf(-(1024.f + zf), sxlo[m], v);
                                v = fmaf(-(64.f + zf), sxhi[m], v);
                            } else {
                                v = fmaf(-(1024.f + zf), sxlo[m], alo[m][t]);
                            }
                            y[m][t] = fmaf(s, v, y[m][t]);
                        }
                    }
                }
                reset();
            }
            if (group_end) {
                pos = 0;
                ++gl;
            }
        }
    };

    // One round covers K <= 32 * U * WAVES; larger K walks several rounds,
    // each issuing its loads right before it consumes them.
    for (int r = 0; r < rounds; ++r) {
        Buf b;
        issue(r, b);
        consume(r, b);
    }

    // Lanes c, c+16, c+32, c+48 hold the same columns: combine over kg.
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int t = 0; t < T; ++t) {
            float v = y[m][t];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            y[m][t] = v;
        }
    __syncthreads();   // staging storage becomes the reduction buffer
    if (kg == 0) {
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < T; ++t) sm.red[wave][m][c + 16 * t] = y[m][t];
    }
    __syncthreads();
    if (S == 1) {
        for (int i = tid; i < M * PW; i += NT) {
            const int m = i / PW, col = i % PW;
            const int n = p * PW + col;
            if (n < N && m < mr) {
                float v = 0.f;
#pragma unroll
                for (int w = 0; w < WAVES; ++w) v += sm.red[w][m][col];
                C[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
            }
        }
        return;
    }
    // Split K: park this slice's partial sums, and let the last slice of the
    // panel to arrive add all of them in slice order (fixed order: bitwise
    // reproducible whichever workgroup comes last) and write the output.
    // Partials and counters are touched only by agent-scope atomic accesses,
    // which write through / read past the per-XCD L2; the wait for the
    // partial stores to complete orders them before the arrival count.  No
    // device-wide fence is used: on this part it would write back the whole
    // L2 of the XCD from every workgroup.
    float* part = ws_part + (int64_t)p * S * M * PW;
    for (int i = tid; i < M * PW; i += NT) {
        const int m = i / PW, col = i % PW;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) v += sm.red[w][m][col];
        __hip_atomic_store(&part[split * M * PW + i], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);      // this thread's partial stores have completed
    __syncthreads();
    __shared__ int last;
    if (tid == 0)
        last = __hip_atomic_fetch_add(&ws_cnt[p], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               (uint32_t)(S - 1);
    __syncthreads();
    if (!last) return;
    for (int i = tid; i < M * PW; i += NT) {
        const int m = i / PW, col = i % PW;
        const int n = p * PW + col;
        float v = 0.f;
        for (int s2 = 0; s2 < S; ++s2)
            v += __hip_atomic_load(&part[s2 * M * PW + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (n < N && m < mr) C[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
    }
    if (tid == 0)   // leave the counter at zero for the next call
        __hip_atomic_store(&ws_cnt[p], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Launch plan.  A workgroup of WAVES waves owns one panel and one K-slice of
// AS atoms.  K is split only when few panels (output columns) each carry much
// work: the partial-sum round trip through the workspace (store, arrival
// count, reload: a few microseconds of latency) pays only when it spreads a
// long stream of atoms, or many rows of A, over more compute units.  The
// work measure na * max(1, M / 2) and its threshold come from kernel-trace
// timings of both forms on MI355X (e.g. K=4096 with 64 or 128 panels at M=1:
// one pass is faster; K=14336 with 64 panels: the split is).
struct GemvPlan {
    int waves, S, AS;
};
constexpr int kGemvU = 8, kMaxSplit = 32;
constexpr int64_t kSplitBelowPanels = 192;      // split K only below this many panels ...
constexpr int64_t kSplitFromWork = 256;         // ... carrying at least this much work each
constexpr int64_t kTargetWorkgroups = 256;

inline int gemv_waves(int64_t M) { return M == 1 ? 16 : 8; }

inline GemvPlan plan_gemv(const Layout& L, int64_t M) {
    const int waves = gemv_waves(M);
    const int64_t ra = (int64_t)waves * kGemvU;
    const int64_t apg = L.group / kAtomK;
    int64_t S = 1;
    if (L.np < kSplitBelowPanels && L.na * std::max<int64_t>(1, M / 2) >= kSplitFromWork) {
        S = (kTargetWorkgroups + L.np - 1) / L.np;
        S = std::min<int64_t>(S, (L.na + ra - 1) / ra);
        S = std::min<int64_t>(S, kMaxSplit);
        S = std::max<int64_t>(S, 1);
    }
    int64_t AS = (L.na + S - 1) / S;
    AS = (AS + apg - 1) / apg * apg;     // slices start on group boundaries
    S = (L.na + AS - 1) / AS;            // no empty slice
    return {waves, (int)S, (int)AS};
}

// Workspace layout: arrival counters first, at a fixed place and sized for
// the largest panel count any shape can have, so every call finds its
// counters where an earlier call (of any shape) left them at zero; then the
// per-slice partial sums, which are always written before they are read.


template <int BITS, int M, int APG>
int launch_g(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, void* ws,
             int mr, hipStream_t s) {
    constexpr int WAVES = M == 1 ? 16 : 8;
    const GemvPlan sp = plan_gemv(L, M);
    const bool split = ws != nullptr && sp.S > 1;
    uint32_t* cnt = split ? static_cast<uint32_t*>(ws) : nullptr;
    float* part = split ? reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsCounterBytes) : nullptr;
    const int S = split ? sp.S : 1;
    const int AS = split ? sp.AS : (int)L.na;
    return launch(gemv_kernel<BITS, M, WAVES, kGemvU, APG>, dim3((unsigned)L.np, (unsigned)S),
                  dim3(WAVES * 64), 0, s, A, pk, C, (int)L.K, (int)L.N, L.group, L.s_off, L.z_off,
                  (int)L.na, (int)L.ng, S, AS, part, cnt, mr);
}

template <int BITS, int M>
int launch_m(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, void* ws,
             hipStream_t s, int mr = M) {
    // group 128 (the AWQ default) gets group boundaries fixed at compile time
    if (L.group == 128) return launch_g<BITS, M, 4>(L, A, pk, C, ws, mr, s);
    return launch_g<BITS, M, 0>(L, A, pk, C, ws, mr, s);
}

template <int BITS>
int launch_bits(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    switch (M) {
        case 1: return launch_m<BITS, 1>(L, A, pk, C, ws, s);
        case 2: return launch_m<BITS, 2>(L, A, pk, C, ws, s);
        case 3: return launch_m<BITS, 3>(L, A, pk, C, ws, s);
        case 4: return launch_m<BITS, 4>(L, A, pk, C, ws, s);
        case 5: return launch_m<BITS, 5>(L, A, pk, C, ws, s);
        case 6: return launch_m<BITS, 6>(L, A, pk, C, ws, s);
        case 7: return launch_m<BITS, 7>(L, A, pk, C, ws, s);
        case 8: return launch_m<BITS, 8>(L, A, pk, C, ws, s);
    }
    if (M <= kSkinnyMaxM) return launch_m<BITS, kSkinnyMaxM>(L, A, pk, C, ws, s, (int)M);
    return TF_ERR_ARG;
}

}  // namespace

int64_t gemv_workspace_bytes(const Layout& L, int64_t M) {
    if (M < 1 || M > kSkinnyMaxM) return 0;
    const int64_t slots = M <= TF_GEMV_MAX_M ? M : kSkinnyMaxM;    // row slots of the kernel
    const GemvPlan sp = plan_gemv(L, slots);
    if (sp.S <= 1) return 0;
    return kWsCounterBytes + align256((int64_t)L.np * sp.S * slots * L.pw * 4);
}

int launch_gemv(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s) {
    return L.bits == 4 ? launch_bits<4>(L, A, packed, C, M, ws, s)
                       : launch_bits<8>(L, A, packed, C, M, ws, s);
}

}  // namespace tf
