// Decode GEMV (Section 2.1: batch-1 generation makes linear layers
// matrix-vector products; Section 4.3 "GEMV microkernel"; Section 4.4).
//
// y[m, n] = sum_k x[m, k] * s[g, n] * (q[k, n] - z[g, n]),  1 <= M <= 8, on
// the vector ALU only.  The same streaming kernel with 16, 32 or 64 row
// slots serves the GEMM entry points for few rows (skinny prefill,
// 4 <= M <= 64) on the matrix cores (v_mfma_f32_16x16x32_f16 / _bf16), where
// the weights, not the matrix cores, bound the time.  With 16 or 32 slots the
// codes themselves (exact 16-bit integers o + q) are the B operand: per group
// the matrix core forms sum A * (o + q) and, against an operand of ones, the
// row sums of A, and the group closes with s * (acc - (o + z) * rowsum), which
// leaves the vector ALU a few instructions per dword instead of the whole
// dequantization.  With 64 slots (too many group sums for the registers) each
// weight is dequantized with the GEMM's code and fed to the matrix core.
//
// Mapping (the GPU form of the principle of Section 4.4: every compute unit
// streams its own weight slice, the activations are shared, each workgroup
// owns distinct outputs and no partial sum leaves it):
//  - a workgroup owns a panel of PW output columns and all of K, or, when the
//    panels alone are too few to fill the chip and a workspace is given, one
//    slice of K;
//  - each wave streams a contiguous run of the slice's atoms (one 16-byte
//    load per lane per atom) through a small ring of registers: the atom D
//    places ahead is requested as each one is consumed.  Issuing a wave's
//    whole share at once queues the entire transfer in the memory system
//    within about a microsecond, and the first-needed bytes then arrive
//    anywhere in it while the vector units wait;
//  - the run is consumed in rounds of U atoms; a round's slice of x and its
//    groups' metadata are loaded one round ahead and staged in wave-private
//    LDS;
//  - a lane owns T columns x 8 rows of an atom: one 16-byte activation slice
//    per row of A feeds its T columns (the widening idea of Section 4.3: one
//    activation fragment reused across many outputs).
// Arithmetic (Eq. 2 summed over a group, where s and z are constant):
//    sum_k x (s (q - z)) = s * (sum_k x c - sum_k x o - z * sum_k x),
// with c = o + q the code read as an exact fp16 integer and o its offset.
//  - M <= 4 ("factored"): 4-bit codes are read as 1024 + q (rows 0,1,4,5 of a
//    lane's 8) or 64 + q (rows 2,3,6,7), 8-bit codes as 1024 + q, and dotted
//    with x by v_dot2_f32_f16 into one fp32 sum per column; the offsets and z
//    are removed once per group with sums of x that each wave forms once per
//    round for all of its columns.
//  - M > 4: each weight is dequantized once to fp16 with the GEMM's code,
//    RNE(s (q - z)), and dotted with all M rows of x.
// All sums are fp32.  Lanes sharing a column combine by cross-lane shuffles,
// the waves through LDS; K-slices through a workspace, added by the last
// slice to finish in slice order.  Every order is fixed, so results are
// bitwise reproducible.
#include "tf_internal.h"

#include <algorithm>

namespace tf {
namespace {

constexpr int kGemvU = 8;        // atoms per wave per round
constexpr int kFactMaxM = 4;     // rows up to which the factored form runs

template <int BITS, int M>
struct GemvCfg {
    static constexpr int T = BITS == 4 ? 4 : 2;      // columns per lane
    static constexpr int PW = BITS == 4 ? 64 : 32;   // panel width
    static constexpr bool FACT = M <= kFactMaxM;
    // 16, 32 or 64 row slots (GEMM calls with few rows): matrix cores, A
    // read per atom, MB blocks of 16 rows
    static constexpr bool MF = M > TF_GEMV_MAX_M;
    static constexpr int MB = MF ? M / 16 : 1;
    // matrix-core factored form (16 or 32 row slots): the codes themselves
    // are the B operand and the scale and zero-point are applied per group
    // (64 slots keep the dequantized operand: the group sums would not fit
    // in registers)
    static constexpr bool MFF = MF && M <= 32;
    static constexpr int XR = MF ? 1 : M;             // rows of x staged in LDS
    static constexpr int CR = FACT ? M : 1;           // rows of slice sums
};

// One wave's staging area in LDS (private to the wave: no barrier needed).
template <int XR, int CR, int PW>
struct WaveStage {
    uint64_t x[XR][64];                 // lane l holds k = 4l..4l+3 of the round's 256
    float2_t cs[CR][64];                // factored form: lane l: sums of 8-k slice l / 2
    u32x4 s[kGemvU * PW * 2 / 16];      // scales of up to U groups
    uint64_t z[kGemvU * PW / 8];        // zero-points of up to U groups
};

// SEG > 0: segments (atoms summed before the scale is applied) have SEG
// atoms, fixed at compile time (one group of 32 SEG rows); SEG = 0: group
// size known at run time.  D: weight atoms a wave keeps in flight; D = U is
// the one-round form (the vector forms with at most U atoms per wave): every
// atom of the run is requested at the start and nothing is refilled.  CH: the
// workgroups that share one panel (vector forms, all of K each): workgroup
// part h computes the columns c + 16 t with t in [h T / CH, (h + 1) T / CH),
// reading only those columns' 16 / CH bytes of each lane's 16, so that few
// panels still give every compute unit its own share of the weight stream.
template <int BITS, int M, int WAVES, int SEG, int D, bool BF, int CH>
__global__ __launch_bounds__(WAVES * 64) void gemv_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int K, int N, int group, int64_t s_off, int64_t z_off, int na, int ng, int S, int AS, int RW,
    float* __restrict__ ws_part, uint32_t* __restrict__ ws_cnt, int mr) {
    // mr <= M rows of A and C exist; row slots past them re-read row mr - 1
    // (in bounds) and are never stored.
    using Cfg = GemvCfg<BITS, M>;
    constexpr int U = kGemvU, T = Cfg::T, PW = Cfg::PW;
    constexpr bool FACT = Cfg::FACT, MF = Cfg::MF, MFF = Cfg::MFF;
    constexpr int NT = WAVES * 64;
    static_assert(!MF || M == 16 || M == 32 || M == 64, "the matrix-core form holds 16, 32 or 64 rows");
    constexpr int MB = Cfg::MB;
    static_assert(SEG == 0 || U % SEG == 0, "segments tile a round");
    static_assert(U % D == 0, "the load ring tiles a round");
    constexpr bool ONE = D == U && !MF;
    static_assert(CH == 1 || (!MF && T % CH == 0), "column parts split a lane's columns");
    constexpr int TE = T / CH;                          // columns a lane computes
    // metadata of the groups one round touches: U / SEG groups, or up to U
    constexpr int NGR = SEG > 0 ? U / SEG : U;
    constexpr int SLANES = NGR * PW * 2 / 16, ZLANES = NGR * PW / 8;
    using Stage = WaveStage<Cfg::XR, Cfg::CR, PW>;
    // The vector forms keep the reduction buffer beside the staging areas
    // (84 KB together at most, W4 with 3 rows; one workgroup per compute unit
    // either way), so a wave that has finished writes its sums while others
    // still read their staging, with no barrier in between; the matrix-core
    // form's reduction buffer (up to 64 rows) reuses the staging storage.
    struct SmemApart {
        Stage st[WAVES];
        float red[WAVES][M][PW];
    };
    union SmemShared {
        Stage st[WAVES];
        float red[WAVES][M][PW];
    };
    using Smem = std::conditional_t<MF, SmemShared, SmemApart>;
    __shared__ __align__(16) Smem sm;

    // With CH parts per panel, the parts of a panel are workgroups b, b + 8,
    // ..., b + 8 (CH - 1): one XCD (workgroups are dealt to the eight XCDs in
    // turn), so every part after the first finds the panel's lines in that
    // XCD's L2.  Workgroups past the last panel (the grid is whole groups of
    // 8 CH) end at once.
    const int p = CH == 1 ? blockIdx.x : blockIdx.x / (8 * CH) * 8 + blockIdx.x % 8;
    const int part_h = CH == 1 ? 0 : blockIdx.x / 8 % CH;
    const int tp0 = part_h * TE;                        // first of this part's columns t of a lane
    if (CH > 1 && p >= (N + PW - 1) / PW) return;
    const int split = blockIdx.y;                       // K-slice of this workgroup
    const int a_end = min(na, split * AS + AS);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar) index math
    const int c = lane & 15, kg = lane >> 4;
    const int apg = group / kAtomK;
    const uint32_t magic = BF ? magic_bf_reg() : magic_reg();
    const uint32_t magic64 = magic64_reg();
    // this wave's run: atoms aw0 .. aw_end-1 of the panel (RW per wave; a
    // multiple of the group's atoms when SEG > 0)
    const int aw0 = split * AS + wave * RW;
    const int aw_end = min(a_end, aw0 + RW);
    const int nw = aw_end - aw0;                        // may be <= 0: an idle wave
    const int nrounds = nw > 0 ? (nw + U - 1) / U : 0;
    // a lane's share of an atom: 16 bytes, or the 16 / CH bytes of its part's columns
    using WT = std::conditional_t<CH == 1, u32x4, std::conditional_t<CH == 2, u32x2, uint32_t>>;
    const WT* wrun = reinterpret_cast<const WT*>(packed + ((int64_t)p * na * 64 + lane) * 16 + 16 / CH * part_h);
    const uint8_t* spanel = packed + s_off + (int64_t)p * ng * PW * 2;
    const uint8_t* zpanel = packed + z_off + (int64_t)p * ng * PW;
    const int64_t s_last = ((int64_t)ng * PW * 2 - 16);     // last 16-byte slot of the panel's scales
    const int64_t z_last = ((int64_t)ng * PW - 8);
    Stage& st = sm.st[wave];
    const uint8_t* sbytes = reinterpret_cast<const uint8_t*>(st.s);
    const uint8_t* zbytes = reinterpret_cast<const uint8_t*>(st.z);

    float y[M][TE];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
        for (int t = 0; t < TE; ++t) y[m][t] = 0.f;

    // Loads.  A round is U atoms of the run; its small loads (the wave's
    // slice of x, its groups' metadata) are issued one round ahead.  Weight
    // atoms stream through a ring of D registers: the atom D places ahead is
    // requested as each one is taken, so the memory queues stay short and
    // data comes back in the order it is used (issuing everything at once
    // lets the first-needed bytes arrive anywhere in the whole transfer).
    // Addresses are clamped into the panel, so every load is in bounds.
    struct Meta {
        uint64_t xr[Cfg::XR];
        u32x4 sr;
        uint64_t zr;
    };
    auto issue_meta = [&](int r, Meta& mt) {
        const int ac = min(aw0 + r * U, na - 1);
        const int k0 = ac * kAtomK;
        if constexpr (!MF) {
#pragma unroll
            for (int m = 0; m < M; ++m) {
                const int k = min(k0 + 4 * lane, K - 4);
                mt.xr[m] = *reinterpret_cast<const uint64_t*>(A + (int64_t)min(m, mr - 1) * K + k);
            }
        }
        // every lane loads (lanes past the needed bytes repeat the last
        // slot): no branch around a load, so the compiler's wait counts stay
        // exact and the ring below keeps D atoms in flight
        const int g0 = ac / apg;
        mt.sr = *reinterpret_cast<const u32x4*>(
            spanel + min((int64_t)g0 * PW * 2 + 16 * min(lane, SLANES - 1), s_last));
        mt.zr = *reinterpret_cast<const uint64_t*>(
            zpanel + min((int64_t)g0 * PW + 8 * min(lane, ZLANES - 1), z_last));
    };
    // atom j of the run; requests past the run repeat its last atom (a cache
    // hit, issued without a branch for the same reason)
    auto load_atom = [&](int j) {
        return __builtin_nontemporal_load(wrun + (int64_t)min(aw0 + min(j, nw - 1), na - 1) * 64 * CH);
    };
    WT ring[D];
    // Matrix-core form: the A operand of v_mfma_f32_16x16x32_f16 for atom j
    // and row block b, row 16 b + c (row slots past mr repeat row mr - 1),
    // k = 32 a + 8 kg + 0..7, read straight from global memory (A is small
    // and stays in L2) through a ring of its own.
    const uint16_t* arow[MB];
#pragma unroll
    for (int b = 0; b < MB; ++b) arow[b] = A + (int64_t)min(16 * b + c, mr - 1) * K + 8 * kg;
    auto load_afrag = [&](int b, int j) {
        return *reinterpret_cast<const u32x4*>(arow[b] + (int64_t)min(aw0 + min(j, nw - 1), na - 1) * kAtomK);
    };
    u32x4 aring[MF ? MB : 1][MF ? D : 1];
    // lane (c, kg) of block (b, t): rows 16 b + 4 kg + 0..3, column c + 16 t
    float4_t macc[MF ? MB : 1][MF ? T : 1];
#pragma unroll
    for (int b = 0; b < (MF ? MB : 1); ++b)
#pragma unroll
        for (int t = 0; t < (MF ? T : 1); ++t) macc[b][t] = float4_t{0.f, 0.f, 0.f, 0.f};

    // One round r of the run.
    auto consume_round = [&](int r, Meta& mt) {
        const int a0 = aw0 + r * U;
        const int g0 = a0 / apg;
        int pos = a0 - g0 * apg;      // runtime segments: atom a0's place in its group
        int gl = 0;                   // current group, relative to g0

        // stage this wave's x slice and metadata (wave-private LDS)
        if constexpr (!MF) {
#pragma unroll
            for (int m = 0; m < M; ++m) st.x[m][lane] = mt.xr[m];
        }
        // (lanes past the needed slots rewrite the last slot with its own
        // value: no branch, which would let the compiler sink the loads into
        // it and wait for every load in flight)
        st.s[min(lane, SLANES - 1)] = mt.sr;
        st.z[min(lane, ZLANES - 1)] = mt.zr;
        if constexpr (FACT) {
            // Sums of x per 8-k slice, once for all columns: sx = sum x and
            // B = sum x * offset.  fp16: offset 1024 for rows 0,1,4,5 and,
            // 4-bit, 64 for rows 2,3,6,7 (lane l holds rows 4(l%2)..+3 of
            // slice l/2: its first pair has offset 1024, its second 1024 or
            // 64).  bf16: 128 for every 4-bit row, 0 for 8-bit codes.
            const uint32_t ones = BF ? 0x3F803F80u : 0x3C003C00u;
            const uint32_t o_lo = BF ? (BITS == 4 ? 0x43004300u : 0u) : 0x64006400u;
            const uint32_t o_hi = BF ? o_lo : (BITS == 4 ? 0x54005400u : 0x64006400u);
#pragma unroll
            for (int m = 0; m < M; ++m) {
                const uint32_t x01 = (uint32_t)mt.xr[m], x23 = (uint32_t)(mt.xr[m] >> 32);
                float sx = dot2<BF>(x23, ones, dot2<BF>(x01, ones, 0.f));
                float bo = (BF && BITS == 8) ? 0.f : dot2<BF>(x23, o_hi, dot2<BF>(x01, o_lo, 0.f));
                sx += __shfl_xor(sx, 1);
                bo += __shfl_xor(bo, 1);
                // both lanes of a slice store its sums (no branch: a masked
                // store lets the compiler move the later reads under the mask)
                st.cs[m][lane] = float2_t{bo, sx};
            }
        }
        // the staged data is read by other lanes of this wave: order the
        // stores before those reads (a wave-scope fence, no workgroup barrier)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        float acc[M][TE];                // factored form: sums of x * code of the open segment
        float bo[M], sx[M];              // ... and the segment's sums of x * offset and of x
        DqConst<BF> kq[TE];              // dequant form: the open segment's scale and zero-point
        // matrix-core factored form: the open segment's sums of A x code and
        // of A (row sums, the same in every column of a block)
        float4_t accg[MFF ? MB : 1][MFF ? T : 1], rsum[MFF ? MB : 1];
        auto open = [&]() {
            if constexpr (MFF) {
#pragma unroll
                for (int b = 0; b < MB; ++b) {
                    rsum[b] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int t = 0; t < T; ++t) accg[b][t] = float4_t{0.f, 0.f, 0.f, 0.f};
                }
            } else if constexpr (FACT) {
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    bo[m] = 0.f;
                    sx[m] = 0.f;
#pragma unroll
                    for (int t = 0; t < TE; ++t) acc[m][t] = 0.f;
                }
            } else {
                const uint16_t* sp = reinterpret_cast<const uint16_t*>(sbytes + (gl * PW + c * T + tp0) * 2);
                const uint8_t* zp = zbytes + gl * PW + c * T + tp0;
#pragma unroll
                for (int t = 0; t < TE; ++t) kq[t] = make_dq_const<BF>(sp[t], zp[t]);
            }
        };
        // close the open segment: y += s * (acc - bo - z * sx); matrix-core
        // factored form: y += s * (acc - (o + z) * (row sum of A)), o the
        // codes' offset
        auto close = [&]() {
            if constexpr (MFF) {
                const uint16_t* sp = reinterpret_cast<const uint16_t*>(sbytes + (gl * PW + c * T) * 2);
                const uint8_t* zp = zbytes + gl * PW + c * T;
                constexpr float off = BF ? (BITS == 4 ? 128.f : 0.f) : 1024.f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const float zo = off + (float)zp[t];
                    const float sf = scale_f32<BF>(sp[t]);
#pragma unroll
                    for (int b = 0; b < MB; ++b)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            macc[b][t][q] = fmaf(sf, fmaf(-zo, rsum[b][q], accg[b][t][q]), macc[b][t][q]);
                }
            } else if constexpr (FACT) {
                const uint16_t* sp = reinterpret_cast<const uint16_t*>(sbytes + (gl * PW + c * T + tp0) * 2);
                const uint8_t* zp = zbytes + gl * PW + c * T + tp0;
#pragma unroll
                for (int t = 0; t < TE; ++t) {
                    const float zf = (float)zp[t];
                    const float sf = scale_f32<BF>(sp[t]);
#pragma unroll
                    for (int m = 0; m < M; ++m)
                        y[m][t] = fmaf(sf, acc[m][t] - fmaf(zf, sx[m], bo[m]), y[m][t]);
                }
            }
        };

        if constexpr (FACT || MFF || SEG > 0) open();
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int j = r * U + i;      // atom of the run
            if (i > 0 && j >= nw) break;
            // take atom j from the ring and request atom j + D in its place
            const WT wv = ring[i % D];
            if constexpr (!ONE) ring[i % D] = load_atom(j + D);
            u32x4 afrag[MF ? MB : 1];
            if constexpr (MF) {
#pragma unroll
                for (int b = 0; b < MB; ++b) {
                    afrag[b] = aring[b][i % D];
                    aring[b][i % D] = load_afrag(b, j + D);
                }
            }
            if constexpr (MFF) {
                // row sums of this atom's A, by the matrix core against ones
                const uint32_t one2 = BF ? 0x3F803F80u : 0x3C003C00u;
                const u32x4 ones = {one2, one2, one2, one2};
#pragma unroll
                for (int b = 0; b < MB; ++b) rsum[b] = mfma16<BF>(afrag[b], ones, rsum[b]);
            }
            // dequant form, group size known at run time: this atom's metadata
            if constexpr (!FACT && !MFF && SEG == 0) open();
            u32x4 xv[Cfg::XR];
            if constexpr (!MF) {
#pragma unroll
                for (int m = 0; m < M; ++m)
                    xv[m] = *reinterpret_cast<const u32x4*>(&st.x[m][(i * kAtomK + 8 * kg) / 4]);
            }
            if constexpr (FACT) {
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const float2_t v = st.cs[m][8 * i + 2 * kg];   // slice (atom i, kg)
                    bo[m] += v[0];
                    sx[m] += v[1];
                }
            }
            // the dwords of this part's columns (dword t of a 4-bit lane is
            // column t, dwords 2 t and 2 t + 1 of an 8-bit lane are column t)
            uint32_t wd[4 / CH];
            if constexpr (CH == 4) {
                wd[0] = wv;
            } else {
#pragma unroll
                for (int q = 0; q < 4 / CH; ++q) wd[q] = wv[q];
            }
#pragma unroll
            for (int t = 0; t < TE; ++t) {
                uint32_t P[4];
                if constexpr (MFF) {
                    // the codes as exact 16-bit integers o + q: fp16 1024 + q,
                    // bf16 128 + q (4-bit) or q (8-bit, converted)
                    if constexpr (BITS == 4) {
                        w4_code_pairs(wd[t], magic, P);
                    } else if constexpr (BF) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t wq = wd[2 * t + q / 2];
                            const bf16x2_t v = {(__bf16)byte_f32(wq, 2 * (q & 1)), (__bf16)byte_f32(wq, 2 * (q & 1) + 1)};
                            P[q] = __builtin_bit_cast(uint32_t, v);
                        }
                    } else {
                        w8_code_pairs(wd[2 * t], P);
                        w8_code_pairs(wd[2 * t + 1], P + 2);
                    }
                    const u32x4 pv = {P[0], P[1], P[2], P[3]};
#pragma unroll
                    for (int b = 0; b < MB; ++b) accg[b][t] = mfma16<BF>(afrag[b], pv, accg[b][t]);
                    continue;
                }
                if constexpr (FACT) {
                    if constexpr (BF && BITS == 4) {
                        w4_code_pairs(wd[t], magic, P);          // rows (2q, 2q+1) as 128 + q
                    } else if constexpr (BF) {
                        // bytes have 8 bits, past bfloat16's exact 128 + v range:
                        // each code converts to fp32 and back, exactly
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t wq = wd[2 * t + q / 2];
                            const bf16x2_t v = {(__bf16)byte_f32(wq, 2 * (q & 1)), (__bf16)byte_f32(wq, 2 * (q & 1) + 1)};
                            P[q] = __builtin_bit_cast(uint32_t, v);
                        }
                    } else if constexpr (BITS == 4) {
                        w4_code_pairs_sum(wd[t], magic, magic64, P);
                    } else {
                        w8_code_pairs(wd[2 * t], P);
                        w8_code_pairs(wd[2 * t + 1], P + 2);
                    }
                } else {
                    const u32x4 wu = dq_operand<BF, BITS>(wd[BITS == 4 ? t : 2 * t], wd[BITS == 4 ? t : 2 * t + 1],
                                                          magic, kq[t]);
                    if constexpr (MF) {
                        // the dequantized dword is the B operand of columns c + 16 t
#pragma unroll
                        for (int b = 0; b < MB; ++b) macc[b][t] = mfma16<BF>(afrag[b], wu, macc[b][t]);
                        continue;
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) P[q] = wu[q];
                }
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    float v = FACT ? acc[m][t] : y[m][t];
#pragma unroll
                    for (int q = 0; q < 4; ++q) v = dot2<BF>(P[q], xv[m][q], v);
                    if constexpr (FACT) acc[m][t] = v; else y[m][t] = v;
                }
            }
            // end of a segment: end of its group, of the round, or of the run
            bool seg_end, grp_end;
            if constexpr (SEG > 0) {
                grp_end = (i + 1) % SEG == 0;
                seg_end = grp_end || j + 1 == nw;
            } else {
                grp_end = ++pos == apg;
                seg_end = grp_end || i == U - 1 || j + 1 == nw;
            }
            if (seg_end) {
                close();
                if (i < U - 1) {
                    if (grp_end) {
                        ++gl;
                        pos = 0;
                    }
                    if constexpr (FACT || MFF || SEG > 0) open();
                }
            }
        }
    };

    if (nrounds > 0) {
        Meta m0, m1;
        issue_meta(0, m0);
#pragma unroll
        for (int d = 0; d < D; ++d) {
            ring[d] = load_atom(d);
            if constexpr (MF)
#pragma unroll
                for (int b = 0; b < MB; ++b) aring[b][d] = load_afrag(b, d);
        }
        if constexpr (ONE) {
            // one round (the launcher's guarantee): no further requests, so
            // the wave waits for no load it does not use before it ends
            consume_round(0, m0);
        } else {
            // The next round's small loads are issued even past the last
            // round, at clamped addresses: without a branch around a load the
            // compiler's wait counts stay exact.  Round 0 is peeled off the
            // loop for the same reason (waits after a loop header are
            // conservative).
            issue_meta(1, m1);
            consume_round(0, m0);
            for (int r = 1; r < nrounds; r += 2) {
                issue_meta(r + 1, m0);
                consume_round(r, m1);
                if (r + 1 < nrounds) {
                    issue_meta(r + 2, m1);
                    consume_round(r + 1, m0);
                }
            }
        }
    }

    if constexpr (MF) {
        // each lane holds distinct outputs: rows 4 kg + 0..3 of columns c + 16 t
        __syncthreads();   // staging storage becomes the reduction buffer
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int b = 0; b < MB; ++b) sm.red[wave][16 * b + 4 * kg + q][c + 16 * t] = macc[b][t][q];
    } else {
        // Lanes c, c+16, c+32, c+48 hold the same columns: combine over kg.
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < TE; ++t) {
                float v = y[m][t];
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                y[m][t] = v;
            }
        if (kg == 0) {
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int t = 0; t < TE; ++t) sm.red[wave][m][c + 16 * (tp0 + t)] = y[m][t];
        }
    }
    __syncthreads();
    if (CH > 1 || S == 1) {
        // this part's columns: c + 16 t for t in [tp0, tp0 + TE), PW / CH in a row
        for (int i = tid; i < M * PW / CH; i += NT) {
            const int m = i / (PW / CH), col = i % (PW / CH) + 16 * tp0;
            const int n = p * PW + col;
            if (n < N && m < mr) {
                float v = 0.f;
#pragma unroll
                for (int w = 0; w < WAVES; ++w) v += sm.red[w][m][col];
                C[(int64_t)m * N + n] = round_out<BF>(v);
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
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) v += sm.red[w][i / PW][i % PW];
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
        if (n < N && m < mr) C[(int64_t)m * N + n] = round_out<BF>(v);
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
    int waves, S, AS, CH;
};
constexpr int kMaxSplit = 32;
constexpr int64_t kSplitBelowPanels = 192;      // split K only below this many panels ...
constexpr int64_t kSplitFromWork = 256;         // ... carrying at least this much work each
constexpr int64_t kTargetWorkgroups = 256;
constexpr int64_t kMfSliceAtoms = 64;

// 16 waves (four per SIMD) while 128 registers hold a lane's state, else 8.
constexpr int gemv_waves_for(int M) { return M <= 3 ? 16 : 8; }
// Weight atoms in flight per wave.  Two measured best on MI355X (graph
// replay, K=4096 N=14336 and K=14336 N=4096, M = 1..16): four or eight
// lengthen the memory queues without raising the rate a compute unit streams.
// A run of one round (at most kGemvU atoms per wave) is instead requested
// whole at the start (the one-round form): no refill requests past its end and
// no metadata for a round that does not come, each a round trip the wave
// would wait for before it ends (measured: K=4096 with N=14336 W4 2%, N=32768
// W4 10%, N=4096 W8 11% faster).
constexpr int gemv_ring_for(int) { return 2; }

// Column parts per panel (vector forms): 2 or 4 workgroups share a panel,
// each reading only its own columns' bytes of every atom over all of K, so
// that few panels still give every compute unit a share of the stream and of
// the dot products, with no partial sums.  Taken while panels x parts fit one
// workgroup per compute unit, for runs of up to kPartsMaxAtoms atoms carrying
// at least kPartsFromWork work (the K split's measure): every part requests
// all of the panel's cache lines, so over long runs a compute unit's line
// rate, not the bytes it uses, sets the time and the K split is faster, and
// on short light runs the extra workgroups only add start-up time.  Measured
// on MI355X (graph replay, against the plan without parts): K = N = 4096,
// W4 M = 1, 4, 8 5.84, 8.66, 12.8 -> 5.66, 7.64, 8.4 us, W8 M = 8 10.5 ->
// 8.6 us; K = 14336, N = 4096 W4 M = 1 13.2 us with 4 parts against 10.0 us
// split; two workgroups per compute unit (K = 4096, N = 14336, M = 1 to 8)
// 1-21% slower.
constexpr int64_t kPartsMaxAtoms = 128;
constexpr int64_t kPartsFromWork = 128;
inline int gemv_parts(const Layout& L, int64_t M) {
    if (M > TF_GEMV_MAX_M || L.na > kPartsMaxAtoms || L.na * std::max<int64_t>(1, M / 2) < kPartsFromWork)
        return 1;
    const int64_t T = L.pw / 16;
    int ch = 1;
    while (2 * ch <= T && L.np * 2 * ch <= kTargetWorkgroups) ch *= 2;
    return ch;
}

inline GemvPlan plan_gemv(const Layout& L, int64_t M) {
    const int waves = gemv_waves_for((int)M);
    const int CH = gemv_parts(L, M);
    if (CH > 1) return {waves, 1, (int)L.na, CH};
    // slices keep at least this many atoms: a round of 16 waves at M = 1, of
    // 8 up to 8 rows; the matrix-core form (little vector work per atom)
    // splits down to kMfSliceAtoms
    const int64_t ra = M > TF_GEMV_MAX_M ? kMfSliceAtoms : (int64_t)(M == 1 ? 16 : 8) * kGemvU;
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
    return {waves, (int)S, (int)AS, 1};
}

// Workspace layout: arrival counters first, at a fixed place and sized for
// the largest panel count any shape can have, so every call finds its
// counters where an earlier call (of any shape) left them at zero; then the
// per-slice partial sums, which are always written before they are read.

template <int BITS, int M, int SEG, bool BF>
int launch_g(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, void* ws,
             int mr, hipStream_t s) {
    constexpr int WAVES = gemv_waves_for(M);
    const GemvPlan sp = plan_gemv(L, M);
    const bool split = ws != nullptr && sp.S > 1;
    uint32_t* cnt = split ? static_cast<uint32_t*>(ws) : nullptr;
    float* part = split ? reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsCounterBytes) : nullptr;
    const int S = split ? sp.S : 1;
    const int AS = split ? sp.AS : (int)L.na;
    int RW = (AS + WAVES - 1) / WAVES;               // atoms per wave
    if (SEG > 0) RW = (RW + SEG - 1) / SEG * SEG;    // runs start on group boundaries
    auto go = [&](auto kernel, int d, int ch) {
        if (log_enabled())
            log_plan("gemv_kernel<%d,%d,%d,%d,%d,%s,%d> rows=%d K=%lld N=%lld G=%d: %s form, %lld panels x %d "
                     "column parts x %d K slices of %d atoms, %d atoms per wave%s", BITS, M, WAVES, SEG, d,
                     BF ? "bf16" : "f16", ch, mr, (long long)L.K, (long long)L.N, L.group,
                     M > TF_GEMV_MAX_M ? "matrix-core" : (d == kGemvU ? "one-round vector" : "vector"),
                     (long long)L.np, ch, S, AS, RW, split ? ", partials summed by the last slice" : "");
        // column parts: whole groups of 8 ch workgroups (those past the last panel end at once)
        const int64_t gx = ch == 1 ? L.np : (L.np + 7) / 8 * 8 * ch;
        return launch(kernel, dim3((unsigned)gx, (unsigned)S), dim3(WAVES * 64), 0, s, A, pk, C,
                      (int)L.K, (int)L.N, L.group, L.s_off, L.z_off, (int)L.na, (int)L.ng, S, AS, RW,
                      part, cnt, mr);
    };
    auto with_parts = [&](auto ch_tag) {
        constexpr int CH = decltype(ch_tag)::value;
        if (RW <= kGemvU) return go(gemv_kernel<BITS, M, WAVES, SEG, kGemvU, BF, CH>, kGemvU, CH);
        return go(gemv_kernel<BITS, M, WAVES, SEG, gemv_ring_for(M), BF, CH>, gemv_ring_for(M), CH);
    };
    if constexpr (M <= TF_GEMV_MAX_M) {
        if (BITS == 4 && sp.CH == 4) return with_parts(std::integral_constant<int, BITS == 4 ? 4 : 1>{});
        if (sp.CH == 2) return with_parts(std::integral_constant<int, 2>{});
        return with_parts(std::integral_constant<int, 1>{});
    }
    return go(gemv_kernel<BITS, M, WAVES, SEG, gemv_ring_for(M), BF, 1>, gemv_ring_for(M), 1);
}

template <int BITS, int M, bool BF>
int launch_m(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, void* ws,
             hipStream_t s, int mr = M) {
    // group 128 (the AWQ default) gets its segments fixed at compile time
    if (L.group == 128) return launch_g<BITS, M, 4, BF>(L, A, pk, C, ws, mr, s);
    return launch_g<BITS, M, 0, BF>(L, A, pk, C, ws, mr, s);
}

template <int BITS, bool BF>
int launch_bits(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    switch (M) {
        case 1: return launch_m<BITS, 1, BF>(L, A, pk, C, ws, s);
        case 2: return launch_m<BITS, 2, BF>(L, A, pk, C, ws, s);
        case 3: return launch_m<BITS, 3, BF>(L, A, pk, C, ws, s);
        case 4: return launch_m<BITS, 4, BF>(L, A, pk, C, ws, s);
        case 5: return launch_m<BITS, 5, BF>(L, A, pk, C, ws, s);
        case 6: return launch_m<BITS, 6, BF>(L, A, pk, C, ws, s);
        case 7: return launch_m<BITS, 7, BF>(L, A, pk, C, ws, s);
        case 8: return launch_m<BITS, 8, BF>(L, A, pk, C, ws, s);
    }
    return TF_ERR_ARG;
}

int64_t workspace_for_slots(const Layout& L, int64_t slots) {
    const GemvPlan sp = plan_gemv(L, slots);
    if (sp.S <= 1) return 0;
    return kWsCounterBytes + align256((int64_t)L.np * sp.S * slots * L.pw * 4);
}

}  // namespace

int64_t gemv_workspace_bytes(const Layout& L, int64_t M) {
    return M >= 1 && M <= TF_GEMV_MAX_M ? workspace_for_slots(L, M) : 0;
}

// row slots of the matrix-core form for M rows: 16, 32 or 64
static int64_t skinny_slots(int64_t M) { return M <= 16 ? 16 : M <= 32 ? 32 : 64; }

int64_t skinny_workspace_bytes(const Layout& L, int64_t M) {
    return M >= 1 && M <= kSkinnyMaxM ? workspace_for_slots(L, skinny_slots(M)) : 0;
}

int launch_gemv(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s, bool bf) {
    if (bf)
        return L.bits == 4 ? launch_bits<4, true>(L, A, packed, C, M, ws, s)
                           : launch_bits<8, true>(L, A, packed, C, M, ws, s);
    return L.bits == 4 ? launch_bits<4, false>(L, A, packed, C, M, ws, s)
                       : launch_bits<8, false>(L, A, packed, C, M, ws, s);
}

namespace {
template <int BITS, bool BF>
int launch_skinny_bits(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C,
                       int64_t M, void* ws, hipStream_t s) {
    switch (skinny_slots(M)) {
        case 16: return launch_m<BITS, 16, BF>(L, A, pk, C, ws, s, (int)M);
        case 32: return launch_m<BITS, 32, BF>(L, A, pk, C, ws, s, (int)M);
        default: return launch_m<BITS, 64, BF>(L, A, pk, C, ws, s, (int)M);
    }
}
}  // namespace

int launch_skinny_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C,
                       int64_t M, void* ws, hipStream_t s, bool bf) {
    if (M < 1 || M > kSkinnyMaxM) return TF_ERR_ARG;
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (bf)
        return L.bits == 4 ? launch_skinny_bits<4, true>(L, A, pk, C, M, ws, s)
                           : launch_skinny_bits<8, true>(L, A, pk, C, M, ws, s);
    return L.bits == 4 ? launch_skinny_bits<4, false>(L, A, pk, C, M, ws, s)
                       : launch_skinny_bits<8, false>(L, A, pk, C, M, ws, s);
}

}  // namespace tf
