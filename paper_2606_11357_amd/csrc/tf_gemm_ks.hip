// Prefill GEMM for the sizes whose output tiles are too few to give every
// compute unit one of the larger tiles (Section 2.1; Section 4.3 "GEMM
// microkernel"; Section 4.4):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 or bf16 MFMA, fp32 sums.
//
// Workgroup tile 64 x 128, four waves, one per SIMD.  Each wave computes the
// whole tile over its own quarter of K (a contiguous run of 128-row chunks)
// and streams it alone: no LDS and no barrier inside the loop, and no
// partial sum leaves the compute unit.
//  - The wave's A fragments (4 row blocks of 16 rows) and the packed atoms of
//    the tile's columns (one per panel per 32-row step) go from memory
//    straight into a register ring of four steps, requested three steps before
//    their use; the metadata of a group is requested with the atoms of the
//    step that opens it.  Requests are issued metadata first, then atoms, then
//    A, in the order the step that waits for them needs them (vector-memory
//    loads complete in order).
//  - A step's 32 MFMAs run column block by column block (8 blocks of 16
//    columns, each against the 4 row blocks); while the four MFMAs of block u
//    run, the wave dequantizes (Eq. 2, rounded once, the same arithmetic as
//    the other GEMMs) the B operand of block u + 1, so the dequantization's
//    vector work issues in the matrix core's shadow.  Each weight is
//    dequantized once per 64 rows of A (Sections 4.1.1 and 4.3: dequantize a
//    tile once and reuse it across the activation rows).
//  - After the loop the four K quarters are added through LDS in quarter
//    order (bitwise reproducible) and the tile of C is written once.
//  - Tiles are dealt so that each XCD takes a contiguous band of them, row
//    tiles varying fastest: the band's weight columns are fetched into that
//    XCD's L2 once for all of its row tiles.
#include <algorithm>

#include "tf_internal.h"

namespace tf {
namespace {

constexpr int kKsBM = 64, kKsBN = 128, kKsBK = 32;
constexpr int kKsWaves = 4, kKsThreads = 64 * kKsWaves;
constexpr int kKsCS = 4;                // steps per chunk (128 rows of K) and ring slots
constexpr int kKsLead = 3;              // steps between a request and its step
constexpr int kKsRB = kKsBM / 16;       // row blocks
constexpr int kKsNB = kKsBN / 16;       // column blocks: B operands per step
constexpr int kKsXcds = 8;

// A step's 32 MFMA slots, block u = slot / 4 (columns 16 u ..), row block
// i = slot % 4.  Requests for step + 3 sit at fixed slots: the metadata (when
// step + 3 opens a group) at kKsMetaSlot, the atoms at kKsAtomSlot, the A
// fragment of row block r at kKsASlot + kKsASlotStride * r.
constexpr int kKsMetaSlot = 0, kKsAtomSlot = 4, kKsASlot = 8, kKsASlotStride = 3;
// The step waits twice: for its own A at block 0, for the next step's atoms
// and metadata at block kKsMetaWaitBlock; the constants of the group the next
// step opens are formed after that, those of block v at slot kKsConstSlot[v]
// (block v's old constants were last used under block v - 1).
constexpr int kKsMetaWaitBlock = 5;
constexpr int kKsConstSlot[8] = {20, 21, 22, 23, 24, 25, 26, 28};
static_assert(kKsMetaSlot < kKsAtomSlot && kKsAtomSlot < kKsASlot, "requests go out metadata, atoms, A");
static_assert(kKsASlot + kKsASlotStride * (kKsRB - 1) < kKsMetaWaitBlock * kKsRB,
              "a step's requests are all issued before its second wait counts them");
constexpr bool ks_const_slots_ok() {
    for (int v = 0; v < kKsNB; ++v) {
        const int blk = kKsConstSlot[v] / kKsRB;
        if (blk < kKsMetaWaitBlock || blk < v || blk >= kKsNB) return false;
    }
    return true;
}
static_assert(ks_const_slots_ok(), "constants formed after the wait and after their old value's last use");

// Buffer resource words (raw buffer, 32-bit format) for the asm loads.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return i32x4{(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}
// Buffer loads issued as asm statements: the compiler then places no wait for
// them, and the kernel's own counted waits (vm_wait, before every first use)
// keep each load's full lead.  Loads complete in the order they are issued.
__device__ __forceinline__ u32x4 ld128(i32x4 r, uint32_t voff, uint32_t soff) {
    u32x4 v;
    asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff));
    return v;
}
__device__ __forceinline__ uint2 ld64(i32x4 r, uint32_t voff, uint32_t soff) {
    uint2 v;
    asm volatile("buffer_load_dwordx2 %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff));
    return v;
}
__device__ __forceinline__ uint32_t ld32(i32x4 r, uint32_t voff, uint32_t soff) {
    uint32_t v;
    asm volatile("buffer_load_dword %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff));
    return v;
}
__device__ __forceinline__ uint32_t ld16(i32x4 r, uint32_t voff, uint32_t soff) {
    uint32_t v;
    asm volatile("buffer_load_ushort %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff));
    return v;
}
// Wait until at most n loads are in flight (n a constant once the step loop
// is unrolled).
__device__ __forceinline__ void vm_wait(int n) {
    switch (n) {
#define TF_VMW(k) \
    case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
        TF_VMW(0) TF_VMW(1) TF_VMW(2) TF_VMW(3) TF_VMW(4) TF_VMW(5) TF_VMW(6) TF_VMW(7) TF_VMW(8)
        TF_VMW(9) TF_VMW(10) TF_VMW(11) TF_VMW(12) TF_VMW(13) TF_VMW(14) TF_VMW(15) TF_VMW(16)
        TF_VMW(17) TF_VMW(18) TF_VMW(19) TF_VMW(20) TF_VMW(21) TF_VMW(22) TF_VMW(23) TF_VMW(24)
        TF_VMW(25) TF_VMW(26) TF_VMW(27) TF_VMW(28) TF_VMW(29) TF_VMW(30) TF_VMW(31) TF_VMW(32)
        TF_VMW(33) TF_VMW(34) TF_VMW(35) TF_VMW(36) TF_VMW(37) TF_VMW(38) TF_VMW(39) TF_VMW(40)
#undef TF_VMW
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}
// Marks a register as (re)defined here, after a wait: its uses cannot move
// above the wait, and it stays allocated until then.
template <typename V>
__device__ __forceinline__ void tie(V& v) { asm volatile("" : "+v"(v)); }

// MPC: metadata groups per chunk (1 when a group spans the chunk, else chunk
// rows / group).
template <int BITS, int MPC, bool BF>
__global__ __launch_bounds__(kKsThreads, 1) void gemm_ks_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int gshift, int64_t s_off, int64_t z_off, int na, int ng, int np,
    int tiles_m, int tiles_n) {
    constexpr int PW = BITS == 4 ? 64 : 32;   // columns per panel (one atom per step)
    constexpr int T = PW / 16;                // column blocks per panel
    constexpr int PANELS = kKsBN / PW;
    constexpr int SPG = kKsCS / MPC;          // steps per metadata group
    constexpr int S = dq_steps<BF, BITS>();   // dequantization micro-steps per operand
    static_assert(kKsRB + 2 * (kKsRB + 3 * PANELS) <= 40, "counted waits stay within vm_wait's range");
    __shared__ __align__(16) float4_t red[kKsWaves][kKsRB * kKsNB][64];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 15, kg = lane >> 4;
    const uint32_t magic = magic_reg();

    // Block b runs on XCD b % 8, which takes the (b % 8)-th contiguous band
    // of tiles; row tiles vary fastest.
    int unit;
    {
        const int total = tiles_m * tiles_n;
        const int b = blockIdx.x;
        const int per = total / kKsXcds, rem = total % kKsXcds;
        const int x = b % kKsXcds, i = b / kKsXcds;
        unit = x * per + min(x, rem) + i;
    }
    // (pinned to scalar registers: integer division runs on the vector ALU,
    // and buffer resources built from a value the compiler cannot prove
    // uniform would be loaded lane by lane)
    const int tm = __builtin_amdgcn_readfirstlane(unit % tiles_m);
    const int tn = __builtin_amdgcn_readfirstlane(unit / tiles_m);
    const int64_t row0 = (int64_t)tm * kKsBM, col0 = (int64_t)tn * kKsBN;

    // This wave's K quarter (the launcher guarantees at least one chunk each).
    const int nch = na / kKsCS;
    const int qch = nch / kKsWaves, rch = nch % kKsWaves;
    const int ch0 = __builtin_amdgcn_readfirstlane(wave * qch + min(wave, rch));
    const int chunks = __builtin_amdgcn_readfirstlane(qch + (wave < rch ? 1 : 0));
    const int st0 = ch0 * kKsCS, steps = chunks * kKsCS;

    // A: fragment of row block i = rows 16 i + c, halves 8 kg .. 8 kg + 7 of
    // the step's 32; rows past M read row M - 1 (in bounds, never stored).
    // Buffer loads: a per-lane offset fixed for the whole loop and a scalar
    // offset per step, so no address arithmetic runs in the loop.
    const int rows = __builtin_amdgcn_readfirstlane(min(M - tm * kKsBM, kKsBM));
    const i32x4 ar = rsrc_words(A + row0 * K, (uint32_t)rows * (uint32_t)K * 2u);
    uint32_t aoff[kKsRB];
#pragma unroll
    for (int i = 0; i < kKsRB; ++i) {
        const uint32_t r = (uint32_t)min(16 * i + c, rows - 1);
        aoff[i] = (r * (uint32_t)K + 8u * kg) * 2u;
    }
    // B: atoms and metadata of the tile's panels; panels past N read the last
    // panel (in bounds, never stored).
    i32x4 wr[PANELS], sr[PANELS], zr[PANELS];
#pragma unroll
    for (int pp = 0; pp < PANELS; ++pp) {
        const int panel = __builtin_amdgcn_readfirstlane(min(tn * PANELS + pp, np - 1));
        wr[pp] = rsrc_words(packed + (int64_t)panel * na * 1024, (uint32_t)na * 1024u);
        sr[pp] = rsrc_words(packed + s_off + (int64_t)panel * ng * PW * 2, (uint32_t)(ng * PW * 2));
        zr[pp] = rsrc_words(packed + z_off + (int64_t)panel * ng * PW, (uint32_t)(ng * PW));
    }
    const uint32_t woff = lane * 16, soff = c * T * 2, zoff = c * T;

    struct Slot {
        u32x4 a[kKsRB];
        u32x4 w[PANELS];
    };
    struct Meta {
        uint32_t s[PANELS][(T + 1) / 2];   // T 16-bit scales of the lane's columns
        uint32_t z[PANELS];                // T zero-point bytes
    };
    auto load_w = [&](int step, Slot& sl) {
        step = min(step, steps - 1);       // clamped: a repeated valid step, never used
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) sl.w[pp] = ld128(wr[pp], woff, (uint32_t)(st0 + step) * 1024u);
    };
    auto load_a = [&](int step, int i, Slot& sl) {
        step = min(step, steps - 1);
        sl.a[i] = ld128(ar, aoff[i], (uint32_t)(st0 + step) * (kKsBK * 2));
    };
    auto load_meta = [&](int step, Meta& mt) {
        step = min(step, steps - 1);
        const uint32_t g = (uint32_t)(((st0 + step) * kKsBK) >> gshift);
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) {
            if constexpr (BITS == 4) {
                const uint2 sv = ld64(sr[pp], soff, g * PW * 2);
                mt.s[pp][0] = sv.x;
                mt.s[pp][1] = sv.y;
                mt.z[pp] = ld32(zr[pp], zoff, g * PW);
            } else {
                mt.s[pp][0] = ld32(sr[pp], soff, g * PW * 2);
                mt.z[pp] = ld16(zr[pp], zoff, g * PW);
            }
        }
    };
    // Loads issued for step t (its metadata when it opens a group, its atoms,
    // its A fragments): what a counted wait leaves in flight per step.
    auto loads_for = [&](int t) { return kKsRB + PANELS + (t % SPG == 0 ? 2 * PANELS : 0); };
    auto tie_meta = [&](Meta& mt) {
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) {
#pragma unroll
            for (int h = 0; h < (T + 1) / 2; ++h) tie(mt.s[pp][h]);
            tie(mt.z[pp]);
        }
    };
    auto tie_slot = [&](Slot& sl) {
#pragma unroll
        for (int i = 0; i < kKsRB; ++i) tie(sl.a[i]);
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) tie(sl.w[pp]);
    };
    // Group constants of column block u (panel u / T, lane column t = u % T).
    auto make_const = [&](const Meta& mt, int u) {
        const int pp = u / T, t = u % T;
        DqConst<BF> kq;
        if constexpr (BF) {
            const uint32_t sw = mt.s[pp][t / 2];
            kq.s = __builtin_bit_cast(float, (t & 1) ? (sw & 0xFFFF0000u) : (sw << 16));
            kq.nzs = -(byte_f32(mt.z[pp], t) * kq.s);
        } else {
            const uint32_t sh = mt.s[pp][t / 2] >> (16 * (t & 1));
            kq.s2 = as_h2(__builtin_amdgcn_perm(sh, sh, 0x01000100u));
            const uint32_t n = __builtin_amdgcn_perm(0xE4E4E4E4u, mt.z[pp], 0x04000400u | (t * 0x00010001u));
            kq.nz = n;
            kq.nz64 = neg_zero64_pair(n);
        }
        return kq;
    };
    // Micro-step k of the B operand of column block u from the atoms of `sl`.
    auto dq_micro = [&](int k, const Slot& sl, int u, const DqConst<BF>& kq, DqSt<BF>& st) {
        const int pp = u / T, t = u % T;
        dq_step<BF, BITS>(k, sl.w[pp][BITS == 4 ? t : 2 * t], sl.w[pp][BITS == 4 ? t : 2 * t + 1], magic, kq, st);
    };

    float4_t acc[kKsRB][kKsNB];
#pragma unroll
    for (int i = 0; i < kKsRB; ++i)
#pragma unroll
        for (int u = 0; u < kKsNB; ++u) acc[i][u] = float4_t{0.f, 0.f, 0.f, 0.f};

    // Prologue: steps 0 .. 2 requested in the loop's order (metadata of the
    // groups they open, atoms, A); constants of step 0's group; B operand of
    // step 0, block 0.  Metadata slot m holds the group that opens at chunk
    // step m * SPG.
    Slot ring[kKsCS];
    Meta meta[MPC];
#pragma unroll
    for (int j = 0; j < kKsLead; ++j) {
        if (j % SPG == 0) load_meta(j, meta[j / SPG]);
        load_w(j, ring[j]);
#pragma unroll
        for (int i = 0; i < kKsRB; ++i) load_a(j, i, ring[j]);
    }
    vm_wait(kKsRB + loads_for(1) + loads_for(2));     // step 0's metadata and atoms
    tie_meta(meta[0]);
    tie_slot(ring[0]);
    DqConst<BF> kc[kKsNB];
#pragma unroll
    for (int u = 0; u < kKsNB; ++u) kc[u] = make_const(meta[0], u);
    u32x4 bop[2];
    {
        DqSt<BF> st;
#pragma unroll
        for (int k = 0; k < S; ++k) dq_micro(k, ring[0], 0, kc[0], st);
        bop[0] = st.out;
    }
    // the accumulators' zeros are written before the gap
#pragma unroll
    for (int i = 0; i < kKsRB; ++i)
#pragma unroll
        for (int u = 0; u < kKsNB; ++u) asm volatile("" : "+a"(acc[i][u]));
    mfma_hazard_gap();

    for (int ch = 0; ch < chunks; ++ch) {
#pragma unroll
        for (int j = 0; j < kKsCS; ++j) {
            const int step = ch * kKsCS + j;
            const int jl = (j + kKsLead) % kKsCS;          // ring slot of step + 3 (held step - 1)
            const bool meta_req = jl % SPG == 0;           // step + 3 opens a group
            const bool new_group = (j + 1) % SPG == 0;     // step + 1 opens a group
            const int jn = (j + 1) % kKsCS;                // ring slot of step + 1
#pragma unroll
            for (int u = 0; u < kKsNB; ++u) {
                // operand dequantized under block u: block u + 1 of this step,
                // or block 0 of the next step under the last block
                const int du = (u + 1) % kKsNB;
                const Slot& src = ring[u + 1 < kKsNB ? j : jn];
                DqSt<BF> st;
#pragma unroll
                for (int i = 0; i < kKsRB; ++i) {
                    const int q = u * kKsRB + i;
                    __builtin_amdgcn_sched_barrier(0);
                    if (i == 0) {
                        // two wait states between the last write of this
                        // block's operand (end of the block before) and its
                        // first MFMA
                        asm volatile("s_nop 1");
                        if (u == 0) {
                            // this step's A: everything requested for steps
                            // up to this one has landed, the requests for the
                            // next two steps stay in flight
                            vm_wait(loads_for(j + 1) + loads_for(j + 2));
#pragma unroll
                            for (int r = 0; r < kKsRB; ++r) tie(ring[j].a[r]);
                        }
                        if (u == kKsMetaWaitBlock) {
                            // the next step's atoms and metadata (its A and
                            // the requests of the last two steps in flight)
                            vm_wait(kKsRB + loads_for(j + 2) + loads_for(j + 3));
#pragma unroll
                            for (int pp = 0; pp < PANELS; ++pp) tie(ring[jn].w[pp]);
                            if (new_group) tie_meta(meta[jn / SPG]);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    if (meta_req && q == kKsMetaSlot) load_meta(step + kKsLead, meta[jl / SPG]);
                    if (q == kKsAtomSlot) load_w(step + kKsLead, ring[jl]);
                    if (q >= kKsASlot && q < kKsASlot + kKsASlotStride * kKsRB && (q - kKsASlot) % kKsASlotStride == 0)
                        load_a(step + kKsLead, (q - kKsASlot) / kKsASlotStride, ring[jl]);
                    // constants of the group step + 1 opens; block v's old
                    // ones were last used under block v - 1
#pragma unroll
                    for (int v = 0; v < kKsNB; ++v)
                        if (new_group && q == kKsConstSlot[v]) kc[v] = make_const(meta[jn / SPG], v);
#pragma unroll
                    for (int k = i * S / kKsRB; k < (i + 1) * S / kKsRB; ++k) dq_micro(k, src, du, kc[du], st);
                    mfma_acc<BF>(acc[i][u], bop[u & 1], ring[j].a[i]);
                }
                bop[du & 1] = st.out;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // the requests of the last three steps (clamped, unused) land before any
    // of their registers is reused
    vm_wait(0);
#pragma unroll
    for (int j = 0; j < kKsCS; ++j) tie_slot(ring[j]);
#pragma unroll
    for (int m = 0; m < MPC; ++m) tie_meta(meta[m]);
    mfma_hazard_gap();

    // Sum the four K quarters in quarter order: every wave parks its sums,
    // then wave w adds row block w of all four and stores it.
#pragma unroll
    for (int i = 0; i < kKsRB; ++i)
#pragma unroll
        for (int u = 0; u < kKsNB; ++u) red[wave][i * kKsNB + u][lane] = acc[i][u];
    __syncthreads();
    const int i = wave;
    const int64_t row = row0 + 16 * i + c;
#pragma unroll
    for (int u = 0; u < kKsNB; ++u) {
        const int b = i * kKsNB + u;
        float4_t v = red[0][b][lane];
#pragma unroll
        for (int w = 1; w < kKsWaves; ++w) v += red[w][b][lane];
        // weights were the first MFMA operand: lane holds row c of the block
        // and columns 4 kg .. 4 kg + 3 (N % 8 == 0, so all four or none fit)
        const int64_t col = col0 + 16 * u + 4 * kg;
        if (row < M && col < N) {
            const uint2 o{round_out2<BF>(v[0], v[1]), round_out2<BF>(v[2], v[3])};
            *reinterpret_cast<uint2*>(C + row * N + col) = o;
        }
    }
}

template <int BITS, int MPC, bool BF>
int launch_ks(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M, hipStream_t s) {
    const int tiles_m = (int)((M + kKsBM - 1) / kKsBM);
    const int tiles_n = (int)((L.N + kKsBN - 1) / kKsBN);
    const int gshift = __builtin_ctz((unsigned)L.group);
    if (log_enabled())
        log_plan("gemm_ks_kernel<%d,%d,%s> M=%lld K=%lld N=%lld G=%d: %dx%d tiles of 64x128, K in 4 quarters "
                 "per workgroup", BITS, MPC, BF ? "bf16" : "f16", (long long)M, (long long)L.K, (long long)L.N,
                 L.group, tiles_m, tiles_n);
    return launch(gemm_ks_kernel<BITS, MPC, BF>, dim3((unsigned)(tiles_m * tiles_n)), dim3(kKsThreads), 0, s, A,
                  pk, C, (int)M, (int)L.K, (int)L.N, gshift, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np,
                  tiles_m, tiles_n);
}

template <int BITS, bool BF>
int launch_ks_bits(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                   hipStream_t s) {
    const int chunk_rows = kKsBK * kKsCS;
    const int mpc = L.group >= chunk_rows ? 1 : chunk_rows / L.group;
    if (mpc == 1) return launch_ks<BITS, 1, BF>(L, A, pk, C, M, s);
    if (mpc == 2) return launch_ks<BITS, 2, BF>(L, A, pk, C, M, s);
    return launch_ks<BITS, 4, BF>(L, A, pk, C, M, s);
}

}  // namespace

bool gemm_ks_supported(const Layout& L) {
    const int chunk_rows = kKsBK * kKsCS;
    return L.K % chunk_rows == 0 && L.K / chunk_rows >= kKsWaves && (L.group & (L.group - 1)) == 0;
}

int launch_gemm_ks(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                   hipStream_t s, bool bf) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (bf)
        return L.bits == 4 ? launch_ks_bits<4, true>(L, A, pk, C, M, s) : launch_ks_bits<8, true>(L, A, pk, C, M, s);
    return L.bits == 4 ? launch_ks_bits<4, false>(L, A, pk, C, M, s) : launch_ks_bits<8, false>(L, A, pk, C, M, s);
}

}  // namespace tf
