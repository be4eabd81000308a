// Prefill GEMM for the sizes whose output tiles are too few to give every
// compute unit one of the larger tiles (Section 2.1; Section 4.3 "GEMM
// microkernel"; Section 4.4):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 or bf16 MFMA, fp32 sums.
//
// Workgroup tile 64 x BN (BN = 128, or 256 for 4-bit weights where the
// wider tiles still fill the chip), four waves, one per SIMD.  Each wave computes the
// whole tile over its own quarter of K (a contiguous run of 128-row chunks),
// and no partial sum leaves the compute unit; inside the loop the waves share
// nothing and never wait for each other.
//  - A goes through a private LDS ring of four buffers per wave, each one pair
//    of 32-row steps (64 rows x 128 bytes), requested three pairs ahead by
//    direct global-to-LDS loads that move 8 whole rows each; the wave reads
//    each step's MFMA fragments (16 rows x 16 bytes per lane) a step ahead.
//    (The fragment layout straight from memory, 16 rows x 64 bytes per load,
//    cost a fifth more time.)
//  - The packed atoms of the tile's columns (one per panel per step) go into
//    a register ring of four steps, requested three steps ahead; the metadata
//    of a group travels with the atoms of the step that opens it.  All loads
//    are asm statements with counted waits, issued metadata, atoms, A in the
//    order their waits need them (vector-memory loads complete in order).
//  - A step's MFMAs run column block by column block (BN / 16 blocks of 16
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

constexpr int kKsBM = 64, kKsBK = 32;
constexpr int kKsWaves = 4, kKsThreads = 64 * kKsWaves;
constexpr int kKsCS = 4;                // steps per chunk (128 rows of K) and ring slots
constexpr int kKsLead = 3;              // steps between a request and its step
constexpr int kKsRB = kKsBM / 16;       // row blocks
constexpr int kKsSumNB = 8;             // column blocks per pass of the quarters' sum
constexpr int kKsXcds = 8;
constexpr int kKsRing = 4;              // A buffers per wave, one pair of steps each
constexpr int kKsPairBytes = kKsBM * 2 * kKsBK * 2;   // 64 rows x 128 bytes
constexpr int kKsALead = 3;             // pairs between a pair's A request and its first step

// A step's 32 MFMA slots, block u = slot / 4 (columns 16 u ..), row block
// i = slot % 4.  Requests sit at fixed slots: the metadata of step + 3 (when
// it opens a group) at kKsMetaSlot, its atoms at kKsAtomSlot, and the step's
// four direct loads of A (half a pair) at kKsASlot + kKsASlotStride * r.
constexpr int kKsMetaSlot = 0, kKsAtomSlot = 4, kKsASlot = 8, kKsASlotStride = 3;
// The step waits twice: for its own fragments (LDS reads) at block 0, for
// the next step's atoms and metadata, and so for every pair of A requested
// before them, at block kKsMetaWaitBlock; the next step's fragments are read
// from kKsReadSlot, and the constants of the group the next step opens are
// formed after that wait, those of block v at slot kKsConstSlot[v] (block v's
// old constants were last used under block v - 1).
constexpr int kKsMetaWaitBlock = 5;
constexpr int kKsReadSlot = 24;         // the next step's fragments, after that wait
constexpr int kKsConstSlot[16] = {20, 21, 22, 23, 24, 25, 26, 28, 32, 36, 40, 44, 48, 52, 56, 60};
static_assert(kKsMetaSlot < kKsAtomSlot && kKsAtomSlot < kKsASlot, "requests go out metadata, atoms, A");
static_assert(kKsASlot + kKsASlotStride * (kKsRB - 1) < kKsMetaWaitBlock * kKsRB,
              "a step's requests are all issued before its second wait counts them");
constexpr bool ks_const_slots_ok(int nb) {
    for (int v = 0; v < nb; ++v) {
        const int blk = kKsConstSlot[v] / kKsRB;
        if (blk < kKsMetaWaitBlock || blk < v || blk >= nb) return false;
    }
    return true;
}
static_assert(ks_const_slots_ok(8) && ks_const_slots_ok(16),
              "constants formed after the wait and after their old value's last use");
static_assert(kKsReadSlot >= kKsMetaWaitBlock * kKsRB && kKsReadSlot < 8 * kKsRB,
              "the next step's fragments are read after the wait that completes their pair");
// The pair holding step s + 1 was requested during steps up to
// 2 (kKsALead - 1) before it, which the wait at step s completes when that is
// at least 4 (everything issued up to step s - 3); a buffer is refilled only
// after the last read of the pair it held.
static_assert(2 * (kKsALead - 1) >= 4 && kKsRing >= kKsALead + 1, "A lead and ring size");

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
// 16 bytes per lane from a buffer straight into LDS at lds + 16 * lane (M0
// holds the LDS address; nothing else in these kernels uses M0).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(i32x4 r, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                 :: "v"(voff), "s"(r), "s"(soff), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop
template <int OFF>
__device__ __forceinline__ u32x4 ds_read16(uint32_t addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
    return v;
}
// Every LDS read of this wave has returned.
__device__ __forceinline__ void lgkm_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// MPC: metadata groups per chunk (1 when a group spans the chunk, else chunk
// rows / group).  BN: tile columns.
template <int BITS, int MPC, bool BF, int BN>
__global__ __launch_bounds__(kKsThreads, 1) void gemm_ks_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int gshift, int64_t s_off, int64_t z_off, int na, int ng, int np,
    int tiles_m, int tiles_n, KsRange rg) {
    constexpr int PW = BITS == 4 ? 64 : 32;   // columns per panel (one atom per step)
    constexpr int T = PW / 16;                // column blocks per panel
    constexpr int PANELS = BN / PW;
    constexpr int NB = BN / 16;               // column blocks: B operands per step
    static_assert(BN == 128 || (BN == 256 && BITS == 4), "tiles of 64 x 128, or 64 x 256 for 4-bit weights");
    constexpr int SPG = kKsCS / MPC;          // steps per metadata group
    constexpr int S = dq_steps<BF, BITS>();   // dequantization micro-steps per operand
    static_assert(kKsRB + 2 * (kKsRB + 3 * PANELS) <= 40, "counted waits stay within vm_wait's range");
    // A's per-wave rings during the loop; the K quarters' sums after it, in
    // passes of 8 column blocks (wave w's quarter of the sum buffer is exactly
    // its own ring)
    __shared__ __align__(16) float4_t lds[kKsWaves][kKsRB * kKsSumNB][64];
    static_assert(sizeof(lds) == kKsWaves * kKsRing * kKsPairBytes, "ring and sum buffer coincide");

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 15, kg = lane >> 4;
    const uint32_t magic = magic_reg();

    // Block b runs on XCD b % 8, which takes the (b % 8)-th contiguous band
    // of the tile list: all tiles with row tiles varying fastest, or, over a
    // range of 256 x 256 tiles, the UPT tiles of 64 x BN of each in turn.
    constexpr int CPT = 256 / BN, UPT = 4 * CPT;
    int unit;
    {
        const int total = rg.count ? rg.count * UPT : tiles_m * tiles_n;
        const int b = blockIdx.x;
        const int per = total / kKsXcds, rem = total % kKsXcds;
        const int x = b % kKsXcds, i = b / kKsXcds;
        unit = x * per + min(x, rem) + i;
    }
    // (pinned to scalar registers: integer division runs on the vector ALU,
    // and buffer resources built from a value the compiler cannot prove
    // uniform would be loaded lane by lane)
    int tm, tn;
    if (rg.count) {
        const int t = rg.tile0 + unit / UPT, sub = unit % UPT;
        const int tm2 = rg.col_major ? t % rg.tiles_m : t / rg.tiles_n;
        const int tn2 = rg.col_major ? t / rg.tiles_m : t % rg.tiles_n;
        tm = __builtin_amdgcn_readfirstlane(4 * tm2 + sub / CPT);
        tn = __builtin_amdgcn_readfirstlane(CPT * tn2 + sub % CPT);
    } else {
        tm = __builtin_amdgcn_readfirstlane(unit % tiles_m);
        tn = __builtin_amdgcn_readfirstlane(unit / tiles_m);
    }
    const int64_t row0 = (int64_t)tm * kKsBM, col0 = (int64_t)tn * BN;
    // a 64 x BN part of a 256 x 256 tile can lie wholly past C (the whole
    // workgroup leaves before any load or barrier)
    if (row0 >= M || col0 >= N) return;

    // This wave's K quarter (the launcher guarantees at least one chunk each).
    const int nch = na / kKsCS;
    const int qch = nch / kKsWaves, rch = nch % kKsWaves;
    const int ch0 = __builtin_amdgcn_readfirstlane(wave * qch + min(wave, rch));
    const int chunks = __builtin_amdgcn_readfirstlane(qch + (wave < rch ? 1 : 0));
    const int st0 = ch0 * kKsCS, steps = chunks * kKsCS;

    // A: the wave's K quarter in pairs of steps (64 rows x 128 bytes), each
    // through one buffer of the wave's LDS ring.  A direct load moves 8 whole
    // rows (lane l: row l / 8 of the 8, 16-byte chunk (l % 8) ^ (row % 8) to
    // LDS position l % 8); rows past M read row M - 1 (in bounds; never
    // stored).  The fragment of row block i for step s (half h of its pair):
    // lane l reads row 16 i + c at chunk 4 h + kg, held at position
    // (4 h + kg) ^ (c % 8).
    const int rows = __builtin_amdgcn_readfirstlane(min(M - tm * kKsBM, kKsBM));
    const i32x4 ar = rsrc_words(A + row0 * K, (uint32_t)rows * (uint32_t)K * 2u);
    const int pairs = steps / 2;
    const uint32_t wlds = __builtin_amdgcn_readfirstlane(
        (uint32_t)reinterpret_cast<uintptr_t>(&lds[0][0][0]) + (uint32_t)wave * (kKsRing * kKsPairBytes));
    // Each direct load's row offset sits in its own per-lane offset (rows past
    // M clamped to the last row, so every read stays inside A whatever part of
    // the address the buffer's range check covers); the pair's K offset is the
    // scalar offset.
    uint32_t vb[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        const uint32_t row = (uint32_t)min(8 * g + (lane >> 3), rows - 1);
        vb[g] = row * (uint32_t)K * 2u + (uint32_t)((lane & 7) ^ (lane >> 3)) * 16u;
    }
    uint32_t rb[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) rb[h] = wlds + (uint32_t)(c * 128 + (((4 * h + kg) ^ (c & 7)) * 16));
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
    // direct load g (0..7, rows 8 g ..) of pair `pair`'s A into its ring buffer
    auto dma_a = [&](int pair, int g) {
        const uint32_t buf = wlds + (uint32_t)(pair & (kKsRing - 1)) * kKsPairBytes + (uint32_t)g * 1024u;
        pair = min(pair, pairs - 1);       // clamped: a repeated valid pair, never read
        dma16(ar, vb[g], (uint32_t)(st0 + 2 * pair) * (kKsBK * 2), buf);
    };
    // the four fragments of step `step` from its pair's buffer
    auto read_af = [&](int step, u32x4 (&af)[kKsRB]) {
        const uint32_t base = rb[step & 1] + (uint32_t)((step >> 1) & (kKsRing - 1)) * kKsPairBytes;
        af[0] = ds_read16<0 * 16 * 128>(base);
        af[1] = ds_read16<1 * 16 * 128>(base);
        af[2] = ds_read16<2 * 16 * 128>(base);
        af[3] = ds_read16<3 * 16 * 128>(base);
    };
    // the direct loads issued during step t: half t % 2 of pair t / 2 + 3
    auto dma_step = [&](int t, int r) { dma_a((t >> 1) + kKsALead, 4 * (t & 1) + r); };
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
    // Loads issued in the step that requests step t's operands: t's metadata
    // when t opens a group, its atoms, and that step's four direct loads of A
    // (half a pair): what a counted wait leaves in flight per step.
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

    float4_t acc[kKsRB][NB];
#pragma unroll
    for (int i = 0; i < kKsRB; ++i)
#pragma unroll
        for (int u = 0; u < NB; ++u) acc[i][u] = float4_t{0.f, 0.f, 0.f, 0.f};

    // Prologue: the requests of steps -6 .. -1 in the loop's order (the
    // direct loads of pairs 0 and 1 and half of 2... as steps -6 .. -4 issue
    // them; then per step -3 .. -1 the metadata and atoms of step + 3 and its
    // half pair), so the loop's counted waits see the same queue at its entry
    // as at its back edge; then step 0's constants, B operand and fragments.
    // Metadata slot m holds the group that opens at chunk step m * SPG.
    Slot ring[kKsCS];
    Meta meta[MPC];
#pragma unroll
    for (int t = -6; t < -3; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) dma_step(t, r);
#pragma unroll
    for (int j = 0; j < kKsLead; ++j) {
        if (j % SPG == 0) load_meta(j, meta[j / SPG]);
        load_w(j, ring[j]);
#pragma unroll
        for (int r = 0; r < 4; ++r) dma_step(j - kKsLead, r);
    }
    vm_wait(4 + loads_for(1) + loads_for(2));     // step 0's metadata, atoms and pair
    tie_meta(meta[0]);
    tie_slot(ring[0]);
    u32x4 af[2][kKsRB];
    read_af(0, af[0]);
    DqConst<BF> kc[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) kc[u] = make_const(meta[0], u);
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
        for (int u = 0; u < NB; ++u) asm volatile("" : "+a"(acc[i][u]));
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
            for (int u = 0; u < NB; ++u) {
                // operand dequantized under block u: block u + 1 of this step,
                // or block 0 of the next step under the last block
                const int du = (u + 1) % NB;
                const Slot& src = ring[u + 1 < NB ? j : jn];
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
                            // this step's fragments (read a step ago)
                            lgkm_wait();
#pragma unroll
                            for (int r = 0; r < kKsRB; ++r) tie(af[j & 1][r]);
                        }
                        if (u == kKsMetaWaitBlock) {
                            // the next step's atoms and metadata, and with
                            // them the A pairs requested before them (the
                            // direct loads that followed them and the
                            // requests of the last two steps in flight)
                            vm_wait(4 + loads_for(j + 2) + loads_for(j + 3));
#pragma unroll
                            for (int pp = 0; pp < PANELS; ++pp) tie(ring[jn].w[pp]);
                            if (new_group) tie_meta(meta[jn / SPG]);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    if (meta_req && q == kKsMetaSlot) load_meta(step + kKsLead, meta[jl / SPG]);
                    if (q == kKsAtomSlot) load_w(step + kKsLead, ring[jl]);
                    if (q >= kKsASlot && q < kKsASlot + kKsASlotStride * 4 && (q - kKsASlot) % kKsASlotStride == 0)
                        dma_step(step, (q - kKsASlot) / kKsASlotStride);
                    if (q == kKsReadSlot) read_af(step + 1, af[(j + 1) & 1]);
                    // constants of the group step + 1 opens; block v's old
                    // ones were last used under block v - 1
#pragma unroll
                    for (int v = 0; v < NB; ++v)
                        if (new_group && q == kKsConstSlot[v]) kc[v] = make_const(meta[jn / SPG], v);
#pragma unroll
                    for (int k = i * S / kKsRB; k < (i + 1) * S / kKsRB; ++k) dq_micro(k, src, du, kc[du], st);
                    mfma_acc<BF>(acc[i][u], bop[u & 1], af[j & 1][i]);
                }
                bop[du & 1] = st.out;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // the requests of the last three steps (clamped, unused) land before any
    // of their registers is reused
    vm_wait(0);
    lgkm_wait();
#pragma unroll
    for (int j = 0; j < kKsCS; ++j) tie_slot(ring[j]);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < kKsRB; ++r) tie(af[h][r]);
#pragma unroll
    for (int m = 0; m < MPC; ++m) tie_meta(meta[m]);
    mfma_hazard_gap();

    // Sum the four K quarters in quarter order, 8 column blocks per pass:
    // every wave parks its sums, then wave w adds row block w of all four and
    // stores it.
    const int i = wave;
    const int64_t row = row0 + 16 * i + c;
#pragma unroll
    for (int h = 0; h < NB / kKsSumNB; ++h) {
        if (h > 0) __syncthreads();     // the previous pass's sums have been read
#pragma unroll
        for (int r = 0; r < kKsRB; ++r)
#pragma unroll
            for (int u = 0; u < kKsSumNB; ++u) lds[wave][r * kKsSumNB + u][lane] = acc[r][h * kKsSumNB + u];
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kKsSumNB; ++u) {
            const int b = i * kKsSumNB + u;
            float4_t v = lds[0][b][lane];
#pragma unroll
            for (int w = 1; w < kKsWaves; ++w) v += lds[w][b][lane];
            // weights were the first MFMA operand: lane holds row c of the
            // block and columns 4 kg .. 4 kg + 3 (N % 8 == 0, so all four or
            // none fit)
            const int64_t col = col0 + 16 * (h * kKsSumNB + u) + 4 * kg;
            if (row < M && col < N) {
                const uint2 o{round_out2<BF>(v[0], v[1]), round_out2<BF>(v[2], v[3])};
                *reinterpret_cast<uint2*>(C + row * N + col) = o;
            }
        }
    }
}

template <int BITS, int MPC, bool BF, int BN>
int launch_ks(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M, const KsRange& rg,
              hipStream_t s) {
    const int tiles_m = (int)((M + kKsBM - 1) / kKsBM);
    const int tiles_n = (int)((L.N + BN - 1) / BN);
    const int gshift = __builtin_ctz((unsigned)L.group);
    const int blocks = rg.count ? rg.count * 4 * (256 / BN) : tiles_m * tiles_n;
    if (log_enabled()) {
        if (rg.count)
            log_plan("  gemm_ks_kernel<%d,%d,%s,%d>: 256x256 tiles %d..%d as %d tiles of 64x%d, K in 4 quarters "
                     "per workgroup", BITS, MPC, BF ? "bf16" : "f16", BN, rg.tile0, rg.tile0 + rg.count - 1, blocks,
                     BN);
        else
            log_plan("gemm_ks_kernel<%d,%d,%s,%d> M=%lld K=%lld N=%lld G=%d: %dx%d tiles of 64x%d, K in 4 quarters "
                     "per workgroup", BITS, MPC, BF ? "bf16" : "f16", BN, (long long)M, (long long)L.K,
                     (long long)L.N, L.group, tiles_m, tiles_n, BN);
    }
    return launch(gemm_ks_kernel<BITS, MPC, BF, BN>, dim3((unsigned)blocks), dim3(kKsThreads), 0, s, A, pk, C,
                  (int)M, (int)L.K, (int)L.N, gshift, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np, tiles_m,
                  tiles_n, rg);
}

template <int BITS, bool BF, int BN>
int launch_ks_bits(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                   const KsRange& rg, hipStream_t s) {
    const int chunk_rows = kKsBK * kKsCS;
    const int mpc = L.group >= chunk_rows ? 1 : chunk_rows / L.group;
    if (mpc == 1) return launch_ks<BITS, 1, BF, BN>(L, A, pk, C, M, rg, s);
    if (mpc == 2) return launch_ks<BITS, 2, BF, BN>(L, A, pk, C, M, rg, s);
    return launch_ks<BITS, 4, BF, BN>(L, A, pk, C, M, rg, s);
}

// 64 x 256 tiles (4-bit weights only): twice the MFMA work per byte a
// compute unit loads, at about 1.5 times a 64 x 128 tile's time (one round of
// either at K = 4096, N = 14336: 32.4 against 21.4 us).  Taken when whole
// rounds of them at that cost beat the 64 x 128 tiles' rounds counted
// fractionally (a short last round of small tiles runs faster than a full
// one).  Measured on MI355X (graph replay, fp16; 64 x 128 -> 64 x 256):
// K = 4096, N = 14336, M = 256 and 512 41.2 -> 37.0 and 80.5 -> 70.3 us;
// K = 4096, N = 4096, M = 1000 43.3 -> 38.7 us; K = 4096, N = 11008, M = 300
// 40.0 -> 35.2 us; left at 64 x 128: N = 14336, M = 128, 384, 640 (21.4, 61,
// 100 against 32.4, 67, 103.5 us) and K = 8192, N = 8192, M = 200 (39.2
// against 56 us).
constexpr int64_t kKsWideCostHalves = 3;    // a 64 x 256 tile's time in halves of a 64 x 128 tile's
bool gemm_ks_wide(const Layout& L, int64_t M, hipStream_t s) {
    if (L.bits != 4) return false;
    const int64_t cus = device_cus(s);
    const int64_t tm = (M + 63) / 64;
    const int64_t t128 = tm * ((L.N + 127) / 128), t256 = tm * ((L.N + 255) / 256);
    return 2 * t128 > kKsWideCostHalves * ((t256 + cus - 1) / cus) * cus;
}

int launch_any(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M, const KsRange& rg,
               hipStream_t s, bool bf, bool wide) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (L.bits == 8)
        return bf ? launch_ks_bits<8, true, 128>(L, A, pk, C, M, rg, s)
                  : launch_ks_bits<8, false, 128>(L, A, pk, C, M, rg, s);
    if (wide)
        return bf ? launch_ks_bits<4, true, 256>(L, A, pk, C, M, rg, s)
                  : launch_ks_bits<4, false, 256>(L, A, pk, C, M, rg, s);
    return bf ? launch_ks_bits<4, true, 128>(L, A, pk, C, M, rg, s)
              : launch_ks_bits<4, false, 128>(L, A, pk, C, M, rg, s);
}

}  // namespace

bool gemm_ks_supported(const Layout& L) {
    const int chunk_rows = kKsBK * kKsCS;
    return L.K % chunk_rows == 0 && L.K / chunk_rows >= kKsWaves && (L.group & (L.group - 1)) == 0;
}

int launch_gemm_ks(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                   hipStream_t s, bool bf) {
    return launch_any(L, A, packed, C, M, KsRange{0, 0, 0, 0, 0}, s, bf, gemm_ks_wide(L, M, s));
}

int launch_gemm_ks_range(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                         const KsRange& rg, hipStream_t s, bool bf) {
    if (rg.count <= 0) return TF_OK;
    return launch_any(L, A, packed, C, M, rg, s, bf, false);
}

}  // namespace tf
