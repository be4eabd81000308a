// Prefill GEMM for large M (Section 2.1; Section 4.3 "GEMM microkernel"):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 MFMA, fp32 accumulate.
//
// One workgroup of four waves per compute unit (one wave per SIMD, so each
// wave has the whole 512-entry register file: 256 accumulators plus operands).
// Workgroup tile 256 x 256; each wave owns all 256 rows x 64 columns (one
// 4-bit panel or two 8-bit panels).  The dequantization of a 32 x 64 weight
// step (Eq. 2, rounded once) is therefore reused across 16 row blocks: about
// one vector-ALU instruction per v_mfma_f32_16x16x32_f16, which the SIMD
// issues while the matrix core works (Sections 4.1.1 and 4.3: dequantize each
// weight tile once and reuse it for every activation row).
//  - A (fp16) goes global -> LDS by direct loads, two K steps at a time:
//    three buffers of 256 rows x 64 halves (128 bytes per row, so each direct
//    load brings eight whole rows of cache lines), rows XOR-swizzled in 16-byte
//    chunks so fragment reads are free of bank conflicts; one barrier per step.
//  - A fragments are read from LDS in two bursts per step, a half step ahead
//    of their use, and the dequantization runs in the parts of the step where
//    no LDS data is returning: measured on MI355X, LDS reads interleaved one
//    by one with vector-ALU work stall the matrix core far more than the same
//    work kept apart.
//  - The wave's packed atoms are loaded three steps ahead into a register
//    ring and dequantized one step ahead, straight into the B-operand layout.
//  - Loads go through buffer resources: the step advances a scalar offset,
//    and rows past M or panels past N read as zero (hardware range check).
//  - Tiles are dealt so each XCD (blocks go round-robin over the 8 XCDs)
//    walks a contiguous band of the tile list; the list runs along whichever
//    operand is larger so that operand is fetched by fewer XCD caches.
#include <algorithm>

#include "tf_internal.h"

namespace tf {
namespace {

constexpr int kBM = 256, kBN = 256, kBK = 32;
constexpr int kThreads = 256;
constexpr int kXcds = 8;
constexpr int kCS = 4;                 // steps per 128-row chunk (atom ring size)
constexpr int kPairK = 2 * kBK;        // K rows per A buffer (two steps)
constexpr int kPairBufs = 3;           // A buffers: the pair being read, the next, one landing
constexpr int kPairBytes = kBM * kPairK * 2;   // 32 KB
constexpr int kRowBytes = kPairK * 2;  // 128 bytes of A per row per buffer
constexpr int kRB = kBM / 16;          // 16-row blocks per wave
constexpr int kSkMinUnits = 8;         // fewest K chunks per block when every tile is split

// A buffer layout: row r of the tile at byte r * 128; its 16-byte chunk of
// halves 8 l .. 8 l + 7 (l = 0..7) at position l ^ a_swz(r).  A fragment read
// covers 16 rows (16 i .. 16 i + 15) at one logical chunk.  Measured on
// MI355X (SQ_LDS_BANK_CONFLICT over this exact read pattern): the XOR with
// row & 7 reads a fragment in 4 LDS cycles without bank conflicts, as a
// contiguous 1 KB read does; adding (row >> 3) & 1 to it costs 4 more.
__device__ __forceinline__ int a_swz(int row) { return row & 7; }

// 16-byte LDS read issued as an asm statement, so the compiler neither waits
// for the direct loads in flight into the other A buffers (it cannot tell the
// buffers of one array apart) nor for the read itself: the kernel waits for
// its reads explicitly (lds_wait) before their first use.
template <int OFF>
__device__ __forceinline__ u32x4 lds_read16_at(uint32_t addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
    return v;
}
// fragment of row block i (16 rows x 128 bytes = 2 KB apart); i is a
// constant once the step's slot loop is unrolled
__device__ __forceinline__ u32x4 lds_read_block(uint32_t addr, int i) {
    switch (i) {
#define TF_BLOCK(n) \
    case n: return lds_read16_at<(n) * 16 * kRowBytes>(addr);
        TF_BLOCK(0) TF_BLOCK(1) TF_BLOCK(2) TF_BLOCK(3) TF_BLOCK(4) TF_BLOCK(5) TF_BLOCK(6) TF_BLOCK(7)
        TF_BLOCK(8) TF_BLOCK(9) TF_BLOCK(10) TF_BLOCK(11) TF_BLOCK(12) TF_BLOCK(13) TF_BLOCK(14) TF_BLOCK(15)
#undef TF_BLOCK
        default: return lds_read16_at<0>(addr);
    }
}
// every LDS read of this wave has returned
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// The weights go in as the first operand and the activations as the second,
// so each accumulator block is a 16 (n) x 16 (m) tile of C transposed: lane l
// holds row m = l % 16 of C and four consecutive columns n = 4 (l / 16) + r,
// which the epilogue stores as one 8-byte write.
// Hazards around mfma_acc (see there): the loop body is its own basic block,
// so mfma_hazard_gap() placed before and after the loop covers the
// accumulator initialisation and the epilogue's reads; inside the loop,
// accumulators are only read by further MFMAs of the same shape (no wait
// needed) and B operands are produced a whole K step (and a barrier) ahead of
// their use.

// End-of-step barrier.  The A tile of step s + 3 reaches LDS by direct
// global-to-LDS loads issued during step s; its first fragments are read
// during step s + 2, so at the end of every step the direct loads issued in
// the step before must have landed (each wave waits for its own, then the
// barrier makes all of them visible).  Vector-memory operations complete in
// order, so the wait leaves in flight exactly the NOW operations this step
// issued (its atom loads, its four direct loads and, on a chunk's last step,
// the metadata loads of the chunk after next), which are needed a step or
// more later: a weight atom three steps on, metadata four.  LDS reads
// issued before the barrier stay in flight (no LDS wait).  s_waitcnt fields:
// vmcnt = NOW (bits 3..0 and 15..14), expcnt and lgkmcnt at their maximum.
__device__ __forceinline__ void barrier_only() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}
template <int NOW>
__device__ __forceinline__ void barrier_after_a_loads() {
    static_assert(NOW >= 4 && NOW < 64, "vmcnt holds 6 bits");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0x0F70 | (NOW & 15) | ((NOW >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Work split.  Data-parallel (sk.groups == 0): block b computes one whole
// tile.  Stream-K (sk.groups = G > 0): the tiles x chunks 128-row K chunks of
// the whole problem, tile-major, are cut into G equal contiguous ranges, one
// per block; a block walks its range tile by tile, so a tile may be computed
// in several K segments by consecutive blocks.  Every segment of a split
// tile parks its fp32 partial tile in the workspace (slot 2v for the first
// segment of block v's range, 2v + 1 for its last), and a second launch on
// the same stream (stream_k_reduce_kernel, spread over all compute units)
// adds each split tile's segments in K order and writes C; the kernel
// boundary orders the parked stores before those loads on every XCD.
// (Summing in the last segment to arrive left one block per tile streaming
// the other parts while the rest of the GPU idled.)

struct StreamK {
    int groups;               // G, 0 = data-parallel
    int units;                // tiles * chunks
    float* part;              // 2 G partial tiles of kBM x kBN floats
    int dp_rounds;            // hybrid: whole tiles per block before the stream-K units
};

__device__ __forceinline__ int sk_owner(int64_t u, int G, int U) {   // block whose range holds u
    return (int)(((u + 1) * G - 1) / U);
}
__device__ __forceinline__ int sk_begin(int v, int G, int U) { return (int)((int64_t)v * U / G); }

// Slots of a K step's 64 that carry dequantization micro-steps: two windows,
// [W, 32) and [W + 32, 64), after the two LDS read bursts (slots 0..7 and
// 32..39) have returned.  fp16 (52 or 48 micro-steps) uses W = 16, one or two
// per slot; bf16 (92 or 80) uses W = 8, at most two per slot.
template <bool BF>
constexpr int dq_window() { return BF ? 8 : 16; }
template <bool BF>
constexpr int dq_slots() { return 2 * (32 - dq_window<BF>()); }
template <bool BF>
constexpr int dq_index(int q) {
    return (q & 31) < dq_window<BF>() ? -1 : (q >> 5) * (32 - dq_window<BF>()) + (q & 31) - dq_window<BF>();
}
// micro-steps [dq_slot_begin, dq_slot_end) of R go to slot q
template <bool BF>
constexpr int dq_slot_begin(int q, int R) { return dq_index<BF>(q) < 0 ? 0 : dq_index<BF>(q) * R / dq_slots<BF>(); }
template <bool BF>
constexpr int dq_slot_end(int q, int R) { return dq_index<BF>(q) < 0 ? 0 : (dq_index<BF>(q) + 1) * R / dq_slots<BF>(); }

template <int BITS, int MPC, bool BF>
__global__ __launch_bounds__(kThreads, 1) void gemm256_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int gshift, int64_t s_off, int64_t z_off, int na, int ng, int np,
    int tiles_m, int tiles_n, int col_major, StreamK sk) {
    constexpr int PW = BITS == 4 ? 64 : 32;
    constexpr int T = PW / 16;                 // columns per lane per atom
    constexpr int PANELS = 64 / PW;            // panels per wave
    constexpr int SPG = kCS / MPC;             // steps per metadata group
    __shared__ __align__(16) uint8_t As[kPairBufs * kPairBytes];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 15, kg = lane >> 4;
    const uint32_t magic = magic_reg();
    const int steps = na;
    const int chunks = steps / kCS;            // the launcher requires K % 128 == 0
    constexpr int kDqSteps = dq_steps<BF, BITS>();
    constexpr int kDqTotal = 4 * kDqSteps;     // micro-steps per K step
    static_assert(kDqTotal <= 2 * dq_slots<BF>(), "at most two micro-steps per slot");

    // An A buffer (256 rows x 64 halves, 32 KB) arrives by eight direct loads
    // per thread, four in each of two steps; load r of wave w fills bytes
    // (8 w + r) KB .. + 1 KB (a direct load writes lane l's 16 bytes at its
    // base + 16 l), i.e. rows 64 w + 8 r .. + 7, eight lanes per row, so each
    // lane fetches the A chunk that belongs at its position (the inverse of
    // a_swz): eight whole 128-byte rows of A per load.
    uint32_t avoff[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        const int row = 64 * wave + 8 * r + (lane >> 3);
        const int lc = (lane & 7) ^ a_swz(row);
        avoff[r] = (uint32_t)row * (uint32_t)K * 2u + (uint32_t)lc * 16u;
    }
    // Fragment of row block i (rows 16 i + c, halves 8 kg .. + 7 of the step):
    // lane byte offset inside a buffer for an even (first) and an odd step;
    // the block adds 2 KB per i as an immediate offset.
    const uint32_t a_lds = (uint32_t)reinterpret_cast<uintptr_t>(As);
    uint32_t a_lane[2];
#pragma unroll
    for (int odd = 0; odd < 2; ++odd)
        a_lane[odd] = a_lds + (uint32_t)(c * kRowBytes + ((kg + 4 * odd) ^ a_swz(c)) * 16);
    struct Meta {
        uint32_t s[MPC][PANELS][(T + 1) / 2];   // T fp16 scales per group and panel
        uint32_t z[MPC][PANELS];                // T zero-point bytes
    };
    // Group constants of each lane column (see DqConst).
    struct Consts {
        DqConst<BF> q[4];
    };
    // constants of lane column u (panel u / T, column t = u % T)
    auto make_const = [&](const Meta& mt, int m, Consts& k, int u) {
        const int pp = u / T, t = u % T;
        DqConst<BF>& kq = k.q[u];
        if constexpr (BF) {
            const uint32_t sw = mt.s[m][pp][t / 2];
            kq.s = __builtin_bit_cast(float, (t & 1) ? (sw & 0xFFFF0000u) : (sw << 16));
            kq.nzs = -(byte_f32(mt.z[m][pp], t) * kq.s);
        } else {
            const uint32_t sh = mt.s[m][pp][t / 2] >> (16 * (t & 1));
            kq.s2 = as_h2(__builtin_amdgcn_perm(sh, sh, 0x01000100u));
            const uint32_t n = __builtin_amdgcn_perm(0xE4E4E4E4u, mt.z[m][pp], 0x04000400u | (t * 0x00010001u));
            kq.nz = n;
            kq.nz64 = neg_zero64_pair(n);
        }
    };
    auto make_consts = [&](const Meta& mt, int m, Consts& k) {
#pragma unroll
        for (int u = 0; u < 4; ++u) make_const(mt, m, k, u);
    };
    // Dequantization micro-step k of B operand u (0..3) from ring slot `slot`.
    auto dq_step_u = [&](int u, int k, const u32x4 (&slot)[PANELS], const Consts& kk, DqSt<BF>& st) {
        const int pp = u / T, t = u % T;
        dq_step<BF, BITS>(k, slot[pp][BITS == 4 ? t : 2 * t], slot[pp][BITS == 4 ? t : 2 * t + 1], magic,
                          kk.q[u], st);
    };
    auto dequant = [&](const u32x4 (&slot)[PANELS], const Consts& kk, u32x4 (&bop)[4]) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            DqSt<BF> st;
#pragma unroll
            for (int k = 0; k < kDqSteps; ++k) dq_step_u(u, k, slot, kk, st);
            bop[u] = st.out;
        }
    };

    // ---- output: 16-row blocks through a per-wave LDS staging area (rows
    // padded to 144 bytes), leaving as 16-byte stores, eight full 128-byte
    // rows per store instruction.  get(i, t) yields accumulator block (i, t):
    // row m = 16 i + c, columns n = 16 t + 4 kg + 0..3 of the wave's tile.
    // The caller has made sure no wave still reads the A buffers underneath.
    auto store_tile = [&](int64_t row0, int64_t col0, auto&& get_block) {
        uint8_t* stage = As + wave * 4096;
        constexpr int kStageRow = 144;
        const bool interior = row0 + kBM <= M && col0 + 64 <= N;
        const int rr = lane >> 3, cc = lane & 7;      // read-back: row rr (+8), 16-byte chunk cc
#pragma unroll
        for (int i = 0; i < kRB; ++i) {
            // one row block at a time: keep the scheduler from hoisting the
            // loads of every block (their registers would not fit)
            __builtin_amdgcn_sched_barrier(0);
            float4_t blk[4];
            get_block(i, blk);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float4_t a = blk[t];
                *reinterpret_cast<uint2*>(stage + c * kStageRow + 32 * t + 8 * kg) =
                    uint2{round_out2<BF>(a[0], a[1]), round_out2<BF>(a[2], a[3])};
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);       // lgkmcnt(0): this wave's stores landed
            u32x4 v[2];
#pragma unroll
            for (int h = 0; h < 2; ++h)
                v[h] = *reinterpret_cast<const u32x4*>(stage + (rr + 8 * h) * kStageRow + 16 * cc);
            __builtin_amdgcn_s_waitcnt(0xC07F);       // reads done before the area is rewritten
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t m = row0 + 16 * i + rr + 8 * h, n = col0 + 8 * cc;   // N % 8 == 0
                if (interior || (m < M && n < N)) *reinterpret_cast<u32x4*>(C + m * N + n) = v[h];
            }
        }
    };

    float4_t acc[kRB][4];

    // ---- one K segment: chunks [c0, c1) of tile `tile` into acc.
    auto segment = [&](int tile, int c0, int c1, int64_t& row0_out, int64_t& col0_out) {
        __syncthreads();   // the previous segment's output staging is done with the LDS
        // (uniform values; readfirstlane keeps the buffer resources in scalars)
        const int tm = __builtin_amdgcn_readfirstlane(col_major ? tile % tiles_m : tile / tiles_n);
        const int tn = __builtin_amdgcn_readfirstlane(col_major ? tile / tiles_m : tile % tiles_n);
        const int64_t row0 = (int64_t)tm * kBM;
        const int64_t col0 = (int64_t)tn * kBN + wave * 64;      // this wave's 64 columns
        row0_out = row0;
        col0_out = col0;

        // A: the tile's rows as one buffer (rows past M read as zero); a pair
        // of steps (256 rows x 64 halves) = 32 direct loads of 1 KB, 8 per
        // thread.
        const int rows = (int)min<int64_t>(kBM, (int64_t)M - row0);
        const __amdgpu_buffer_rsrc_t a_rsrc = make_rsrc(A + row0 * K, (uint32_t)rows * (uint32_t)K * 2u);
        const int pairs = steps / 2;
        auto dma_a = [&](int pair, uint32_t buf, int r) {  // direct load r (0..7) of a pair's A into buffer byte offset buf
            const uint32_t soff = (uint32_t)min(pair, pairs - 1) * kRowBytes;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                a_rsrc, (__attribute__((address_space(3))) void*)(As + buf + (8 * wave + r) * 1024), 16,
                avoff[r], soff, 0, 0);
        };
        // B: packed panels and metadata as buffers; a panel past N is an
        // empty buffer (reads zero; its columns are never stored).
        __amdgpu_buffer_rsrc_t wr[PANELS], sr[PANELS], zr[PANELS];
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) {
            const int64_t panel = col0 / PW + pp;
            const bool in = panel < np;
            const int64_t pc = in ? panel : 0;
            wr[pp] = make_rsrc(packed + pc * na * kAtomBytes, in ? (uint32_t)na * kAtomBytes : 0u);
            sr[pp] = make_rsrc(packed + s_off + pc * ng * PW * 2, in ? (uint32_t)(ng * PW * 2) : 0u);
            zr[pp] = make_rsrc(packed + z_off + pc * ng * PW, in ? (uint32_t)(ng * PW) : 0u);
        }
        u32x4 ring[kCS][PANELS];
        auto load_atom = [&](int step, u32x4 (&slot)[PANELS]) {
            const uint32_t soff = (uint32_t)min(step, steps - 1) * kAtomBytes;
#pragma unroll
            for (int pp = 0; pp < PANELS; ++pp) slot[pp] = load16(wr[pp], (uint32_t)lane * 16u, soff);
        };
        auto load_meta = [&](int ch, Meta& mt) {
            ch = min(ch, chunks - 1);
#pragma unroll
            for (int m = 0; m < MPC; ++m) {
                const uint32_t g = (uint32_t)((ch * kCS + m * SPG) * kAtomK) >> gshift;
#pragma unroll
                for (int pp = 0; pp < PANELS; ++pp) {
                    if constexpr (BITS == 4) {
                        const uint2 sv = __builtin_bit_cast(
                            uint2, __builtin_amdgcn_raw_buffer_load_b64(sr[pp], (uint32_t)c * 8u, g * (PW * 2), 0));
                        mt.s[m][pp][0] = sv.x;
                        mt.s[m][pp][1] = sv.y;
                        mt.z[m][pp] = __builtin_amdgcn_raw_buffer_load_b32(zr[pp], (uint32_t)c * 4u, g * PW, 0);
                    } else {
                        mt.s[m][pp][0] =
                            __builtin_amdgcn_raw_buffer_load_b32(sr[pp], (uint32_t)c * 4u, g * (PW * 2), 0);
                        mt.z[m][pp] = __builtin_amdgcn_raw_buffer_load_b16(zr[pp], (uint32_t)c * 2u, g * PW, 0);
                    }
                }
            }
        };

#pragma unroll
        for (int i = 0; i < kRB; ++i)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[i][t] = float4_t{0.f, 0.f, 0.f, 0.f};

        // Prologue (s0 = first step, pair p0 = s0 / 2): A of pairs p0, p0+1
        // (steps s0..s0+3) into buffers b0, b1; atoms of steps s0..s0+3 and
        // metadata of the first two chunks requested; B operands of step s0;
        // everything landed, then the A fragments of blocks 0..7 of step s0
        // read.  Within a chunk ch the steps use buffers b0, b0, b1, b1 (pairs
        // 2 ch, 2 ch + 1); the direct loads of pair 2 ch + 2 go to b2 during
        // its first two steps, those of pair 2 ch + 3 to b0 (free once its
        // second step is done) during the last two; then the three rotate.
        const int s0 = c0 * kCS;
        uint32_t b0 = 0, b1 = kPairBytes, b2 = 2 * kPairBytes;
#pragma unroll
        for (int r = 0; r < 8; ++r) dma_a(s0 / 2, b0, r);
#pragma unroll
        for (int r = 0; r < 8; ++r) dma_a(s0 / 2 + 1, b1, r);
#pragma unroll
        for (int j = 0; j < kCS; ++j) load_atom(s0 + j, ring[j]);
        Meta mcur, mnext;
        load_meta(c0, mcur);
        load_meta(c0 + 1, mnext);
        Consts kc;
        make_consts(mcur, 0, kc);
        u32x4 bop[4];
        dequant(ring[0], kc, bop);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        // A fragments: block i of every step in af[i]; blocks 8..15 are read
        // at the start of their step, blocks 0..7 half a step before theirs.
        u32x4 af[kRB];
#pragma unroll
        for (int i = 0; i < kRB / 2; ++i) af[i] = lds_read_block(a_lane[0] + b0, i);
        lds_wait();
        mfma_hazard_gap();

        // One K step s (j = s mod 4), as 64 MFMA slots (row block i = slot / 4,
        // column block t = slot % 4), each followed by at most one other
        // instruction group, fixed by scheduling fences:
        //   slot 0        wait for this step's blocks 0..7 (read half a step ago)
        //   slots 0..7    A fragments of blocks 8..15 of step s
        //   slot 32       wait for them
        //   slots 32..39  A fragments of blocks 0..7 of step s+1
        //   fp16: slots 8+2r direct load r (0..3) of half of the A pair two
        //   ahead; slots 9..15 the constants of a new group; slot 41 the atom
        //   loads for step s+4 (into the ring slot of step s, whose operands
        //   were formed during s-1); slot 43 the metadata reload.
        //   bf16: slot 0 the atoms, slots 16+4r the direct loads.
        //   [W, 32), [W + 32, 64)
        //                 the dequantization micro-steps of step s+1's B
        //                 operands, one vector instruction each, issued while
        //                 the matrix core works and no LDS data returns
        // then one barrier (after even steps, once the direct loads of the
        // pair about to be read ahead have landed).
        // slots of the atom load, the metadata reload (fp16) and the four
        // direct loads
        constexpr int kAtomSlot = BF ? 0 : 41, kMetaSlot = 43;
        constexpr int kDmaSlot = BF ? 16 : 8, kDmaStride = BF ? 4 : 2;
        for (int ch = c0; ch < c1; ++ch) {
#pragma unroll
            for (int j = 0; j < kCS; ++j) {
                const int step = ch * kCS + j;
                const int odd = j & 1;
                const uint32_t bcur = j < 2 ? b0 : b1;                    // this step's pair
                const uint32_t bnxt = j == 0 ? b0 : (j == 3 ? b2 : b1);   // step s+1's pair
                const uint32_t bdma = j < 2 ? b2 : b0;                    // pair 2 ch + 2 + j / 2
                const int dpair = 2 * ch + 2 + (j >> 1);
                // The next step starts a new metadata group (the next chunk's
                // first, from metadata that landed a chunk ago, or the next
                // group of this chunk): its constants are formed before this
                // step's dequantization window, and the chunk's last step
                // reloads the metadata registers after they are consumed (a
                // load into registers still to be copied would have to wait).
                // fp16 spreads this work over the quiet slots 8..15 and 40
                // (no LDS returns, no dequantization); bf16, whose window
                // starts at slot 8, does it before the step.
                const bool new_group = j == kCS - 1 || (j + 1) % SPG == 0;
                const Meta& msrc = j == kCS - 1 ? mnext : mcur;
                const int mgrp = j == kCS - 1 ? 0 : (j + 1) / SPG;
                if constexpr (BF) {
                    if (new_group) make_consts(msrc, mgrp, kc);
                    if (j == kCS - 1) {
                        if constexpr (MPC > 1) mcur = mnext;
                        load_meta(ch + 2, mnext);
                    }
                }
                u32x4 bnext[4];
                DqSt<BF> st[4];
#pragma unroll
                for (int q = 0; q < 4 * kRB; ++q) {
                    const int i = q / 4, t = q % 4;
                    __builtin_amdgcn_sched_barrier(0);
                    if (q == 0 || q == 2 * kRB) lds_wait();
                    mfma_acc<BF>(acc[i][t], bop[t], af[i]);
                    if (q == kAtomSlot) load_atom(step + 4, ring[j]);
                    if constexpr (!BF) {
                        if (new_group && q >= 9 && q < 16 && q % 2 == 1) make_const(msrc, mgrp, kc, (q - 9) / 2);
                        if (j == kCS - 1 && q == 40) {
                            if constexpr (MPC > 1) mcur = mnext;
                        }
                        if (j == kCS - 1 && q == kMetaSlot) load_meta(ch + 2, mnext);
                    }
                    if (q < kRB / 2) af[kRB / 2 + q] = lds_read_block(a_lane[odd] + bcur, kRB / 2 + q);
                    if (q >= 2 * kRB && q < 2 * kRB + kRB / 2)
                        af[q - 2 * kRB] = lds_read_block(a_lane[odd ^ 1] + bnxt, q - 2 * kRB);
                    if (q >= kDmaSlot && q < kDmaSlot + 4 * kDmaStride && (q - kDmaSlot) % kDmaStride == 0)
                        dma_a(dpair, bdma, 4 * odd + (q - kDmaSlot) / kDmaStride);
#pragma unroll
                    for (int o = dq_slot_begin<BF>(q, kDqTotal); o < dq_slot_end<BF>(q, kDqTotal); ++o) {
                        const int u = o / kDqSteps, k = o % kDqSteps;
                        dq_step_u(u, k, ring[(j + 1) % kCS], kc, st[u]);
                        if (k == kDqSteps - 1) bnext[u] = st[u].out;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < 4; ++t) bop[t] = bnext[t];
                // The direct loads of a pair must have landed before the step
                // whose next-step reads take its first fragments: pair 2 ch + 1
                // (loaded during the previous chunk's last two steps) before
                // step j = 1 reads ahead, pair 2 ch + 2 (loaded during j = 0,
                // 1) before j = 3 does.  So only the even steps end with a
                // wait, for every load but those issued after the previous
                // step's direct loads (loads complete in order): fp16 issues
                // its atoms (one load per panel) and metadata (two per group
                // and panel, chunk's last step) after its direct loads, so a
                // slow weight fetch holds up the wait one step later than
                // it would otherwise; bf16 issues them before.  The odd
                // steps' barrier only orders the reuse of a buffer.
                constexpr int kMetaLoads = 2 * MPC * PANELS;
                if (j % 2 == 1) {
                    barrier_only();
                } else if constexpr (BF) {
                    barrier_after_a_loads<PANELS + 4>();
                } else {
                    if (j == 0) barrier_after_a_loads<PANELS + kMetaLoads + 4 + PANELS>();
                    else barrier_after_a_loads<PANELS + 4 + PANELS>();
                }
            }
            const uint32_t bt = b0;        // the chunk's three buffers rotate
            b0 = b2;
            b2 = b1;
            b1 = bt;
        }
        mfma_hazard_gap();
        __builtin_amdgcn_s_waitcnt(0);   // direct loads issued for steps past the segment have landed
        __syncthreads();   // every wave done with the A buffers (the output staging reuses them)
    };

    // Work of this block: whole tiles first, then a range [ua, ub) of 128-row
    // K chunks ("units", tile-major) of the stream-K part.
    const int G = sk.groups, U = sk.units, b = blockIdx.x;
    int v = 0, ua = 0, ub = 0, nwhole, dpu = 0;
    int dp_tile0;                  // data-parallel: this block's tile
    if (G == 0) {
        // Data-parallel: XCD band of the tile list; block b runs on XCD b % 8
        // and takes the (b / 8)-th tile of that XCD's contiguous band.
        const int total = tiles_m * tiles_n;
        const int per = total / kXcds, rem = total % kXcds;
        const int x = b % kXcds, i = b / kXcds;
        dp_tile0 = x * per + min(x, rem) + i;
        nwhole = 1;
    } else {
        // Stream-K: virtual block index v numbers the blocks XCD by XCD, so
        // each XCD walks a contiguous part of the unit list.  Hybrid: the
        // first dp_rounds * G tiles go whole, tile r * G + v to block v, and
        // the stream-K units cover the tiles after them.
        v = (G % kXcds == 0) ? (b % kXcds) * (G / kXcds) + b / kXcds : b;
        nwhole = sk.dp_rounds;
        dp_tile0 = v;
        dpu = sk.dp_rounds * G * chunks;
        ua = dpu + sk_begin(v, G, U);
        ub = dpu + sk_begin(v + 1, G, U);
    }
    auto whole = [&](int i, float4_t (&blk)[4]) {
#pragma unroll
        for (int t = 0; t < 4; ++t) blk[t] = acc[i][t];
    };
    int64_t row0, col0;
    // (one call site of `segment`, whose body is large)
    for (int k = 0, u = ua; k < nwhole || u < ub;) {
        int tile, c0, c1;
        const int useg = u;                               // first unit of a stream-K segment
        if (k < nwhole) {
            tile = dp_tile0 + k * G;
            c0 = 0;
            c1 = chunks;
            ++k;
        } else {
            tile = u / chunks;
            c0 = u % chunks;
            c1 = min(chunks, c0 + (ub - u));
            u += c1 - c0;
        }
        segment(tile, c0, c1, row0, col0);
        if (c0 == 0 && c1 == chunks) {
            store_tile(row0, col0, whole);
        } else {
            // Park the partial: wave w's 256 x 64 part at w * 16384 floats,
            // block (i, t) as 64 consecutive float4 (one per lane); slot 2v
            // holds this block's first segment, 2v + 1 its last.
            // stream_k_reduce_kernel, launched next on the same stream, adds
            // each split tile's segments.
            const int slot = 2 * v + (useg == ua ? 0 : 1);
            float* part = sk.part + (int64_t)slot * (kBM * kBN);
            const __amdgpu_buffer_rsrc_t pr = make_rsrc(part + wave * (kBM * 64), kBM * 64 * 4);
#pragma unroll
            for (int i = 0; i < kRB; ++i)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, acc[i][t]), pr,
                                                           (uint32_t)(((i * 4 + t) * 64 + lane) * 16), 0, 0);
        }
    }
}

// Stream-K reduction: one thread per float4 of a split tile's parked parts
// (the main kernel's layout: wave part w of 256 x 64 floats, block (i, t) as
// 64 consecutive float4; lane (c, kg) holds row 16 i + c, columns
// 16 t + 4 kg + 0..3, C transposed by the operand order), summed over the
// tile's segments in K order (the owner of its first unit first) and
// written as four outputs rounded once.  Tiles are the stream-K tiles after
// the whole-tile rounds; a tile inside one block's range was stored whole.
template <bool BF>
__global__ __launch_bounds__(256) void stream_k_reduce_kernel(
    const float4_t* __restrict__ part, uint16_t* __restrict__ C, int M, int N, int tiles_m,
    int tiles_n, int col_major, int G, int U, int chunks, int tile0, int64_t total) {
    constexpr int kPerTile = kBM * kBN / 4;        // float4 per part of one tile
    constexpr int kPerWave = kBM * 64 / 4;         // float4 per wave part
    const int64_t f = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (f >= total) return;
    const int tile = tile0 + (int)(f / kPerTile);
    const int e = (int)(f % kPerTile);
    const int t0 = (tile - tile0) * chunks;        // the tile's first unit, stream-K numbering
    const int vlo = sk_owner(t0, G, U), vhi = sk_owner(t0 + chunks - 1, G, U);
    if (vlo == vhi) return;                        // one block's range: stored whole
    float4_t r = {0.f, 0.f, 0.f, 0.f};
    for (int w = vlo; w <= vhi; ++w) {
        const int sw = 2 * w + (sk_begin(w, G, U) >= t0 ? 0 : 1);
        r += part[(int64_t)sw * kPerTile + e];
    }
    const int wave = e / kPerWave, rem = e % kPerWave;
    const int blk = rem >> 6, lane = rem & 63;
    const int i = blk >> 2, t = blk & 3, c = lane & 15, kg = lane >> 4;
    const int tm = col_major ? tile % tiles_m : tile / tiles_n;
    const int tn = col_major ? tile / tiles_m : tile % tiles_n;
    const int64_t m = (int64_t)tm * kBM + 16 * i + c;
    const int64_t n = (int64_t)tn * kBN + wave * 64 + 16 * t + 4 * kg;     // N % 8 == 0
    if (m < M && n < N)
        *reinterpret_cast<uint2*>(C + m * N + n) = uint2{round_out2<BF>(r[0], r[1]), round_out2<BF>(r[2], r[3])};
}

// Walk the tile list along N (column-major) when the weights outweigh the
// activations: each XCD band then covers fewer weight panels.
int col_major_for(const Layout& L, int64_t M) {
    const int64_t a_bytes = M * L.K * 2, w_bytes = L.total;
    return w_bytes > a_bytes ? 1 : 0;
}

template <int BITS, int MPC, bool BF>
int launch_mpc(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
               StreamK sk, int tiles_m, int tiles_n, hipStream_t s) {
    const int gshift = __builtin_ctz((unsigned)L.group);
    const int col_major = col_major_for(L, M);
    const unsigned grid = sk.groups ? (unsigned)sk.groups : (unsigned)(tiles_m * tiles_n);
    return launch(gemm256_kernel<BITS, MPC, BF>, dim3(grid), dim3(kThreads), 0, s, A, pk, C, (int)M,
                  (int)L.K, (int)L.N, gshift, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np,
                  tiles_m, tiles_n, col_major, sk);
}

}  // namespace

bool gemm256_supported(const Layout& L) {
    return L.K % (kBK * kCS) == 0 && (L.group & (L.group - 1)) == 0;
}

// Stream-K is planned when the 256 x 256 tiles do not fill whole waves of
// kSkMaxGroups blocks; its workspace is the shared counter region at offset 0
// (the other kernels' arrival counters; this one leaves it untouched), then
// two parked partial tiles per block.
int64_t gemm256_workspace_bytes(const Layout& L, int64_t M) {
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((L.N + kBN - 1) / kBN);
    if (!gemm256_supported(L) || tiles % kSkMaxGroups == 0) return 0;
    return kWsCounterBytes + (int64_t)2 * kSkMaxGroups * kBM * kBN * 4;
}

namespace {
template <bool BF>
int launch_bf(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
              StreamK sk, int tiles_m, int tiles_n, hipStream_t s) {
    const int chunk_rows = kBK * kCS;
    const int mpc = L.group >= chunk_rows ? 1 : chunk_rows / L.group;
    if (L.bits == 4) {
        if (mpc == 1) return launch_mpc<4, 1, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
        if (mpc == 2) return launch_mpc<4, 2, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
        return launch_mpc<4, 4, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
    }
    if (mpc == 1) return launch_mpc<8, 1, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
    if (mpc == 2) return launch_mpc<8, 2, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
    return launch_mpc<8, 4, BF>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
}

}  // namespace

// Where whole tiles leave too short a last wave, the few tiles after the
// whole waves go to the K-split GEMM (8 workgroups of 64 x 128 per tile, no
// partial tiles) instead of stream-K, while K is short and the remainder at
// most three rounds of its workgroups.  Measured on MI355X against the
// stream-K hybrid (K = 4096, N = 14336, graph replay, alternating builds):
// remainders of 8 - 80 tiles 2.2 - 14.3% faster (M = 1280: 137.3 -> 117.7 us),
// 136 tiles (1088 workgroups, M = 1792) 2.7% slower.
constexpr int64_t kKsRestMaxK = 8192, kKsRestMaxTiles = 96;
static bool ks_rest_ok(const Layout& L, int64_t rest) {
    return gemm_ks_supported(L) && L.K <= kKsRestMaxK && rest <= kKsRestMaxTiles;
}

int launch_gemm256(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                   void* ws, size_t ws_bytes, hipStream_t s, bool bf) {
    const int tiles_m = (int)((M + kBM - 1) / kBM);
    const int tiles_n = (int)((L.N + kBN - 1) / kBN);
    const int tiles = tiles_m * tiles_n, chunks = (int)(L.K / (kBK * kCS));
    const int64_t need = gemm256_workspace_bytes(L, M);
    const int cus = device_cus(s);
    StreamK sk{0, 0, nullptr, 0};
    // Otherwise (with a workspace) stream-K; splitting every tile keeps at
    // least kSkMinUnits K chunks per block.  With at least one full wave of
    // tiles the full waves stay whole tiles and only the tiles after them are
    // split ("hybrid"): fewer partial tiles than splitting everything, no
    // idle units in the last wave.
    // Whole tiles while they keep at least 80% of the launch's block slots
    // busy (ceil(tiles / cus) waves of cus blocks) and their last wave holds
    // at least 40% of the blocks.  Measured on MI355X (hybrid against whole
    // tiles): K=4096, N=14336 at M = 4864, 5888, 7168 (last wave 16%, 3%,
    // 12.5% full) 5-6% faster; at M = 2816 (41%) 1.4%, at M = 2048 (75%) 11%
    // slower; K=14336, N=4096 at M = 6656 (62.5%) 4% faster; stream-K over
    // fewer tiles than blocks (M = 3328, 81%) 11% slower.
    const int64_t waves = (tiles + cus - 1) / cus;
    const int64_t last = tiles - (waves - 1) * cus;        // tiles in the last wave
    const bool dp_ok = 5 * (int64_t)tiles >= 4 * waves * cus && 5 * last >= 2 * cus;
    KsRange rest{0, 0, tiles_m, tiles_n, col_major_for(L, M)};
    int Gr = std::min(cus, kSkMaxGroups);
    if (Gr > kXcds) Gr -= Gr % kXcds;
    if (!dp_ok && tiles >= Gr && ks_rest_ok(L, tiles % Gr)) {
        // whole-tile rounds of this kernel, then the remaining tiles as 64 x 128
        // tiles with K split over each workgroup's waves: no partial tiles
        const int dp_rounds = tiles / Gr;
        sk = StreamK{Gr, 0, nullptr, dp_rounds};
        rest.tile0 = dp_rounds * Gr;
        rest.count = tiles - rest.tile0;
    } else if (ws && need > 0 && (int64_t)ws_bytes >= need && !dp_ok) {
        int G = std::min(cus, kSkMaxGroups);
        if (G > kXcds) G -= G % kXcds;
        int dp_rounds = tiles / G;
        // the stream-K part gives every block at least one K chunk (a shorter
        // remainder joins the last whole wave); however many segments that
        // cuts its tiles into, the reduction launch sums them over all CUs
        // (measured on MI355X: 6-14% faster than splitting every tile at
        // M = 1280..3584 with K=4096, N=14336 and M = 4352, 4608 with
        // K=14336, N=4096; a floor of 4 chunks per block loses half of that)
        if (dp_rounds > 0 && (int64_t)(tiles - dp_rounds * G) * chunks < G) --dp_rounds;
        const int64_t units = (int64_t)(tiles - dp_rounds * G) * chunks;
        if (dp_rounds == 0) G = (int)std::min<int64_t>(G, std::max<int64_t>(1, units / kSkMinUnits));
        if (G > kXcds) G -= G % kXcds;
        sk = StreamK{G, (int)units, reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsCounterBytes),
                     dp_rounds};
    }
    if (log_enabled())
        log_plan("gemm256_kernel<%d,%d,%s> M=%lld K=%lld N=%lld G=%d: %dx%d tiles of 256x256, %d K chunks, "
                 "%s, %d CUs, order %s",
                 L.bits, L.group >= kBK * kCS ? 1 : kBK * kCS / L.group, bf ? "bf16" : "f16", (long long)M,
                 (long long)L.K, (long long)L.N, L.group, tiles_m, tiles_n, chunks,
                 sk.groups == 0 ? "whole tiles"
                 : rest.count > 0 ? "whole-tile rounds, then the K-split GEMM over the rest"
                 : sk.dp_rounds > 0 ? "hybrid (whole-tile rounds, then stream-K)" : "stream-K",
                 cus, col_major_for(L, M) ? "column-major" : "row-major");
    if (log_enabled() && sk.groups && rest.count == 0)
        log_plan("  stream-K: %d blocks, %d whole-tile rounds, %d units, reduction launch over %d tiles",
                 sk.groups, sk.dp_rounds, sk.units, tiles - sk.dp_rounds * sk.groups);
    const int rc = bf ? launch_bf<true>(L, A, pk, C, M, sk, tiles_m, tiles_n, s)
                      : launch_bf<false>(L, A, pk, C, M, sk, tiles_m, tiles_n, s);
    if (rc || sk.groups == 0) return rc;
    if (rest.count > 0) return launch_gemm_ks_range(L, A, pk, C, M, rest, s, bf);
    const int tile0 = sk.dp_rounds * sk.groups;                  // first stream-K tile
    const int64_t total = (int64_t)(tiles - tile0) * (kBM * kBN / 4);
    const dim3 grid((unsigned)((total + 255) / 256));
    const float4_t* part = reinterpret_cast<const float4_t*>(sk.part);
    const int cm = col_major_for(L, M);
    if (bf)
        return launch(stream_k_reduce_kernel<true>, grid, dim3(256), 0, s, part, C, (int)M, (int)L.N, tiles_m,
                      tiles_n, cm, sk.groups, sk.units, chunks, tile0, total);
    return launch(stream_k_reduce_kernel<false>, grid, dim3(256), 0, s, part, C, (int)M, (int)L.N, tiles_m,
                  tiles_n, cm, sk.groups, sk.units, chunks, tile0, total);
}

bool gemm256_fills_device(const Layout& L, int64_t M, hipStream_t s) {
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((L.N + kBN - 1) / kBN);
    return 4 * tiles >= 3 * (int64_t)device_cus(s);
}

}  // namespace tf
