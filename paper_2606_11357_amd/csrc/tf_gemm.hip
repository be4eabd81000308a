// Prefill GEMM (Section 2.1; Section 4.3 "GEMM microkernel"):
//   C[M, N] = A[M, K] x dequant(packed)[K, N], fp16 MFMA, fp32 accumulate.
//
// Workgroup tile BM x BN = 128 x 256, four waves side by side along N; each
// wave owns 128 rows x 64 columns (one 4-bit panel or two 8-bit panels).
// K is walked in chunks of 128 rows = 4 steps of 32 rows (one packed atom per
// panel per step).
//  - B never exists as fp16 in memory: each wave loads the packed atoms of its
//    own columns, unpacks and dequantizes them (Eq. 2, rounded once) straight
//    into the register layout of the v_mfma_f32_16x16x32_f16 B operand, and
//    reuses every dequantized operand across its 8 row sub-tiles (Sections
//    4.1.1 and 4.3: dequantize a weight tile once, reuse it for every
//    activation row).  The next chunk's atoms and metadata are loaded a whole
//    chunk ahead; the group constants are formed once per chunk.
//  - A (fp16) goes global -> registers -> LDS through three LDS buffers (16-row
//    blocks chunk-major): the loads for step s+2 leave while step s is multiplied and are
//    written to LDS one step later, so each load has more than a step to land;
//    one barrier per step.
//  - Tiles are numbered so that each XCD (workgroups are dealt round-robin
//    over the 8 XCDs) works on a contiguous band of tiles sharing rows of A,
//    which then stay in that XCD's L2.
//  - When the tiles are too few to occupy the device and a workspace is
//    given, each tile's K is cut into S slices of whole chunks, one workgroup
//    each; every slice parks its fp32 partial tile in the workspace, and a
//    second launch on the same stream (splitk_reduce_kernel) adds the slices
//    of every tile in slice order (bitwise reproducible) and writes C, spread
//    over all compute units.  (Letting the last slice of each tile do that
//    sum left one workgroup per tile streaming S - 1 partial tiles, one
//    latency-bound row block at a time, while the rest of the GPU idled.)
#include "tf_internal.h"

#include <algorithm>

namespace tf {
namespace {

constexpr int kBM = 128, kBN = 256, kBK = 32;
// Steps per chunk (128 rows of K); also the size of the packed-atom ring.
template <int BITS>
constexpr int chunk_steps() { return 4; }
constexpr int kGemmThreads = 256;
constexpr int kXcds = 8;
constexpr int kABufs = 3;

// LDS slot (16-byte chunks) of chunk `ch` (0..3) of A row `row` (64-byte
// rows; see lds_a_slot).
__device__ __forceinline__ int a_slot(int row, int ch) { return lds_a_slot(row, ch); }

// MPC: metadata groups per chunk (1 when a group spans the whole chunk, else
// chunk rows / group); the group of step j is j / (chunk steps / MPC).
// Most K slices per tile (measured on MI355X over the split shapes of the
// M = 256..768 MLP sweep and W8 K = N = 4096: 8 beats 4 where K is long and
// the tiles few, and ties elsewhere; 2 and 1 lose everywhere).
constexpr int kMaxSplit = 8;

// Split-K arguments: S slices per tile of cps chunks each (S = 1: no split);
// the partial tiles in the workspace.
struct SplitK {
    int S, cps;
    float* part;
};

template <int BITS, int MPC, bool BF>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(
    const uint16_t* __restrict__ A, const uint8_t* __restrict__ packed, uint16_t* __restrict__ C,
    int M, int K, int N, int gshift, int64_t s_off, int64_t z_off, int na, int ng, int np,
    int tiles_m, int tiles_n, SplitK sk) {
    constexpr int PW = BITS == 4 ? 64 : 32;
    constexpr int T = PW / 16;                 // columns per lane per atom
    constexpr int PANELS = 64 / PW;            // panels per wave
    constexpr int kChunkSteps = chunk_steps<BITS>();
    constexpr int SPG = kChunkSteps / MPC;     // steps per metadata group
    __shared__ __align__(16) u32x4 As[kABufs][kBM * kBK / 8];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 15, kg = lane >> 4;
    const uint32_t magic = magic_reg();

    // XCD-aware order: block b runs on XCD b % 8; XCD x takes the x-th
    // contiguous band of the row-major list of (tile, slice) units, so the
    // slices of a tile and neighbouring tiles share that XCD's L2.
    const int total = tiles_m * tiles_n * sk.S;
    int unit;
    {
        const int b = blockIdx.x;
        const int per = total / kXcds, rem = total % kXcds;
        const int x = b % kXcds, i = b / kXcds;
        unit = x * per + min(x, rem) + i;
    }
    const int tile = unit / sk.S, split = unit % sk.S;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    constexpr int CS0 = chunk_steps<BITS>();
    const int ch0 = split * sk.cps;                            // first chunk of this slice
    const int chunks = min(na / CS0 - ch0, sk.cps);            // chunks of this slice (>= 1)
    const int st0 = ch0 * CS0;                                 // first step of this slice
    const int64_t row0 = (int64_t)tm * kBM;
    const int64_t col0 = (int64_t)tn * kBN + wave * 64;      // this wave's 64 columns

    float4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[i][t] = float4_t{0.f, 0.f, 0.f, 0.f};

    // ---- A: 128 rows x 32 halves per step = 512 chunks, 2 per thread; thread
    // chunk idx is the one LDS slot idx holds, so each wave stores 1 KB of
    // consecutive slots.  Rows past M read row M-1 instead (in bounds; those
    // rows are never stored).
    const uint16_t* arow[2];
    int aslot[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int idx = tid + kGemmThreads * r;
        const int64_t grow = min<int64_t>(row0 + lds_a_row(idx), (int64_t)M - 1);
        arow[r] = A + grow * K + lds_a_chunk(idx) * 8 + (int64_t)st0 * kBK;
        aslot[r] = idx;
    }
    const int steps = chunks * CS0;            // one 32-row step per atom
    auto load_a = [&](int step, u32x4 (&av)[2]) {
        step = min(step, steps - 1);           // clamped: a repeated valid step, never used
#pragma unroll
        for (int r = 0; r < 2; ++r) av[r] = *reinterpret_cast<const u32x4*>(arow[r] + step * kBK);
    };
    auto store_a = [&](int buf, const u32x4 (&av)[2]) {
#pragma unroll
        for (int r = 0; r < 2; ++r) As[buf][aslot[r]] = av[r];
    };

    // ---- B: the wave's packed atoms and its columns' metadata.  Panels past N
    // read the last panel instead (in bounds; their columns are never stored).
    const u32x4* wp[PANELS];
    const uint8_t* sp[PANELS];
    const uint8_t* zp[PANELS];
    bool live = false;
#pragma unroll
    for (int pp = 0; pp < PANELS; ++pp) {
        int64_t panel = col0 / PW + pp;
        live = live || panel < np;
        panel = min<int64_t>(panel, np - 1);
        wp[pp] = reinterpret_cast<const u32x4*>(packed) + (panel * na + st0) * 64 + lane;
        sp[pp] = packed + s_off + (panel * ng * PW + c * T) * 2;
        zp[pp] = packed + z_off + panel * ng * PW + c * T;
    }
    // Packed atoms live in a ring of kChunkSteps slots: the atom of step s sits
    // in slot s % kChunkSteps, is loaded three steps ahead and is dequantized
    // one step ahead, while the MFMAs of the step before it run.  Raw metadata
    // is loaded a chunk ahead; group constants are formed once per group.
    constexpr int CS = kChunkSteps;           // the launcher requires K % (32 * CS) == 0
    u32x4 ring[CS][PANELS];
    auto load_atom = [&](int step, u32x4 (&slot)[PANELS]) {
        step = min(step, steps - 1);           // clamped: a repeated valid step, never used
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp) slot[pp] = wp[pp][step * 64];
    };
    struct Meta {
        uint32_t s[MPC][PANELS][(T + 1) / 2];   // T fp16 scales per group and panel
        uint32_t z[MPC][PANELS];                // T zero-point bytes
    };
    auto load_meta = [&](int ch, Meta& mt) {
        ch = min(ch, chunks - 1);
#pragma unroll
        for (int m = 0; m < MPC; ++m) {
            const int g = (((ch0 + ch) * CS + m * SPG) * kAtomK) >> gshift;
#pragma unroll
            for (int pp = 0; pp < PANELS; ++pp) {
                if constexpr (BITS == 4) {
                    const uint2 sv = *reinterpret_cast<const uint2*>(sp[pp] + g * PW * 2);
                    mt.s[m][pp][0] = sv.x;
                    mt.s[m][pp][1] = sv.y;
                    mt.z[m][pp] = *reinterpret_cast<const uint32_t*>(zp[pp] + g * PW);
                } else {
                    mt.s[m][pp][0] = *reinterpret_cast<const uint32_t*>(sp[pp] + g * PW * 2);
                    mt.z[m][pp] = *reinterpret_cast<const uint16_t*>(zp[pp] + g * PW);
                }
            }
        }
    };
    // Group constants of each lane column (see DqConst).
    struct Consts {
        DqConst<BF> q[4];
    };
    auto make_consts = [&](const Meta& mt, int m, Consts& k) {
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp)
#pragma unroll
            for (int t = 0; t < T; ++t) {
                DqConst<BF>& kq = k.q[pp * T + t];
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
            }
    };
    auto dequant = [&](const u32x4 (&slot)[PANELS], const Consts& k, u32x4 (&bop)[4]) {
#pragma unroll
        for (int pp = 0; pp < PANELS; ++pp)
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const int u = pp * T + t;
                bop[u] = dq_operand<BF, BITS>(slot[pp][BITS == 4 ? t : 2 * t],
                                              slot[pp][BITS == 4 ? t : 2 * t + 1], magic, k.q[u]);
            }
    };

    // Prologue: A for steps 0 and 1 in flight, step 0 in LDS; atoms of steps
    // 0..2 and metadata of chunks 0 and 1 requested; B operands of step 0.
    u32x4 ra[2][2];
    load_a(0, ra[0]);
    load_a(1, ra[1]);
    static_assert(CS == 4, "the atom ring needs four slots for its three-step lead");
#pragma unroll
    for (int j = 0; j < 3; ++j) load_atom(j, ring[j]);
    Meta mcur, mnext;
    load_meta(0, mcur);
    load_meta(1, mnext);
    store_a(0, ra[0]);
    Consts kc;
    make_consts(mcur, 0, kc);
    u32x4 bop[4];
    dequant(ring[0], kc, bop);

    for (int ch = 0; ch < chunks; ++ch) {
#pragma unroll
        for (int j = 0; j < CS; ++j) {
            const int step = ch * CS + j;
            const int buf = step % kABufs;
            load_a(step + 2, ra[j & 1]);                  // step + 2 has the same parity as step
            load_atom(step + 3, ring[(j + 3) % CS]);      // that slot held step - 1, used already
            if (j == CS - 1) {
                // constants for the first step of the next chunk; the metadata
                // of the chunk after it is requested
                mcur = mnext;
                load_meta(ch + 2, mnext);
                make_consts(mcur, 0, kc);
            } else if ((j + 1) % SPG == 0) {
                make_consts(mcur, (j + 1) / SPG, kc);     // next step starts a new group
            }
            __syncthreads();                              // As[buf] written; As[(step + 1) % 3] free
            u32x4 bnext[4];
            dequant(ring[(j + 1) % CS], kc, bnext);       // B operands of step + 1
            if (live) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const u32x4 af = As[buf][a_slot(16 * i + c, kg)];
#pragma unroll
                    for (int t = 0; t < 4; ++t) acc[i][t] = mfma16<BF>(af, bop[t], acc[i][t]);
                }
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) bop[t] = bnext[t];
            store_a((step + 1) % kABufs, ra[(j + 1) & 1]);   // A for step + 1, loaded a step ago
        }
    }

    // ---- epilogue: lane holds column c of each 16x16 block, rows 4 kg + r
    auto store_block = [&](int i, int t, const float4_t& v) {
        const int64_t col = col0 + 16 * t + c;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t row = row0 + 16 * i + 4 * kg + r;
            if (row < M && col < N) C[row * N + col] = round_out<BF>(v[r]);
        }
    };
    if (sk.S == 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int t = 0; t < 4; ++t) store_block(i, t, acc[i][t]);
        return;
    }
    // Park this slice's partial tile (wave w's 128 x 64 part, block (i, t) as
    // 64 consecutive float4, one per lane); splitk_reduce_kernel, launched
    // next on the same stream, adds the slices.
    {
        const __amdgpu_buffer_rsrc_t pr =
            make_rsrc(sk.part + ((int64_t)tile * sk.S + split) * (kBM * kBN) + wave * (kBM * 64), kBM * 64 * 4);
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, acc[i][t]), pr,
                                                       (uint32_t)(((i * 4 + t) * 64 + lane) * 16), 0, 0);
    }
}

// Split-K reduction: one thread per float4 of a tile's parked partial (the
// main kernel's layout: wave part w of kBM x 64 floats, block (i, t) as 64
// consecutive float4, lane (c, kg) holding rows 16 i + 4 kg + 0..3 of column
// 16 t + c), summed over the S slices in slice order; the four outputs are
// rounded once.  Consecutive threads read consecutive float4.
template <bool BF>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float4_t* __restrict__ part,
                                                            uint16_t* __restrict__ C, int M, int N,
                                                            int tiles_n, int S, int64_t total) {
    constexpr int kPerTile = kBM * kBN / 4;        // float4 per slice of one tile
    constexpr int kPerWave = kBM * 64 / 4;         // float4 per wave part
    const int64_t f = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (f >= total) return;
    const int64_t tile = f / kPerTile;
    const int e = (int)(f - tile * kPerTile);
    const int w = e / kPerWave, rem = e - w * kPerWave;
    const int blk = rem >> 6, lane = rem & 63;
    const int i = blk >> 2, t = blk & 3, c = lane & 15, kg = lane >> 4;
    const float4_t* p = part + tile * S * kPerTile + e;
    float4_t r = p[0];
    for (int sl = 1; sl < S; ++sl) r += p[(int64_t)sl * kPerTile];
    const int64_t tm = tile / tiles_n, tn = tile - tm * tiles_n;
    const int64_t col = tn * kBN + w * 64 + 16 * t + c;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int64_t row = tm * kBM + 16 * i + 4 * kg + q;
        if (row < M && col < N) C[row * N + col] = round_out<BF>(r[q]);
    }
}

// Generic kernel for the cases the main one leaves out (K not a multiple of
// the chunk or a group size that is not a power of two): 128 x 128 tiles,
// 32-row steps, single-buffered.
constexpr int kBM1 = 128, kBN1 = 128, kBK1 = 32;

__device__ __forceinline__ int a_swz1(int row, int chunk) { return lds_a_slot(row, chunk); }

template <int BITS, bool BF>
__global__ __launch_bounds__(kGemmThreads) void gemm_kernel_generic(
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
    const uint32_t magic = magic_reg();

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
            const int row = lds_a_row(idx), ch = lds_a_chunk(idx);   // the chunk slot idx holds
            const int64_t grow = row0 + row;
            av[r] = grow < M ? *reinterpret_cast<const u32x4*>(A + grow * K + (int64_t)a * kBK1 + ch * 8)
                             : u32x4{0u, 0u, 0u, 0u};
        }
        u32x4 b[4];
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
                const DqConst<BF> kq = make_dq_const<BF>(sb[t], zb[t]);
                if constexpr (BITS == 4)
                    b[t] = dq_operand<BF, 4>(wv[t], 0u, magic, kq);
                else
                    b[pp * T + t] = dq_operand<BF, 8>(wv[2 * t], wv[2 * t + 1], magic, kq);
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int idx = tid + kGemmThreads * r;
            As[idx] = av[r];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const u32x4 af = As[a_swz1(wm * 64 + 16 * i + c, kg)];
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[i][t] = mfma16<BF>(af, b[t], acc[i][t]);
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
                    C[row * N + col] = round_out<BF>(acc[i][t][r]);
            }
        }
}

// Split plan of the main kernel: K is cut only when a workspace is given and
// the tiles are fewer than kSplitBelowTiles, into at most kMaxSplit slices of
// at least kMinSliceChunks chunks, aiming at one unit per compute unit.
struct SplitPlan {
    int S, cps;
};
constexpr int kSplitBelowTiles = 256;
constexpr int kTargetUnits = 256;
constexpr int kMinSliceChunks = 4;

template <int BITS>
SplitPlan plan_split(const Layout& L, int64_t M) {
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((L.N + kBN - 1) / kBN);
    const int chunks = (int)(L.K / (kBK * chunk_steps<BITS>()));
    int S = 1;
    if (tiles < kSplitBelowTiles) {
        S = (int)std::min<int64_t>((kTargetUnits + tiles - 1) / tiles, chunks / kMinSliceChunks);
        S = std::max(std::min(S, kMaxSplit), 1);
    }
    const int cps = (chunks + S - 1) / S;
    return {(chunks + cps - 1) / cps, cps};    // no empty slice
}

// Workspace of a split plan: the shared counter region at offset 0 (the
// other kernels' arrival counters; this one leaves it untouched), then one
// fp32 partial tile per (tile, slice).
int64_t split_workspace_bytes(const Layout& L, int64_t M, const SplitPlan& sp) {
    if (sp.S <= 1) return 0;
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((L.N + kBN - 1) / kBN);
    return kWsCounterBytes + tiles * sp.S * (int64_t)(kBM * kBN * 4);
}

bool main_kernel_fits(const Layout& L, int bits) {
    const int chunk_rows = kBK * 4;
    return L.K % chunk_rows == 0 && (L.group & (L.group - 1)) == 0 && bits > 0;
}

template <int BITS, int MPC, bool BF>
int launch_main(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                void* ws, hipStream_t s) {
    const int tiles_m = (int)((M + kBM - 1) / kBM);
    const int tiles_n = (int)((L.N + kBN - 1) / kBN);
    const int gshift = __builtin_ctz((unsigned)L.group);
    SplitPlan sp = plan_split<BITS>(L, M);
    if (!ws) sp = {1, (int)(L.K / (kBK * chunk_steps<BITS>()))};
    SplitK sk{sp.S, sp.cps, nullptr};
    if (sp.S > 1) sk.part = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kWsCounterBytes);
    if (log_enabled())
        log_plan("gemm_kernel<%d,%d,%s> M=%lld K=%lld N=%lld G=%d: %dx%d tiles of 128x256, %d K slices of "
                 "%d chunks%s", BITS, MPC, BF ? "bf16" : "f16", (long long)M, (long long)L.K, (long long)L.N,
                 L.group, tiles_m, tiles_n, sp.S, sp.cps, sp.S > 1 ? ", reduction launch" : "");
    const int rc = launch(gemm_kernel<BITS, MPC, BF>, dim3((unsigned)(tiles_m * tiles_n * sp.S)),
                          dim3(kGemmThreads), 0, s, A, pk, C, (int)M, (int)L.K, (int)L.N, gshift, L.s_off,
                          L.z_off, (int)L.na, (int)L.ng, (int)L.np, tiles_m, tiles_n, sk);
    if (rc || sp.S == 1) return rc;
    const int64_t total = (int64_t)tiles_m * tiles_n * (kBM * kBN / 4);
    return launch(splitk_reduce_kernel<BF>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                  reinterpret_cast<const float4_t*>(sk.part), C, (int)M, (int)L.N, tiles_n, sp.S, total);
}

template <int BITS, bool BF>
int launch_bits(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                void* ws, hipStream_t s) {
    constexpr int CS = chunk_steps<BITS>();
    const int chunk_rows = kBK * CS;
    const bool pow2_group = (L.group & (L.group - 1)) == 0;
    if (L.K % chunk_rows == 0 && pow2_group) {
        const int mpc = L.group >= chunk_rows ? 1 : chunk_rows / L.group;
        if (mpc == 1) return launch_main<BITS, 1, BF>(L, A, pk, C, M, ws, s);
        if (mpc == 2) return launch_main<BITS, 2, BF>(L, A, pk, C, M, ws, s);
        if constexpr (CS >= 4) return launch_main<BITS, 4, BF>(L, A, pk, C, M, ws, s);
    }
    dim3 grid((unsigned)((L.N + kBN1 - 1) / kBN1), (unsigned)((M + kBM1 - 1) / kBM1));
    if (log_enabled())
        log_plan("gemm_kernel_generic<%d,%s> M=%lld K=%lld N=%lld G=%d: %ux%u tiles of 128x128", BITS,
                 BF ? "bf16" : "f16", (long long)M, (long long)L.K, (long long)L.N, L.group, grid.y, grid.x);
    return launch(gemm_kernel_generic<BITS, BF>, grid, dim3(kGemmThreads), 0, s, A, pk, C, (int)M,
                  (int)L.K, (int)L.N, L.group, L.s_off, L.z_off, (int)L.na, (int)L.ng, (int)L.np);
}

}  // namespace

// The 256 x 256 kernel runs, for the sizes below, when its tiles fill the
// device or a workspace lets it split K (it is then the only GEMM that uses
// a workspace).
// The 256-row GEMM from M = 1024 on, and from M = 256 where K is long: its
// stream-K split measured 12% and 29% faster than the 128-row split-K at
// M = 512 and 768 (K = 14336, N = 4096) and equal at M = 256, while at
// K = 4096 the 128-row kernel stays ahead below M = 1024 (M = 512 and 768 at
// N = 14336 by 15% and 5%; W8 M = 512, K = N = 4096 by 13%).
constexpr int64_t kGemm256MinM = 1024, kGemm256MinMLongK = 256, kLongK = 8192;
static bool gemm256_size(const Layout& L, int64_t M) {
    return gemm256_supported(L) && (M >= kGemm256MinM || (M >= kGemm256MinMLongK && L.K >= kLongK));
}
static bool use_gemm256(const Layout& L, int64_t M, const void* ws, hipStream_t s) {
    return gemm256_size(L, M) && (ws != nullptr || gemm256_fills_device(L, M, s));
}

// Workspace either GEMM may use for this problem: the 256-row kernel's
// stream-K (gemm256_size), else the 128-row kernel's split-K.
// The 64 x 128 GEMM with K split over each workgroup's waves (one workgroup
// per compute unit, no partial sums in a workspace) wherever it beats the
// 128-row GEMM.  Measured on MI355X (graph replay, fp16, M = 65 .. 1000 at
// K = 1024 .. 14336, both widths): it wins up to 1120 tiles (0.43 - 0.92 of
// the 128-row time; 896 tiles ties) and loses from 1344 (1.09 - 1.18); with
// long K on few tiles (K = 14336, N = 4096: 64 - 96 tiles) one workgroup's
// run of K is too long against the 128-row split-K (1.08 - 1.18), while
// K = 8192 on 256 tiles still wins (0.75).
constexpr int64_t kKsMaxTiles = 1200, kKsMinTilesLongK = 192, kKsLongK = 8192;
static bool use_gemm_ks(const Layout& L, int64_t M) {
    if (gemm256_size(L, M) || !gemm_ks_supported(L)) return false;
    const int64_t tiles = ((M + 63) / 64) * ((L.N + 127) / 128);
    return tiles <= kKsMaxTiles && (L.K <= kKsLongK || tiles >= kKsMinTilesLongK);
}

int64_t gemm_workspace_bytes(const Layout& L, int64_t M) {
    if (gemm256_size(L, M)) return gemm256_workspace_bytes(L, M);
    if (use_gemm_ks(L, M)) return 0;
    if (!main_kernel_fits(L, L.bits)) return 0;
    const SplitPlan sp = L.bits == 4 ? plan_split<4>(L, M) : plan_split<8>(L, M);
    return split_workspace_bytes(L, M, sp);
}

int launch_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, size_t ws_bytes, hipStream_t s, bool bf) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (use_gemm256(L, M, ws, s)) return launch_gemm256(L, A, pk, C, M, ws, ws_bytes, s, bf);
    if (use_gemm_ks(L, M)) return launch_gemm_ks(L, A, pk, C, M, s, bf);
    // a workspace too small for this kernel's split (sized for another
    // kernel of a larger M) selects the single-pass form
    if (ws && (int64_t)ws_bytes < gemm_workspace_bytes(L, M)) ws = nullptr;
    if (bf)
        return L.bits == 4 ? launch_bits<4, true>(L, A, pk, C, M, ws, s)
                           : launch_bits<8, true>(L, A, pk, C, M, ws, s);
    return L.bits == 4 ? launch_bits<4, false>(L, A, pk, C, M, ws, s)
                       : launch_bits<8, false>(L, A, pk, C, M, ws, s);
}

}  // namespace tf
