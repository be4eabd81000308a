// Internal definitions shared by the HIP sources of libtilefuse: the packed
// weight layout (host and device), launch helper, and the device-side
// unpack / dequantize primitives every kernel uses.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>
#include <type_traits>

#include "tilefuse.h"

namespace tf {

// ---------------------------------------------------------------------------
// Packed layout, version 1 (the GPU counterpart of offline pre-tiling,
// Section 4.2: tile-major, K-major inside a tile, metadata per tile).
//
// Columns are grouped into panels of PW columns (64 for 4-bit, 32 for 8-bit);
// a panel is cut along K into atoms of 32 rows.  One atom is 1 KiB, exactly
// one 16-byte load per lane of a 64-lane wavefront:
//
//   lane l = 16 * kg + c   (c = 0..15, kg = 0..3), dword t = 0..3 of the lane
//   4-bit: column  64 p + c + 16 t,       rows 32 a + 8 kg + 0..7
//          nibble position j (bits 4j..4j+3) holds row offset
//          2j (j < 4) or 2(j-4)+1 (j >= 4), so nibbles j and j+4 are a K-pair
//   8-bit: column  32 p + c + 16 (t / 2), rows 32 a + 8 kg + 4 (t % 2) + 0..3,
//          one byte per row, lowest byte first
//
// The eight rows of one lane and column are exactly the 8 k-values one lane
// holds for the B operand of v_mfma_f32_16x16x32_f16 (column = lane % 16,
// k = 8 (lane / 16) + 0..7), and, for the GEMV, 8 consecutive k that meet one
// 16-byte slice of the activation row.
//
// Regions (byte offsets from the packed base, each 256-byte aligned):
//   weights: atom (p, a) at (p * NA + a) * 1024, NA = K / 32
//   scales : fp16, block (p, g) of PW entries at ((p * NG + g) * PW) * 2
//   zeros  : uint8, block (p, g) of PW entries at  (p * NG + g) * PW
// Inside a metadata block entry e = c * T + t (T = PW / 16) belongs to
// column PW p + c + 16 t, so each lane reads its T scales / zeros in one load.
// Columns past N (last panel) hold q = z = 0 and s = 0, i.e. weight 0.
// ---------------------------------------------------------------------------
constexpr int kLayoutVersion = 1;

// Workspace of the matmul entry points: arrival counters first, in a region
// of fixed size at offset 0 (every call leaves the counters it used at zero,
// so one zero-filled buffer serves calls of any shape), then partial sums.
constexpr int64_t kWsCounterBytes = (TF_MAX_DIM / 32) * 4;
// Most workgroups a stream-K GEMM launch uses (sizes its workspace).
constexpr int kSkMaxGroups = 256;
// GEMM calls with kSkinnyMinM..kSkinnyMaxM rows run the streaming kernel's
// matrix-core form (16, 32 or 64 row slots); fewer rows run the decode GEMV.
constexpr int kSkinnyMinM = 4;
constexpr int kSkinnyMaxM = 64;
constexpr int kAtomK = 32;
constexpr int kAtomBytes = 1024;

struct Layout {
    int bits;
    int64_t K, N;
    int group;
    int64_t pw;    // panel width in columns
    int64_t T;     // columns per lane in one atom (pw / 16)
    int64_t np;    // number of panels
    int64_t na;    // atoms per panel (K / 32)
    int64_t ng;    // groups (K / group)
    int64_t w_off, s_off, z_off, total;
};

__host__ __device__ inline int64_t align256(int64_t v) { return (v + 255) & ~int64_t(255); }

__host__ __device__ inline Layout make_layout(int bits, int64_t K, int64_t N, int group) {
    Layout L;
    L.bits = bits;
    L.K = K;
    L.N = N;
    L.group = group;
    L.pw = bits == 4 ? 64 : 32;
    L.T = L.pw / 16;
    L.np = (N + L.pw - 1) / L.pw;
    L.na = K / kAtomK;
    L.ng = K / group;
    L.w_off = 0;
    L.s_off = align256(L.np * L.na * kAtomBytes);
    L.z_off = L.s_off + align256(L.np * L.ng * L.pw * 2);
    L.total = L.z_off + align256(L.np * L.ng * L.pw);
    return L;
}

// ---------------------------------------------------------------------------
// Launch through hipLaunchKernel so the launch status is returned directly
// (no dependence on the sticky per-thread last-error state).
// ---------------------------------------------------------------------------
template <typename... KArgs, typename... Args>
inline int launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem,
                  hipStream_t stream, Args... args) {
    std::tuple<KArgs...> held(static_cast<KArgs>(args)...);
    void* argv[sizeof...(KArgs)];
    std::apply([&](auto&... a) {
        int i = 0;
        ((argv[i++] = static_cast<void*>(&a)), ...);
    }, held);
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv,
                                   shmem, stream);
    return e == hipSuccess ? TF_OK : TF_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Device primitives.
// ---------------------------------------------------------------------------
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef float float2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes): loads past the end return 0.
// Word 3 = 32-bit data format, no swizzle, for this GPU family.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// Cache policy of split-K partial sums: sc1, device-coherent (writes reach
// memory visible to every XCD, reads do not hit a stale line).
constexpr int kSc1 = 16;

__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }
__device__ __forceinline__ uint32_t as_u32(half2_t v) { return __builtin_bit_cast(uint32_t, v); }

// fp16 bit patterns: 0x6400 | v is exactly 1024 + v for 0 <= v < 1024.
constexpr uint32_t kMagic2 = 0x64006400u;


// kMagic2 held in a register the compiler cannot see through: VOP3
// instructions cannot carry literal constants on this target, and with both
// operands literal the compiler splits (w & mask) | magic into two
// instructions; with the magic in a register it emits one v_and_or_b32.
__device__ __forceinline__ uint32_t magic_reg() {
    uint32_t m;
    asm("v_mov_b32 %0, 0x64006400" : "=v"(m));
    return m;
}

// 0x54005400: fp16 64.0 in both halves.  Its mantissa unit is 1/16, so a
// nibble placed in bits 4..7 of a half reads as 64 + q, exactly.
__device__ __forceinline__ uint32_t magic64_reg() {
    uint32_t m;
    asm("v_mov_b32 %0, 0x54005400" : "=v"(m));
    return m;
}

// Unpack primitives (Section 4.3).  `magic` = kMagic2 (pass magic_reg()).
// Low nibbles of both halves: (1024 + q, 1024 + q') for the nibbles in bits
// 0..3 and 16..19 of x.
__device__ __forceinline__ uint32_t w4_pair_lo(uint32_t x, uint32_t magic) {
    return (x & 0x000F000Fu) | magic;
}
// Nibbles in bits 4..7 and 20..23 of x, read without a shift:
// (1024 + 16 q, 1024 + 16 q'), still exact fp16 integers.
__device__ __forceinline__ uint32_t w4_pair_hi_x16(uint32_t x, uint32_t magic) {
    return (x & 0x00F000F0u) | magic;
}
// Nibbles in bits 4..7 and 20..23 of x as (64 + q, 64 + q') with
// magic64 = magic64_reg(): exact fp16 integers, no shift.
__device__ __forceinline__ uint32_t w4_pair_hi_64(uint32_t x, uint32_t magic64) {
    return (x & 0x00F000F0u) | magic64;
}
// Bytes b, b+1 of an 8-bit dword as (1024 + q, 1024 + q'): v_perm_b32 picks
// bytes of the second operand with selector values 0-3 and of the first
// (0x64 bytes) with 4; `hi` selects bytes 2, 3 instead of 0, 1.
__device__ __forceinline__ uint32_t w8_pair(uint32_t w, bool hi) {
    return __builtin_amdgcn_perm(0x64646464u, w, hi ? 0x04030402u : 0x04010400u);
}

// One packed 4-bit dword -> four half2 K-pairs (1024 + q[k], 1024 + q[k+1])
// for row offsets (0,1), (2,3), (4,5), (6,7).
__device__ __forceinline__ void w4_code_pairs(uint32_t w, uint32_t magic, uint32_t out[4]) {
    out[0] = w4_pair_lo(w, magic);
    out[1] = w4_pair_lo(w >> 4, magic);
    out[2] = w4_pair_lo(w >> 8, magic);
    out[3] = w4_pair_lo(w >> 12, magic);
}

// Cheaper variant for sums (five instructions per dword): out[0], out[2] are
// rows (0,1), (4,5) as 1024 + q; out[1], out[3] are rows (2,3), (6,7) as
// 64 + q.
__device__ __forceinline__ void w4_code_pairs_sum(uint32_t w, uint32_t magic, uint32_t magic64,
                                                  uint32_t out[4]) {
    const uint32_t w8 = w >> 8;
    out[0] = w4_pair_lo(w, magic);
    out[1] = w4_pair_hi_64(w, magic64);
    out[2] = w4_pair_lo(w8, magic);
    out[3] = w4_pair_hi_64(w8, magic64);
}

// One 8-bit dword (rows r..r+3, lowest byte first) -> two half2 pairs
// (1024 + q[r], 1024 + q[r+1]) and (1024 + q[r+2], 1024 + q[r+3]).
__device__ __forceinline__ void w8_code_pairs(uint32_t w, uint32_t out[2]) {
    out[0] = w8_pair(w, false);
    out[1] = w8_pair(w, true);
}

// -(1024 + z) as an fp16 pair, exact for 0 <= z <= 255.
__device__ __forceinline__ uint32_t neg_zero_pair(uint32_t z) {
    uint32_t h = 0xE400u | z;          // sign bit | (1024 + z)
    return h | (h << 16);
}

// -(64 + z) as an fp16 pair from neg_zero_pair(z): -(1024 + z) + 960, exact.
__device__ __forceinline__ uint32_t neg_zero64_pair(uint32_t negz2) {
    const half2_t c960 = {(_Float16)960.0f, (_Float16)960.0f};
    return as_u32(as_h2(negz2) + c960);
}

// Dequantization of eight weights (one MFMA B operand) as a fixed sequence of
// single vector instructions ("micro-steps"), so that a kernel can place them
// one by one between matrix instructions.  dq_w4_dword / dq_w8_dwords run
// the whole sequence; every kernel and tf_dequant use this code.
//
// 4-bit, 13 steps:
//   0      w8 = w >> 8
//   1..4   unpack: rows (0,1), (4,5) as 1024 + q; rows (2,3), (6,7) read without
//          a shift as 1024 + 16 q (see w4_pair_hi_x16)
//   5, 6   (1024 + q) - (1024 + z) = q - z, exact
//   7, 8   (1024 + 16 q) / 16 - (64 + z) by one fused multiply-add: its exact
//          value q - z is an fp16 integer, so its single rounding is exact
//   9..12  one fp16 multiply by s: RNE(s * (q - z)) (Eq. 2), rounded once
// negz2 = neg_zero_pair(z), negz64 = neg_zero64_pair(negz2), s2 = (s, s).
struct DqState {
    uint32_t w8;
    uint32_t p[4];   // four half2 K-pairs
    u32x4 out;       // the finished operand, pair j in dword j
};
constexpr int kDqW4Steps = 13, kDqW8Steps = 12;

__device__ __forceinline__ void dq_w4_step(int k, uint32_t w, uint32_t magic, uint32_t negz2,
                                           uint32_t negz64, half2_t s2, DqState& st) {
#pragma clang fp contract(off)
    const half2_t sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f};
    switch (k) {
        case 0: st.w8 = w >> 8; break;
        case 1: st.p[0] = w4_pair_lo(w, magic); break;
        case 2: st.p[1] = w4_pair_hi_x16(w, magic); break;
        case 3: st.p[2] = w4_pair_lo(st.w8, magic); break;
        case 4: st.p[3] = w4_pair_hi_x16(st.w8, magic); break;
        case 5: st.p[0] = as_u32(as_h2(st.p[0]) + as_h2(negz2)); break;
        case 6: st.p[2] = as_u32(as_h2(st.p[2]) + as_h2(negz2)); break;
        case 7: st.p[1] = as_u32(__builtin_elementwise_fma(as_h2(st.p[1]), sixteenth, as_h2(negz64))); break;
        case 8: st.p[3] = as_u32(__builtin_elementwise_fma(as_h2(st.p[3]), sixteenth, as_h2(negz64))); break;
        default: st.out[k - 9] = as_u32(as_h2(st.p[k - 9]) * s2); break;
    }
}

// 8-bit, 12 steps on two dwords (rows 0..3, 4..7):
//   0..3   unpack to four pairs 1024 + q (see w8_code_pairs)
//   4..7   (1024 + q) - (1024 + z) = q - z, exact (|q - z| <= 255)
//   8..11  one fp16 multiply by s (Eq. 2), rounded once
__device__ __forceinline__ void dq_w8_step(int k, uint32_t w0, uint32_t w1, uint32_t negz2,
                                           half2_t s2, DqState& st) {
#pragma clang fp contract(off)
    switch (k) {
        case 0: st.p[0] = w8_pair(w0, false); break;
        case 1: st.p[1] = w8_pair(w0, true); break;
        case 2: st.p[2] = w8_pair(w1, false); break;
        case 3: st.p[3] = w8_pair(w1, true); break;
        case 4: case 5: case 6: case 7:
            st.p[k - 4] = as_u32(as_h2(st.p[k - 4]) + as_h2(negz2));
            break;
        default: st.out[k - 8] = as_u32(as_h2(st.p[k - 8]) * s2); break;
    }
}

// Eight dequantized fp16 weights from one 4-bit dword, each RNE(s * (q - z)).
__device__ __forceinline__ half8_t dq_w4_dword(uint32_t w, uint32_t magic, uint32_t negz2,
                                               uint32_t negz64, half2_t s2) {
    DqState st;
#pragma unroll
    for (int k = 0; k < kDqW4Steps; ++k) dq_w4_step(k, w, magic, negz2, negz64, s2, st);
    return __builtin_bit_cast(half8_t, st.out);
}

// Eight dequantized fp16 weights from two 8-bit dwords (rows 0..3, 4..7).
__device__ __forceinline__ half8_t dq_w8_dwords(uint32_t w0, uint32_t w1, uint32_t negz2,
                                                half2_t s2) {
    DqState st;
#pragma unroll
    for (int k = 0; k < kDqW8Steps; ++k) dq_w8_step(k, w0, w1, negz2, s2, st);
    return __builtin_bit_cast(half8_t, st.out);
}

// 16-byte LDS slot of chunk `ch` (0..3) of activation row `row` in a tile of
// 64-byte rows (32 fp16 / bf16 values of K per row), a whole number of 16-row
// blocks.  Each 16-row block is stored chunk-major: chunk 0 of its 16 rows,
// then chunk 1, and so on.  The matrix-core kernels read one 16-row block per
// ds_read_b128 (lane c of quarter kg reads row r0 + c, chunk kg), so the 64
// lanes of a wavefront read 1 KB of consecutive bytes, which the LDS serves
// without bank conflicts; the block's writers (a direct load or a store of
// 64 lanes) likewise cover 1 KB of consecutive slots.  (Measured on MI355X
// with a read-only probe: the former layout, chunks XOR-swizzled inside each
// row, took 4 bank-conflict cycles per ds_read_b128 and ran 68% slower than
// this one.)
__device__ __forceinline__ int lds_a_slot(int row, int ch) { return ((row >> 4) << 6) + (ch << 4) + (row & 15); }
// The row and chunk that slot x holds (the inverse of lds_a_slot).
__device__ __forceinline__ int lds_a_row(int x) { return ((x >> 6) << 4) + (x & 15); }
__device__ __forceinline__ int lds_a_chunk(int x) { return (x >> 4) & 3; }

// ---------------------------------------------------------------------------
// BF16 activations and scales (Sections 2.2 and 4.3: the paper's kernels take
// BF16 activations, BF16 scales, and hold the dequantized weights in BF16).
// Kernels are instantiated for fp16 (BF = false) and bfloat16 (BF = true);
// both travel as 16-bit patterns, accumulation is fp32 either way.
//
// This GPU has no packed bfloat16 arithmetic, so the BF16 dequantization runs
// in fp32: each code becomes an fp32 integer (v_cvt_f32_ubyte), one fused
// multiply-add forms s * q - z * s = s * (q - z) exactly (s has 8 significant
// bits and |q - z| < 2^8, so the product and z * s fit fp32's 24), and
// v_cvt_pk_bf16_f32 rounds each pair to bfloat16, nearest even (Eq. 2,
// rounded once).
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// bfloat16 bits -> fp32 (exact: the pattern is the high half of a binary32)
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __builtin_bit_cast(float, bits16 << 16);
}
// The scale in fp32 from its 16-bit pattern.
template <bool BF>
__device__ __forceinline__ float scale_f32(uint32_t bits16) {
    if constexpr (BF) return bf16_to_f32(bits16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}
// fp32 -> output element, rounded to nearest even.
template <bool BF>
__device__ __forceinline__ uint16_t round_out(float v) {
    if constexpr (BF) return __builtin_bit_cast(uint16_t, (__bf16)v);
    else return __builtin_bit_cast(uint16_t, (_Float16)v);
}
// Two fp32 values -> one dword of two output elements (a in the low half).
template <bool BF>
__device__ __forceinline__ uint32_t round_out2(float a, float b) {
    if constexpr (BF) {
        const bf16x2_t v = {(__bf16)a, (__bf16)b};
        return __builtin_bit_cast(uint32_t, v);
    } else {
        const half2_t v = {(_Float16)a, (_Float16)b};
        return as_u32(v);
    }
}
// c + a.lo * b.lo + a.hi * b.hi with fp32 accumulation (v_dot2 of two 16-bit pairs).
template <bool BF>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    if constexpr (BF)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                               __builtin_bit_cast(bf16x2_t, b), c, false);
    else return __builtin_amdgcn_fdot2(as_h2(a), as_h2(b), c, false);
}
// acc += a x b on the matrix core, 16 x 16 x 32, 16-bit inputs.
template <bool BF>
__device__ __forceinline__ float4_t mfma16(const u32x4& a, const u32x4& b, const float4_t& c) {
    if constexpr (BF)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                      __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
}

// acc += a x b on the matrix core with the accumulator pinned to one AGPR
// quad (source C and destination the same registers).  An asm statement
// because, with hundreds of loop-carried accumulators, the register
// allocator otherwise copies them between AGPRs and VGPRs at every step; not
// volatile, so it still schedules freely.  The compiler does not see the
// matrix instruction inside, so it inserts none of the wait states the ISA
// requires around it: a caller keeps at least two wait states between a
// vector-ALU write of an operand and the MFMA that reads it, and puts
// mfma_hazard_gap() between the accumulators' initialisation and the first
// MFMA and between the last MFMA and the first read of the accumulators.
template <bool BF>
__device__ __forceinline__ void mfma_acc(float4_t& acc, const u32x4& a, const u32x4& b) {
    if constexpr (BF)
        asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
    else
        asm("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// 32 wait states, more than any matrix-instruction dependency requires.
__device__ __forceinline__ void mfma_hazard_gap() {
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7");
}

// bfloat16 pattern 0x4300 | v is exactly 128 + v for 0 <= v < 128: a nibble
// in bits 0..3 of each half of x reads as (128 + q, 128 + q').
constexpr uint32_t kMagicBf2 = 0x43004300u;
__device__ __forceinline__ uint32_t magic_bf_reg() {
    uint32_t m;
    asm("v_mov_b32 %0, 0x43004300" : "=v"(m));
    return m;
}

// Per-column dequantization constants of one group.
//  fp16: (s, s), -(1024 + z) and -(64 + z) as fp16 pairs (see dq_w4_step);
//  bf16: s and -(z * s) in fp32 (exact).
template <bool BF>
struct DqConst;
template <>
struct DqConst<false> {
    half2_t s2;
    uint32_t nz, nz64;
};
template <>
struct DqConst<true> {
    float s, nzs;
};
template <bool BF>
__device__ __forceinline__ DqConst<BF> make_dq_const(uint32_t sbits16, uint32_t z) {
    DqConst<BF> k;
    if constexpr (BF) {
        k.s = bf16_to_f32(sbits16);
        k.nzs = -((float)z * k.s);
    } else {
        k.s2 = as_h2(sbits16 | (sbits16 << 16));
        k.nz = neg_zero_pair(z);
        k.nz64 = neg_zero64_pair(k.nz);
    }
    return k;
}

// BF16 dequantization micro-steps (one vector instruction each, like
// dq_w4_step / dq_w8_step).  Packed nibble j holds row 2j (j < 4) or
// 2(j - 4) + 1, so after lo = w & 0x0F0F0F0F and hi = (w >> 4) & 0x0F0F0F0F
// the bytes hold rows lo: 0, 4, 1, 5 and hi: 2, 6, 3, 7.
// 4-bit, 23 steps: 0..2 split into lo, hi; then per output pair j (rows
// 2j, 2j + 1), five steps: two byte -> fp32 conversions, two exact fmas,
// one rounding conversion of the pair.
// 8-bit, 20 steps on w0 (rows 0..3) and w1 (rows 4..7): five per pair.
struct DqStateBf {
    uint32_t lo, hi;
    float f0, f1;
    u32x4 out;
};
constexpr int kDqW4StepsBf = 23, kDqW8StepsBf = 20;

__device__ __forceinline__ float byte_f32(uint32_t v, int b) {
    return (float)((v >> (8 * b)) & 0xFFu);      // v_cvt_f32_ubyte{b}
}

// pair j's source word and bytes (4-bit: after the split)
__device__ __forceinline__ void dq_bf_pair_step(int k, uint32_t src, int b0, int b1, int j,
                                                const DqConst<true>& kc, DqStateBf& st) {
    switch (k) {
        case 0: st.f0 = byte_f32(src, b0); break;
        case 1: st.f1 = byte_f32(src, b1); break;
        case 2: st.f0 = __builtin_fmaf(st.f0, kc.s, kc.nzs); break;
        case 3: st.f1 = __builtin_fmaf(st.f1, kc.s, kc.nzs); break;
        default: {
            const bf16x2_t v = {(__bf16)st.f0, (__bf16)st.f1};
            st.out[j] = __builtin_bit_cast(uint32_t, v);
        }
    }
}

__device__ __forceinline__ void dq_w4_step_bf(int k, uint32_t w, const DqConst<true>& kc,
                                              DqStateBf& st) {
    // (the empty asm statements hide from the compiler that the bytes are
    // below 16: knowing it, it extracts each nibble with v_bfe_u32 and
    // converts byte 0, two instructions per weight, instead of one
    // v_cvt_f32_ubyte{b})
    if (k == 0) { st.lo = w & 0x0F0F0F0Fu; asm("" : "+v"(st.lo)); return; }
    if (k == 1) { st.hi = w >> 4; return; }
    if (k == 2) { st.hi &= 0x0F0F0F0Fu; asm("" : "+v"(st.hi)); return; }
    const int j = (k - 3) / 5, r = (k - 3) % 5;
    // pairs: (lo.b0, lo.b2), (hi.b0, hi.b2), (lo.b1, lo.b3), (hi.b1, hi.b3)
    dq_bf_pair_step(r, (j & 1) ? st.hi : st.lo, j >> 1, (j >> 1) + 2, j, kc, st);
}

__device__ __forceinline__ void dq_w8_step_bf(int k, uint32_t w0, uint32_t w1,
                                              const DqConst<true>& kc, DqStateBf& st) {
    const int j = k / 5, r = k % 5;
    dq_bf_pair_step(r, j < 2 ? w0 : w1, 2 * (j & 1), 2 * (j & 1) + 1, j, kc, st);
}

// Generic interface over both element types: the state, the number of
// micro-steps, one step, and the whole operand (eight weights of one column,
// 16-bit elements, rows 0..7 in order, two per dword).  w1 is the second
// dword of an 8-bit operand (unused for 4-bit).  `magic` = magic_reg() (fp16).
template <bool BF>
using DqSt = typename std::conditional<BF, DqStateBf, DqState>::type;

template <bool BF, int BITS>
constexpr int dq_steps() {
    return BF ? (BITS == 4 ? kDqW4StepsBf : kDqW8StepsBf) : (BITS == 4 ? kDqW4Steps : kDqW8Steps);
}

template <bool BF, int BITS>
__device__ __forceinline__ void dq_step(int k, uint32_t w0, uint32_t w1, uint32_t magic,
                                        const DqConst<BF>& kc, DqSt<BF>& st) {
    if constexpr (BF) {
        if constexpr (BITS == 4) dq_w4_step_bf(k, w0, kc, st);
        else dq_w8_step_bf(k, w0, w1, kc, st);
    } else {
        if constexpr (BITS == 4) dq_w4_step(k, w0, magic, kc.nz, kc.nz64, kc.s2, st);
        else dq_w8_step(k, w0, w1, kc.nz, kc.s2, st);
    }
}

template <bool BF, int BITS>
__device__ __forceinline__ u32x4 dq_operand(uint32_t w0, uint32_t w1, uint32_t magic,
                                            const DqConst<BF>& kc) {
    DqSt<BF> st;
#pragma unroll
    for (int k = 0; k < dq_steps<BF, BITS>(); ++k) dq_step<BF, BITS>(k, w0, w1, magic, kc, st);
    return st.out;
}

}  // namespace tf

// Host services shared by the launchers (tf_api.hip).
namespace tf {
// Compute units of the device that `stream` belongs to (NULL: the current
// device), queried once per device and cached; 256 if the runtime cannot
// tell.  Safe to call from several threads at once.
int device_cus(hipStream_t stream);
// Whether TF_LOG=1 is set (read once); log_plan() then writes one line per
// matmul call to stderr naming the kernel and launch plan it chose.
bool log_enabled();
void log_plan(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
}  // namespace tf

// Launchers implemented in the kernel sources (called by tf_api.hip after
// argument validation).
namespace tf {
int launch_pack_w4(const int32_t* qw, const int32_t* qz, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s);
int launch_pack_w8(const uint8_t* qw, const uint8_t* zr, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s);
int launch_pack_w8_sym(const int8_t* qw, const uint16_t* sc, const Layout& L, void* packed,
                       hipStream_t s);
int launch_unpack(const Layout& L, const void* packed, uint8_t* q_out, uint8_t* z_out,
                  hipStream_t s);
int launch_dequant(const Layout& L, const void* packed, int out_dtype, void* w_out,
                   hipStream_t s);
int64_t gemv_workspace_bytes(const Layout& L, int64_t M);
int64_t skinny_workspace_bytes(const Layout& L, int64_t M);
int launch_gemv(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s, bool bf);
int launch_skinny_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C,
                       int64_t M, void* ws, hipStream_t s, bool bf);
int64_t gemm_workspace_bytes(const Layout& L, int64_t M);
bool gemm256_supported(const Layout& L);
bool gemm256_fills_device(const Layout& L, int64_t M, hipStream_t s);
int64_t gemm256_workspace_bytes(const Layout& L, int64_t M);
int launch_gemm256(const Layout& L, const uint16_t* A, const uint8_t* pk, uint16_t* C, int64_t M,
                   void* ws, size_t ws_bytes, hipStream_t s, bool bf);
// The 64 x 128 GEMM with K split over the workgroup's waves (no workspace).
bool gemm_ks_supported(const Layout& L);
int launch_gemm_ks(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                   hipStream_t s, bool bf);
// The same kernel over a range of the 256-row GEMM's 256 x 256 tiles: count
// tiles from tile0 in that GEMM's order (row-major or column-major over
// tiles_m x tiles_n), each as 8 tiles of 64 x 128.
struct KsRange {
    int tile0, count, tiles_m, tiles_n, col_major;
};
int launch_gemm_ks_range(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                         const KsRange& rg, hipStream_t s, bool bf);
int launch_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, size_t ws_bytes, hipStream_t s, bool bf);
int launch_silu_mul(const uint16_t* gu, int64_t M, int64_t N, uint16_t* h, hipStream_t s, bool bf);
}  // namespace tf
