// Internal definitions shared by the HIP sources of libtilefuse: the packed
// weight layout (host and device), launch helper, and the device-side
// unpack / dequantize primitives every kernel uses.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

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
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// Unpack (Section 4.3): one packed 4-bit dword -> four half2 K-pairs holding
// (1024 + q[k], 1024 + q[k+1]) for row offsets (0,1), (2,3), (4,5), (6,7).
// `magic` = kMagic2 (pass magic_reg()).
__device__ __forceinline__ void w4_code_pairs(uint32_t w, uint32_t magic, uint32_t out[4]) {
    out[0] = (w & 0x000F000Fu) | magic;
    out[1] = ((w >> 4) & 0x000F000Fu) | magic;
    out[2] = ((w >> 8) & 0x000F000Fu) | magic;
    out[3] = ((w >> 12) & 0x000F000Fu) | magic;
}

// Cheaper variant for sums: the odd pairs are read without a shift, as
// (1024 + 16 q[k], 1024 + 16 q[k+1]) (nibble in bits 4..7 of each half, still
// an exact fp16 integer).  out[0], out[2]: rows (0,1), (4,5) as 1024 + q;
// out[1], out[3]: rows (2,3), (6,7) as 1024 + 16 q.  `magic` = kMagic2.
__device__ __forceinline__ void w4_code_pairs_x16(uint32_t w, uint32_t magic, uint32_t out[4]) {
    const uint32_t w8 = w >> 8;
    out[0] = (w & 0x000F000Fu) | magic;
    out[1] = (w & 0x00F000F0u) | magic;
    out[2] = (w8 & 0x000F000Fu) | magic;
    out[3] = (w8 & 0x00F000F0u) | magic;
}

// Unpack one 8-bit dword (rows r..r+3, lowest byte first) -> two half2 pairs
// (1024 + q[r], 1024 + q[r+1]) and (1024 + q[r+2], 1024 + q[r+3]).
// v_perm_b32 selector bytes 0-3 pick bytes of the second operand, 4-7 bytes
// of the first; 0x64 comes from the constant.
__device__ __forceinline__ void w8_code_pairs(uint32_t w, uint32_t out[2]) {
    out[0] = __builtin_amdgcn_perm(0x64646464u, w, 0x04010400u);
    out[1] = __builtin_amdgcn_perm(0x64646464u, w, 0x04030402u);
}

// -(1024 + z) as an fp16 pair, exact for 0 <= z <= 255.
__device__ __forceinline__ uint32_t neg_zero_pair(uint32_t z) {
    uint32_t h = 0xE400u | z;          // sign bit | (1024 + z)
    return h | (h << 16);
}

// Eq. 2 on a code pair, rounded once: (1024+q) - (1024+z) = q - z exactly in
// fp16 (|q - z| <= 255), then one fp16 multiply by s: RNE(s * (q - z)).
__device__ __forceinline__ half2_t dq_pair(uint32_t codes, uint32_t negz2, half2_t s2) {
#pragma clang fp contract(off)
    half2_t d = as_h2(codes) + as_h2(negz2);
    return d * s2;
}

// -(64 + z) as an fp16 pair from neg_zero_pair(z): -(1024 + z) + 960, exact.
__device__ __forceinline__ uint32_t neg_zero64_pair(uint32_t negz2) {
    const half2_t c960 = {(_Float16)960.0f, (_Float16)960.0f};
    return as_u32(as_h2(negz2) + c960);
}

// Eight dequantized fp16 weights (one MFMA B operand) from one 4-bit dword,
// each RNE(s * (q - z)) rounded once (Eq. 2).  Rows (0,1) and (4,5) are read
// as 1024 + q and reduced by (1024 + z); rows (2,3) and (6,7) are read without
// a shift as 1024 + 16 q and reduced by one fused multiply-add,
// (1024 + 16 q) / 16 - (64 + z), whose exact value q - z is an fp16 integer,
// so the single rounding of the fma is exact.  Then one multiply by s.
// negz2 = neg_zero_pair(z), negz64 = neg_zero64_pair(negz2), s2 = (s, s).
__device__ __forceinline__ half8_t dq_w4_dword(uint32_t w, uint32_t magic, uint32_t negz2,
                                               uint32_t negz64, half2_t s2) {
#pragma clang fp contract(off)
    uint32_t c[4];
    w4_code_pairs_x16(w, magic, c);
    const half2_t sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2_t d0 = as_h2(c[0]) + as_h2(negz2);
    const half2_t d2 = as_h2(c[2]) + as_h2(negz2);
    const half2_t d1 = __builtin_elementwise_fma(as_h2(c[1]), sixteenth, as_h2(negz64));
    const half2_t d3 = __builtin_elementwise_fma(as_h2(c[3]), sixteenth, as_h2(negz64));
    const half2_t p0 = d0 * s2, p1 = d1 * s2, p2 = d2 * s2, p3 = d3 * s2;
    return half8_t{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// Eight dequantized fp16 weights from two 8-bit dwords (rows 0..3, 4..7).
__device__ __forceinline__ half8_t dq_w8_dwords(uint32_t w0, uint32_t w1, uint32_t negz2,
                                                half2_t s2) {
    uint32_t c0[2], c1[2];
    w8_code_pairs(w0, c0);
    w8_code_pairs(w1, c1);
    half2_t p0 = dq_pair(c0[0], negz2, s2), p1 = dq_pair(c0[1], negz2, s2);
    half2_t p2 = dq_pair(c1[0], negz2, s2), p3 = dq_pair(c1[1], negz2, s2);
    return half8_t{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

}  // namespace tf

// Launchers implemented in the kernel sources (called by tf_api.hip after
// argument validation).
namespace tf {
int launch_pack_w4(const int32_t* qw, const int32_t* qz, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s);
int launch_pack_w8(const uint8_t* qw, const uint8_t* zr, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s);
int launch_unpack(const Layout& L, const void* packed, uint8_t* q_out, uint8_t* z_out,
                  hipStream_t s);
int launch_dequant(const Layout& L, const void* packed, int out_dtype, void* w_out,
                   hipStream_t s);
int64_t gemv_workspace_bytes(const Layout& L, int64_t M);
int launch_gemv(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, hipStream_t s);
int64_t gemm_workspace_bytes(const Layout& L, int64_t M);
int launch_gemm(const Layout& L, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                void* ws, size_t ws_bytes, hipStream_t s);
}  // namespace tf
