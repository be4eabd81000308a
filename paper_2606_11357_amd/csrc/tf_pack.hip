// Offline pre-tiling (Section 4.2) into the packed layout described in
// tf_internal.h, and the debug kernels that read it back through the same
// device unpack / dequantize primitives as the matmul kernels (Section 4.3).
#include "tf_internal.h"

namespace tf {
namespace {

// Row offset (0..7) held by nibble position j of a packed 4-bit dword.
__device__ __forceinline__ int w4_row_of_nibble(int j) { return j < 4 ? 2 * j : 2 * (j - 4) + 1; }

// One thread per output dword of the weights region.
__global__ void pack_w4_weights(const int32_t* __restrict__ qw, uint32_t* __restrict__ out,
                                int64_t K, int64_t N, int64_t na, int64_t total_dwords) {
    int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (d >= total_dwords) return;
    int64_t atom = d >> 8;
    int within = (int)(d & 255);
    int lane = within >> 2, t = within & 3;
    int64_t p = atom / na, a = atom % na;
    int c = lane & 15, kg = lane >> 4;
    int64_t n = p * 64 + c + 16 * t;
    uint32_t word = 0;
    if (n < N) {
        int64_t k0 = a * kAtomK + 8 * kg;
        const uint32_t* src = reinterpret_cast<const uint32_t*>(qw);
        int shift = 4 * (int)(n & 7);
        for (int j = 0; j < 8; ++j) {
            int64_t k = k0 + w4_row_of_nibble(j);
            uint32_t q = (src[k * (N / 8) + (n >> 3)] >> shift) & 0xFu;
            word |= q << (4 * j);
        }
    }
    out[d] = word;
}

// flip = 0x80808080 turns signed INT8 codes into unsigned codes q + 128
// (two's complement: flipping the sign bit adds 128).
__global__ void pack_w8_weights(const uint8_t* __restrict__ qw, uint32_t* __restrict__ out,
                                int64_t K, int64_t N, int64_t na, int64_t total_dwords,
                                uint32_t flip) {
    int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (d >= total_dwords) return;
    int64_t atom = d >> 8;
    int within = (int)(d & 255);
    int lane = within >> 2, t = within & 3;
    int64_t p = atom / na, a = atom % na;
    int c = lane & 15, kg = lane >> 4;
    int64_t n = p * 32 + c + 16 * (t >> 1);
    uint32_t word = 0;
    if (n < N) {
        int64_t k0 = a * kAtomK + 8 * kg + 4 * (t & 1);
        for (int b = 0; b < 4; ++b) word |= (uint32_t)qw[(k0 + b) * N + n] << (8 * b);
        word ^= flip;
    }
    out[d] = word;
}

// One thread per metadata entry: scales copied bit for bit, zero-points
// unpacked to one byte each.  s_gstride = N for per-group scales [K/G, N], 0
// for one scale per column [N]; with neither zero-point array, zconst.
__global__ void pack_meta(const uint16_t* __restrict__ sc, const int32_t* __restrict__ qz4,
                          const uint8_t* __restrict__ z8, uint16_t* __restrict__ s_out,
                          uint8_t* __restrict__ z_out, int64_t N, int64_t ng, int pw,
                          int64_t entries, int64_t s_gstride, int zconst) {
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= entries) return;
    int64_t p = e / (ng * pw);
    int64_t g = (e / pw) % ng;
    int i = (int)(e % pw);
    int T = pw / 16;
    int c = i / T, t = i % T;
    int64_t n = p * pw + c + 16 * t;
    uint16_t s = 0;
    uint8_t z = 0;
    if (n < N) {
        s = sc[g * s_gstride + n];
        if (qz4) {
            uint32_t w = reinterpret_cast<const uint32_t*>(qz4)[g * (N / 8) + (n >> 3)];
            z = (uint8_t)((w >> (4 * (int)(n & 7))) & 0xFu);
        } else if (z8) {
            z = z8[g * N + n];
        } else {
            z = (uint8_t)zconst;
        }
    }
    s_out[e] = s;
    z_out[e] = z;
}

// Column and row of code (lane, dword t, position j) of an atom.
struct CodePos {
    int64_t n, k;
};

__device__ __forceinline__ CodePos w4_pos(int64_t p, int64_t a, int lane, int t, int j) {
    // j: row offset 0..7 inside the lane's 8-row slice
    return {p * 64 + (lane & 15) + 16 * t, a * kAtomK + 8 * (lane >> 4) + j};
}
__device__ __forceinline__ CodePos w8_pos(int64_t p, int64_t a, int lane, int t, int b) {
    return {p * 32 + (lane & 15) + 16 * (t >> 1), a * kAtomK + 8 * (lane >> 4) + 4 * (t & 1) + b};
}

// tf_unpack: one thread per packed dword; the codes come out of the same
// magic-number unpack the matmul kernels use, then 1024 is removed.
__global__ void unpack_weights(int bits, const uint32_t* __restrict__ wreg, uint8_t* __restrict__ q_out,
                               int64_t N, int64_t na, int64_t total_dwords) {
    int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (d >= total_dwords) return;
    int64_t atom = d >> 8;
    int within = (int)(d & 255);
    int lane = within >> 2, t = within & 3;
    int64_t p = atom / na, a = atom % na;
    uint32_t w = wreg[d];
    if (bits == 4) {
        uint32_t cp[4];
        w4_code_pairs(w, magic_reg(), cp);
        for (int pr = 0; pr < 4; ++pr) {
            for (int h = 0; h < 2; ++h) {
                CodePos pos = w4_pos(p, a, lane, t, 2 * pr + h);
                if (pos.n < N)
                    q_out[pos.k * N + pos.n] = (uint8_t)((cp[pr] >> (16 * h)) & 0x3FFu);
            }
        }
    } else {
        uint32_t cp[2];
        w8_code_pairs(w, cp);
        for (int pr = 0; pr < 2; ++pr) {
            for (int h = 0; h < 2; ++h) {
                CodePos pos = w8_pos(p, a, lane, t, 2 * pr + h);
                if (pos.n < N)
                    q_out[pos.k * N + pos.n] = (uint8_t)((cp[pr] >> (16 * h)) & 0x3FFu);
            }
        }
    }
}

__global__ void unpack_zeros(const uint8_t* __restrict__ zreg, uint8_t* __restrict__ z_out, int64_t N,
                             int64_t ng, int pw, int64_t entries) {
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= entries) return;
    int64_t p = e / (ng * pw);
    int64_t g = (e / pw) % ng;
    int i = (int)(e % pw);
    int T = pw / 16;
    int64_t n = p * pw + i / T + 16 * (i % T);
    if (n < N) z_out[g * N + n] = zreg[e];
}

// tf_dequant: one thread per 8 codes of one column (one MFMA B operand),
// dequantized with the matmul kernels' own code.  mode 0: fp16 scales, fp16
// weights; 1: fp16 scales, exact fp32 weights; 2: bf16 scales, bf16 weights.
__global__ void dequant_weights(int bits, const uint8_t* __restrict__ packed, int64_t s_off,
                                int64_t z_off, int64_t N, int64_t na, int64_t ng, int group,
                                int mode, void* __restrict__ w_out, int64_t slices) {
    int64_t sidx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (sidx >= slices) return;
    // slice = (atom, lane, column-slot); 64 lanes x 4 (4-bit) or 2 (8-bit) slots
    const int T = bits == 4 ? 4 : 2;
    const int pw = bits == 4 ? 64 : 32;
    int64_t atom = sidx / (64 * T);
    int rem = (int)(sidx % (64 * T));
    int lane = rem / T, t = rem % T;
    int64_t p = atom / na, a = atom % na;
    int c = lane & 15;
    int64_t n = p * pw + c + 16 * t;
    if (n >= N) return;
    int64_t k0 = a * kAtomK + 8 * (lane >> 4);
    int64_t g = (a * kAtomK) / group;
    int64_t meta = (p * ng + g) * pw + c * T + t;
    uint16_t sbits = reinterpret_cast<const uint16_t*>(packed + s_off)[meta];
    uint32_t z = packed[z_off + meta];
    const uint32_t* atomw = reinterpret_cast<const uint32_t*>(packed) + atom * 256 + lane * 4;
    if (mode == 2) {
        const DqConst<true> kq = make_dq_const<true>(sbits, z);
        const u32x4 wb = bits == 4 ? dq_operand<true, 4>(atomw[t], 0u, 0u, kq)
                                   : dq_operand<true, 8>(atomw[2 * t], atomw[2 * t + 1], 0u, kq);
        uint16_t* o = reinterpret_cast<uint16_t*>(w_out);
        for (int j = 0; j < 8; ++j) o[(k0 + j) * N + n] = (uint16_t)(wb[j >> 1] >> (16 * (j & 1)));
        return;
    }
    half8_t w8;
    uint32_t codes[4];
    if (bits == 4) {
        uint32_t w = atomw[t];
        const uint32_t magic = magic_reg();
        const uint32_t nz = neg_zero_pair(z);
        w8 = dq_w4_dword(w, magic, nz, neg_zero64_pair(nz), as_h2(sbits | ((uint32_t)sbits << 16)));
        w4_code_pairs(w, magic, codes);
    } else {
        uint32_t w0 = atomw[2 * t], w1 = atomw[2 * t + 1];
        w8 = dq_w8_dwords(w0, w1, neg_zero_pair(z), as_h2(sbits | ((uint32_t)sbits << 16)));
        w8_code_pairs(w0, codes);
        w8_code_pairs(w1, codes + 2);
    }
    if (mode == 1) {
        // exact: (q - z) is formed exactly in fp16 by the same pair subtraction
        // and its product with the fp16 scale needs at most 19 significant bits
        float s = (float)__builtin_bit_cast(_Float16, sbits);
        float* o = reinterpret_cast<float*>(w_out);
        for (int j = 0; j < 8; ++j) {
            half2_t d = as_h2(codes[j >> 1]) + as_h2(neg_zero_pair(z));
            o[(k0 + j) * N + n] = (float)d[j & 1] * s;
        }
    } else {
        _Float16* o = reinterpret_cast<_Float16*>(w_out);
        for (int j = 0; j < 8; ++j) o[(k0 + j) * N + n] = w8[j];
    }
}

inline unsigned blocks_for(int64_t n, int threads) { return (unsigned)((n + threads - 1) / threads); }

}  // namespace

int launch_pack_w4(const int32_t* qw, const int32_t* qz, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s) {
    uint8_t* base = static_cast<uint8_t*>(packed);
    int64_t dwords = L.np * L.na * 256;
    int rc = launch(pack_w4_weights, dim3(blocks_for(dwords, 256)), dim3(256), 0, s, qw,
                    reinterpret_cast<uint32_t*>(base + L.w_off), L.K, L.N, L.na, dwords);
    if (rc) return rc;
    int64_t entries = L.np * L.ng * L.pw;
    return launch(pack_meta, dim3(blocks_for(entries, 256)), dim3(256), 0, s, sc, qz,
                  (const uint8_t*)nullptr, reinterpret_cast<uint16_t*>(base + L.s_off),
                  base + L.z_off, L.N, L.ng, (int)L.pw, entries, L.N, 0);
}

int launch_pack_w8(const uint8_t* qw, const uint8_t* zr, const uint16_t* sc, const Layout& L,
                   void* packed, hipStream_t s) {
    uint8_t* base = static_cast<uint8_t*>(packed);
    int64_t dwords = L.np * L.na * 256;
    int rc = launch(pack_w8_weights, dim3(blocks_for(dwords, 256)), dim3(256), 0, s, qw,
                    reinterpret_cast<uint32_t*>(base + L.w_off), L.K, L.N, L.na, dwords, 0u);
    if (rc) return rc;
    int64_t entries = L.np * L.ng * L.pw;
    return launch(pack_meta, dim3(blocks_for(entries, 256)), dim3(256), 0, s, sc,
                  (const int32_t*)nullptr, zr, reinterpret_cast<uint16_t*>(base + L.s_off),
                  base + L.z_off, L.N, L.ng, (int)L.pw, entries, L.N, 0);
}

// Signed INT8 with one scale per column (Eq. 1): stored as the 8-bit layout
// with codes q + 128, zero-point 128 and the column's scale in every group,
// so s * ((q + 128) - 128) = s * q through the same kernels.
int launch_pack_w8_sym(const int8_t* qw, const uint16_t* sc, const Layout& L, void* packed,
                       hipStream_t s) {
    uint8_t* base = static_cast<uint8_t*>(packed);
    int64_t dwords = L.np * L.na * 256;
    int rc = launch(pack_w8_weights, dim3(blocks_for(dwords, 256)), dim3(256), 0, s,
                    reinterpret_cast<const uint8_t*>(qw), reinterpret_cast<uint32_t*>(base + L.w_off),
                    L.K, L.N, L.na, dwords, 0x80808080u);
    if (rc) return rc;
    int64_t entries = L.np * L.ng * L.pw;
    return launch(pack_meta, dim3(blocks_for(entries, 256)), dim3(256), 0, s, sc,
                  (const int32_t*)nullptr, (const uint8_t*)nullptr,
                  reinterpret_cast<uint16_t*>(base + L.s_off), base + L.z_off, L.N, L.ng, (int)L.pw,
                  entries, (int64_t)0, 128);
}

int launch_unpack(const Layout& L, const void* packed, uint8_t* q_out, uint8_t* z_out,
                  hipStream_t s) {
    const uint8_t* base = static_cast<const uint8_t*>(packed);
    int64_t dwords = L.np * L.na * 256;
    int rc = launch(unpack_weights, dim3(blocks_for(dwords, 256)), dim3(256), 0, s, L.bits,
                    reinterpret_cast<const uint32_t*>(base + L.w_off), q_out, L.N, L.na, dwords);
    if (rc) return rc;
    int64_t entries = L.np * L.ng * L.pw;
    return launch(unpack_zeros, dim3(blocks_for(entries, 256)), dim3(256), 0, s, base + L.z_off,
                  z_out, L.N, L.ng, (int)L.pw, entries);
}

int launch_dequant(const Layout& L, const void* packed, int out_dtype, void* w_out,
                   hipStream_t s) {
    int64_t slices = L.np * L.na * 64 * L.T;
    return launch(dequant_weights, dim3(blocks_for(slices, 256)), dim3(256), 0, s, L.bits,
                  static_cast<const uint8_t*>(packed), L.s_off, L.z_off, L.N, L.na, L.ng,
                  L.group, out_dtype == TF_F32 ? 1 : out_dtype == TF_BF16 ? 2 : 0, w_out, slices);
}

}  // namespace tf
