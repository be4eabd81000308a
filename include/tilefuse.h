/*
 * tilefuse.h -- C ABI of the fused weight-only quantized matmul for gfx950.
 *
 * The operation (TileFuse, Sections 2.1-2.2 and 4.2-4.3):
 *
 *     C[m, n] = sum_k A[m, k] * w_hat[k, n],      C = A x B (Section 2.1)
 *     w_hat[k, n] = s[g, n] * (q[k, n] - z[g, n]), g = floor(k / G)  (Eq. 2)
 *
 * A is fp16 [M, K] row-major, the weights are 4-bit (W4A16) or 8-bit (W8A16)
 * integer codes with one fp16 scale and one integer zero-point per group of G
 * consecutive k in one column n (Section 2.2), accumulation is fp32 and C is
 * fp16 [M, N] row-major, rounded to nearest even.  The weights never exist in
 * memory as fp16: each kernel unpacks and dequantizes them on the fly (Section
 * 4.3, fused unpack -> dequantize -> multiply-accumulate).
 *
 * Weights are first rearranged once, offline, into a device-private layout
 * (tf_pack_w4 / tf_pack_w8; the GPU counterpart of the offline pre-tiling of
 * Section 4.2).  The packed buffer is opaque; pass the same (K, N, group) to
 * the matmul calls that were given to the pack call.
 *
 * Conventions for every entry point:
 *  - All array pointers are DEVICE pointers (hipMalloc / torch CUDA tensors).
 *  - fp16 values travel as uint16_t bit patterns.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    Calls only enqueue work on `stream` and return; the caller synchronizes.
 *  - The caller allocates and frees every buffer; the library keeps no device
 *    memory.  Its only global state is a per-device cache of the compute-unit
 *    count (read atomically; the launch plans depend on it), so calls are
 *    thread-safe.  Plans are made for the device of the `stream` argument.
 *  - Arguments are validated before any HIP call; a rejected call enqueues
 *    nothing.  Only TF_ERR_HIP comes from the runtime (launch failure).
 *  - Outputs must not overlap inputs.
 *  - No C++ exception crosses this boundary.  The library prints nothing,
 *    except with the environment variable TF_LOG=1 (read once, at the first
 *    matmul call): each matmul call then writes one line to stderr naming the
 *    kernel it launched and its plan (tiles, K slices, stream-K blocks).
 */
#ifndef TILEFUSE_H
#define TILEFUSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (returned as int; negative means failure). */
enum tf_status {
    TF_OK = 0,
    TF_ERR_NULL = -1,   /* a required pointer is NULL                          */
    TF_ERR_SHAPE = -2,  /* M < 1, K or N <= 0, K % group != 0, N % 8 != 0,
                           or a dimension above TF_MAX_DIM                      */
    TF_ERR_GROUP = -3,  /* group is not a positive multiple of 32              */
    TF_ERR_ALIGN = -4,  /* a pointer is not 16-byte aligned                    */
    TF_ERR_ARG = -5,    /* other bad argument: bits not 4/8, GEMV with M > 8,
                           unknown dtype, workspace too small                  */
    TF_ERR_HIP = -6     /* the HIP runtime reported an error at launch         */
};

/* Output dtypes of tf_dequant. */
enum tf_dtype { TF_F16 = 1, TF_F32 = 2, TF_BF16 = 3 };

/* Largest accepted K and N (each) and M; keeps every byte offset in int64
 * and every per-kernel index in 32 bits. */
#define TF_MAX_DIM 65536
#define TF_MAX_M (1 << 20)
/* Largest M accepted by the GEMV entry points (decode, Section 2.1). */
#define TF_GEMV_MAX_M 8

/* Library version of the packed layout; bumps whenever the layout changes. */
int tf_layout_version(void);

/* Human-readable text for a status code (static storage, never NULL). */
const char* tf_status_str(int status);

/*
 * Size in bytes of the packed buffer for a (bits, K, N, group) weight.
 * bits is 4 or 8.  Returns > 0, or a negative tf_status on bad arguments.
 */
int64_t tf_packed_bytes(int bits, int64_t K, int64_t N, int group);

/*
 * Offline pre-tiling of a 4-bit AWQ weight (Section 4.2: weights are known at
 * deployment, so the rearrangement is done once and is not on the timed path).
 *   qweight  int32 [K, N/8]   nibble i (bits 4i..4i+3) of word j = q[k, 8j+i]
 *   qzeros   int32 [K/G, N/8] same packing, z[g, 8j+i]
 *   scales   fp16  [K/G, N]   s[g, n]
 *   packed   tf_packed_bytes(4, K, N, group) bytes, written entirely
 * Requires N % 8 == 0, group % 32 == 0, K % group == 0, 16-byte aligned
 * pointers.  Integer rearrangement only: scales are copied bit for bit.
 */
int tf_pack_w4(const int32_t* qweight, const int32_t* qzeros, const uint16_t* scales,
               int64_t K, int64_t N, int group, void* packed, void* stream);

/*
 * Offline pre-tiling of an 8-bit weight with per-group zero-points.
 *   qweight  uint8 [K, N]     q[k, n]
 *   zeros    uint8 [K/G, N]   z[g, n]
 *   scales   fp16  [K/G, N]   s[g, n]
 *   packed   tf_packed_bytes(8, K, N, group) bytes
 * Same constraints as tf_pack_w4 (N % 8 == 0 keeps rows 8-byte aligned).
 * The symmetric form of Eq. 1 is the case z = 0 (pass a zero-filled array).
 */
int tf_pack_w8(const uint8_t* qweight, const uint8_t* zeros, const uint16_t* scales,
               int64_t K, int64_t N, int group, void* packed, void* stream);

/*
 * Offline pre-tiling of the W8A16 form of Section 2.2 (W8A16 paragraph):
 * signed INT8 weights with one scale per output channel and no zero-point,
 * dequantized by Eq. 1 as w_hat[k, n] = s[n] * q[k, n].
 *   qweight  int8  [K, N]     q[k, n] in -128..127
 *   scales   fp16  [N]        s[n]
 *   packed   tf_packed_bytes(8, K, N, group) bytes
 * Stored as the 8-bit layout with codes q + 128, zero-point 128 and the
 * column's scale repeated in every group of `group` rows, so the 8-bit
 * matmul and debug entry points (bits = 8, the same group) apply unchanged:
 * s * ((q + 128) - 128) = s * q exactly.  `group` only sets that internal
 * grouping (128 is the usual choice; it needs K % group == 0).  Same
 * constraints and errors as tf_pack_w8.
 */
int tf_pack_w8_sym(const int8_t* qweight, const uint16_t* scales, int64_t K, int64_t N, int group,
                   void* packed, void* stream);

/*
 * Workspace the matmul entry points can use for this problem, in bytes (0
 * when the kernels chosen for it need none).  Negative tf_status on bad
 * arguments.  The workspace holds per-K-slice partial sums (fp32) and, for
 * the decode GEMV and the weight-streaming matrix-core form, arrival counters;
 * it lets those kernels split K over more workgroups than there are output
 * panels, and the tiled GEMMs split K (partials summed by a second launch in
 * slice order) or share tiles between blocks (stream-K).
 *
 * Contract for every `workspace` argument below:
 *  - NULL selects kernels that need none (workspace_bytes is then ignored);
 *  - otherwise it is a device buffer of at least tf_workspace_bytes(...)
 *    bytes, 16-byte aligned and ZERO-FILLED before its first use; each call
 *    returns the arrival counters it used to zero, so the same buffer serves
 *    any later call (of any shape it is large enough for) without clearing;
 *  - calls that may run concurrently must not share one workspace.
 */
int64_t tf_workspace_bytes(int bits, int64_t M, int64_t K, int64_t N, int group);

/*
 * The same query under the name of the GEMM's workspace (the prefill GEMM
 * is the main user of a workspace: stream-K or split-K partial tiles).  It
 * returns exactly tf_workspace_bytes(bits, M, K, N, group), which already
 * covers every kernel the GEMM and GEMV entry points can choose for M rows,
 * so one buffer of that size serves either call.
 */
int64_t tf_gemm_workspace_bytes(int bits, int64_t M, int64_t K, int64_t N, int group);

/*
 * Prefill GEMM (Section 2.1: M grows with the prompt length):
 *   C_f16[M, N] = A_f16[M, K] x dequant(packed)[K, N], fp32 accumulate, RNE.
 * Any M >= 1.  M <= 3 runs the decode GEMV; 4 <= M <= 64 a weight-streaming
 * kernel on the matrix cores (16, 32 or 64 row slots); larger M the tiled
 * matrix-core GEMMs.  The tiled GEMMs and the 64-slot form feed the matrix
 * cores the dequantized fp16 weight RNE(s * (q - z)), rounded once; up to
 * 32 rows the streaming kernel feeds the codes themselves and applies scale
 * and zero-point to each group's sums (Eq. 2 summed over a group), so no
 * weight is rounded (as in the decode GEMV up to 4 rows).
 * workspace: see tf_workspace_bytes.
 */
int tf_w4a16_gemm(const uint16_t* A_f16, const void* packed, uint16_t* C_f16,
                  int64_t M, int64_t K, int64_t N, int group,
                  void* workspace, size_t workspace_bytes, void* stream);
int tf_w8a16_gemm(const uint16_t* A_f16, const void* packed, uint16_t* C_f16,
                  int64_t M, int64_t K, int64_t N, int group,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decode GEMV (Section 2.1: batch-1 generation turns linear layers into
 * matrix-vector products), 1 <= M <= TF_GEMV_MAX_M rows of A.
 * Same operands and result as the GEMM; vector ALU only, fp32 accumulate.
 * With a workspace (see tf_workspace_bytes) K is split over many
 * workgroups and the slices are added in a fixed order, so for a given
 * shape and workspace choice the result is bitwise identical run to run
 * (with and without a workspace the fp32 summation order differs).
 */
int tf_w4a16_gemv(const uint16_t* A_f16, const void* packed, uint16_t* C_f16,
                  int64_t M, int64_t K, int64_t N, int group,
                  void* workspace, size_t workspace_bytes, void* stream);
int tf_w8a16_gemv(const uint16_t* A_f16, const void* packed, uint16_t* C_f16,
                  int64_t M, int64_t K, int64_t N, int group,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * tf_w4a16_gemv without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that forbid hipMalloc).  Same operands, checks, kernels and
 * result as tf_w4a16_gemv with a workspace: where the decode GEMV splits K,
 * its partial sums and arrival counters live in a scratch array of 1 MiB in
 * the library's static device memory, one per GPU, held until the process
 * ends (every shape the GEMV entry points accept needs at most about 0.9 MiB;
 * a larger need returns TF_ERR_ARG).  The call allocates nothing: the first
 * call on a device looks up that device's copy of the array and enqueues one
 * small kernel on `stream` that zeroes its counters (again at the next call
 * outside stream capture if the first was captured); every call leaves the
 * counters at zero.  All calls on one GPU share its array, so calls that may
 * run concurrently on one GPU (different streams, not ordered by events)
 * race and must not overlap.
 */
int tf_w4a16_gemv_noalloc(const uint16_t* A_f16, const void* packed, uint16_t* C_f16,
                          int64_t M, int64_t K, int64_t N, int group, void* stream);

/*
 * BF16 activations and scales (the paper's dtype: Section 2.2 takes BF16
 * activations, Section 4.2 stores BF16 scales beside each weight tile,
 * Section 4.3 holds the dequantized weights in BF16 before the multiply):
 *   C_bf16[M, N] = A_bf16[M, K] x RNE_bf16(s_bf16 * (q - z))[K, N],
 * fp32 accumulate, C rounded to bfloat16, nearest even.
 * The packed buffer is the same format: tf_pack_w4 / tf_pack_w8 /
 * tf_pack_w8_sym copy the 16-bit scale patterns verbatim, so packing with
 * bfloat16 scale bits gives a buffer for these entry points (and packing
 * with fp16 bits one for the entry points above; the buffer does not record
 * which).  Same shapes, alignment, workspace contract and tf_workspace_bytes
 * as the fp16 entry points; the same kernels are chosen for each M.
 * s * (q - z) is formed exactly in fp32 and rounded once to bfloat16.
 */
int tf_w4a16_gemm_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16,
                       int64_t M, int64_t K, int64_t N, int group,
                       void* workspace, size_t workspace_bytes, void* stream);
int tf_w8a16_gemm_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16,
                       int64_t M, int64_t K, int64_t N, int group,
                       void* workspace, size_t workspace_bytes, void* stream);
int tf_w4a16_gemv_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16,
                       int64_t M, int64_t K, int64_t N, int group,
                       void* workspace, size_t workspace_bytes, void* stream);
int tf_w8a16_gemv_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16,
                       int64_t M, int64_t K, int64_t N, int group,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * Debug / test exports.  They read the packed buffer through the same device
 * unpack and dequantize code as the matmul kernels.
 *   tf_unpack : q_out uint8 [K, N] and z_out uint8 [K/G, N] (Section 4.3 unpack)
 *   tf_dequant: W_out [K, N] of s * (q - z) (Eq. 2), dtype TF_F16 (rounded
 *               once, nearest even) or TF_F32 (exact), both reading the
 *               scales as fp16; or TF_BF16: scales read as bfloat16, the
 *               weight rounded once to bfloat16 as the BF16 entry points do.
 */
int tf_unpack(int bits, const void* packed, int64_t K, int64_t N, int group,
              uint8_t* q_out, uint8_t* z_out, void* stream);
int tf_dequant(int bits, const void* packed, int64_t K, int64_t N, int group,
               int out_dtype, void* W_out, void* stream);

/*
 * Gated activation of a transformer MLP, for a layer-level composite around
 * the matmuls (gate/up GEMM -> this -> down GEMM); not part of the paper's
 * method:
 *   H[m, n] = silu(G[m, n]) * U[m, n],   silu(g) = g / (1 + exp(-g)),
 * where G = GU[:, 0:N] and U = GU[:, N:2N] are the two halves of one fp16
 * [M, 2N] row-major matrix (the output of a GEMM whose weight concatenates
 * the gate and up projections along N).  Computed in fp32; H is fp16 [M, N]
 * row-major, rounded to nearest even.  Requires N % 8 == 0 and 16-byte
 * aligned pointers; H must not overlap GU.
 */
int tf_silu_mul(const uint16_t* GU_f16, int64_t M, int64_t N, uint16_t* H_f16, void* stream);
/* The same with bfloat16 GU and H (the layer composite in the paper's dtype). */
int tf_silu_mul_bf16(const uint16_t* GU_bf16, int64_t M, int64_t N, uint16_t* H_bf16, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TILEFUSE_H */
