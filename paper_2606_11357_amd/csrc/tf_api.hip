// C-ABI entry points of libtilefuse: argument validation (always before any
// HIP call), layout sizing, and dispatch to the kernel launchers; and the
// host services the launchers share (device properties, plan logging).
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <mutex>

#include "tf_internal.h"

namespace tf {

int device_cus(hipStream_t stream) {
    constexpr int kMaxDevices = 64;
    constexpr int kFallback = 256;          // MI355X: 256 compute units
    // one slot per device; every writer stores the same value, read and
    // written atomically
    static std::atomic<int> cus[kMaxDevices];
    int dev = -1;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return kFallback;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return kFallback;
    cus[dev].store(n, std::memory_order_relaxed);
    return n;
}

bool log_enabled() {
    static const bool on = [] {
        const char* e = std::getenv("TF_LOG");
        return e != nullptr && e[0] == '1' && e[1] == '\0';
    }();
    return on;
}

void log_plan(const char* fmt, ...) {
    if (!log_enabled()) return;
    char line[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(line, sizeof line, fmt, ap);
    va_end(ap);
    std::fprintf(stderr, "[tilefuse] %s\n", line);
}

}  // namespace tf

namespace {

using tf::Layout;

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

// Shape / format checks shared by every entry point.
int check_weight(int bits, int64_t K, int64_t N, int group) {
    if (bits != 4 && bits != 8) return TF_ERR_ARG;
    if (group <= 0 || group % tf::kAtomK != 0) return TF_ERR_GROUP;
    if (K <= 0 || N <= 0 || K > TF_MAX_DIM || N > TF_MAX_DIM) return TF_ERR_SHAPE;
    if (K % group != 0 || N % 8 != 0) return TF_ERR_SHAPE;
    return TF_OK;
}

// Bytes of workspace the matmul kernels of this problem can use (the GEMM
// and GEMV entry points may pick different kernels for the same M: the
// larger need of the two).
int64_t workspace_bytes(const Layout& L, int64_t M) {
    if (M > tf::kSkinnyMaxM) return tf::gemm_workspace_bytes(L, M);
    const int64_t gemv = tf::gemv_workspace_bytes(L, M);
    const int64_t skinny = M >= tf::kSkinnyMinM ? tf::skinny_workspace_bytes(L, M) : 0;
    return gemv > skinny ? gemv : skinny;
}

int check_matmul(int bits, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
                 int64_t K, int64_t N, int group) {
    if (!A || !packed || !C) return TF_ERR_NULL;
    int rc = check_weight(bits, K, N, group);
    if (rc) return rc;
    if (M < 1 || M > TF_MAX_M) return TF_ERR_SHAPE;
    if (misaligned(A) || misaligned(packed) || misaligned(C)) return TF_ERR_ALIGN;
    return TF_OK;
}

// Workspace rules shared by the matmul entry points: NULL selects the
// single-pass kernels; otherwise it must be large enough and aligned.
int check_workspace(const Layout& L, int64_t M, const void* ws, size_t ws_bytes) {
    if (!ws) return TF_OK;
    if ((int64_t)ws_bytes < workspace_bytes(L, M)) return TF_ERR_ARG;
    if (misaligned(ws)) return TF_ERR_ALIGN;
    return TF_OK;
}

int gemm_entry(int bits, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
               int64_t K, int64_t N, int group, void* ws, size_t ws_bytes, void* stream, bool bf) {
    int rc = check_matmul(bits, A, packed, C, M, K, N, group);
    if (rc) return rc;
    Layout L = tf::make_layout(bits, K, N, group);
    rc = check_workspace(L, M, ws, ws_bytes);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (M < tf::kSkinnyMinM) return tf::launch_gemv(L, A, packed, C, M, ws, s, bf);
    if (M <= tf::kSkinnyMaxM) return tf::launch_skinny_gemm(L, A, packed, C, M, ws, s, bf);
    return tf::launch_gemm(L, A, packed, C, M, ws, ws_bytes, s, bf);
}

int gemv_entry(int bits, const uint16_t* A, const void* packed, uint16_t* C, int64_t M,
               int64_t K, int64_t N, int group, void* ws, size_t ws_bytes, void* stream, bool bf) {
    int rc = check_matmul(bits, A, packed, C, M, K, N, group);
    if (rc) return rc;
    if (M > TF_GEMV_MAX_M) return TF_ERR_ARG;
    Layout L = tf::make_layout(bits, K, N, group);
    rc = check_workspace(L, M, ws, ws_bytes);
    if (rc) return rc;
    return tf::launch_gemv(L, A, packed, C, M, ws, static_cast<hipStream_t>(stream), bf);
}

// ---- Scratch of the allocation-free decode GEMV (tf_w4a16_gemv_noalloc):
// one array of kScratchBytes per device in the library's static device
// memory, held until the process ends.  Host code never passes the array's
// name to a kernel (in host code it is a host-side stand-in): it asks the
// runtime once per device for the array's device address and uses that.
constexpr int64_t kScratchBytes = int64_t(1) << 20;
constexpr int kScratchDevices = 64;

__global__ void clear_words_kernel(uint32_t* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

struct ScratchSlot {
    void* ptr;        // device address of `scratch` on this device, once known
    bool cleared;     // counters cleared by a launch outside stream capture
};
std::mutex g_scratch_mu;
ScratchSlot g_scratch[kScratchDevices];

int silu_mul_entry(const uint16_t* GU, int64_t M, int64_t N, uint16_t* H, void* stream, bool bf) {
    if (!GU || !H) return TF_ERR_NULL;
    if (M < 1 || M > TF_MAX_M || N <= 0 || N > TF_MAX_DIM || N % 8 != 0) return TF_ERR_SHAPE;
    if (misaligned(GU) || misaligned(H)) return TF_ERR_ALIGN;
    return tf::launch_silu_mul(GU, M, N, H, static_cast<hipStream_t>(stream), bf);
}

}  // namespace

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

// The scratch of the device `s` belongs to.  The first call on a device looks
// up its address (with that device current) and enqueues a clear of the
// arrival counters on `s`; every GEMV leaves the counters it used at zero, so
// later calls need no clear.  A clear recorded into a graph under capture
// does not count as done (the graph may never be launched): the next call
// outside capture clears again.
int scratch_for(hipStream_t s, void** out) {
    int dev = -1;
    if (hipStreamGetDevice(s, &dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return TF_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchSlot& slot = g_scratch[dev];
    if (slot.ptr == nullptr) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return TF_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return TF_ERR_HIP;
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev && hipSetDevice(cur) != hipSuccess) return TF_ERR_HIP;
        if (e != hipSuccess || p == nullptr) return TF_ERR_HIP;
        slot.ptr = p;
    }
    if (!slot.cleared) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(s, &cs) != hipSuccess) return TF_ERR_HIP;
        constexpr int kWords = (int)(tf::kWsCounterBytes / 4);
        const int rc = tf::launch(clear_words_kernel, dim3((kWords + 255) / 256), dim3(256), 0, s,
                                  static_cast<uint32_t*>(slot.ptr), kWords);
        if (rc) return rc;
        if (cs == hipStreamCaptureStatusNone) slot.cleared = true;
    }
    *out = slot.ptr;
    return TF_OK;
}

}  // namespace

extern "C" {

int tf_layout_version(void) { return tf::kLayoutVersion; }

const char* tf_status_str(int status) {
    switch (status) {
        case TF_OK: return "ok";
        case TF_ERR_NULL: return "null pointer argument";
        case TF_ERR_SHAPE: return "bad shape (M, K, N, K % group, N % 8 or size limit)";
        case TF_ERR_GROUP: return "group size must be a positive multiple of 32";
        case TF_ERR_ALIGN: return "pointer not 16-byte aligned";
        case TF_ERR_ARG: return "bad argument (bits, M for GEMV, dtype or workspace size)";
        case TF_ERR_HIP: return "HIP runtime error at launch";
        default: return "unknown status";
    }
}

int64_t tf_packed_bytes(int bits, int64_t K, int64_t N, int group) {
    int rc = check_weight(bits, K, N, group);
    if (rc) return rc;
    return tf::make_layout(bits, K, N, group).total;
}

int tf_pack_w4(const int32_t* qweight, const int32_t* qzeros, const uint16_t* scales, int64_t K,
               int64_t N, int group, void* packed, void* stream) {
    if (!qweight || !qzeros || !scales || !packed) return TF_ERR_NULL;
    int rc = check_weight(4, K, N, group);
    if (rc) return rc;
    if (misaligned(qweight) || misaligned(qzeros) || misaligned(scales) || misaligned(packed))
        return TF_ERR_ALIGN;
    return tf::launch_pack_w4(qweight, qzeros, scales, tf::make_layout(4, K, N, group), packed,
                              static_cast<hipStream_t>(stream));
}

int tf_pack_w8(const uint8_t* qweight, const uint8_t* zeros, const uint16_t* scales, int64_t K,
               int64_t N, int group, void* packed, void* stream) {
    if (!qweight || !zeros || !scales || !packed) return TF_ERR_NULL;
    int rc = check_weight(8, K, N, group);
    if (rc) return rc;
    if (misaligned(qweight) || misaligned(zeros) || misaligned(scales) || misaligned(packed))
        return TF_ERR_ALIGN;
    return tf::launch_pack_w8(qweight, zeros, scales, tf::make_layout(8, K, N, group), packed,
                              static_cast<hipStream_t>(stream));
}

int tf_pack_w8_sym(const int8_t* qweight, const uint16_t* scales, int64_t K, int64_t N, int group,
                   void* packed, void* stream) {
    if (!qweight || !scales || !packed) return TF_ERR_NULL;
    int rc = check_weight(8, K, N, group);
    if (rc) return rc;
    if (misaligned(qweight) || misaligned(scales) || misaligned(packed)) return TF_ERR_ALIGN;
    return tf::launch_pack_w8_sym(qweight, scales, tf::make_layout(8, K, N, group), packed,
                                  static_cast<hipStream_t>(stream));
}

int64_t tf_workspace_bytes(int bits, int64_t M, int64_t K, int64_t N, int group) {
    int rc = check_weight(bits, K, N, group);
    if (rc) return rc;
    if (M < 1 || M > TF_MAX_M) return TF_ERR_SHAPE;
    return workspace_bytes(tf::make_layout(bits, K, N, group), M);
}

int64_t tf_gemm_workspace_bytes(int bits, int64_t M, int64_t K, int64_t N, int group) {
    return tf_workspace_bytes(bits, M, K, N, group);
}

int tf_w4a16_gemm(const uint16_t* A_f16, const void* packed, uint16_t* C_f16, int64_t M,
                  int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                  void* stream) {
    return gemm_entry(4, A_f16, packed, C_f16, M, K, N, group, workspace, workspace_bytes, stream,
                      false);
}

int tf_w4a16_gemm_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16, int64_t M,
                       int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return gemm_entry(4, A_bf16, packed, C_bf16, M, K, N, group, workspace, workspace_bytes, stream,
                      true);
}

int tf_w8a16_gemm(const uint16_t* A_f16, const void* packed, uint16_t* C_f16, int64_t M,
                  int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                  void* stream) {
    return gemm_entry(8, A_f16, packed, C_f16, M, K, N, group, workspace, workspace_bytes, stream,
                      false);
}

int tf_w8a16_gemm_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16, int64_t M,
                       int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return gemm_entry(8, A_bf16, packed, C_bf16, M, K, N, group, workspace, workspace_bytes, stream,
                      true);
}

int tf_w4a16_gemv(const uint16_t* A_f16, const void* packed, uint16_t* C_f16, int64_t M,
                  int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                  void* stream) {
    return gemv_entry(4, A_f16, packed, C_f16, M, K, N, group, workspace, workspace_bytes, stream,
                      false);
}

int tf_w4a16_gemv_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16, int64_t M,
                       int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return gemv_entry(4, A_bf16, packed, C_bf16, M, K, N, group, workspace, workspace_bytes, stream,
                      true);
}

int tf_w4a16_gemv_noalloc(const uint16_t* A_f16, const void* packed, uint16_t* C_f16, int64_t M,
                          int64_t K, int64_t N, int group, void* stream) {
    int rc = check_matmul(4, A_f16, packed, C_f16, M, K, N, group);
    if (rc) return rc;
    if (M > TF_GEMV_MAX_M) return TF_ERR_ARG;
    const Layout L = tf::make_layout(4, K, N, group);
    if (tf::gemv_workspace_bytes(L, M) > kScratchBytes) return TF_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* ws = nullptr;
    rc = scratch_for(s, &ws);
    if (rc) return rc;
    return tf::launch_gemv(L, A_f16, packed, C_f16, M, ws, s, false);
}

int tf_w8a16_gemv(const uint16_t* A_f16, const void* packed, uint16_t* C_f16, int64_t M,
                  int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                  void* stream) {
    return gemv_entry(8, A_f16, packed, C_f16, M, K, N, group, workspace, workspace_bytes, stream,
                      false);
}

int tf_w8a16_gemv_bf16(const uint16_t* A_bf16, const void* packed, uint16_t* C_bf16, int64_t M,
                       int64_t K, int64_t N, int group, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return gemv_entry(8, A_bf16, packed, C_bf16, M, K, N, group, workspace, workspace_bytes, stream,
                      true);
}

int tf_unpack(int bits, const void* packed, int64_t K, int64_t N, int group, uint8_t* q_out,
              uint8_t* z_out, void* stream) {
    if (!packed || !q_out || !z_out) return TF_ERR_NULL;
    int rc = check_weight(bits, K, N, group);
    if (rc) return rc;
    if (misaligned(packed)) return TF_ERR_ALIGN;
    return tf::launch_unpack(tf::make_layout(bits, K, N, group), packed, q_out, z_out,
                             static_cast<hipStream_t>(stream));
}

int tf_dequant(int bits, const void* packed, int64_t K, int64_t N, int group, int out_dtype,
               void* W_out, void* stream) {
    if (!packed || !W_out) return TF_ERR_NULL;
    int rc = check_weight(bits, K, N, group);
    if (rc) return rc;
    if (out_dtype != TF_F16 && out_dtype != TF_F32 && out_dtype != TF_BF16) return TF_ERR_ARG;
    if (misaligned(packed) || misaligned(W_out)) return TF_ERR_ALIGN;
    return tf::launch_dequant(tf::make_layout(bits, K, N, group), packed, out_dtype, W_out,
                              static_cast<hipStream_t>(stream));
}

int tf_silu_mul(const uint16_t* GU_f16, int64_t M, int64_t N, uint16_t* H_f16, void* stream) {
    return silu_mul_entry(GU_f16, M, N, H_f16, stream, false);
}

int tf_silu_mul_bf16(const uint16_t* GU_bf16, int64_t M, int64_t N, uint16_t* H_bf16, void* stream) {
    return silu_mul_entry(GU_bf16, M, N, H_bf16, stream, true);
}

}  // extern "C"
