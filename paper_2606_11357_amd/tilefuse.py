"""Python binding of libtilefuse (ctypes; argument marshalling only).

Every computation runs in the library's HIP kernels; torch supplies device
memory and the current stream.  The names mirror the C ABI in
``include/tilefuse.h``.  There is no fallback: if the shared library is not
built, importing the binding fails with an error that says how to build it.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# TILEFUSE_LIB names another build of the same library to load instead (the
# host-sanitizer build the CPU tests run the argument checks under).
LIB_PATH = os.environ.get("TILEFUSE_LIB") or os.path.join(PKG, "libtilefuse.so")

TF_OK = 0
TF_ERR_NULL = -1
TF_ERR_SHAPE = -2
TF_ERR_GROUP = -3
TF_ERR_ALIGN = -4
TF_ERR_ARG = -5
TF_ERR_HIP = -6
TF_F16 = 1
TF_F32 = 2
TF_BF16 = 3
GEMV_MAX_M = 8

EXPORTS = (
    "tf_layout_version", "tf_status_str", "tf_packed_bytes", "tf_pack_w4", "tf_pack_w8",
    "tf_pack_w8_sym", "tf_workspace_bytes", "tf_gemm_workspace_bytes", "tf_w4a16_gemm",
    "tf_w8a16_gemm", "tf_w4a16_gemv", "tf_w8a16_gemv", "tf_w4a16_gemv_noalloc", "tf_w4a16_gemm_bf16", "tf_w8a16_gemm_bf16", "tf_w4a16_gemv_bf16",
    "tf_w8a16_gemv_bf16", "tf_unpack", "tf_dequant", "tf_silu_mul", "tf_silu_mul_bf16",
)


class TileFuseError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


_lib = None


def load() -> ctypes.CDLL:
    """Load libtilefuse.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with "
                          "`python -m paper_2606_11357_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
    sig = {
        "tf_layout_version": (I, []),
        "tf_status_str": (ctypes.c_char_p, [I]),
        "tf_packed_bytes": (I64, [I, I64, I64, I]),
        "tf_pack_w4": (I, [P, P, P, I64, I64, I, P, P]),
        "tf_pack_w8": (I, [P, P, P, I64, I64, I, P, P]),
        "tf_pack_w8_sym": (I, [P, P, I64, I64, I, P, P]),
        "tf_workspace_bytes": (I64, [I, I64, I64, I64, I]),
        "tf_gemm_workspace_bytes": (I64, [I, I64, I64, I64, I]),
        "tf_w4a16_gemm": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w8a16_gemm": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w4a16_gemv": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w8a16_gemv": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w4a16_gemv_noalloc": (I, [P, P, P, I64, I64, I64, I, P]),
        "tf_w4a16_gemm_bf16": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w8a16_gemm_bf16": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w4a16_gemv_bf16": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_w8a16_gemv_bf16": (I, [P, P, P, I64, I64, I64, I, P, SZ, P]),
        "tf_unpack": (I, [I, P, I64, I64, I, P, P, P]),
        "tf_dequant": (I, [I, P, I64, I64, I, I, P, P]),
        "tf_silu_mul": (I, [P, I64, I64, P, P]),
        "tf_silu_mul_bf16": (I, [P, I64, I64, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().tf_status_str(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != TF_OK:
        raise TileFuseError(status, where)


# ---------------------------------------------------------------------------
# torch-facing wrappers
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _need_cuda(*tensors):
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise ValueError("tensors must be on the GPU (the library has no CPU path)")
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def packed_bytes(bits: int, K: int, N: int, group: int = 128) -> int:
    n = load().tf_packed_bytes(bits, K, N, group)
    if n < 0:
        raise TileFuseError(int(n), "tf_packed_bytes")
    return int(n)


def workspace_bytes(bits: int, M: int, K: int, N: int, group: int = 128) -> int:
    n = load().tf_workspace_bytes(bits, M, K, N, group)
    if n < 0:
        raise TileFuseError(int(n), "tf_workspace_bytes")
    return int(n)


_default_ws = {}


def default_workspace(device, nbytes: int):
    """A zero-filled workspace of at least `nbytes`, cached per device.

    Every call returns the workspace's arrival counters to zero, so the cached
    buffer serves later calls of any shape without clearing; it must not be
    shared by calls running concurrently on different streams (pass your own
    workspace for that).
    """
    torch = _torch()
    key = torch.device(device).index if torch.device(device).index is not None else torch.cuda.current_device()
    buf = _default_ws.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.zeros(max(nbytes, 1 << 20), dtype=torch.uint8, device=device)
        _default_ws[key] = buf
    return buf


def pack_w4(qweight, qzeros, scales, K: int, N: int, group: int = 128, out=None):
    """Pre-tile an AWQ 4-bit weight (int32 [K, N/8], int32 [K/G, N/8], fp16 or bf16
    [K/G, N]; the scale bits are copied as they are)."""
    torch = _torch()
    _need_cuda(qweight, qzeros, scales)
    if out is None:
        out = torch.empty(packed_bytes(4, K, N, group), dtype=torch.uint8, device=qweight.device)
    _check(load().tf_pack_w4(_ptr(qweight), _ptr(qzeros), _ptr(scales), K, N, group, _ptr(out),
                             _stream(qweight.device)), "tf_pack_w4")
    return out


def pack_w8(qweight, zeros, scales, K: int, N: int, group: int = 128, out=None):
    """Pre-tile an 8-bit weight (uint8 [K, N], uint8 [K/G, N], fp16 or bf16 [K/G, N])."""
    torch = _torch()
    _need_cuda(qweight, zeros, scales)
    if out is None:
        out = torch.empty(packed_bytes(8, K, N, group), dtype=torch.uint8, device=qweight.device)
    _check(load().tf_pack_w8(_ptr(qweight), _ptr(zeros), _ptr(scales), K, N, group, _ptr(out),
                             _stream(qweight.device)), "tf_pack_w8")
    return out


def pack_w8_sym(qweight, scales, K: int, N: int, group: int = 128, out=None):
    """Pre-tile a signed INT8 weight with one scale per output channel
    (int8 [K, N], fp16 or bf16 [N]); use it with the 8-bit matmul calls and `group`."""
    torch = _torch()
    _need_cuda(qweight, scales)
    if out is None:
        out = torch.empty(packed_bytes(8, K, N, group), dtype=torch.uint8, device=qweight.device)
    _check(load().tf_pack_w8_sym(_ptr(qweight), _ptr(scales), K, N, group, _ptr(out),
                                 _stream(qweight.device)), "tf_pack_w8_sym")
    return out


def _matmul(bits, kind, A, packed, K, N, group, out, workspace):
    """A fp16 or bfloat16 [M, K] selects the entry point (the packed scales must
    hold the same dtype's bits); the output has A's dtype.
    workspace: None -> the cached per-device default, False -> none (single-pass
    kernels), or a caller tensor (zero-filled before its first use)."""
    torch = _torch()
    _need_cuda(A, packed, out)
    M = A.shape[0]
    if A.dtype not in (torch.float16, torch.bfloat16) or A.dim() != 2 or A.shape[1] != K:
        raise ValueError("A must be fp16 or bf16 [M, K]")
    if out is None:
        out = torch.empty((M, N), dtype=A.dtype, device=A.device)
    elif out.dtype != A.dtype or tuple(out.shape) != (M, N):
        raise ValueError("out must have A's dtype and shape [M, N]")
    if workspace is None:
        need = workspace_bytes(bits, M, K, N, group)
        workspace = default_workspace(A.device, need) if need else False
    if workspace is False:
        ws_ptr, ws_bytes = None, 0
    else:
        _need_cuda(workspace)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
    name = f"tf_w{bits}a16_{kind}" + ("_bf16" if A.dtype == torch.bfloat16 else "")
    rc = getattr(load(), name)(_ptr(A), _ptr(packed), _ptr(out), M, K, N, group, ws_ptr, ws_bytes,
                               _stream(A.device))
    _check(rc, name)
    return out


def w4a16_gemm(A, packed, K: int, N: int, group: int = 128, out=None, workspace=None):
    return _matmul(4, "gemm", A, packed, K, N, group, out, workspace)


def w8a16_gemm(A, packed, K: int, N: int, group: int = 128, out=None, workspace=None):
    return _matmul(8, "gemm", A, packed, K, N, group, out, workspace)


def w4a16_gemv(A, packed, K: int, N: int, group: int = 128, out=None, workspace=None):
    return _matmul(4, "gemv", A, packed, K, N, group, out, workspace)


def w8a16_gemv(A, packed, K: int, N: int, group: int = 128, out=None, workspace=None):
    return _matmul(8, "gemv", A, packed, K, N, group, out, workspace)


def w4a16_gemv_noalloc(A, packed, K: int, N: int, group: int = 128, out=None):
    """The decode GEMV through tf_w4a16_gemv_noalloc: no workspace argument, the
    library's static per-device scratch instead (A fp16 [M, K], 1 <= M <= 8)."""
    torch = _torch()
    _need_cuda(A, packed, out)
    M = A.shape[0]
    if A.dtype != torch.float16 or A.dim() != 2 or A.shape[1] != K:
        raise ValueError("A must be fp16 [M, K]")
    if out is None:
        out = torch.empty((M, N), dtype=A.dtype, device=A.device)
    elif out.dtype != A.dtype or tuple(out.shape) != (M, N):
        raise ValueError("out must have A's dtype and shape [M, N]")
    _check(load().tf_w4a16_gemv_noalloc(_ptr(A), _ptr(packed), _ptr(out), M, K, N, group, _stream(A.device)),
           "tf_w4a16_gemv_noalloc")
    return out


def unpack(bits: int, packed, K: int, N: int, group: int = 128):
    """Codes q [K, N] and zero-points z [K/G, N] read back from a packed buffer."""
    torch = _torch()
    _need_cuda(packed)
    q = torch.empty((K, N), dtype=torch.uint8, device=packed.device)
    z = torch.empty((K // group, N), dtype=torch.uint8, device=packed.device)
    _check(load().tf_unpack(bits, _ptr(packed), K, N, group, _ptr(q), _ptr(z),
                            _stream(packed.device)), "tf_unpack")
    return q, z


def dequant(bits: int, packed, K: int, N: int, group: int = 128, dtype=None):
    """Dequantized weights [K, N]: fp16 rounded once or exact fp32 (fp16 scales),
    or bfloat16 rounded once (bfloat16 scales)."""
    torch = _torch()
    dtype = dtype or torch.float16
    _need_cuda(packed)
    code = {torch.float16: TF_F16, torch.float32: TF_F32, torch.bfloat16: TF_BF16}[dtype]
    w = torch.empty((K, N), dtype=dtype, device=packed.device)
    _check(load().tf_dequant(bits, _ptr(packed), K, N, group, code, _ptr(w),
                             _stream(packed.device)), "tf_dequant")
    return w


def silu_mul(gu, out=None):
    """H = silu(gu[:, :N]) * gu[:, N:] for an fp16 or bfloat16 [M, 2N] CUDA
    tensor (the gate and up halves side by side); returns [M, N] of gu's dtype."""
    torch = _torch()
    _need_cuda(gu, out)
    if gu.dtype not in (torch.float16, torch.bfloat16) or gu.dim() != 2 or gu.shape[1] % 2 != 0:
        raise ValueError("gu must be fp16 or bf16 [M, 2N]")
    M, N = gu.shape[0], gu.shape[1] // 2
    if out is None:
        out = torch.empty((M, N), dtype=gu.dtype, device=gu.device)
    elif out.dtype != gu.dtype:
        raise ValueError("out must have gu's dtype")
    name = "tf_silu_mul_bf16" if gu.dtype == torch.bfloat16 else "tf_silu_mul"
    _check(getattr(load(), name)(_ptr(gu), M, N, _ptr(out), _stream(gu.device)), name)
    return out
