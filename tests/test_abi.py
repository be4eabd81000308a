"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes the packed layout, and rejects bad arguments before it
makes any HIP call (so these calls are safe without a device)."""
from __future__ import annotations

import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_11357_amd import tilefuse as tfb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tilefuse.h")

# fake device addresses: never dereferenced, because validation fails first
P = ctypes.c_void_p(0x10000)          # 16-byte aligned
P_ODD = ctypes.c_void_p(0x10008)      # 8-byte aligned only
NULL = None


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tf_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return tfb.load()


def test_header_declares_expected_entry_points():
    assert header_functions() == sorted(tfb.EXPORTS)


def test_library_exports_every_header_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", tfb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (tf_[a-z0-9_]+)$", out, flags=re.M))
    for name in header_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_version_and_status_strings(lib):
    assert lib.tf_layout_version() == 1
    for code in (tfb.TF_OK, tfb.TF_ERR_NULL, tfb.TF_ERR_SHAPE, tfb.TF_ERR_GROUP,
                 tfb.TF_ERR_ALIGN, tfb.TF_ERR_ARG, tfb.TF_ERR_HIP):
        s = tfb.status_str(code)
        assert s and s != "unknown status"
    assert tfb.status_str(12345) == "unknown status"


def _layout_bytes(bits, K, N, G):
    """Independent sizing of the packed layout: weights + fp16 scales + u8 zeros,
    per panel of 64 (4-bit) or 32 (8-bit) columns, regions 256-byte aligned."""
    pw = 64 if bits == 4 else 32
    npan = -(-N // pw)
    a256 = lambda v: -(-v // 256) * 256
    return a256(npan * K * pw * bits // 8) + a256(npan * (K // G) * pw * 2) + a256(npan * (K // G) * pw)


@pytest.mark.parametrize("bits,K,N,G", [(4, 4096, 14336, 128), (8, 4096, 4096, 128),
                                        (4, 2048, 2048, 128), (4, 32768, 8192, 128),
                                        (4, 256, 136, 64), (8, 96, 40, 32)])
def test_packed_bytes(lib, bits, K, N, G):
    assert lib.tf_packed_bytes(bits, K, N, G) == _layout_bytes(bits, K, N, G)


def test_packed_bytes_headline_numbers(lib):
    # K=4096, N=14336: 29,360,128 B of codes (same as the AWQ qweight), fp16
    # scales 917,504 B (same), zero-points one byte each: 458,752 B
    assert lib.tf_packed_bytes(4, 4096, 14336, 128) == 29360128 + 917504 + 458752


@pytest.mark.parametrize("args,want", [
    ((3, 256, 64, 128), tfb.TF_ERR_ARG),
    ((4, 256, 64, 0), tfb.TF_ERR_GROUP),
    ((4, 256, 64, 48), tfb.TF_ERR_GROUP),
    ((4, 256, 64, -128), tfb.TF_ERR_GROUP),
    ((4, 0, 64, 128), tfb.TF_ERR_SHAPE),
    ((4, 256, 0, 128), tfb.TF_ERR_SHAPE),
    ((4, 384, 64, 256), tfb.TF_ERR_SHAPE),      # K % G != 0
    ((4, 256, 60, 128), tfb.TF_ERR_SHAPE),      # N % 8 != 0
    ((8, 256, 12, 128), tfb.TF_ERR_SHAPE),
    ((4, 65536 + 128, 64, 128), tfb.TF_ERR_SHAPE),
])
def test_packed_bytes_rejects(lib, args, want):
    assert lib.tf_packed_bytes(*args) == want


MATMUL_OK = dict(A=P, packed=P, C=P, M=4, K=256, N=64, G=128)


def _gemv(lib, bits, dt="", **kw):
    a = {**MATMUL_OK, **kw}
    fn = getattr(lib, f"tf_w{bits}a16_gemv{dt}")
    return fn(a["A"], a["packed"], a["C"], a["M"], a["K"], a["N"], a["G"], NULL, 0, NULL)


def _gemm(lib, bits, ws=NULL, ws_bytes=0, dt="", **kw):
    a = {**MATMUL_OK, **kw}
    fn = getattr(lib, f"tf_w{bits}a16_gemm{dt}")
    return fn(a["A"], a["packed"], a["C"], a["M"], a["K"], a["N"], a["G"], ws, ws_bytes, NULL)


BAD_MATMUL = [
    (dict(A=NULL), tfb.TF_ERR_NULL),
    (dict(packed=NULL), tfb.TF_ERR_NULL),
    (dict(C=NULL), tfb.TF_ERR_NULL),
    (dict(M=0), tfb.TF_ERR_SHAPE),
    (dict(M=-1), tfb.TF_ERR_SHAPE),
    (dict(K=0), tfb.TF_ERR_SHAPE),
    (dict(N=-64), tfb.TF_ERR_SHAPE),
    (dict(K=320), tfb.TF_ERR_SHAPE),           # K % 128 != 0
    (dict(N=68), tfb.TF_ERR_SHAPE),            # N % 8 != 0
    (dict(G=100), tfb.TF_ERR_GROUP),
    (dict(A=P_ODD), tfb.TF_ERR_ALIGN),
    (dict(packed=P_ODD), tfb.TF_ERR_ALIGN),
    (dict(C=P_ODD), tfb.TF_ERR_ALIGN),
]


@pytest.mark.parametrize("dt", ["", "_bf16"])
@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("kw,want", BAD_MATMUL, ids=[str(b[0]) for b in BAD_MATMUL])
def test_matmul_rejects(lib, bits, kw, want, dt):
    assert _gemv(lib, bits, dt=dt, **kw) == want
    assert _gemm(lib, bits, dt=dt, **kw) == want


@pytest.mark.parametrize("dt", ["", "_bf16"])
@pytest.mark.parametrize("bits", [4, 8])
def test_gemv_rejects_large_m(lib, bits, dt):
    assert _gemv(lib, bits, dt=dt, M=9) == tfb.TF_ERR_ARG
    assert _gemv(lib, bits, dt=dt, M=4096) == tfb.TF_ERR_ARG


def test_workspace_query(lib):
    for bits, M, K, N in [(4, 2048, 4096, 14336), (8, 512, 4096, 4096), (4, 16, 2048, 2048),
                          (4, 1, 4096, 14336), (8, 8, 4096, 4096)]:
        n = lib.tf_workspace_bytes(bits, M, K, N, 128)
        assert n >= 0 and n % 256 == 0
    # many panels: one workgroup per panel fills the chip, no K split
    assert lib.tf_workspace_bytes(4, 1, 4096, 14336, 128) == 0
    # few panels and long K (down-projection): K is split, partial sums + counters
    assert lib.tf_workspace_bytes(4, 1, 14336, 4096, 128) > 64 * 64 * 4
    assert lib.tf_workspace_bytes(4, 0, 256, 64, 128) == tfb.TF_ERR_SHAPE
    assert lib.tf_workspace_bytes(4, 16, 256, 64, 100) == tfb.TF_ERR_GROUP


KIB = 1024
COUNTERS = 8 * KIB          # arrival counters at offset 0: one u32 per 32 columns of TF_MAX_DIM


@pytest.mark.parametrize("bits,M,K,N,want", [
    # 256-row GEMM whose 256 x 256 tiles do not fill whole waves of 256
    # blocks: two parked fp32 partial tiles per block
    (4, 2048, 4096, 14336, COUNTERS + 2 * 256 * 256 * 256 * 4),
    (4, 2048, 14336, 4096, COUNTERS + 2 * 256 * 256 * 256 * 4),
    (4, 1024, 4096, 14336, COUNTERS + 2 * 256 * 256 * 256 * 4),
    (4, 2048, 4096, 16384, 0),                       # 512 tiles: whole waves, no split
    # 128-row GEMM split-K (long K on few tiles): one 128 x 256 fp32 partial
    # per (tile, slice), 16 tiles x 8 slices
    (4, 128, 14336, 4096, COUNTERS + 16 * 8 * 128 * 256 * 4),
    # 64 x 128 GEMM with K split over each workgroup's waves: the K quarters
    # are summed in LDS, no workspace
    (8, 512, 4096, 4096, 0),
    (8, 256, 4096, 4096, 0),
    (4, 128, 4096, 14336, 0),
    # decode GEMV on 64 panels of 64 columns, K split in 4 slices: one fp32
    # partial per (panel, slice, row)
    (4, 1, 14336, 4096, COUNTERS + 64 * 4 * 1 * 64 * 4),
    (4, 3, 14336, 4096, COUNTERS + 64 * 4 * 3 * 64 * 4),
    # GEMM entry with 40 rows: the streaming matrix-core form, 64 row slots
    (4, 40, 14336, 4096, COUNTERS + 64 * 4 * 64 * 64 * 4),
    (4, 1, 4096, 14336, 0),                          # 224 panels fill the chip: no split
])
def test_workspace_sizes(lib, bits, M, K, N, want):
    """The workspace each documented plan asks for: the counter region, then
    the fp32 partials its K split parks."""
    assert lib.tf_workspace_bytes(bits, M, K, N, 128) == want


@pytest.mark.parametrize("bits", [4, 8])
def test_workspace_rejects(lib, bits):
    need = lib.tf_workspace_bytes(bits, 1, 14336, 2048, 128)
    assert need > 0
    fn = lib.tf_w4a16_gemv if bits == 4 else lib.tf_w8a16_gemv
    assert fn(P, P, P, 1, 14336, 2048, 128, P, need - 16, NULL) == tfb.TF_ERR_ARG
    assert fn(P, P, P, 1, 14336, 2048, 128, P_ODD, need, NULL) == tfb.TF_ERR_ALIGN
    fn = lib.tf_w4a16_gemm if bits == 4 else lib.tf_w8a16_gemm
    assert fn(P, P, P, 1, 14336, 2048, 128, P, need - 16, NULL) == tfb.TF_ERR_ARG


def test_pack_rejects(lib):
    ok = (P, P, P, 256, 64, 128, P, NULL)
    for fn in (lib.tf_pack_w4, lib.tf_pack_w8):
        for i in (0, 1, 2, 6):
            a = list(ok)
            a[i] = NULL
            assert fn(*a) == tfb.TF_ERR_NULL
            a[i] = P_ODD
            assert fn(*a) == tfb.TF_ERR_ALIGN
        assert fn(P, P, P, 256, 60, 128, P, NULL) == tfb.TF_ERR_SHAPE
        assert fn(P, P, P, 200, 64, 128, P, NULL) == tfb.TF_ERR_SHAPE
        assert fn(P, P, P, 256, 64, 16, P, NULL) == tfb.TF_ERR_GROUP


def test_pack_w8_sym_rejects(lib):
    ok = (P, P, 256, 64, 128, P, NULL)
    for i in (0, 1, 5):
        a = list(ok)
        a[i] = NULL
        assert lib.tf_pack_w8_sym(*a) == tfb.TF_ERR_NULL
        a[i] = P_ODD
        assert lib.tf_pack_w8_sym(*a) == tfb.TF_ERR_ALIGN
    assert lib.tf_pack_w8_sym(P, P, 256, 60, 128, P, NULL) == tfb.TF_ERR_SHAPE
    assert lib.tf_pack_w8_sym(P, P, 200, 64, 128, P, NULL) == tfb.TF_ERR_SHAPE
    assert lib.tf_pack_w8_sym(P, P, 256, 64, 16, P, NULL) == tfb.TF_ERR_GROUP


def test_unpack_dequant_reject(lib):
    assert lib.tf_unpack(4, NULL, 256, 64, 128, P, P, NULL) == tfb.TF_ERR_NULL
    assert lib.tf_unpack(4, P, 256, 64, 128, NULL, P, NULL) == tfb.TF_ERR_NULL
    assert lib.tf_unpack(5, P, 256, 64, 128, P, P, NULL) == tfb.TF_ERR_ARG
    assert lib.tf_unpack(4, P_ODD, 256, 64, 128, P, P, NULL) == tfb.TF_ERR_ALIGN
    assert lib.tf_dequant(4, P, 256, 64, 128, 7, P, NULL) == tfb.TF_ERR_ARG
    assert lib.tf_dequant(8, P, 256, 64, 128, tfb.TF_F16, NULL, NULL) == tfb.TF_ERR_NULL
    assert lib.tf_dequant(8, P, 256, 64, 128, tfb.TF_F32, P_ODD, NULL) == tfb.TF_ERR_ALIGN
    assert lib.tf_dequant(4, P, 250, 64, 128, tfb.TF_F32, P, NULL) == tfb.TF_ERR_SHAPE
    assert lib.tf_dequant(4, P, 256, 64, 128, tfb.TF_BF16, P_ODD, NULL) == tfb.TF_ERR_ALIGN
    assert lib.tf_dequant(4, P, 256, 64, 128, 4, P, NULL) == tfb.TF_ERR_ARG


def test_binding_refuses_cpu_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(4, 256, dtype=torch.float16)
    with pytest.raises(ValueError):
        tfb.w4a16_gemv(x, torch.zeros(16, dtype=torch.uint8), 256, 64)


@pytest.mark.parametrize("args,want", [
    ((NULL, 4, 64, P, NULL), tfb.TF_ERR_NULL), ((P, 4, 64, NULL, NULL), tfb.TF_ERR_NULL),
    ((P, 0, 64, P, NULL), tfb.TF_ERR_SHAPE), ((P, 4, 60, P, NULL), tfb.TF_ERR_SHAPE),
    ((P, 4, 0, P, NULL), tfb.TF_ERR_SHAPE), ((P_ODD, 4, 64, P, NULL), tfb.TF_ERR_ALIGN),
    ((P, 4, 64, P_ODD, NULL), tfb.TF_ERR_ALIGN)])
def test_silu_mul_rejects(lib, args, want):
    assert lib.tf_silu_mul(*args) == want
    assert lib.tf_silu_mul_bf16(*args) == want


@pytest.mark.parametrize("args", [(4, 2048, 4096, 14336, 128), (8, 512, 4096, 4096, 128), (4, 1, 14336, 4096, 128),
                                  (4, 40, 14336, 4096, 128), (8, 3, 4096, 4096, 64), (4, 0, 256, 64, 128),
                                  (4, 16, 256, 64, 100), (5, 16, 256, 64, 128)])
def test_gemm_workspace_query_is_the_workspace_query(lib, args):
    """tf_gemm_workspace_bytes answers exactly what tf_workspace_bytes does,
    sizes and errors alike."""
    assert lib.tf_gemm_workspace_bytes(*args) == lib.tf_workspace_bytes(*args)


@pytest.mark.parametrize("kw,want", BAD_MATMUL + [(dict(M=9), tfb.TF_ERR_ARG)],
                         ids=[str(b[0]) for b in BAD_MATMUL] + ["M=9"])
def test_gemv_noalloc_rejects(lib, kw, want):
    """The allocation-free GEMV makes the same checks, before any HIP call."""
    a = {**MATMUL_OK, **kw}
    assert lib.tf_w4a16_gemv_noalloc(a["A"], a["packed"], a["C"], a["M"], a["K"], a["N"], a["G"], NULL) == want
