"""Static checks of the hand-scheduled GEMM kernels' machine code (CPU only).

Both MFMA GEMMs issue their matrix instructions as asm statements with
AGPR-pinned accumulators, so the compiler inserts none of the wait states the
ISA requires around them; the K-split GEMM also issues its buffer loads as
asm statements and waits for them with its own counted s_waitcnt, so the
compiler inserts none of those waits either.  These tests compile the two
kernel files to gfx950 assembly with the library's own flags and check every
instantiation:

  * K-split GEMM (64 x 128 and 64 x 256 tiles): no VGPR that a buffer load
    targets is read or overwritten before a wait that leaves that load
    complete (vector-memory loads complete in issue order), over the
    prologue, three passes of the step loop and the epilogue;
  * both GEMMs: at least two wait states between a vector-ALU write of an MFMA's
    A or B operand and the MFMA, and between an accumulator write
    (v_accvgpr_write) and an MFMA reading it; at least 18 between an MFMA
    writing an accumulator and any other instruction reading it (checked over
    the code in order and over two passes of every loop).

Each checker is also run on small planted violations.
"""
import os
import re
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2606_11357_amd import build as B  # noqa: E402

KERNELS = {"tf_gemm_ks.hip": "gemm_ks_kernel", "tf_gemm256.hip": "gemm256_kernel"}


def _compile_asm(src, out):
    cmd = [B.HIPCC, *B.FLAGS, *B.EXTRA.get(os.path.basename(src), []), "--cuda-device-only", "-S", src, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(r.stderr[-3000:])
    return out


@pytest.fixture(scope="module")
def asm():
    if not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    tmp = tempfile.mkdtemp(prefix="tf_asm_")
    srcs = {f: os.path.join(B.CSRC, f) for f in KERNELS}
    with ThreadPoolExecutor(len(srcs)) as ex:
        outs = dict(zip(srcs, ex.map(lambda f: _compile_asm(srcs[f], os.path.join(tmp, f + ".s")), srcs)))
    texts = {f: open(p).read() for f, p in outs.items()}
    shutil.rmtree(tmp, ignore_errors=True)
    return texts


# ---------------------------------------------------------------- parsing

def functions(text, needle):
    """(name, [(op, operand text, label-or-None)]) for each kernel whose name contains needle."""
    out = []
    for m in re.finditer(r"^(_Z\S+):[^\n]*\n(.*?)^\.Lfunc_end", text, re.S | re.M):
        if needle in m.group(1):
            out.append((m.group(1), parse(m.group(2))))
    return out


def parse(body):
    ins = []
    for line in body.splitlines():
        code = line.split(";")[0].strip()
        lab = re.match(r"^(\.LBB\w+):", line)
        if lab:
            ins.append(("#label", lab.group(1), "Loop Header" in line))
            continue
        if not code or code.startswith("."):
            continue
        op = code.split()[0]
        ins.append((op, code[len(op):].strip(), None))
    return ins


def regs(tok, kind="v"):
    out = set()
    for m in re.finditer(r"\b%s\[(\d+):(\d+)\]|\b%s(\d+)\b" % (kind, kind), tok):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def split_args(a):
    return [x.strip() for x in a.split(",")] if a else []


def loops(ins):
    """(start, end) index ranges of every loop: header label .. its back-edge branch."""
    out = []
    for k, (op, a, hdr) in enumerate(ins):
        if op == "#label" and hdr:
            for e in range(k + 1, len(ins)):
                if ins[e][0].startswith("s_cbranch") and ins[e][1] == a:
                    out.append((k, e))
                    break
    return out


def code(seq):
    return [(op, a) for op, a, _ in seq if op != "#label"]


# ---------------------------------------------------------------- checkers

def check_vm_waits(seq):
    """Violations of the counted waits: a use or overwrite of a VGPR whose
    buffer load or LDS read may still be in flight (each kind completes in
    issue order; an LDS read counts as pending until an lgkmcnt wait leaves
    fewer LDS reads in flight, whatever scalar loads share that counter)."""
    queue, lgkm, bad = [], [], []
    for op, a in seq:
        args = split_args(a)
        if op == "s_waitcnt":
            m = re.search(r"vmcnt\((\d+)\)", a)
            if m:
                n = int(m.group(1))
                queue = queue[max(0, len(queue) - n):]
            m = re.search(r"lgkmcnt\((\d+)\)", a)
            if m:
                n = int(m.group(1))
                lgkm = lgkm[max(0, len(lgkm) - n):]
            continue
        if op.startswith("ds_read"):
            dst = regs(args[0])
            if any(q & (dst | regs(args[1])) for q in queue + lgkm):
                bad.append((op, a))
            lgkm.append(dst)
            continue
        if op.startswith("buffer_load"):
            # a direct-to-LDS load counts in the same queue but targets no VGPR
            # (its first operand is then the offset it reads)
            to_lds = a.endswith(" lds")
            dst = set() if to_lds else regs(args[0])
            srcs = set().union(*[regs(x) for x in (args if to_lds else args[1:])])
            if any(q & (dst | srcs) for q in queue):
                bad.append((op, a))
            queue.append(dst)
            continue
        if op.startswith("v_mfma"):
            srcs, dsts = regs(args[1]) | regs(args[2]), set()
        elif op.startswith("v_") or op.startswith("ds_") or op.startswith("global_") or op.startswith("buffer_"):
            srcs = set().union(*[regs(x) for x in args[1:]]) if len(args) > 1 else set()
            dsts = regs(args[0]) if op.startswith("v_") else set()
            if not op.startswith("v_"):
                srcs |= regs(args[0]) if args else set()
        else:
            srcs = set().union(*[regs(x) for x in args]) if args else set()
            dsts = set()
        if any(q & (srcs | dsts) for q in queue + lgkm):
            bad.append((op, a))
    return bad


def wait_states(op, a):
    return int(a, 0) + 1 if op == "s_nop" else 1


def check_mfma_hazards(seq):
    """Violations of the MFMA wait states (see the module docstring)."""
    valu_w, acc_w, mfma_w, clock, bad = {}, {}, {}, 0, []
    for op, a in seq:
        args = split_args(a)
        if op.startswith("v_mfma"):
            if any(r in valu_w and clock - valu_w[r] < 2 for r in regs(args[1]) | regs(args[2])):
                bad.append(("VALU write -> MFMA A/B", op, a))
            if any(r in acc_w and clock - acc_w[r] < 2 for r in regs(args[3], "a")):
                bad.append(("accumulator write -> MFMA C", op, a))
            for r in regs(args[0], "a"):
                mfma_w[r] = clock
        else:
            reads = args[1:] if op.startswith("v_") else args
            if any(r in mfma_w and clock - mfma_w[r] < 18
                   for r in (set().union(*[regs(x, "a") for x in reads]) if reads else set())):
                bad.append(("MFMA -> accumulator read", op, a))
            if op == "v_accvgpr_write_b32":
                for r in regs(args[0], "a"):
                    acc_w[r] = clock
            elif op.startswith("v_") and args:
                for r in regs(args[0]):
                    valu_w[r] = clock
        clock += wait_states(op, a)
    return bad


# ---------------------------------------------------------------- tests

def test_ks_counted_waits(asm):
    fns = functions(asm["tf_gemm_ks.hip"], KERNELS["tf_gemm_ks.hip"])
    # 1/2/4 groups per chunk x fp16/bf16 x (4-bit: 64 x 128 and 64 x 256 tiles, 8-bit: 64 x 128)
    assert len(fns) == 18
    for name, ins in fns:
        lp = loops(ins)
        assert len(lp) == 1, name               # one step loop, no waterfall loops
        s, e = lp[0]
        seq = code(ins[:s]) + 3 * code(ins[s:e + 1]) + code(ins[e + 1:])
        assert sum(op.startswith("buffer_load") for op, _ in seq) > 0
        assert check_vm_waits(seq) == [], name


INSTANTIATIONS = {"tf_gemm_ks.hip": 18, "tf_gemm256.hip": 12}


@pytest.mark.parametrize("f", sorted(KERNELS))
def test_mfma_wait_states(asm, f):
    fns = functions(asm[f], KERNELS[f])
    assert len(fns) == INSTANTIATIONS[f]
    for name, ins in fns:
        assert sum(op.startswith("v_mfma") for op, _, _ in ins) >= 64, name
        assert check_mfma_hazards(code(ins)) == [], name
        for s, e in loops(ins):
            assert check_mfma_hazards(2 * code(ins[s:e + 1])) == [], name


def test_checkers_catch_planted_violations():
    ok = [("buffer_load_dwordx4", "v[4:7], v1, s[8:11], s12 offen"), ("s_waitcnt", "vmcnt(0)"),
          ("v_mov_b32", "v2, v4")]
    assert check_vm_waits(ok) == []
    early = [("buffer_load_dwordx4", "v[4:7], v1, s[8:11], s12 offen"),
             ("buffer_load_dwordx4", "v[8:11], v1, s[8:11], s13 offen"), ("s_waitcnt", "vmcnt(1)"),
             ("v_mov_b32", "v2, v8")]                 # waits for the first load only
    assert len(check_vm_waits(early)) == 1
    overwrite = [("buffer_load_dwordx4", "v[4:7], v1, s[8:11], s12 offen"), ("v_mov_b32", "v5, 0")]
    assert len(check_vm_waits(overwrite)) == 1
    behind_lds = [("buffer_load_dwordx4", "v[4:7], v1, s[8:11], s12 offen"),
                  ("buffer_load_dwordx4", "v2, s[8:11], s13 offen lds"), ("s_waitcnt", "vmcnt(1)"),
                  ("v_mov_b32", "v3, v4")]            # the direct load keeps one slot: v4 is complete
    assert check_vm_waits(behind_lds) == []
    assert len(check_vm_waits(behind_lds[:2] + [("s_waitcnt", "vmcnt(2)"), ("v_mov_b32", "v3, v4")])) == 1
    lds = [("ds_read_b128", "v[4:7], v1 offset:16"), ("ds_read_b128", "v[8:11], v1 offset:32")]
    assert check_vm_waits(lds + [("s_waitcnt", "lgkmcnt(1)"), ("v_mov_b32", "v2, v4")]) == []
    assert len(check_vm_waits(lds + [("s_waitcnt", "lgkmcnt(1)"), ("v_mov_b32", "v2, v8")])) == 1
    mf = ("v_mfma_f32_16x16x32_f16", "a[0:3], v[10:13], v[20:23], a[0:3]")
    assert len(check_mfma_hazards([("v_pk_mul_f16", "v11, v1, v2"), mf])) == 1
    assert check_mfma_hazards([("v_pk_mul_f16", "v11, v1, v2"), ("s_nop", "1"), mf]) == []
    assert len(check_mfma_hazards([("v_accvgpr_write_b32", "a2, 0"), mf])) == 1
    assert len(check_mfma_hazards([mf, ("s_nop", "7"), ("ds_write_b128", "v1, a[0:3]")])) == 1
    assert check_mfma_hazards([mf, ("s_nop", "7"), ("s_nop", "7"), ("s_nop", "7"),
                               ("ds_write_b128", "v1, a[0:3]")]) == []
