"""Static check of the gfx950 code hipcc emits for the kernels that load
through inline asm (no GPU needed).

The decode attention's MFMA score kernel (K fragments) and the MFMA
projection kernel (activation fragments) issue some vector-memory loads as
inline asm, outside the compiler's load tracking, and wait for them with
their own s_waitcnt; the prefill GEMM does the same with its fragment reads
from LDS, waiting for each row tile's read with a partial lgkmcnt.  That is sound only while the compiler leaves the
loaded registers alone until the wait: an instruction that reads such a
register earlier -- a copy at a loop's back edge, a spill into an
accumulation register -- takes data that has not arrived, and one that
writes it is overwritten when the load lands.  So in every instantiation,
from each asm load to the next s_waitcnt with a vmcnt (the kernels' own
waits cover their asm loads), no instruction may touch its destination
registers.  The walk is linear through the function, which matches these
kernels, whose loads and waits share a basic block.

Two earlier builds that gave wrong results both fail this check: a pooling
variant of the attention whose compiler copied the next slab's K at the
loop's back edge (NaN once a wavefront took two slabs), and four-k-step
projection rounds with six column tiles, whose registers spilled into
accumulation registers before the wait."""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2606_09514_amd import build as hip_build

SOURCES = {"k_attn.hip": "_ZN5buddy16attn_mfma_kernel", "k_mfma.hip": "_ZN5buddy11mfma_kernel",
           "k_gemm.hip": "_ZN5buddy11gemm_kernel"}
REG = re.compile(r"\bv(\d+)\b|\bv\[(\d+):(\d+)\]")


def device_asm(src: str) -> str:
    flags = [f for f in hip_build.FLAGS if f != "-fPIC"]
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        subprocess.run([hip_build.HIPCC, *flags, "--cuda-device-only", "-S",
                        os.path.join(hip_build.CSRC, src), "-o", out],
                       check=True, capture_output=True)
        with open(out) as f:
            return f.read()


def vregs(operand: str) -> set:
    out = set()
    for m in REG.finditer(operand):
        if m.group(1):
            out.add(int(m.group(1)))
        else:
            out.update(range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def operands(text: str):
    parts = text.split(None, 1)
    if len(parts) == 1:
        return parts[0], []
    ops, depth, cur = [], 0, ""
    for ch in parts[1]:
        depth += ch == "["
        depth -= ch == "]"
        if ch == "," and depth == 0:
            ops.append(cur.strip())
            cur = ""
        else:
            cur += ch
    if cur.strip():
        ops.append(cur.strip())
    return parts[0], ops


LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def hazards(lines) -> list:
    """Instructions that read or write an asm load's registers before the
    wait that covers it: the next vmcnt wait for a global load; for an LDS
    read, the first lgkmcnt(n) wait with at most n asm LDS reads issued after
    it (LDS reads return in issue order)."""
    in_asm, pending, bad = False, set(), []
    lds = []   # destination register sets of asm LDS reads, in issue order
    for ln in lines:
        raw = ln.strip()
        if raw.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if raw.startswith(";;#ASMEND"):
            in_asm = False
            continue
        text = ln.split(";")[0].strip()
        if not text or text.endswith(":") or text.startswith("."):
            continue
        op, ops = operands(text)
        if op == "s_waitcnt":
            if "vmcnt" in text:
                pending.clear()
            m = LGKM.search(text)
            if m:
                n = int(m.group(1))
                lds = lds[len(lds) - n:] if n < len(lds) else lds
            continue
        if in_asm and op == "global_load_dwordx4":
            pending |= vregs(ops[0])
            continue
        if op.startswith("s_") or not ops:
            continue
        store = not op.startswith("v_") and any(k in op for k in ("store", "ds_write", "atomic"))
        touched = set().union(*[vregs(o) for o in ops])
        if not store:
            touched |= vregs(ops[0])
        if touched & (pending.union(*lds) if lds else pending):
            bad.append(text)
        if in_asm and op == "ds_read_b128":
            lds.append(vregs(ops[0]))
    return bad


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(hip_build.HIPCC):
        pytest.skip("hipcc not available")
    out = {}
    for src, prefix in SOURCES.items():
        asm = device_asm(src)
        for m in re.finditer(r"^(" + re.escape(prefix) + r"\S*):", asm, re.M):
            start = m.end()
            out[m.group(1)] = asm[start:asm.index(".Lfunc_end", start)].splitlines()
    return out


def test_every_asm_load_instantiation_is_checked(kernels):
    # the attention's four instantiations (two group sizes, masked and not,
    # pooling) and every MFMA projection tiling
    assert sum(k.startswith(SOURCES["k_attn.hip"]) for k in kernels) >= 4
    assert sum(k.startswith(SOURCES["k_mfma.hip"]) for k in kernels) >= 60
    # the prefill GEMM's eight (epilogue x tile) instantiations, each with
    # its fragment reads from LDS as asm
    gemm = [b for k, b in kernels.items() if k.startswith(SOURCES["k_gemm.hip"])]
    assert len(gemm) >= 8
    assert all(sum(ln.strip().startswith("ds_read_b128") for ln in b) >= 8 for b in gemm)
    asm_loads = sum(1 for body in kernels.values() for ln in body
                    if ln.strip().startswith("global_load_dwordx4") and "off" in ln)
    assert asm_loads > 0


def test_no_register_of_an_untracked_load_is_touched_before_its_wait(kernels):
    bad = {name: h[:3] for name, body in kernels.items() if (h := hazards(body))}
    assert not bad, bad


def test_attention_k_loads_feed_the_score_mfma_directly(kernels):
    # the unmasked score kernels: the asm K loads write the score MFMA's A
    # operands themselves (no copy at all)
    for g in (4, 8):
        body = kernels[f"_ZN5buddy16attn_mfma_kernelILi{g}ELb0ELb0EEEvNS_8AttnArgsE"]
        in_asm, k_dst, a_ops = False, [], set()
        for ln in body:
            s = ln.strip()
            if s.startswith(";;#ASMSTART"):
                in_asm = True
            elif s.startswith(";;#ASMEND"):
                in_asm = False
            elif in_asm:
                m = re.match(r"global_load_dwordx4 (v\[\d+:\d+\]),", s)
                if m:
                    k_dst.append(m.group(1))
            else:
                m = re.match(r"v_mfma_f32_16x16x32_bf16 v\[\d+:\d+\], (v\[\d+:\d+\]),", s)
                if m:
                    a_ops.add(m.group(1))
        assert len(k_dst) >= 8 and len(a_ops) == 4, (k_dst, a_ops)
        assert set(k_dst) <= a_ops, (k_dst, sorted(a_ops))


def test_the_walk_flags_what_it_should():
    """The checker itself, on hand-written instruction streams: registers of
    an asm load read or overwritten before the wait that covers it are
    flagged; after that wait they are free.  For LDS reads, lgkmcnt(n)
    covers all but the last n asm reads issued."""
    A, E = ";;#ASMSTART", ";;#ASMEND"
    glob = [A, "global_load_dwordx4 v[4:7], v2, off", E]
    assert hazards(glob + ["v_mov_b32_e32 v9, v5"]) == ["v_mov_b32_e32 v9, v5"]
    assert hazards(glob + ["v_mov_b32_e32 v6, v9"]) == ["v_mov_b32_e32 v6, v9"]
    assert hazards(glob + ["s_waitcnt vmcnt(0)", "v_mov_b32_e32 v9, v5"]) == []
    assert hazards(glob + ["v_mov_b32_e32 v9, v8"]) == []
    lds = [A, "ds_read_b128 v[10:13], v1 offset:0", "ds_read_b128 v[14:17], v1 offset:1024",
           "ds_read_b128 v[18:21], v1 offset:2048", E]
    mfma = "v_mfma_f32_16x16x32_bf16 v[30:33], v[{}], v[40:43], v[30:33]"
    # after lgkmcnt(2) only the first read has landed
    assert hazards(lds + ["s_waitcnt lgkmcnt(2)", mfma.format("10:13")]) == []
    assert hazards(lds + ["s_waitcnt lgkmcnt(2)", mfma.format("14:17")]) == [mfma.format("14:17")]
    assert hazards(lds + ["s_waitcnt lgkmcnt(1)", mfma.format("14:17")]) == []
    assert hazards(lds + ["s_waitcnt lgkmcnt(1)", mfma.format("18:21")]) == [mfma.format("18:21")]
    assert hazards(lds + ["s_waitcnt lgkmcnt(0)", mfma.format("18:21")]) == []
    # a copy of a pending register, and a second read into it, are flagged
    assert hazards(lds + ["v_mov_b32_e32 v50, v19"]) == ["v_mov_b32_e32 v50, v19"]
    again = "ds_read_b128 v[18:21], v1 offset:4096"
    assert hazards(lds + [A, again, E]) == [again]
    # compiler-issued LDS reads (outside asm) are the compiler's to track
    assert hazards(["ds_read_b128 v[10:13], v1", mfma.format("10:13")]) == []
