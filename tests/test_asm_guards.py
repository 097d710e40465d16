"""Static check of the gfx950 code hipcc emits for the decode attention's
MFMA score kernel (no GPU needed).

Without an execution map the kernel loads each slab's K fragments with
inline-asm loads that the compiler does not track, and waits for them
itself (s_waitcnt) just before the score MFMAs.  That is sound only while
the compiler leaves the loaded registers where the asm put them until the
wait: a copy of them (for instance at the loop's back edge, when the next
slab's loads went to other registers) would read data that has not arrived.
So every asm K load must write registers that the score MFMAs read as their
A operand directly.  A variant with 32 more live registers broke exactly
this (NaN scores once a wavefront took two slabs), which is why that variant
uses compiler-tracked loads instead."""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2606_09514_amd import build as hip_build

SRC = os.path.join(hip_build.CSRC, "k_attn.hip")
KERNELS = [f"_ZN5buddy16attn_mfma_kernelILi{g}ELb0ELb0EEEvNS_8AttnArgsE" for g in (4, 8)]


@pytest.fixture(scope="module")
def device_asm():
    if not os.path.exists(hip_build.HIPCC):
        pytest.skip("hipcc not available")
    flags = [f for f in hip_build.FLAGS if f != "-fPIC"]
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k_attn.s")
        subprocess.run([hip_build.HIPCC, *flags, "--cuda-device-only", "-S", SRC, "-o", out],
                       check=True, capture_output=True)
        with open(out) as f:
            return f.read()


def function_body(asm: str, name: str) -> list:
    start = asm.index(f"\n{name}:")
    end = asm.index(".Lfunc_end", start)
    return asm[start:end].splitlines()


@pytest.mark.parametrize("name", KERNELS)
def test_asm_k_loads_feed_the_score_mfma_directly(device_asm, name):
    lines = function_body(device_asm, name)
    in_asm, k_dst, a_ops = False, [], set()
    for ln in lines:
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
    # the first slab's four loads and the loop's four
    assert len(k_dst) >= 8, k_dst
    assert len(a_ops) == 4, a_ops
    stray = [r for r in k_dst if r not in a_ops]
    assert not stray, f"asm K loads into {stray}, score MFMAs read {sorted(a_ops)}"
