"""The wide decode-attention kernel reaches its first K/V load after one memory round trip, and a pass over
consecutive rows issues its K/V loads without 64-bit address arithmetic (no GPU needed).

Before a workgroup can issue its first K/V load it needs its sequence's retained-set description (range table,
or layout and policy, or count) and the launch fields (K/V bases and strides, limits).  The kernel fetches the
former with a vector load and pins the latter in scalar registers in one batch, so that a single wait on the
scalar loads overlaps the vector load.  Scalar waits cannot be partial, and the compiler may split the scalar
loads around a wait of its own (a scratch value placed in a register a load is still filling, or a launch
field loaded again under register pressure): each such split puts another memory round trip, about 0.3-0.7 us,
in front of the first K/V load.  This test compiles the kernels with the build's flags and checks the property
on the generated code of the range-table, fused-step and index-list variants.

A pass whose 32 ranks lie in one piece of the retained set reads 32 consecutive rows.  Its 16 loads (8 K, 8 V)
then take the first row's address as a scalar base and a 32-bit offset per lane (the scalar-base form of the
load), one offset per row shared by K and V; a 64-bit address per load and lane would cost about ten vector
instructions each, all before or between the loads that start the pass's memory traffic.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2606_01483_amd import _build

WIDE = r"^(_ZN6murmur23decode_attn_wide_kernelILi{k}EE\S*):"
VARIANTS = {0: "index list", 1: "range table", 2: "fused step (layout and policy)"}


@pytest.fixture(scope="module")
def asm():
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "kernels.s")
        subprocess.run([hipcc, *_build.KERNEL_FLAGS, "--cuda-device-only", "-S",
                        os.path.join(_build.CSRC, "kernels.hip"), "-o", out], check=True, capture_output=True)
        return open(out).read()


def kernel_body(asm_text: str, k: int) -> str:
    m = re.search(WIDE.format(k=k), asm_text, re.M)
    assert m, f"no decode_attn_wide_kernel<{k}> in the generated code"
    return asm_text[m.end():asm_text.index(".Lfunc_end", m.end())]


def prologue(asm_text: str, k: int) -> str:
    """Code of variant k from its entry (past the fallback block that loads the preloaded arguments, which
    hardware with argument preloading skips) to its first direct-to-LDS K/V load."""
    m = re.search(WIDE.format(k=k), asm_text, re.M)
    assert m, f"no decode_attn_wide_kernel<{k}> in the generated code"
    body = asm_text[m.end():asm_text.index(".Lfunc_end", m.end())]
    body = body[body.index(".p2align\t8"):]
    dma = [i for i in (body.find("global_load_lds"), body.find(" lds\n")) if i >= 0]
    assert dma, f"decode_attn_wide_kernel<{k}> issues no direct-to-LDS load"
    return body[:min(dma)]


@pytest.mark.parametrize("k", sorted(VARIANTS))
def test_one_round_trip_before_the_first_kv_load(asm, k):
    code = prologue(asm, k)
    waits = re.findall(r"s_waitcnt[^\n]*lgkmcnt", code)
    assert len(waits) == 1, f"{VARIANTS[k]}: {len(waits)} scalar waits before the first K/V load"
    first_wait = code.index(waits[0])
    vload = re.search(r"\tglobal_load_dword ", code)
    assert vload and vload.start() < first_wait, f"{VARIANTS[k]}: the sequence's words are not loaded ahead of the wait"


SADDR_LOAD = re.compile(r"global_load_lds_dwordx4 v\d+, s\[\d+:\d+\]")


@pytest.mark.parametrize("k", [1, 2])
def test_consecutive_rows_take_scalar_base_loads(asm, k):
    lines = [ln.strip() for ln in kernel_body(asm, k).splitlines() if ln.startswith("\t")]
    loads = [i for i, ln in enumerate(lines) if SADDR_LOAD.match(ln)]
    # the full-tile pass: 16 scalar-base loads in a row, a few instructions (offset add, LDS address in m0,
    # wait states) apart, with no 64-bit vector address arithmetic among them
    best = 0
    for a in range(len(loads)):
        b = a
        while b + 1 < len(loads) and loads[b + 1] - loads[b] <= 5 and not any(
                ln.startswith(("v_lshl_add_u64", "v_mad_u64_u32", "v_lshlrev_b64")) for ln in lines[loads[b]:loads[b + 1]]):
            b += 1
        best = max(best, b - a + 1)
    assert best >= 16, f"{VARIANTS[k]}: longest run of scalar-base K/V loads is {best}, expected 16"
