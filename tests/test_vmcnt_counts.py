"""The streamed Gated DeltaNet state pass (gdn_state_dma_kernel) waits on the
vector-memory counter with counts derived from its own constants: per chunk,
NIW global_load_lds pieces of the chunk NSTAGE - 1 ahead, then NKH state stores
(every sstride-th chunk) and NSU U^T stores; vmcnt(n) lets exactly those stay in
flight.  The counts are only right if the compiler issues exactly those
vector-memory instructions in the chunk loop and no others (a register spill, a
split or merged load or an extra global load would shift them and the wait would
silently under-wait).  This test compiles the kernel source to gfx950 assembly
with the library's own flags and checks the chunk loop of every instantiation
the library launches, on the CPU.
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2606_01294_amd import build as B

C = 64


def expected(DK, NPR, NH):
    """(stream-load instructions in the loop, stores in the loop) from the kernel's
    constants; a piece shared by several waves is one lane-masked load in each."""
    NW, BVS = NPR * NH, 16 * NPR
    DKH = DK // NH
    NKH = DKH // 32
    NIK, NIT, NIV = C * DK * 2 // 1024, C * C * 2 // 1024, C * BVS * 2 // 1024
    NIVW = (NIV + NW - 1) // NW
    NIW = NIK // NW + NIT // NW + NIVW + 1
    NSU = 2 if NH == 1 else 1
    return NIW, NKH + NSU


# the instantiations the library launches (template <DK, NPR, NH, NSTAGE, RS, RSU>)
INSTANCES = [(256, 2, 4, 2, 1, 1), (256, 1, 4, 3, 1, 1), (128, 4, 2, 3, 1, 1), (128, 2, 4, 3, 1, 1)]


@pytest.fixture(scope="module")
def gdn_asm():
    src = os.path.join(B.CSRC, "ccq_gdn.hip")
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "ccq_gdn.s")
        cmd = [B._hipcc()] + B.COMMON + B.DEVICE + ["--cuda-device-only", "-S", src, "-o", out]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            pytest.skip("hipcc unavailable for gfx950 here: " + res.stderr[-300:])
        return open(out).read()


def chunk_loop(asm, sym):
    """Instructions of the kernel's outermost loop (the chunk loop): from the loop
    header label to the last branch back to it."""
    body = asm.split("\n" + sym + ":", 1)[1].split("s_endpgm", 1)[0].split("\n")
    head = [i for i, line in enumerate(body) if "Loop Header: Depth=1" in line]
    assert len(head) == 1, "one chunk loop expected in %s" % sym
    label = body[head[0]].split(":", 1)[0].strip()
    back = [i for i, line in enumerate(body) if re.search(r"s_cbranch\w*\s+" + re.escape(label) + r"\b", line)
            or re.search(r"s_branch\s+" + re.escape(label) + r"\b", line)]
    assert back, "no branch back to %s" % label
    return [line.split(";")[0].strip() for line in body[head[0]:max(back) + 1]]


@pytest.mark.parametrize("inst", INSTANCES, ids=lambda t: "dk%d-npr%d-nh%d-ns%d-rs%d-rsu%d" % t)
def test_state_pass_loop_issues_the_counted_vector_memory_ops(gdn_asm, inst):
    DK, NPR, NH, NS, RS, RSU = inst
    sym = "_ZN3ccq20gdn_state_dma_kernelILi%dELi%dELi%dELi%dELb%dELb%dEEEvNS_7GdnArgsE" % inst
    assert ("\n" + sym + ":") in gdn_asm, "instantiation %s not emitted" % sym
    loop = chunk_loop(gdn_asm, sym)
    mnem = [line.split()[0] for line in loop if line and not line.startswith((".", ";"))]
    vmem = [m for m in mnem if m.startswith(("global_", "buffer_", "scratch_", "flat_"))]
    loads = [m for m in vmem if m == "global_load_lds_dwordx4"]
    stores = [m for m in vmem if m.startswith("global_store_")]
    other = [m for m in vmem if m not in ("global_load_lds_dwordx4",) and not m.startswith("global_store_")]
    n_loads, n_stores = expected(DK, NPR, NH)
    assert not other, "unexpected vector-memory instructions in the chunk loop: %s" % other
    assert len(loads) == n_loads, (len(loads), n_loads)
    assert len(stores) == n_stores, (len(stores), n_stores)
