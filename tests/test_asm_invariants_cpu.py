"""Invariants of the compiled gfx950 code that the C++ source relies on but cannot state.

The index store publishes a slot with a 16-byte store written as inline assembly
(`store_pair_coherent`, paper_2609_38706_amd/csrc/k_table.hip) and does not wait for it: the
compiler does not count that store, which is sound only while every wait the compiler itself
places after it is `s_waitcnt vmcnt(0)` (a wait for a count above zero could then let an older
load through early).  This compiles the file for gfx950 and checks it for every kernel that
contains the store: no `vmcnt(N)` with N > 0 from the top of the loop that holds the store on.
Needs hipcc (the build's compiler), no GPU."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2609_38706_amd import _build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return None


def _kernels_with_store(asm: str):
    """(name, body) of every function whose body holds the inline-asm coherent pair store."""
    out = []
    for m in re.finditer(r"^(_ZN\S+):\s*;.*?$(.*?)^\.Lfunc_end", asm, re.M | re.S):
        body = m.group(2)
        if re.search(r"global_store_dwordx4 [^\n]*sc1", body) and "ASMSTART" in body:
            out.append((m.group(1), body))
    return out


@pytest.mark.skipif(_hipcc() is None, reason="hipcc not available")
def test_no_partial_vmem_wait_after_the_uncounted_store(tmp_path):
    src = os.path.join(ROOT, "paper_2609_38706_amd", "csrc", "k_table.hip")
    out = tmp_path / "k_table.s"
    flags = [f for f in _build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    cmd = [_hipcc()] + flags + ["--cuda-device-only", "-S", "-I", os.path.join(ROOT, "include"),
                                "-I", os.path.join(ROOT, "paper_2609_38706_amd", "csrc"), "-o", str(out), src]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels = _kernels_with_store(out.read_text())
    assert kernels, "no kernel with the coherent pair store found"
    for name, body in kernels:
        late = _partial_waits_after_store(body)
        assert not late, f"{name}: partial VMEM waits after the uncounted store: {late[:3]}"


def _partial_waits_after_store(body: str):
    """`vmcnt(N)` waits with N > 0 from the top of the loop that holds the first coherent pair
    store on (the last loop header before it; a wait at the top of that loop runs after the store
    of the previous iteration)."""
    first_store = re.search(r"global_store_dwordx4 [^\n]*sc1", body).start()
    headers = [m.start() for m in re.finditer(r"Loop Header", body) if m.start() < first_store]
    start = headers[-1] if headers else first_store
    return [m.group(0) for m in re.finditer(r"s_waitcnt[^\n]*vmcnt\((\d+)\)", body)
            if m.start() >= start and int(m.group(1)) > 0]


def test_the_check_finds_a_planted_partial_wait():
    prologue = "\ts_waitcnt vmcnt(2)\n.LBB0_1:  ; =>This Inner Loop Header: Depth=1\n\ts_branch .LBB0_1\n"
    loop = ".LBB0_5:  ; =>This Inner Loop Header: Depth=1\n\tglobal_load_dwordx2 v[0:1], v[2:3], off\n"
    store = "\t;;#ASMSTART\n\tglobal_store_dwordx4 v[4:5], v[6:9], off sc1\n\t;;#ASMEND\n"
    ok = prologue + loop + "\ts_waitcnt vmcnt(0)\n" + store + "\ts_cbranch_scc1 .LBB0_5\n"
    assert _partial_waits_after_store(ok) == []                     # the prologue's wait is before the loop
    bad_in_loop = prologue + loop + "\ts_waitcnt vmcnt(1)\n" + store + "\ts_cbranch_scc1 .LBB0_5\n"
    assert _partial_waits_after_store(bad_in_loop) == ["s_waitcnt vmcnt(1)"]
    bad_after = ok + "\ts_waitcnt vmcnt(3) lgkmcnt(0)\n"
    assert _partial_waits_after_store(bad_after) == ["s_waitcnt vmcnt(3)"]
