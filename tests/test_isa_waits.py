"""Static check of the scans' partial memory waits (CPU only: compiles to
gfx950 assembly, runs nothing).

At the end of every chunk the scans publish the next chunk's LDS-DMA data
with `s_waitcnt vmcnt(N)` followed by a barrier, N > 0 leaving that many of
the wave's newest vector-memory operations in flight.  Vector memory
operations complete in issue order, so this is correct only if those N
newest operations were all issued after the last LDS-DMA (they are register
prefetches and stores, whose own uses the compiler waits for).  This test
compiles both scan kernels and checks, for every such wait in every template
instance, that at least N vector-memory instructions lie between the last
LDS-DMA instruction and the wait.
"""
import os
import re
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2509_25223_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _asm(src: str) -> str:
    from paper_2509_25223_amd import build as B
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [HIPCC] + [f for f in B.FLAGS if f not in ("-fPIC",)] + [
            "-x", "hip", "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return open(out).read()


def _publishing_waits(body):
    """(N, ops after the last LDS-DMA, index) for each vmcnt(N > 0) wait
    that reaches a barrier before any other vector-memory op or vmcnt wait."""
    out = []
    for k, line in enumerate(body):
        m = re.match(r"s_waitcnt vmcnt\((\d+)\)", line)
        if not m or int(m.group(1)) == 0:
            continue
        publishes = False
        for x in body[k + 1:]:
            op = x.split()[0]
            if op == "s_barrier":
                publishes = True
                break
            if op.startswith(("global_", "buffer_")) or "vmcnt" in x:
                break
        if not publishes:
            continue
        after = 0
        for x in reversed(body[:k]):
            op = x.split()[0]
            if op.startswith(("global_", "buffer_")):
                if "_lds" in op:
                    break
                after += 1
        out.append((int(m.group(1)), after, k))
    return out


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("src,kernel", [("fwd_scan.hip", "fwd_scan_kernel"),
                                        ("bwd_scan.hip", "bwd_scan_kernel")])
def test_partial_waits_leave_no_dma_in_flight(src, kernel):
    s = _asm(src)
    names = re.findall(r"^(_Z\w*%s\w*):" % kernel, s, re.M)
    assert names, "no %s instances found" % kernel
    checked = 0
    for name in names:
        i = s.index(name + ":")
        j = s.index(".Lfunc_end", i)
        body = [l.strip() for l in s[i:j].split("\n")
                if l.strip() and not l.strip().startswith((";", "."))
                and not l.strip().endswith(":")]
        for n, after, _ in _publishing_waits(body):
            assert after >= n, (name, n, after)
            checked += 1
    assert checked > 0
