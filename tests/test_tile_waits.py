"""The explicit vector-memory waits of the tile kernel, checked against the
compiled gfx950 code (CPU only: hipcc compiles, nothing runs).

The tile kernel orders its LDS activation stages with hand-counted
`s_waitcnt vmcnt(N)`: loads complete in issue order, so at the wait every
load issued before the last N has landed.  N is a count of the loads the
source issues per group; if the compiler issues fewer (it drops a load whose
value is unused, as it did for the {s, z} word of unquantized weights), the
wait lets a direct-to-LDS load of the next stage still be in flight when the
waves read it.  This test reads every such wait (tagged in the assembly with
its stage count) and counts the vector-memory instructions between it and the
direct-to-LDS loads whose data it must cover:

  NS = 2, loop:      the stage loaded at the start of this group  -> N <= a
  NS = 3, loop:      the stage loaded one group earlier           -> N <= b
  NS = 3, prologue:  stage 0 and the codes of group 0             -> N <= a + n
  NS = 2, prologue:  stage 0 and the codes of group 0             -> N <= a / 2

with a (b) the instructions issued after the latest (the previous) group of
direct-to-LDS loads and n the size of the latest group.
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
sys.path.insert(0, os.path.join(ROOT, "paper_2503_21135_amd"))

VMEM = ("buffer_load", "global_load", "buffer_store", "global_store", "scratch_", "buffer_atomic", "global_atomic")
WAIT = re.compile(r"s_waitcnt vmcnt\((\d+)\) ; tile-wait ns=(\d) pro=(\d)")


def check_asm(text):
    """Returns (number of waits checked per kind, list of violations)."""
    groups, sizes = [], []   # per direct-to-LDS group: instructions issued since, group size
    in_dma = False
    seen = {}
    bad = []
    for lineno, raw in enumerate(text.splitlines(), 1):
        line = raw.strip()
        m = WAIT.search(line)
        if m:
            n, ns, pro = (int(v) for v in m.groups())
            if ns == 0:
                continue
            if len(groups) < (2 if (ns == 3 and not pro) else 1):
                bad.append((lineno, "no direct-to-LDS loads before the wait"))
                continue
            a, na = groups[-1], sizes[-1]
            b = groups[-2] if len(groups) > 1 else None
            if pro:
                ok = n <= a + na if ns == 3 else n <= a // 2
            else:
                ok = n <= b if ns == 3 else n <= a
            seen[(ns, pro)] = seen.get((ns, pro), 0) + 1
            if not ok:
                bad.append((lineno, "vmcnt(%d) ns=%d pro=%d: a=%d b=%s n=%d" % (n, ns, pro, a, b, na)))
            continue
        if line.startswith(";") or not line:
            continue
        op = line.split()[0]
        if not op.startswith(VMEM):
            continue
        dma = op.startswith("buffer_load") and line.split(";")[0].rstrip().endswith(" lds")
        if dma:
            if in_dma:
                groups = [g + 1 for g in groups[:-1]] + [groups[-1]]
                sizes[-1] += 1
            else:
                groups = [g + 1 for g in groups] + [0]
                sizes.append(1)
            in_dma = True
        else:
            groups = [g + 1 for g in groups]
            in_dma = False
    return seen, bad


def _compile(nm, out_dir):
    import build as B
    src = os.path.join(ROOT, "paper_2503_21135_amd", "csrc", "ffn_tile.hip")
    out = os.path.join(out_dir, "tile%d.s" % nm)
    cmd = [B.HIPCC] + B.FLAGS + ["-DMOE_FFN_NM=%d" % nm, "--cuda-device-only", "-S",
                                 "-I", os.path.join(ROOT, "include"),
                                 "-I", os.path.join(ROOT, "paper_2503_21135_amd", "csrc"), src, "-o", out]
    subprocess.run(cmd, check=True, capture_output=True)
    return open(out).read()


@pytest.fixture(scope="module")
def tile_asm():
    import build as B
    if not shutil.which(B.HIPCC) and not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not found")
    with tempfile.TemporaryDirectory() as d:
        with ThreadPoolExecutor(2) as ex:
            return dict(zip((2, 4), ex.map(lambda nm: _compile(nm, d), (2, 4))))


@pytest.mark.parametrize("nm", [2, 4])
def test_tile_waits_cover_the_lds_stages(tile_asm, nm):
    seen, bad = check_asm(tile_asm[nm])
    assert not bad, bad[:5]
    # every kind of wait is present (the tags survived), loop waits of both depths
    assert seen.get((3, 0), 0) > 0 and seen.get((3, 1), 0) > 0, seen
    if nm == 4:   # 8-bit and 6-bit rows at group 128 take two stages
        assert seen.get((2, 0), 0) > 0 and seen.get((2, 1), 0) > 0, seen


def test_checker_catches_a_dropped_load():
    """A two-stage loop wait that counts one load more than was issued."""
    ok = """
    buffer_load_dwordx4 v1, s[0:3], s4 offen lds
    buffer_load_dwordx4 v[2:5], v6, s[8:11], s12 offen
    buffer_load_dword v7, v6, s[8:11], s12 offen
    s_waitcnt vmcnt(2) ; tile-wait ns=2 pro=0
    """
    seen, bad = check_asm(ok)
    assert seen == {(2, 0): 1} and not bad
    dropped = ok.replace("    buffer_load_dword v7, v6, s[8:11], s12 offen\n", "")
    _, bad = check_asm(dropped)
    assert len(bad) == 1
