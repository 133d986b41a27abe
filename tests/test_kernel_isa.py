"""Static checks on the gfx950 code of the attention kernel (CPU: hipcc cross-compiles).

The kernel waits for its direct-to-LDS tile copies with explicit vmcnt counts
that assume the copies are the only vector-memory instructions in flight inside
the key-block loop.  A register spill (scratch load/store) or any other vector
load/store placed in the loop by the compiler would silently shift those counts.
These tests compile the kernel to assembly and check, for every instantiation:
no VGPR spills, no scratch, and no vector-memory instruction in a loop other than
global_load_lds_dwordx4.
"""

import os
import re
import shutil
import subprocess
import tempfile
from collections import Counter

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_23019_amd", "csrc", "attn_fwd.hip")
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    from paper_2606_23019_amd import build
    tmp = tempfile.mkdtemp()
    try:
        out = os.path.join(tmp, "attn.s")
        cmd = [HIPCC] + [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")] + [
            "-I", os.path.join(ROOT, "include"), "-I", os.path.dirname(SRC),
            "--cuda-device-only", "-S", "-o", out, SRC]
        subprocess.run(cmd, check=True, capture_output=True)
        text = open(out).read()
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    funcs, cur = {}, None
    for line in text.split("\n"):
        m = re.match(r"^(_ZN2sa\S+bsattn_fwd_(?:pp_)?kernel\S+):", line)
        if m:
            cur = m.group(1)
            funcs[cur] = []
            continue
        if cur and line.startswith(".Lfunc_end"):
            cur = None
            continue
        if cur:
            funcs[cur].append(line)
    meta = {}
    for block in text.split("  - .agpr_count")[1:]:
        name = re.search(r"\.name:\s+(\S+)", block)
        if name:
            meta[name.group(1)] = dict(
                spill=int(re.search(r"\.vgpr_spill_count:\s+(\d+)", block).group(1)),
                private=int(re.search(r"\.private_segment_fixed_size:\s+(\d+)", block).group(1)))
    return funcs, meta


def test_every_instantiation_found(kernels):
    funcs, meta = kernels
    # 3 one-item tile shapes + the 128 x 128 ping-pong kernel, x 2 head dims, masked with bf16
    # or fp32 out, and maskless (bf16 out)
    assert len(funcs) == 24, sorted(funcs)
    assert set(meta) >= set(funcs)


def test_no_spills_or_scratch(kernels):
    funcs, meta = kernels
    for name in funcs:
        assert meta[name]["spill"] == 0 and meta[name]["private"] == 0, (name, meta[name])


def test_only_tile_copies_use_vmcnt_inside_loops(kernels):
    funcs, _ = kernels
    for name, lines in funcs.items():
        marked = [i for i, l in enumerate(lines) if "in Loop:" in l or "Loop Header" in l]
        assert marked, "no loop found in %s" % name
        lo, hi = min(marked), max(marked) + 1
        while hi < len(lines) and not re.match(r"^\.LBB", lines[hi]):
            hi += 1
        ops = Counter(l.split()[0] for l in lines[lo:hi]
                      if re.match(r"^\s+(global_|buffer_|scratch_|flat_)", l))
        assert set(ops) == {"global_load_lds_dwordx4"}, (name, dict(ops))
