"""Build the HIP library ``libsa_bsattn.so`` in-tree for gfx950.

Run ``python -m paper_2606_23019_amd.build`` (or ``__graft_entry__.build()``).
Every call recompiles; the library lands next to this file so that it
travels with the source tree.
"""

import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
LIB_NAME = "libsa_bsattn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
ARCH = "gfx950"

SOURCES = ["api.cpp", "prepass.hip", "mask_inst.hip", "fidelity.hip", "resize.hip", "attn_fwd.hip"]
# sustained MFMA rate probe, a measurement helper of bench.py (not in the C ABI)
MFMA_PEAK_SOURCES = ["mfma_peak.hip"]
MFMA_PEAK_PATH = os.path.join(PKG_DIR, "libsa_mfma_peak.so")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=" + ARCH,
    # keep hipcc from forming packed fp32 instructions by itself
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in VGPRs: the softmax reads the logits with vector ALU
    # instructions, and AGPR results would need a copy per element
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-fvisibility=hidden", "-Wall", "-Wno-unused-function",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _compile(sources, lib_path, verbose):
    srcs = [os.path.join(CSRC, s) for s in sources]
    tmp = lib_path + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + ["-I", os.path.join(ROOT, "include"), "-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "is not a recognized feature" not in l)
    if r.returncode != 0:
        if os.path.exists(tmp):
            os.unlink(tmp)
        raise RuntimeError("hipcc failed (%d):\n%s" % (r.returncode, out))
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib_path)
    return lib_path


def build(verbose=False):
    """Compile all sources into LIB_PATH (atomically replaced), and the MFMA-rate
    probe the benchmark reads its measured peak from into MFMA_PEAK_PATH; return
    LIB_PATH."""
    _compile(SOURCES, LIB_PATH, verbose)
    _compile(MFMA_PEAK_SOURCES, MFMA_PEAK_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
