"""Build libhs.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2110_08941_amd.build

Every source is compiled each time (a few tens of seconds); objects go to
_build/ at the repository root and the library to paper_2110_08941_amd/libhs.so.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libhs.so")
BUILD = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I" + os.path.join(ROOT, "include"), "-Wall", "-Wno-unused-function"]
# Host arithmetic of the repartition must not be contracted (bit-exact with the
# reference arithmetic in the header).
PER_FILE = {"api.cpp": ["-ffp-contract=off"]}
SOURCES = ["igemm.hip", "igemm_fast.hip", "conv2.hip", "conv64.hip", "stem.hip", "wgrad3.hip", "layers.hip", "stats.hip", "opt.hip", "static_scratch.hip", "probe.hip", "model.cpp", "api.cpp"]


def _compile(src):
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC] + COMMON + PER_FILE.get(src, []) + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (r.stdout + r.stderr).splitlines()
            if "packed-fp32-ops" not in l and l.strip()]
    return src, obj, r.returncode, "\n".join(msgs)


def build(verbose=False):
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        raise RuntimeError("hipcc not found")
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), 8)) as ex:
        results = list(ex.map(_compile, SOURCES))
    objs = []
    for src, obj, rc, msg in results:
        if rc != 0:
            raise RuntimeError("hipcc failed on %s:\n%s" % (src, msg))
        if msg and verbose:
            print(msg)
        objs.append(obj)
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
