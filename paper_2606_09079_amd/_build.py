"""Builds ``liblsa.so`` in place from the HIP sources for gfx950."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
# LSA_LIB points the binding at another build of the same sources (for example an
# installed copy); by default the in-tree library is used.
LIB_PATH = os.environ.get("LSA_LIB") or os.path.join(HERE, "liblsa.so")
SOURCES = ("score.hip", "topk.hip", "attn.hip", "recall.hip", "tier.hip", "golden.hip", "kvpack.hip", "lsa_api.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         # no packed-fp32 instructions anywhere in the device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(quiet: bool = True) -> str:
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, *FLAGS, *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stderr}")
    if not quiet:
        print(res.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH
