"""Builds libregenvc_attn.so for gfx950 with hipcc (in-tree, no JIT cache).

Run as ``python -m paper_2607_28144_amd.build``; it compiles every time it is
called.  Packed-fp32 VALU instructions are switched off for all device code.
"""
import os
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
REPO_DIR = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
LIB_NAME = "libregenvc_attn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
SOURCES = ["api.cpp", "attn_fwd.hip", "lse_merge.hip", "norm_rope.hip", "dit_api.cpp", "dit.hip", "vae_api.cpp",
           "vae.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile the shared library; returns its path.  Raises on failure."""
    out_tmp = LIB_PATH + ".tmp"
    cmd = [
        hipcc(),
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-shared",
        "-Wall",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # MFMA results in VGPRs: the score tiles feed VALU softmax code directly,
        # and read-only operands may then live in AGPRs
        "-mllvm", "-amdgpu-mfma-vgpr-form",
        "-I", os.path.join(REPO_DIR, "include"),
        "-I", CSRC,
        "-o", out_tmp,
    ] + [os.path.join(CSRC, s) for s in SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature: that warning is harmless
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), flush=True)
    os.replace(out_tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
