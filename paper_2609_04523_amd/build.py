"""Build the gfx950 HIP library ``libmk_attn.so`` in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmk_attn.so")
# one translation unit per kernel family, compiled in parallel, then linked
SOURCES = [os.path.join(CSRC, f) for f in
           ("mk_attn.hip", "fwd_launch_d128.hip", "fwd_launch_d64.hip",
            "fwd_varlen_launch.hip", "fwd_rpa_launch.hip", "fwd_vt_launch.hip", "dec_launch.hip", "bwd_launch.hip",
            "mla_launch.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # keep hipcc from forming packed fp32 instructions on its own
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
]


def _noise_free(stderr: str) -> str:
    # hipcc's host pass does not know the packed-fp32 feature and says so
    noise = "'-packed-fp32-ops' is not a recognized feature"
    return "\n".join(l for l in stderr.splitlines() if noise not in l)


def build(out: str = LIB, extra: list[str] | None = None, verbose: bool = False) -> str:
    import tempfile
    with tempfile.TemporaryDirectory(prefix="mk_attn_build_") as tmp:
        objs, procs = [], []
        for src in SOURCES:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [HIPCC, *FLAGS, *(extra or []), "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.PIPE, text=True)))
            objs.append(obj)
        failed = []
        for src, p in procs:
            _, err = p.communicate()
            err = _noise_free(err)
            if p.returncode != 0:
                failed.append(f"{os.path.basename(src)}:\n{err}")
            elif err.strip() and verbose:
                print(err, file=sys.stderr)
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out + ".tmp"]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed ({res.returncode}):\n{_noise_free(res.stderr)}")
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
