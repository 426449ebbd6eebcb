"""Build libsva.so for gfx950 from the HIP sources in csrc/ (in-tree).

    python -m paper_2606_23743_amd.build [--jobs N] [--save-temps DIR]

Every source is compiled to an object with hipcc in parallel, then linked into
paper_2606_23743_amd/libsva.so (written to a temporary name and renamed, so a
failed build never leaves a half-written library behind).
"""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsva.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from emitting packed fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libsva.so)")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def build(jobs: int = 8, save_temps: str | None = None, verbose: bool = False) -> str:
    cc = hipcc()
    srcs = sources()
    with tempfile.TemporaryDirectory(prefix="sva_build_") as tmp:
        def compile_one(src):
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [cc, *HIPCC_FLAGS, "-c", src, "-o", obj]
            if save_temps:
                os.makedirs(save_temps, exist_ok=True)
                cmd += ["-save-temps=obj"]
                obj_dir = save_temps
                cmd[-1] = os.path.join(obj_dir, os.path.basename(src) + ".o")
                obj = cmd[-1]
            r = subprocess.run(cmd, capture_output=True, text=True)
            noise = [ln for ln in (r.stderr or "").splitlines() if "packed-fp32-ops" not in ln]
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed for {src}:\n" + "\n".join(noise))
            if verbose and noise:
                print("\n".join(noise), file=sys.stderr)
            return obj

        with ThreadPoolExecutor(max(1, jobs)) as ex:
            objs = list(ex.map(compile_one, srcs))
        tmp_lib = LIB + ".tmp"
        cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp_lib, *objs]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + r.stderr)
        os.replace(tmp_lib, LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--save-temps", default=None)
    ap.add_argument("-v", "--verbose", action="store_true")
    args = ap.parse_args(argv)
    print(build(args.jobs, args.save_temps, args.verbose))


if __name__ == "__main__":
    main()
