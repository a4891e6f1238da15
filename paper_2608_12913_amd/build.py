"""Build libdcd.so (gfx950) in place with hipcc, and the benchmark's measurement
probes into a library of their own, libdcd_probe.so."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libdcd.so")
PROBE_LIB = os.path.join(PKG, "libdcd_probe.so")
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
         # packed fp32 VALU forms are kept out of every kernel
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link libdcd.so (csrc/) and libdcd_probe.so
    (probe/); always rebuilds."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    libs = {LIB: sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip"))),
            PROBE_LIB: sorted(glob.glob(os.path.join(PKG, "probe", "*.hip")))}
    procs = []
    objs = {lib: [] for lib in libs}
    for lib, srcs in libs.items():
        for src in srcs:
            procs.append((lib, src, os.path.join(objdir, os.path.basename(src) + ".o")))
    running = []
    for lib, src, obj in procs:
        objs[lib].append(obj)
        cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        running.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in running:
        out, _ = p.communicate()
        text = "\n".join(l for l in out.decode(errors="replace").splitlines()
                         if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(f"{s}:\n{t}" for s, t in failed))
    for lib, lobjs in objs.items():
        tmp = lib + ".tmp"
        subprocess.check_call([HIPCC, "-shared", f"--offload-arch={ARCH}", *lobjs, "-o", tmp])
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
