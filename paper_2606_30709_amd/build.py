"""Build libhga.so (the HIP library behind include/hga.h) for gfx950.

Every translation unit is compiled by hipcc for gfx950 only, then linked
against the HIP runtime that PyTorch loads (torch/lib/libamdhip64.so), so the
library and torch share one runtime, one device context and one allocator
view in a process.  Run ``python -m paper_2606_30709_amd.build``.
"""

from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libhga.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
CXXFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def torch_lib_dir() -> str:
    import importlib.util
    spec = importlib.util.find_spec("torch")
    if spec is None or spec.origin is None:
        raise RuntimeError("torch is required to locate its HIP runtime")
    return os.path.join(os.path.dirname(spec.origin), "lib")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, src_dir: str = CSRC, out: str = LIB,
          defines: tuple = ()) -> str:
    """Compile every source of ``src_dir`` and link ``out``."""
    srcs = sorted(glob.glob(os.path.join(src_dir, "*.hip"))) + \
        sorted(glob.glob(os.path.join(src_dir, "*.cpp")))
    tlib = torch_lib_dir()
    hip_rt = os.path.join(tlib, "libamdhip64.so")
    if not os.path.exists(hip_rt):
        raise RuntimeError(f"HIP runtime not found at {hip_rt}")
    tmp = tempfile.mkdtemp(prefix="hga_build_")
    try:
        objs = []
        procs = []
        for s in srcs:
            o = os.path.join(tmp, os.path.basename(s) + ".o")
            lang = ["-x", "hip"] if s.endswith(".hip") else []
            cmd = [HIPCC] + CXXFLAGS + ["-I", src_dir] + [f"-D{d}" for d in defines] + \
                lang + ["-c", s, "-o", o]
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.STDOUT, text=True)))
            objs.append(o)
        for cmd, p in procs:
            log, _ = p.communicate()
            log = "\n".join(l for l in log.splitlines() if "packed-fp32-ops" not in l)
            if p.returncode != 0:
                raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{log}")
            if verbose and log.strip():
                print(log)
        tmp_lib = out + ".tmp"
        _run(["g++", "-shared", "-o", tmp_lib] + objs +
             [hip_rt, f"-Wl,-rpath,{tlib}", "-Wl,--no-undefined", "-Wl,-z,defs"])
        os.replace(tmp_lib, out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
