"""Build liblstmss.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "liblstmss.so")
SOURCES = ["lstmss_api.cpp", "cell.hip", "gemm1.hip", "wgrad_f32.hip", "wgrad_bf16.hip", "gemm.hip",
           "train.hip", "bidir.hip", "noalloc.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _flags():
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
            # packed fp32 instructions stay off (see the notes on gfx950 in the design document)
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include")]


def _filtered(r):
    return "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False) -> str:
    """Compile every source to an object (in parallel), then link liblstmss.so."""
    with tempfile.TemporaryDirectory(prefix="lstmss_build_") as tmpdir:
        procs = []
        for src in SOURCES:
            obj = os.path.join(tmpdir, src + ".o")
            cmd = [HIPCC] + _flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
            procs.append((src, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                     stderr=subprocess.PIPE, text=True)))
        objs, logs = [], []
        for src, obj, p in procs:
            out, err = p.communicate()
            r = subprocess.CompletedProcess(p.args, p.returncode, out, err)
            if r.returncode != 0:
                raise RuntimeError("hipcc failed on %s:\n%s" % (src, _filtered(r)))
            logs.append(_filtered(r))
            objs.append(obj)
        tmp = LIB + ".tmp%d" % os.getpid()
        r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs,
                           capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc link failed:\n" + _filtered(r))
    out = "\n".join(l for l in logs if l.strip())
    if verbose and out.strip():
        print(out, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
