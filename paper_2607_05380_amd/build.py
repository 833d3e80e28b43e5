"""Build step: compiles the HIP sources into the in-tree shared library
``paper_2607_05380_amd/libtabpack.so`` for gfx950 with hipcc."""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = ["kernels_gemm.hip", "kernels_aux.hip", "kernels_muon.hip", "kernels_embed.hip", "select_static.hip", "host.cpp"]
LIB = os.path.join(HERE, "libtabpack.so")

FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include")]


def build(verbose=False, jobs=3):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    with tempfile.TemporaryDirectory(prefix="tabpack_build_") as tmp:
        procs = []
        objs = []
        for src in SRC:
            obj = os.path.join(tmp, src + ".o")
            lang = ["-x", "hip"] if src.endswith(".cpp") else []
            cmd = [hipcc] + FLAGS + lang + ["-c", os.path.join(HERE, "csrc", src), "-o", obj]
            objs.append(obj)
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        for cmd, p in procs:
            out = p.communicate()[0].decode()
            if p.returncode != 0:
                sys.stderr.write(out)
                raise RuntimeError("compile failed: " + " ".join(cmd))
            if verbose and out.strip():
                sys.stderr.write(out)
        tmp_lib = LIB + ".tmp"
        cmd = [hipcc, "-shared", "--offload-arch=gfx950", "-o", tmp_lib] + objs
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
        if r.returncode != 0:
            sys.stderr.write(r.stdout.decode())
            raise RuntimeError("link failed")
        os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
