"""Build the native libraries in-tree for gfx950.

libmk.so      the composed-module library (HIP kernels + C ABI, with the input
              generator linked in for mk_gen_fill), via hipcc
libmkgen.so   the seeded input generator (plain C, gcc)

Objects go to _build/ (git-ignored); every source is recompiled on each call.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed-fp32 VALU forms are disabled for every device compile.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
             "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-munsafe-fp-atomics"]


def _sources():
    return sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile(src):
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC] + HIP_FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{r.stdout}\n{r.stderr}")
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if err:
        sys.stderr.write(err + "\n")
    return obj


def _compile_gen():
    """The input generator (plain C) linked into libmk.so for mk_gen_fill."""
    obj = os.path.join(BUILD, "mkgen.c.o")
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-Wall", "-Wno-unknown-pragmas", "-c",
                           os.path.join(PKG, "inputs", "mkgen.c"), "-o", obj])
    return obj


def build_libmk(jobs=8):
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, _sources()))
    objs.append(_compile_gen())
    out = os.path.join(PKG, "libmk.so")
    tmp = out + ".tmp"
    subprocess.check_call([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs)
    os.replace(tmp, out)
    return out


def build_gen():
    src = os.path.join(PKG, "inputs", "mkgen.c")
    out = os.path.join(PKG, "inputs", "libmkgen.so")
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-Wall",
                           "-o", tmp, src, "-lm"])
    os.replace(tmp, out)
    return out


def build_all(jobs=8):
    build_gen()
    return build_libmk(jobs)


if __name__ == "__main__":
    print(build_all())
