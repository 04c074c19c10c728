"""The host-side code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): the plan, the C ABI's host paths, the implementation table, the
input generator and the oracle are compiled with clang and
-fsanitize=address,undefined (device objects as built), and the host-side
test files -- plan bookkeeping for every grouping of the five workloads, error
paths, the swap / budget rules, the generator, the oracle's pins -- run again
against those builds in a child process with the sanitizer runtime preloaded.
Any report (out-of-bounds access, use after free, signed overflow, invalid
shift, misaligned access ...) aborts the child."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_20501_amd", "csrc")
LLVM = "/opt/rocm/llvm/bin"
HOST_SOURCES = ["plan.cpp", "abi.cpp", "impls.cpp", "gen.cpp"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1", "-fPIC"]


def asan_runtime():
    out = subprocess.run([os.path.join(LLVM, "clang"), "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(out):
        hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        out = hits[0] if hits else ""
    return out


def device_objects():
    """The device-code objects of the regular build (rebuilt if missing or
    older than their sources)."""
    from paper_2607_20501_amd import build
    hips = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    objs = [os.path.join(build.BUILD, f + ".o") for f in hips]
    gen = os.path.join(build.BUILD, "mkgen.c.o")
    stale = any(not os.path.exists(o) or os.path.getmtime(o) < os.path.getmtime(
        os.path.join(CSRC, f)) for f, o in zip(hips, objs))
    if stale or not os.path.exists(gen):
        build.build_libmk()
    return objs + [gen]


@pytest.mark.timeout(900)
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    rt = asan_runtime()
    if not os.path.exists(os.path.join(LLVM, "clang++")) or not os.path.exists(rt):
        pytest.fail("clang or its AddressSanitizer runtime is missing")
    objs = []
    for src in HOST_SOURCES:
        o = str(tmp_path / (src + ".o"))
        subprocess.check_call([os.path.join(LLVM, "clang++"), "-std=c++17", "-D__HIP_PLATFORM_AMD__",
                               "-I/opt/rocm/include"] + SAN + ["-c", os.path.join(CSRC, src),
                                                               "-o", o])
        objs.append(o)
    libmk = str(tmp_path / "libmk_san.so")
    subprocess.check_call([os.path.join(LLVM, "clang++"), "-shared", "-shared-libasan"] + SAN +
                          ["-o", libmk] + objs + device_objects() +
                          ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    libmko = str(tmp_path / "libmko_san.so")
    subprocess.check_call([os.path.join(LLVM, "clang"), "-std=c99", "-D_DEFAULT_SOURCE",
                           "-shared", "-shared-libasan", "-fopenmp"] + SAN +
                          ["-I", os.path.join(ROOT, "oracle"), "-o", libmko,
                           os.path.join(ROOT, "oracle", "mko.c"), "-lm"])
    env = dict(os.environ, LD_PRELOAD=rt, MK_LIBRARY=libmk, MKO_LIBRARY=libmko,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    files = ["tests/test_plan.py", "tests/test_policy.py", "tests/test_inputs.py",
             "tests/test_oracle_pins.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-m", "not gpu"] + files, cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=840)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    for marker in ("ERROR: AddressSanitizer", "runtime error:"):
        assert marker not in report, report[-4000:]
    assert " passed" in r.stdout
