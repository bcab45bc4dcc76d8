"""Host sanitizer build and run (CPU only, no GPU needed).

    python paper_2607_16973_amd/sanitize.py

1. Builds _build/san/libtq_san.so from the library sources with
   AddressSanitizer and UndefinedBehaviorSanitizer on the host code only
   (every -fsanitize flag follows -Xarch_host; the gfx950 device code is
   compiled as usual).  The two host solvers are compiled by clang++ here
   (without OpenMP), so that one sanitizer runtime serves the whole library.
2. Builds _build/san/libtq_oracle_san.so from the oracle's C with gcc's
   AddressSanitizer and UndefinedBehaviorSanitizer.
3. Runs, each in a child process with the matching runtime preloaded and
   the build named by TQ_LIBRARY / TQ_ORACLE_LIBRARY:
   - tests/test_lib_host.py and tests/test_index_file.py (argument
     validation, host codebook and rotation solvers, index file parsing and
     every rejection path) against libtq_san.so;
   - the oracle encode pins (tests/test_oracle_encode.py,
     tests/test_oracle_tqplus.py) against libtq_oracle_san.so.
   Any sanitizer report aborts the child (halt_on_error), which fails the run.
Leak detection is off: the Python interpreter itself keeps allocations alive
at exit.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SAN = os.path.join(PKG, "_build", "san")
LIB = os.path.join(SAN, "libtq_san.so")
ORACLE_LIB = os.path.join(SAN, "libtq_oracle_san.so")
CLANG = "/opt/rocm/llvm/bin/clang++"

sys.path.insert(0, PKG)
import build as libbuild  # noqa: E402


def _host_san():
    out = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer"):
        out += ["-Xarch_host", f]
    return out


def build_library() -> str:
    os.makedirs(SAN, exist_ok=True)
    hipcc = libbuild._hipcc()
    objs = []
    for src in libbuild.HIP_SOURCES:
        obj = os.path.join(SAN, src + ".o")
        objs.append(obj)
        libbuild._run([hipcc] + libbuild.hip_flags() + libbuild.EXTRA_FLAGS.get(src, []) +
                      _host_san() + ["-g", "-c", os.path.join(CSRC, src), "-o", obj])
    for src in libbuild.HOST_SOURCES:
        obj = os.path.join(SAN, src + ".o")
        objs.append(obj)
        libbuild._run([CLANG, "-O1", "-g", "-std=c++17", "-fPIC", "-Wno-unknown-pragmas",
                       "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                       "-fno-omit-frame-pointer", "-I", libbuild.INCLUDE, "-I", CSRC,
                       "-c", os.path.join(CSRC, src), "-o", obj])
    libbuild._run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-shared-libsan"] +
                  _host_san()[:4] + ["-o", LIB] + objs)
    return LIB


def build_oracle() -> str:
    os.makedirs(SAN, exist_ok=True)
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", "-fno-fast-math",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer",
                           os.path.join(ROOT, "oracle", "csrc", "tq_oracle.c"),
                           "-o", ORACLE_LIB, "-lm"])
    return ORACLE_LIB


def _runtime(cmd):
    return subprocess.check_output(cmd, text=True).strip()


def run_tests(env_extra, preload, tests) -> int:
    env = dict(os.environ)
    env.update(env_extra)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu"] + tests
    print("+", " ".join("%s=%s" % kv for kv in env_extra.items()), "LD_PRELOAD=" + preload,
          " ".join(cmd), flush=True)
    return subprocess.call(cmd, cwd=ROOT, env=env)


def main() -> int:
    lib = build_library()
    olib = build_oracle()
    clang_rt = _runtime([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"])
    gcc_rt = _runtime(["gcc", "-print-file-name=libasan.so"])
    gcc_ubsan = _runtime(["gcc", "-print-file-name=libubsan.so"])
    rc = run_tests({"TQ_LIBRARY": lib}, clang_rt,
                   ["tests/test_lib_host.py", "tests/test_index_file.py"])
    rc2 = run_tests({"TQ_ORACLE_LIBRARY": olib}, gcc_rt + ":" + gcc_ubsan,
                    ["tests/test_oracle_encode.py", "tests/test_oracle_tqplus.py"])
    print("library (ASan+UBSan host):", "clean" if rc == 0 else "FAILED rc=%d" % rc)
    print("oracle C (ASan+UBSan):", "clean" if rc2 == 0 else "FAILED rc=%d" % rc2)
    return 0 if rc == 0 and rc2 == 0 else 1


if __name__ == "__main__":
    sys.exit(main())
