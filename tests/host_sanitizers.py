"""Run the CPU test suite against a build of libkf.so whose host code is
compiled with AddressSanitizer and UndefinedBehaviorSanitizer.

    python tests/host_sanitizers.py

The host code (csrc/kf_host.cpp: validation, planning, the C ABI) is
compiled by g++ with -fsanitize=address,undefined and linked with the device
objects of the last regular build (_build/*.hip.o, made by
paper_2605_30359_amd.build), into _build/sanitized/libkf.so.  The CPU tests
(pytest -m "not gpu") then run in a child process with the sanitizer
runtimes preloaded and the binding pointed at that library; any report
fails the run.  The device code is not instrumented, and no GPU is used.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2605_30359_amd")
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
OUT = os.path.join(BUILD, "sanitized")
ROCM = "/opt/rocm"


def _gcc_runtime(name: str) -> str:
    path = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True, check=True).stdout.strip()
    if not os.path.isabs(path):
        raise SystemExit(f"g++ has no {name}")
    return path


def build() -> str:
    objs = sorted(glob.glob(os.path.join(BUILD, "*.hip.o")))
    if not objs:
        raise SystemExit("no device objects under _build/: run python -m paper_2605_30359_amd.build first")
    os.makedirs(OUT, exist_ok=True)
    host_obj = os.path.join(OUT, "kf_host.o")
    flags = ["-std=c++17", "-O1", "-g", "-fPIC", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
             f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    subprocess.run(["g++"] + flags + ["-c", os.path.join(CSRC, "kf_host.cpp"), "-o", host_obj], check=True)
    lib = os.path.join(OUT, "libkf.so")
    subprocess.run(["g++", "-shared", "-fsanitize=address,undefined", "-o", lib, host_obj] + objs +
                   [f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib"], check=True)
    return lib


def main() -> int:
    lib = build()
    env = dict(os.environ)
    env["LD_PRELOAD"] = " ".join([_gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")])
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"  # the interpreter's own allocations are not ours
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    code = ("import sys, pytest\n"
            "from paper_2605_30359_amd import kf\n"
            f"kf.LIB_PATH = {lib!r}\n"
            "kf.lib()\n"
            "maps = [l.split()[-1] for l in open('/proc/self/maps') if 'libkf' in l]\n"
            f"assert set(maps) == {{{lib!r}}}, maps\n"
            "sys.exit(pytest.main(['tests', '-x', '-q', '-m', 'not gpu', '-p', 'no:cacheprovider']))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env)
    print(f"host sanitizers: CPU suite exit status {r.returncode} against {lib}")
    return r.returncode


if __name__ == "__main__":
    sys.exit(main())
