"""Host AddressSanitizer and UndefinedBehaviorSanitizer runs of the CPU suite.

CPU only; not collected by pytest.  Run ``python tests/host_sanitizers.py``.

1. The oracle (``oracle/oracle.c``) is built by gcc with
   ``-fsanitize=address,undefined -fno-sanitize-recover=all``. Its CPU tests
   then run in a child Python with gcc's sanitizer runtimes preloaded.
2. ``libprox.so`` is built with the host code of ``api.hip`` (the argument
   checks and dispatch) instrumented the same way by hipcc. The device code
   and the other sources are built as usual. ``tests/test_api_cpu.py``, which
   calls every entry point with invalid arguments and never reaches a HIP
   call, then runs with clang's sanitizer runtime preloaded.

Leak detection is off: the interpreter's own allocations are not ours.
Exits non-zero on the first sanitizer report or test failure.
"""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2607_27591_amd import build as B   # noqa: E402  (compiler flags and sources)

ORACLE_TESTS = ["test_oracle_pins.py", "test_oracle_geglu.py", "test_oracle_threshold.py",
                "test_oracle_w4.py", "test_cost_model.py", "test_calibrate_cpu.py"]
API_TESTS = ["test_api_cpu.py"]
ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

# Runs pytest with one library swapped for its sanitized build.
CHILD = r"""
import os, sys
sys.path.insert(0, {root!r})
{setup}
import pytest
sys.exit(pytest.main(["-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider", *{files!r}]))
"""


def run_child(setup: str, files: list, preload: list) -> int:
    env = dict(os.environ, **ENV, LD_PRELOAD=":".join(preload))
    code = CHILD.format(root=ROOT, setup=setup,
                        files=[os.path.join(ROOT, "tests", f) for f in files])
    return subprocess.run([sys.executable, "-c", code], env=env, cwd=ROOT).returncode


def gcc_runtime(name: str) -> str:
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()
    if not os.path.isabs(path):
        raise RuntimeError(f"gcc has no {name}")
    return path


def clang_asan_runtime() -> str:
    out = subprocess.run([B.HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True).stdout.strip()
    if os.path.isabs(out) and os.path.exists(out):
        return out
    base = "/opt/rocm/llvm/lib/clang"
    for ver in sorted(os.listdir(base)) if os.path.isdir(base) else []:
        for sub in ("lib/linux/libclang_rt.asan-x86_64.so",
                    "lib/x86_64-unknown-linux-gnu/libclang_rt.asan.so"):
            p = os.path.join(base, ver, sub)
            if os.path.exists(p):
                return p
    raise RuntimeError("clang's ASan runtime not found")


def check_instrumented(lib: str) -> None:
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True,
                          check=True).stdout
    for want in ("__asan_init", "__ubsan_handle_"):
        if want not in syms:
            raise RuntimeError(f"{lib} is not instrumented ({want} missing)")


def oracle_run(tmp: str) -> int:
    lib = os.path.join(tmp, "liboracle_asan.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                    "-fopenmp", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "oracle.c"), "-o", lib, "-lm"], check=True)
    check_instrumented(lib)
    print(f"[sanitizers] oracle built: {lib}", flush=True)
    return run_child(f"import oracle\noracle._LIB = {lib!r}", ORACLE_TESTS,
                     [gcc_runtime("libasan.so"), gcc_runtime("libubsan.so")])


def api_run(tmp: str) -> int:
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-g"]

    def compile_one(src: str) -> str:
        obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
        extra = host_san if src == "api.hip" else []
        r = subprocess.run([B.HIPCC, *B.CFLAGS, *extra, "-c", os.path.join(B.CSRC, src),
                            "-o", obj], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        return obj

    with ThreadPoolExecutor(max_workers=min(len(B.SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(compile_one, B.SOURCES))
    lib = os.path.join(tmp, "libprox_asan.so")
    subprocess.run([B.HIPCC, "-shared", f"--offload-arch={B.ARCH}", "-fPIC", *objs, "-o", lib],
                   check=True)
    check_instrumented(lib)
    print(f"[sanitizers] libprox built with host-instrumented api.hip: {lib}", flush=True)
    return run_child("from paper_2607_27591_amd import prox\n"
                     f"prox.LIB_PATH = {lib!r}", API_TESTS, [clang_asan_runtime()])


def main() -> int:
    tmp = tempfile.mkdtemp(prefix="prox_san_")
    try:
        rc = oracle_run(tmp)
        print(f"[sanitizers] oracle suite: exit {rc}", flush=True)
        if rc == 0:
            rc = api_run(tmp)
            print(f"[sanitizers] API validation suite: exit {rc}", flush=True)
        return rc
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


if __name__ == "__main__":
    sys.exit(main())
