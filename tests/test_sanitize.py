"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only,
no GPU): the oracle's C code re-runs its pin suite, and the C ABI's host side
re-runs the argument checks of test_abi.py, each from a sanitizer build in a
child process (the sanitizer runtime preloaded ahead of the interpreter's
libraries, leak detection off: the interpreter itself keeps its allocations).
Any report aborts the child (no recovery), which fails the test."""
import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2207_05808_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _env(runtime, **extra):
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = runtime + (" " + pre if pre else "")   # the sanitizer runtime must come first
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env.update(extra)
    return env


def _child(cmd, env):
    r = subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-4000:] + "\n" + r.stderr[-4000:])


def test_oracle_pins_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    runtime = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(runtime) or not os.path.exists(runtime):
        pytest.skip("gcc's AddressSanitizer runtime not found")
    import oracle
    so = oracle.build(str(tmp_path / "liboracle_san.so"),
                      extra_flags=("-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                                   "-fno-sanitize-recover=all"))
    _child([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider",
            os.path.join(ROOT, "tests", "test_oracle_pins.py")],
           _env(runtime, MADDNESS_ORACLE_LIB=so))


def test_abi_host_code_under_sanitizers(tmp_path):
    runtimes = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not os.path.exists(HIPCC) or not runtimes:
        pytest.skip("hipcc or its AddressSanitizer runtime not found")
    # host code instrumented; device code unoptimized (these checks launch nothing)
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xarch_device", "-O0",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    objs = [str(tmp_path / (os.path.basename(s) + ".o")) for s in srcs]

    def comp(so):
        s, o = so
        r = subprocess.run([HIPCC, *flags, "-c", s, "-o", o], capture_output=True, text=True)
        return r.returncode, s, r.stderr[-3000:]

    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        for rc, s, err in ex.map(comp, zip(srcs, objs)):
            assert rc == 0, f"{s}: {err}"
    lib = str(tmp_path / "libmaddness_san.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                        "-Xarch_host", "-fsanitize=undefined", *objs, "-o", lib], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    runner = ("import sys; sys.path.insert(0, sys.argv[1]); "
              "from paper_2207_05808_amd import _lib; _lib.LIB_PATH = sys.argv[2]; "
              "import pytest; sys.exit(pytest.main(['-q', '-x', '-s', '-p', 'no:cacheprovider', sys.argv[3]]))")
    _child([sys.executable, "-c", runner, ROOT, lib, os.path.join(ROOT, "tests", "test_abi.py")],
           _env(runtimes[-1]))
