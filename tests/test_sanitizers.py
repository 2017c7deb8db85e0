"""Host-side sanitizer runs (CPU only): the oracle's pin tests against an
AddressSanitizer + UndefinedBehaviorSanitizer build of the oracle, and the
C ABI's host tests (argument validation, packing helpers, exports) against a
build of the library whose host code is instrumented the same way.  Device
code is never instrumented.  Each run is a child process with the sanitizer
runtime preloaded; a report makes it exit non-zero."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run_pytest(test_file, env_extra, tmp_path):
    env = dict(os.environ)
    env.update(SAN_ENV)
    env.update(env_extra)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-s", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", test_file)], cwd=str(tmp_path), env=env,
                       capture_output=True, text=True, timeout=900)
    out = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-pthread"] + san +
                          [os.path.join(ROOT, "oracle", "qnn_oracle.c"), "-o", lib])
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    ubsan = subprocess.check_output(["gcc", "-print-file-name=libubsan.so"], text=True).strip()
    _run_pytest("test_oracle_pins.py", {"QNN_ORACLE_LIB": lib, "LD_PRELOAD": asan + ":" + ubsan}, tmp_path)


def test_abi_host_under_asan_ubsan(tmp_path):
    objs = glob.glob(os.path.join(ROOT, "_build", "*.o"))
    if not objs:
        pytest.skip("the library's objects are not built (run __graft_entry__.build())")
    rts = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rts:
        pytest.skip("no clang AddressSanitizer runtime")
    inst = {"qnn_abi.o", "calib.o"}
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
             "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_1908_11263_amd", "csrc")]
    linked = [o for o in objs if os.path.basename(o) not in inst]
    for name in inst:
        src = os.path.join(ROOT, "paper_1908_11263_amd", "csrc", name[:-2] + ".hip")
        obj = str(tmp_path / name)
        subprocess.check_call([HIPCC] + flags + ["-c", src, "-o", obj], stderr=subprocess.DEVNULL)
        linked.append(obj)
    lib = str(tmp_path / "libqnn_san.so")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host",
                           "-fsanitize=address,undefined", "-shared-libsan", "-o", lib] + linked)
    _run_pytest("test_abi_host.py", {"QNN_LIBRARY": lib, "LD_PRELOAD": rts[0]}, tmp_path)
