"""Host sanitizers (AddressSanitizer and UndefinedBehaviorSanitizer) on the host code: the
float64 oracle, run under its pins, and the C ABI's validation layer (hs_api.hip's host code,
every check of which runs before any HIP call), run under the host ABI tests. Each is built
into a temporary directory and exercised in a child process with the sanitizer runtime
preloaded; any report fails the test. CPU only: nothing here touches a GPU."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
           "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}


def _run_pytest(args, env_extra):
    env = dict(os.environ)
    env.update(SAN_ENV)
    env.update(env_extra)
    # -s: the child's pytest must not capture the sanitizer's report on fd 2
    out = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p",
                          "no:cacheprovider", "-m", "not gpu"] + args, cwd=ROOT, env=env,
                         capture_output=True,
                         text=True, timeout=600)
    text = out.stdout + out.stderr
    assert out.returncode == 0, text[-4000:]
    assert "AddressSanitizer" not in text and "runtime error" not in text, text[-4000:]
    return text


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
                           "-ffp-contract=off", "-std=c11", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           os.path.join(ROOT, "oracle", "hs_oracle.c"), "-o", str(lib), "-lm"])
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    ubsan = subprocess.check_output(["gcc", "-print-file-name=libubsan.so"], text=True).strip()
    _run_pytest(["tests/test_oracle_pins.py"],
                {"HS_ORACLE_LIB": str(lib), "LD_PRELOAD": asan + ":" + ubsan})


def _clang_asan_runtime():
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return rt[0] if rt else None


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc") or _clang_asan_runtime() is None,
                    reason="hipcc or clang's sanitizer runtime not found")
def test_abi_validation_under_asan_and_ubsan(tmp_path):
    # hs_api.hip rebuilt with the sanitizers on its host code only (each flag after -Xarch_host),
    # linked with the other objects of the regular build
    sys.path.insert(0, ROOT)
    from paper_2510_20064_amd import build as B

    objdir = os.path.join(ROOT, "paper_2510_20064_amd", "_build")
    others = [os.path.join(objdir, f.replace(".hip", ".o")) for f in B.SOURCES
              if f != "hs_api.hip"]
    if not all(os.path.exists(o) for o in others):
        pytest.skip("the library's objects are not built (run the build first)")

    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-Xarch_host", "-g"]
    api_o = tmp_path / "hs_api_san.o"
    subprocess.check_call([B.HIPCC] + B.FLAGS + san +
                          ["-I", os.path.join(ROOT, "include"), "-I", B.CSRC, "-c",
                           os.path.join(B.CSRC, "hs_api.hip"), "-o", str(api_o)])
    lib = tmp_path / "libhedgespec_san.so"
    subprocess.check_call([B.HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan"] +
                          san + [str(api_o)] + others + ["-o", str(lib)])
    _run_pytest(["tests/test_abi_host.py"],
                {"HS_LIBRARY": str(lib), "LD_PRELOAD": _clang_asan_runtime()})
