"""The host side of the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: the sanitized build of _build.py
(api.cpp through g++ with -fsanitize=address,undefined, linked with the HIP
kernel objects) runs (1) a C++ driver over the validate-mode checks of block
lists and sample offsets and (2) the whole ABI test module."""
import glob
import os
import subprocess
import sys

import pytest

from paper_2609_23169_amd import _build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))


def _runtime(name):
    p = subprocess.run([_build.GXX, f"-print-file-name={name}"], capture_output=True, text=True)
    return p.stdout.strip()


@pytest.fixture(scope="module")
def sanitized_lib():
    objs = sorted(glob.glob(os.path.join(_build.OBJ, "*.o")))
    if not any(o.endswith("bsattn_fwd.o") for o in objs):
        pytest.skip("kernel objects not built (run __graft_entry__.build() first)")
    try:
        return _build.build_sanitized(objs)
    except RuntimeError as e:   # no host compiler with sanitizer runtimes
        pytest.skip(f"sanitized build unavailable: {e}")


def _env(lib):
    env = dict(os.environ)
    env.update(ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    if lib:
        env["UT_LIBRARY"] = lib
    return env


def test_validate_checks_under_sanitizers(sanitized_lib, tmp_path):
    exe = str(tmp_path / "check_validate")
    cmd = [_build.GXX, "-std=c++17", "-g", *_build.SAN_FLAGS, "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", _build.CSRC,
           os.path.join(HERE, "host", "check_validate.cpp"), sanitized_lib,
           f"-Wl,-rpath,{os.path.dirname(sanitized_lib)}", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([exe], capture_output=True, text=True, env=_env(None), timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr[-3000:]
    assert "0 failure(s)" in r.stdout


def test_abi_module_under_sanitizers(sanitized_lib):
    env = _env(sanitized_lib)
    env["LD_PRELOAD"] = " ".join(p for p in (_runtime("libasan.so"), _runtime("libubsan.so")) if p)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_abi.py")],
                       capture_output=True, text=True, env=env, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
