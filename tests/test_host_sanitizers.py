"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU): the whole library is built with the sanitizers on its host side only
(device code unchanged) and host_fuzz.py drives its host-only entry points and
the device entry points' argument checks with random and extreme arguments
in a child process that halts on the first report.  Skipped where a GPU is
visible (the device entry points would then launch with fake pointers) or the
toolchain lacks the sanitizer runtime."""
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "paper_2609_29364_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ASAN_RT = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _gpu_visible():
    import torch
    return torch.cuda.device_count() > 0   # does not initialise a device


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if not os.path.exists(HIPCC) or not ASAN_RT:
        pytest.skip("hipcc or the clang ASan runtime is missing")
    if _gpu_visible():
        pytest.skip("a GPU is visible")
    from paper_2609_29364_amd.build import SOURCES
    out = tmp_path_factory.mktemp("asan")
    flags = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang",
             "-target-feature", "-Xclang", "-packed-fp32-ops",
             f"-I{os.path.join(ROOT, 'include')}"] + SAN

    def compile_one(src):
        obj = str(out / (src + ".o"))
        r = subprocess.run([HIPCC] + flags + ["-x", "hip", "-c", os.path.join(SRC, src), "-o", obj],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return obj

    with ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    lib = str(out / "libnebulasd.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host",
                        "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-shared-libasan", "-o", lib] + objs, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return lib


def test_host_code_runs_clean_under_sanitizers(sanitized_lib):
    env = dict(os.environ, LD_PRELOAD=ASAN_RT[-1],
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, os.path.join(HERE, "host_fuzz.py"), sanitized_lib, "7",
                        "1500"], capture_output=True, text=True, env=env, timeout=600)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0 and "host fuzz: clean" in r.stdout, tail
