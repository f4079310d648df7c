"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

- The C ABI: every source of libmxq built with the sanitizers on its host
  code only (device code compiles as usual and is never run: there is no
  GPU here), linked with tests/sanitize/abi_host_driver.cpp, which runs the
  size queries, the argument checks and, for valid arguments, the path up
  to the kernel launch (refused by the runtime without a device).
- The C oracle: built with gcc's sanitizers and driven by
  tests/sanitize/oracle_driver.c over every width, mode and special value.
Any sanitizer report makes the run fail."""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_17733_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["api.cpp", "quantize.hip", "quantize_act.hip", "gemm_prefill.hip",
           "gemm_partials.hip", "decode.hip", "unpack.hip", "peaks.hip", "calib.hip",
           "attn.hip"]
# sanitizers on the host pass only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-x", "hip", "-O1", "-g", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s%s" % (" ".join(cmd), r.stdout[-4000:], r.stderr[-4000:])
    return r


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_host_paths_under_sanitizers(tmp_path):
    def compile_one(src):
        path = src if os.path.isabs(src) else os.path.join(CSRC, src)
        obj = os.path.join(tmp_path, os.path.basename(src) + ".o")
        _run([HIPCC] + FLAGS + HOST_SAN + ["-c", path, "-o", obj])
        return obj
    driver = os.path.join(ROOT, "tests", "sanitize", "abi_host_driver.cpp")
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(compile_one, SOURCES + [driver]))
    exe = os.path.join(tmp_path, "abi_driver")
    _run([HIPCC, "--offload-arch=gfx950"] + HOST_SAN + ["-o", exe] + objs)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", HIP_VISIBLE_DEVICES="")
    r = _run([exe], env=env, timeout=300)
    assert "abi host driver: ok" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = os.path.join(tmp_path, "oracle_driver")
    _run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
          "-fno-omit-frame-pointer", "-o", exe,
          os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "mxq_oracle.c"), "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = _run([exe], env=env, timeout=300)
    assert "oracle driver: ok" in r.stdout
