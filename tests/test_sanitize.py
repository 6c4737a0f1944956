"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviourSanitizer (CPU only).

* tests/sanitize/oracle_driver.c runs every entry point of the oracle (all
  modes, flags, statistics, ragged and empty shapes, windows, GQA, the decode
  form, the logits, codecs and exponentials) built with gcc
  -fsanitize=address,undefined.
* tests/sanitize/host_driver.cpp calls the C ABI of the library with invalid,
  extreme and valid arguments.  The library's sources are compiled host-only
  (no device code: the kernels' registration is given empty offload bundles,
  and nothing is launched) with the sanitizers on the host side only.

Any sanitizer report aborts the driver (-fno-sanitize-recover=all)."""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2609_39361_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, cwd, timeout=300, env=None):
    r = subprocess.run(cmd, cwd=cwd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=timeout,
                       env=env)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-6000:]}"
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", exe, os.path.join(HERE, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "lamp_oracle.c"), "-lm"], cwd=str(tmp_path))
    out = _run([exe], cwd=str(tmp_path), env=SAN_ENV)
    assert "all calls clean" in out


HOST_SOURCES = ["lamp_kernels.hip", "lamp_fwd.hip", "lamp_fwd16.hip", "lamp_fwd16_sr.hip", "lamp_decode.hip",
                "lamp_rates.hip", "lamp_noalloc.hip", "lamp_host.cpp"]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
       "-fno-sanitize-recover=all"]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_host_code_under_sanitizers(tmp_path):
    from paper_2609_39361_amd import build as B
    assert sorted(B.SOURCES) == sorted(HOST_SOURCES), "a library source is not built here"
    work = str(tmp_path)
    flags = ["-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer",
             "-I", os.path.join(ROOT, "include")] + SAN

    def compile_one(src):
        obj = os.path.join(work, os.path.splitext(os.path.basename(src))[0] + ".o")
        _run([HIPCC] + flags + ["-c", src, "-o", obj], cwd=work)
        return obj

    srcs = [os.path.join(CSRC, s) for s in HOST_SOURCES] + [os.path.join(HERE, "host_driver.cpp")]
    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, srcs))
    # host-only objects refer to the device code of their translation unit by
    # a per-unit symbol: give each an empty offload bundle (no code objects)
    undef = _run(["nm", "-u"] + objs, cwd=work)
    names = sorted(set(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", undef)))
    stub = os.path.join(work, "fatbin_stub.c")
    with open(stub, "w") as f:
        for n in names:
            f.write(f'__attribute__((aligned(4096))) const char {n}[32] = "__CLANG_OFFLOAD_BUNDLE__";\n')
    _run(["gcc", "-c", stub, "-o", stub[:-2] + ".o"], cwd=work)
    exe = os.path.join(work, "host_san")
    _run([HIPCC] + SAN[:4] + ["-o", exe] + objs + [stub[:-2] + ".o"], cwd=work)
    out = _run([exe], cwd=work, timeout=120, env=SAN_ENV)
    assert "all calls clean" in out
