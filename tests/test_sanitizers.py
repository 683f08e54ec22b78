"""CPU sanitizer leg: the oracle (plain C) and the host side of libpresto
(argument checks, workspace sizing, error reporting) built with
AddressSanitizer and UndefinedBehaviorSanitizer, without recovery, and run
through drivers that exercise them on small and extreme inputs.

* tests/sanitize/oracle_driver.c + oracle/oracle.c (gcc): every oracle entry
  point on seeded inputs with edge rows (ties, -inf rows, NaN, empty
  contexts, a budget larger than the candidate tree).
* tests/sanitize/api_driver.cpp + the library sources (hipcc; only the host
  code is instrumented, the device code is built as usual and never
  launched): every entry point with arguments the host rejects, empty
  batches and workspace queries at their extremes.

The builds are cached per source digest in the system temp directory.
"""
import hashlib
import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2607_22634_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LIB_SOURCES = ["api", "topk", "ngram", "round", "tree_build", "tree_attn", "accept"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _digest(paths):
    h = hashlib.sha256()
    for p in sorted(paths):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def test_oracle_under_asan_ubsan():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    srcs = [os.path.join(SAN, "oracle_driver.c"), os.path.join(ROOT, "oracle", "oracle.c"),
            os.path.join(ROOT, "oracle", "oracle.h")]
    out = os.path.join(tempfile.gettempdir(), f"presto_san_oracle_{_digest(srcs)}")
    if not os.path.exists(out):
        _run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
              "-fno-omit-frame-pointer", "-ffp-contract=off", "-fopenmp", "-std=c11",
              "-I", os.path.join(ROOT, "oracle"), srcs[0], srcs[1], "-o", out + ".tmp", "-lm"])
        os.replace(out + ".tmp", out)
    r = _run([out], env=ENV, timeout=300)
    assert "oracle driver: ok" in r.stdout


def test_host_api_under_asan_ubsan():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    srcs = [os.path.join(CSRC, f + ".hip") for f in LIB_SOURCES]
    hdrs = [os.path.join(CSRC, "common.hpp"), os.path.join(ROOT, "include", "presto.h"),
            os.path.join(SAN, "api_driver.cpp")]
    build = os.path.join(tempfile.gettempdir(), f"presto_san_api_{_digest(srcs + hdrs)}")
    exe = os.path.join(build, "api_driver")
    if not os.path.exists(exe):
        os.makedirs(build, exist_ok=True)
        inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
        host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=all"]

        def compile_one(name):
            obj = os.path.join(build, name + ".o")
            _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                  "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san, *inc,
                  "-c", os.path.join(CSRC, name + ".hip"), "-o", obj])
            return obj

        with ThreadPoolExecutor(min(len(LIB_SOURCES), os.cpu_count() or 1)) as ex:
            objs = list(ex.map(compile_one, LIB_SOURCES))
        drv = os.path.join(build, "driver.o")
        _run([HIPCC, "-O1", "-g", "-std=c++17", *host_san, *inc, "-c", hdrs[2], "-o", drv])
        _run([HIPCC, "--offload-arch=gfx950", "-fsanitize=address", "-fsanitize=undefined",
              "-fno-gpu-sanitize", drv, *objs, "-o", exe + ".tmp"])
        os.replace(exe + ".tmp", exe)
    r = _run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=0"), timeout=300)
    assert "api driver: ok" in r.stdout
