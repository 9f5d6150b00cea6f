"""AddressSanitizer and UndefinedBehaviorSanitizer runs of the host code, on the CPU.

1. The oracle (oracle/oracle.c) and the library's host sources (the encoder and the blob
   validation of encode.cpp and capi.cpp; the GPU encoder's device half is replaced by
   stubs) are built with both sanitizers into one driver.  It encodes small tensors with
   both encoders (every container, tile sizes down to one vector, b = 9, the escalation
   path, the per-row refinement), checks that the blobs agree byte for byte, decodes them
   with the oracle to every output type, then feeds thousands of malformed blobs
   (truncations, bit flips, random words) through ep_blob_info and the oracle decoder.
   Leak detection is on.
2. A set of the oracle's CPU pins runs against a sanitized build of the oracle, with the
   sanitizer runtimes preloaded into the Python process.

Both builds use g++/gcc on host code only; no device code is involved.
"""
import os
import shutil
import subprocess
import sys

import pytest

pytestmark = pytest.mark.slow

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


def _gcc_runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.fixture(scope="module")
def sanbuild(tmp_path_factory):
    if not shutil.which("gcc") or not shutil.which("g++"):
        pytest.skip("gcc/g++ not available")
    if not _gcc_runtime("libasan.so") or not _gcc_runtime("libubsan.so"):
        pytest.skip("sanitizer runtimes not installed")
    d = tmp_path_factory.mktemp("asan")
    csrc = os.path.join(ROOT, "paper_2609_34185_amd", "csrc")
    objs = []

    def cc(compiler, src, std, extra=()):
        obj = str(d / (os.path.basename(src) + ".o"))
        subprocess.check_call([compiler, *SAN, std, *extra, "-c", src, "-o", obj])
        objs.append(obj)

    cc("gcc", os.path.join(ROOT, "oracle", "oracle.c"), "-std=c11")
    for f in ("encode.cpp", "capi.cpp"):
        cc("g++", os.path.join(csrc, f), "-std=c++17", ["-pthread", "-ffp-contract=off"])
    cc("g++", os.path.join(ROOT, "tests", "sanitize", "genc_stub.cpp"), "-std=c++17")
    cc("g++", os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"), "-std=c++17")
    driver = str(d / "host_driver")
    subprocess.check_call(["g++", *SAN, "-pthread", *objs, "-lm", "-o", driver])
    lib = str(d / "liboracle_san.so")
    subprocess.check_call(["gcc", *SAN, "-std=c11", "-shared", "-fPIC",
                           os.path.join(ROOT, "oracle", "oracle.c"), "-lm", "-o", lib])
    return dict(driver=driver, oracle=lib)


def test_host_code_under_sanitizers(sanbuild):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([sanbuild["driver"], "4000"], capture_output=True, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "sanitized host run: ok" in r.stdout
    assert "encode cases: 14" in r.stdout


def test_oracle_pins_under_sanitizers(sanbuild):
    preload = ":".join([_gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")])
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0",
               ORACLE_LIB=sanbuild["oracle"])
    tests = [os.path.join(ROOT, "tests", f) for f in
             ("test_oracle_lattice.py", "test_oracle_model.py", "test_second_decoder.py",
              "test_oracle_rdo.py", "test_oracle_gemm.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:xdist", *tests],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert " passed" in r.stdout and "failed" not in r.stdout
