"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer, and the
C ABI's host-side size checks under UndefinedBehaviorSanitizer (CPU builds;
no device code runs).  The harnesses sit in tests/sanitize/."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = os.path.join(HERE, "sanitize")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    return r.returncode, r.stdout + r.stderr


@pytest.mark.parametrize("prime", [2**31 - 1, 15 * 2**27 + 1])
def test_oracle_under_asan_and_ubsan(tmp_path, prime):
    exe = str(tmp_path / "oracle_harness")
    rc, out = _run(["gcc", "-O1", "-g", "-std=c99", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", f"-DORC_P={prime}ULL", "-DORC_COUNT_OPS", "-o", exe,
                    os.path.join(SAN, "oracle_harness.c")])
    assert rc == 0, out
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    rc, out = _run([exe], env=env, timeout=300)
    assert rc == 0 and out.startswith("ok"), out


def test_abi_size_checks_under_ubsan(tmp_path):
    """The library's translation units built with UBSan on the host side only
    (device code is compiled as usual), linked with a harness that calls
    every size and argument check with extreme values."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    from paper_2609_10264_amd import build as B
    objs = []
    flags = [f for f in B.HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g", "-Xarch_host", "-fsanitize=undefined",
                                                          "-Xarch_host", "-fno-sanitize-recover=undefined"]
    srcs = B.sources()
    for src in srcs:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        rc, out = _run([hipcc, *flags, "-c", src, "-o", obj])
        assert rc == 0, out
        objs.append(obj)
    harness = str(tmp_path / "abi_harness.o")
    rc, out = _run([hipcc, *flags, "-x", "hip", "-c", os.path.join(SAN, "abi_harness.cpp"), "-o", harness])
    assert rc == 0, out
    exe = str(tmp_path / "abi_harness")
    rc, out = _run([hipcc, f"--offload-arch={B.ARCH}", "-fsanitize=undefined", "-o", exe, harness, *objs])
    assert rc == 0, out
    rc, out = _run([exe], timeout=120)
    assert rc == 0 and "ok" in out, out
