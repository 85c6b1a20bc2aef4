"""The host ABI tests again, against a build of the library whose host code
carries AddressSanitizer and UndefinedBehaviorSanitizer: every validation
path of include/spec.h (bad configs, bad page tables, null contexts, workspace
sizing of every workload) runs with out-of-bounds, use-after-free and
undefined-behaviour checks on.  The build lands in _build/sanitize/ and is
reused while the sources are unchanged.  No GPU is needed."""
import hashlib
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT_DIR = os.path.join(ROOT, "_build", "sanitize")


def _digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


@pytest.fixture(scope="module")
def sanitized_lib():
    from paper_2606_31160_amd import build as PB
    if not os.path.exists(PB.hipcc()) and shutil.which(PB.hipcc()) is None:
        pytest.skip("hipcc not found")
    try:
        rt = PB.sanitizer_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    srcs = [os.path.join(PB.CSRC, f) for f in sorted(os.listdir(PB.CSRC))] + [os.path.join(ROOT, "include", "spec.h")]
    lib = os.path.join(OUT_DIR, f"libspecdec_asan_{_digest(srcs)}.so")
    if not os.path.exists(lib):
        os.makedirs(OUT_DIR, exist_ok=True)
        for old in os.listdir(OUT_DIR):
            if old.startswith("libspecdec_asan_"):
                os.remove(os.path.join(OUT_DIR, old))
        PB.build(sanitize=True, out=lib)
    return lib, rt


def test_host_abi_under_address_and_undefined_behaviour_sanitizers(sanitized_lib):
    lib, rt = sanitized_lib
    env = dict(os.environ)
    env.update({
        "SPECDEC_LIBRARY": lib,
        "LD_PRELOAD": rt,
        # the interpreter itself is not instrumented: its own allocations are
        # not leak-checked
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out and "failed" not in out, out[-2000:]
