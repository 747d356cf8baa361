"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(gcc, CPU only), every pin run against that build in a child process: an
out-of-bounds access, a use after free or undefined arithmetic anywhere the
pins reach ends the child with the sanitizer's report.  A copy of the oracle
with a planted out-of-bounds write shows that the child does fail when the
sanitizers find something."""
import os
import subprocess
import sys
import tempfile

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all"]

CHILD = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import oracle
from oracle_pins import ALL_PINS
lib = oracle.load({lib!r})
for pin in ALL_PINS:
    pin(lib)
    print(pin.__name__, "ok", flush=True)
"""


def _runtime():
    path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _build(src: str, out: str):
    flags = [f for f in oracle.CFLAGS if f != "-O2"]
    subprocess.check_call(["gcc", *flags, *SAN_FLAGS, src, "-o", out, "-lm"])


def _run_pins(lib_path: str):
    env = dict(os.environ)
    env["LD_PRELOAD"] = _runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib_path)
    return subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600)


@pytest.fixture(scope="module")
def runtime():
    if _runtime() is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")


def test_pins_pass_under_sanitizers(runtime):
    with tempfile.TemporaryDirectory() as tmp:
        lib = os.path.join(tmp, "liboracle_san.so")
        _build(os.path.join(os.path.dirname(oracle.__file__), "gmc_oracle.c"), lib)
        r = _run_pins(lib)
        assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
        assert r.stdout.count(" ok") == len(__import__("oracle_pins").ALL_PINS)
        assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr


def test_sanitizers_catch_a_planted_overrun(runtime):
    """The aggregation's accumulator one element short: the sanitized child
    must fail with AddressSanitizer's heap-buffer-overflow report."""
    with open(os.path.join(os.path.dirname(oracle.__file__), "gmc_oracle.c")) as f:
        src = f.read()
    old = "float* acc = (float*)malloc((size_t)(d > 0 ? d : 1) * sizeof(float));"
    assert src.count(old) == 1
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, "m.c")
        with open(path, "w") as f:
            f.write(src.replace(old, "float* acc = (float*)malloc((size_t)(d > 1 ? d - 1 : 1) * sizeof(float));"))
        lib = os.path.join(tmp, "liboracle_bad.so")
        _build(path, lib)
        r = _run_pins(lib)
        assert r.returncode != 0
        assert "AddressSanitizer" in r.stderr
