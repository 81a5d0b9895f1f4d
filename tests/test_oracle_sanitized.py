"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): the whole pin suite (``test_oracle.py``) runs again in a child
process against that build, and must pass with no sanitizer report (any
out-of-bounds access, use after free or undefined arithmetic in the oracle's
C ends the child with a report).

The instrumented library replaces the default one through the oracle
package's ``IABN_ORACLE_LIB``; the sanitizer runtimes are preloaded into the
child's Python so that numpy's buffers, which the oracle reads and writes,
are tracked as well.  Leak checking is off (the interpreter itself keeps
memory until exit)."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "iabn_oracle.c")


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _run_pins(tmp_path, src):
    """Builds ``src`` with the sanitizers and runs the pin suite against it;
    returns (completed process, sanitizer report text)."""
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("gcc's sanitizer runtimes are not installed")
    lib = str(tmp_path / "liboracle_iabn_sanitized.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer", "-ffp-contract=off", "-Wall", "-Wextra",
                    "-o", lib, src, "-lm"], check=True)
    env = dict(os.environ)
    env.update({
        "IABN_ORACLE_LIB": lib,
        "LD_PRELOAD": asan + ":" + ubsan,
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:log_path=" + str(tmp_path / "asan"),
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1:log_path=" + str(tmp_path / "ubsan"),
        "OMP_NUM_THREADS": "4",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    reports = sorted(p for p in os.listdir(tmp_path) if p.startswith(("asan", "ubsan")))
    return r, "".join(open(tmp_path / p).read() for p in reports)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_pin_suite_under_sanitizers(tmp_path):
    r, reports = _run_pins(tmp_path, SRC)
    assert not reports, "sanitizer reports:\n" + reports[:4000]
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_sanitizers_catch_a_planted_overrun(tmp_path):
    """The same run over a copy of the oracle whose batch statistics read one
    element past each row: the child must end with an AddressSanitizer report."""
    src = open(SRC).read()
    row_loop = "for (int64_t i = 0; i < HW; ++i) csum_add(&s, x[IDX(n, c, i)]);"
    assert src.count(row_loop) >= 1
    bad = tmp_path / "iabn_oracle_overrun.c"
    bad.write_text(src.replace(row_loop, row_loop.replace("i < HW", "i <= HW"), 1))
    r, reports = _run_pins(tmp_path, str(bad))
    assert r.returncode != 0
    assert "AddressSanitizer" in reports and "overflow" in reports, reports[:2000]
