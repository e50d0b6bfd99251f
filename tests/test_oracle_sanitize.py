"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/c/oracle_sanitize.c includes oracle/lbi_oracle.c and runs it over its
whole interface against exact integer references; it is built here with
gcc -fsanitize=address,undefined (any report aborts the run) and must exit
0 with no sanitizer output.  A planted out-of-bounds read in a copy of the
oracle (on the CPU) shows that the build does catch such a mistake.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "c", "oracle_sanitize.c")
FLAGS = ["-std=gnu99", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-ffp-contract=off"]


def _have_sanitizers(tmp_path) -> bool:
    src = tmp_path / "probe.c"
    src.write_text("int main(void){return 0;}\n")
    res = subprocess.run(["gcc", *FLAGS, str(src), "-o", str(tmp_path / "probe")],
                         capture_output=True, text=True)
    return res.returncode == 0


def _build_and_run(tmp_path, driver_src):
    exe = tmp_path / "oracle_sanitize"
    res = subprocess.run(["gcc", *FLAGS, f"-I{os.path.join(ROOT, 'tests', 'c')}", str(driver_src),
                          "-o", str(exe), "-lm"], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="4")
    return subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)


@pytest.fixture
def sanitizers(tmp_path):
    if shutil.which("gcc") is None or not _have_sanitizers(tmp_path):
        pytest.skip("gcc with AddressSanitizer/UBSan not available")


def test_oracle_under_address_and_undefined_sanitizers(tmp_path, sanitizers):
    run = _build_and_run(tmp_path, DRIVER)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out
    assert "Sanitizer" not in out and "runtime error" not in out, out
    assert "all checks passed" in run.stdout


def test_sanitizer_build_catches_a_planted_overread(tmp_path, sanitizers):
    """The same driver over a copy of the oracle whose recurrence reads one
    element past lambda_K: the sanitized build must report it."""
    src = open(os.path.join(ROOT, "oracle", "lbi_oracle.c")).read()
    bad = src.replace("x[i] = widen(lamK, dtype, beta * r + i);",
                      "x[i] = widen(lamK, dtype, beta * r + i + 1);")
    assert bad != src
    odir = tmp_path / "oracle"
    odir.mkdir()
    (odir / "lbi_oracle.c").write_text(bad)
    cdir = tmp_path / "tests" / "c"
    cdir.mkdir(parents=True)
    drv = open(DRIVER).read()
    (cdir / "oracle_sanitize.c").write_text(drv)
    run = _build_and_run(tmp_path, cdir / "oracle_sanitize.c")
    assert run.returncode != 0
    assert "AddressSanitizer" in run.stdout + run.stderr
