"""The bfloat16 packing rule over all 2^32 binary32 patterns (host C program
tests/c/bf16_exhaustive.c): its integer form against the nearest-value
definition, then the oracle against the definition on a spread sample.  No GPU."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import daso_oracle as O

SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "bf16_exhaustive.c")


def _build(tmp_path, name, *defs):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / name)
    omp = ["-fopenmp"] if subprocess.run([gcc, "-fopenmp", "-E", "-x", "c", "/dev/null"],
                                         capture_output=True).returncode == 0 else []
    subprocess.run([gcc, "-O2", "-std=c11", "-Wall", *omp, *defs, SRC, "-o", exe, "-lm"], check=True)
    return exe


def test_integer_form_equals_definition_on_every_pattern(tmp_path):
    exe = _build(tmp_path, "bf16x")
    res = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert res.stdout.strip() == "mismatches 0 checked 4294967296", res.stdout + res.stderr
    assert res.returncode == 0


def test_exhaustive_check_reports_a_planted_truncation(tmp_path):
    exe = _build(tmp_path, "bf16x_planted", "-DPLANT_TRUNCATION")
    res = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert res.returncode == 1
    assert int(res.stdout.split()[1]) > 10 ** 9


def test_oracle_matches_the_definition_on_a_spread_sample(tmp_path):
    exe = _build(tmp_path, "bf16x")
    stride, count = 65_521 * 1_031, 1 << 20            # odd stride: a spread of the 2^32 patterns
    res = subprocess.run([exe, "sample", str(stride), str(count)], capture_output=True, text=True, timeout=300)
    want = np.array([int(v, 16) for v in res.stdout.split()], dtype=np.uint16)
    u = (np.arange(count, dtype=np.uint64) * np.uint64(stride)) & np.uint64(0xFFFFFFFF)
    got = O.bf16_rne(u.astype(np.uint32).view(np.float32))
    assert want.shape == (count,)
    assert np.array_equal(got, want)
