"""The C ABI used from plain C (tests/c/fused_step_capi.c): no Python, no torch
in the process that runs the step; its outputs are compared with the oracle."""
import os
import struct
import subprocess

import numpy as np
import pytest

from oracle import daso_oracle as O
from paper_2104_05588_amd import build as B
from workloads import generate as Gen
from workloads import recipes as R

F32 = np.float32


def _client():
    if not os.path.exists(B.CAPI_CLIENT) or not os.path.exists(B.LIB):
        B.build()
    return B.CAPI_CLIENT


def test_client_is_built_and_checks_its_arguments():
    exe = _client()
    res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert res.returncode == 2 and "usage" in res.stderr


def _write_case(path, inp, buckets, lr, mu, wd, flags=0):
    n = inp["params"].shape[0]
    g, P = len(inp["grads"]), len(inp["stale"])
    with open(path, "wb") as f:
        f.write(struct.pack("<qiiifffI", n, g, P, len(buckets), lr, mu, wd, flags))
        for (s, k, S) in buckets:
            f.write(struct.pack("<qqii", s, k, S, 0))
        for a in inp["grads"]:
            f.write(np.ascontiguousarray(a, F32).tobytes())
        f.write(np.ascontiguousarray(inp["params"], F32).tobytes())
        f.write(np.ascontiguousarray(inp["momentum"], F32).tobytes())
        for a in inp["stale"]:
            f.write(np.ascontiguousarray(a, np.uint16).tobytes())


def _read_out(path, n, nb):
    raw = open(path, "rb").read()
    x = np.frombuffer(raw, F32, n, 0)
    m = np.frombuffer(raw, F32, n, 4 * n)
    w = np.frombuffer(raw, np.uint16, n, 8 * n)
    st = np.frombuffer(raw, np.dtype([("g", "<f8"), ("d", "<f8"), ("nf", "<u8")]), nb, 10 * n)
    return x, m, w, [(float(r["g"]), float(r["d"]), int(r["nf"])) for r in st]


@pytest.mark.gpu
@pytest.mark.parametrize("case", ["tiny", "odd"])
def test_client_fused_step_matches_oracle(tmp_path, case):
    exe = _client()
    if case == "tiny":
        w = R.workload("tiny")
        inp = Gen.host_inputs(w)
        bks = [(b.start, b.numel, b.S) for b in w.buckets]
    else:
        rng = np.random.default_rng(9)
        n = 100_003
        x = (rng.standard_normal(n) * 0.02).astype(F32)
        inp = {"params": x, "momentum": (rng.standard_normal(n) * 1e-3).astype(F32),
               "grads": [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(3)],
               "stale": [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(5)]}
        bks = [(0, 40_001, 2), (40_001, 60_002, 0)]
    print(f"\n[case] C client {case} n={inp['params'].shape[0]}", flush=True)
    _write_case(tmp_path / "in.bin", inp, bks, 0.1, 0.9, 0.0)
    res = subprocess.run([exe, str(tmp_path / "in.bin"), str(tmp_path / "out.bin")], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    x, m, wire, stats = _read_out(tmp_path / "out.bin", inp["params"].shape[0], len(bks))
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
    assert np.array_equal(x.view(np.uint32), want["params"].view(np.uint32))
    assert np.array_equal(m.view(np.uint32), want["momentum"].view(np.uint32))
    assert np.array_equal(wire, want["wire"])
    for g_, w_ in zip(stats, want["stats"]):
        assert abs(g_[0] - w_[0]) <= 1e-10 * w_[0] and abs(g_[1] - w_[1]) <= 1e-10 * max(w_[1], 1e-300)
        assert g_[2] == w_[2]
