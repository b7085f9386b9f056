"""DASO end to end through the C ABI alone (tests/c/daso_cluster_capi.c): the
native schedule controllers of four simulated nodes and the fused kernels run
six epochs with no Python in the loop; the C program's final parameters and
momentum must equal, bit for bit, an oracle simulation of the same training
built from the CPU oracle and the reference schedule."""
import os
import struct
import subprocess

import numpy as np
import pytest

from oracle import daso_oracle as O
from oracle import daso_schedule as OS
from paper_2104_05588_amd import build as B

F32 = np.float32


def _program():
    if not os.path.exists(B.CAPI_CLUSTER) or not os.path.exists(B.LIB):
        B.build()
    return B.CAPI_CLUSTER


def _oracle_cluster(cfg, losses, spans, x0, grads, lr, mu):
    """Every node runs the oracle's fused step each batch; sent wires are
    merged S batches later (Eq. (1)); blocking exchanges average at once."""
    plans = OS.plan_training(cfg, losses)
    nodes = len(x0)
    xs = [x.copy() for x in x0]
    ms = [np.zeros_like(x) for x in x0]
    sent = {}
    for t, plan in enumerate(plans):
        acts = plan["actions"]
        merge = bool(acts & OS.MERGE)
        S = plan["S"] if merge else 0
        bks = [(s, k, S) for (s, k) in spans]
        wires = []
        for k in range(nodes):
            out = O.fused_sync_step(grads[t][k], xs[k], ms[k], sent[t - S] if merge else [], bks, lr, mu)
            xs[k], ms[k] = out["params"], out["momentum"]
            wires.append(out["wire"])
        if acts & OS.BLOCKING:
            for k in range(nodes):
                xs[k] = O.global_merge(xs[k], wires, [(s, kk, 0) for (s, kk) in spans])[0]
        if acts & OS.SEND:
            sent[t] = wires
    return xs, ms, [p["actions"] for p in plans]


def test_c_program_is_built_and_checks_its_arguments():
    res = subprocess.run([_program()], capture_output=True, text=True, timeout=60)
    assert res.returncode == 2 and "usage" in res.stderr


@pytest.mark.gpu
def test_c_program_runs_daso_end_to_end(tmp_path):
    exe = _program()
    nodes, g, n = 4, 4, 10_007
    spans = [(0, 4_001), (4_001, n - 4_001)]
    E, warm, cool, nb, Bi, Wi, pat, tol = 6, 1, 1, 6, 4, 2, 1, 0.0
    lr, mu = F32(0.1), F32(0.9)
    losses = [1.0, 0.9, 0.9, 0.9, 0.8, 0.8]       # plateaus in the cycling epochs change B and W
    rng = np.random.default_rng(4242)
    x0 = [(rng.standard_normal(n) * 0.02).astype(F32) for _ in range(nodes)]
    grads = [[[(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(g)] for _ in range(nodes)]
             for _ in range(E * nb)]

    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(inp, "wb") as f:
        f.write(struct.pack("<11i", nodes, g, n, len(spans), E, warm, cool, nb, Bi, Wi, pat))
        f.write(struct.pack("<dff", tol, lr, mu))
        for (s, k) in spans:
            f.write(struct.pack("<qq", s, k))
        f.write(np.asarray(losses, np.float64).tobytes())
        for x in x0:
            f.write(x.tobytes())
        for t in range(E * nb):
            for k in range(nodes):
                for r in range(g):
                    f.write(grads[t][k][r].tobytes())
    print("[case] C program, 4 nodes x 6 epochs", flush=True)
    res = subprocess.run([exe, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr

    raw = open(outp, "rb").read()
    got_x = [np.frombuffer(raw, F32, n, 4 * n * k) for k in range(nodes)]
    got_m = [np.frombuffer(raw, F32, n, 4 * n * (nodes + k)) for k in range(nodes)]
    got_acts = np.frombuffer(raw, np.int32, E * nb, 8 * n * nodes).tolist()

    cfg = OS.Config(E, warm, cool, nb, Bi, Wi, 1, 0, pat, tol)
    want_x, want_m, want_acts = _oracle_cluster(cfg, losses, spans, x0, grads, lr, mu)
    assert got_acts == want_acts
    for bit in (OS.BLOCKING, OS.SEND, OS.MERGE):          # every kind of batch occurred
        assert any(a & bit for a in want_acts), bit
    for k in range(nodes):
        assert np.array_equal(got_x[k].view(np.uint32), want_x[k].view(np.uint32)), k
        assert np.array_equal(got_m[k].view(np.uint32), want_m[k].view(np.uint32)), k
