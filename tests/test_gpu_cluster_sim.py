"""DASO end to end on one GPU: a cluster of simulated nodes, each driven by the
native schedule through DasoSync, with exchanges simulated as buffer hand-offs
that land S batches later.  Every node's parameters and momentum must equal,
bit for bit, the same simulation built from the CPU oracle and the reference
schedule."""
import numpy as np
import pytest
import torch

import paper_2104_05588_amd as daso
from oracle import daso_oracle as O
from oracle import daso_schedule as OS

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.mark.parametrize("exchange", ["bf16", "cast_blocking"])
def test_simulated_cluster_matches_oracle(exchange):
    """exchange="bf16": every exchange in bf16; "cast_blocking": bf16 for the
    blocking exchanges only, fp32 for the non-blocking ones (Section 3)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nodes, g, n = 4, 4, 40_003
    spans = [(0, 15_001), (15_001, n - 15_001)]
    E, warm, cool, nb = 6, 1, 1, 6
    cfg = dict(total_epochs=E, warmup_epochs=warm, cooldown_epochs=cool, batches_per_epoch=nb, B_init=4,
               W_init=2, group_count=1, local_rank=0, patience=1, plateau_rel_tol=0.0)
    losses = [1.0, 0.9, 0.9, 0.9, 0.8, 0.8]          # plateaus in the cycling epochs change B and W
    plans_ref = OS.plan_training(OS.Config(**cfg), losses)

    rng = np.random.default_rng(2021)
    x0 = [(rng.standard_normal(n) * 0.02).astype(F32) for _ in range(nodes)]
    grads_all = [[[(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(g)] for _ in range(nodes)]
                 for _ in range(E * nb)]

    # GPU side
    syncs = [daso.DasoSync(daso.Schedule(**cfg), torch.from_numpy(x0[k].copy()).cuda(),
                           torch.zeros(n, device="cuda"), spans, 0.1, 0.9, exchange=exchange) for k in range(nodes)]
    sent = {}
    # oracle side
    xs = [x.copy() for x in x0]
    ms = [np.zeros(n, F32) for _ in range(nodes)]
    sent_ref = {}
    wire_ref = [None] * nodes                        # the oracle's wire of each node

    kinds = set()
    for t in range(E * nb):
        plans = [s.next_plan() for s in syncs]
        ref = plans_ref[t]
        assert all(p == ref for p in plans), (t, plans[0], ref)
        acts = ref["actions"]
        kinds.add(acts)
        merge = bool(acts & OS.MERGE)
        S = ref["S"] if merge else 0
        uncast = exchange == "cast_blocking" and ref["phase"] == OS.CYCLING
        bks = [(s, k, S) for (s, k) in spans]
        grads_dev = [[torch.from_numpy(a).cuda() for a in grads_all[t][k]] for k in range(nodes)]
        for k in range(nodes):
            syncs[k].step(ref, grads_dev[k], arrived=sent[t - S] if merge else None)
            out = O.fused_sync_step(grads_all[t][k], xs[k], ms[k], sent_ref[t - S] if merge else [], bks, 0.1, 0.9,
                                    exchange="f32" if uncast else "bf16")
            xs[k], ms[k] = out["params"], out["momentum"]
            if acts & (OS.SEND | OS.BLOCKING):
                wire_ref[k] = out["wire"]
        if acts & OS.BLOCKING:
            copies = [s.wire.clone() for s in syncs]
            copies_ref = list(wire_ref)
            for k in range(nodes):
                syncs[k].blocking_average(copies)
                xs[k] = O.global_merge(xs[k], copies_ref, [(s, kk, 0) for (s, kk) in spans])[0]
        if acts & OS.SEND:
            sent[t] = [(s.wire_f32 if uncast else s.wire).clone() for s in syncs]
            sent_ref[t] = list(wire_ref)
        if ref["batch"] == nb - 1:
            for s in syncs:
                s.end_epoch(losses[ref["epoch"]])
    torch.cuda.synchronize()
    for bit in (OS.BLOCKING, OS.SEND, OS.MERGE):     # every kind of batch occurred
        assert any(a & bit for a in kinds), (bit, kinds)
    for k in range(nodes):
        assert np.array_equal(syncs[k].params.cpu().numpy().view(np.uint32), xs[k].view(np.uint32)), k
        assert np.array_equal(syncs[k].momentum.cpu().numpy().view(np.uint32), ms[k].view(np.uint32)), k
    # the cluster stays together: after the blocking cool-down every node holds the same state
    for k in range(1, nodes):
        assert np.array_equal(xs[k], xs[0])


def test_checkpoint_and_resume_reproduce_the_uninterrupted_run():
    """Stop a simulated cluster after 20 of 36 batches (mid-epoch, with copies in
    flight), keep params, momentum and the sent copies, resume in fresh objects
    whose controllers are fast-forwarded with the losses seen so far: the final
    state equals the uninterrupted run's bit for bit."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nodes, g, n = 3, 2, 20_011
    spans = [(0, 9_001), (9_001, n - 9_001)]
    E, nb = 6, 6
    cfg = dict(total_epochs=E, warmup_epochs=1, cooldown_epochs=1, batches_per_epoch=nb, B_init=4,
               W_init=2, group_count=1, local_rank=0, patience=1, plateau_rel_tol=0.0)
    losses = [1.0, 0.9, 0.9, 0.9, 0.8, 0.8]
    rng = np.random.default_rng(77)
    x0 = [(rng.standard_normal(n) * 0.02).astype(F32) for _ in range(nodes)]
    grads = [[[torch.from_numpy((rng.standard_normal(n) * 1e-3).astype(F32)).cuda() for _ in range(g)]
              for _ in range(nodes)] for _ in range(E * nb)]

    def make(params, momentum):
        return [daso.DasoSync(daso.Schedule(**cfg), params[k], momentum[k], spans, 0.1, 0.9) for k in range(nodes)]

    def run(syncs, sent, first, last):
        for t in range(first, last):
            plan = syncs[0].next_plan()
            for s in syncs[1:]:
                assert s.next_plan() == plan
            acts = plan["actions"]
            merge = bool(acts & daso.ACT_MERGE)
            for k in range(nodes):
                syncs[k].step(plan, grads[t][k], arrived=sent[t - plan["S"]] if merge else None)
            if acts & daso.ACT_BLOCKING:
                copies = [s.wire.clone() for s in syncs]
                for s in syncs:
                    s.blocking_average(copies)
            if acts & daso.ACT_SEND:
                sent[t] = [s.wire.clone() for s in syncs]
            if plan["batch"] == nb - 1:
                for s in syncs:
                    s.end_epoch(losses[plan["epoch"]])

    print("[case] checkpoint and resume after 20 of 36 batches", flush=True)
    # the uninterrupted run
    whole = make([torch.from_numpy(x.copy()).cuda() for x in x0], [torch.zeros(n, device="cuda") for _ in x0])
    run(whole, {}, 0, E * nb)
    # the interrupted one: checkpoint after batch 20, resume in fresh objects
    part = make([torch.from_numpy(x.copy()).cuda() for x in x0], [torch.zeros(n, device="cuda") for _ in x0])
    sent = {}
    run(part, sent, 0, 20)
    torch.cuda.synchronize()
    ckpt = ([s.params.cpu().clone() for s in part], [s.momentum.cpu().clone() for s in part],
            {t: [c.cpu().clone() for c in cs] for t, cs in sent.items()})
    del part, sent
    resumed = make([p.cuda() for p in ckpt[0]], [m.cuda() for m in ckpt[1]])
    for s in resumed:
        s.fast_forward(20, losses)
    run(resumed, {t: [c.cuda() for c in cs] for t, cs in ckpt[2].items()}, 20, E * nb)
    torch.cuda.synchronize()
    for a, b in zip(whole, resumed):
        assert torch.equal(a.params.view(torch.int32), b.params.view(torch.int32))
        assert torch.equal(a.momentum.view(torch.int32), b.momentum.view(torch.int32))
