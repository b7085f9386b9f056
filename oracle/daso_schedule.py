"""Plain reference of DASO's phase and exchange schedule (Section 3).

TEST INFRASTRUCTURE ONLY: used by the tests to check the library's native
controller; nothing in the product path imports it.

What the paper states:
  * training has three phases over a fixed number of epochs: warm-up and
    cool-down (a chosen count of opening and closing epochs) use blocking
    global synchronisation; the cycling phase between them is non-blocking;
  * in the blocking case all synchronisation steps happen after each batch;
  * in cycling, B forward-backward passes separate global synchronisations and
    the exchanged states are used W batches later, merged by Eq. (1) with S = W;
  * B is set by hand, W starts at B/4;
  * whenever the loss stops improving B and W are halved, never below one; a
    further plateau with both at one restores their starting values;
  * the groups (one GPU per node with the same local rank) take turns at the
    global exchange, and the member that merged hands the result to the other
    GPUs of its node.

Readings where the text is silent (the same as the library's):
  * W starts at max(1, B // 4) unless given;
  * a plateau is `patience` consecutive cycling epochs whose loss is not below
    best - tol * |best|, best being the last loss that was; after a change the
    count restarts; new B and W apply from the next epoch (the count of batches
    since the last exchange restarts with them);
  * the first cycling exchange starts after the B-th cycling batch;
  * an exchange is not started if its copies would arrive after the last cycling
    batch, or in a batch where another exchange's copies arrive;
  * blocking exchanges rotate between the groups too, one per batch.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

WARMUP, CYCLING, COOLDOWN = 0, 1, 2
SEND, MERGE, BLOCKING, RECV_BCAST = 1, 2, 4, 8


@dataclass
class Config:
    total_epochs: int
    warmup_epochs: int
    cooldown_epochs: int
    batches_per_epoch: int
    B_init: int
    W_init: int = 0          # 0: B_init // 4, at least 1
    group_count: int = 1
    local_rank: int = 0
    patience: int = 1
    plateau_rel_tol: float = 0.0


def phase_of(cfg: Config, epoch: int) -> int:
    if epoch < cfg.warmup_epochs:
        return WARMUP
    if epoch >= cfg.total_epochs - cfg.cooldown_epochs:
        return COOLDOWN
    return CYCLING


def plan_training(cfg: Config, losses: Sequence[float]) -> List[Dict[str, int]]:
    """Every batch's plan for this GPU, given the loss reported after each epoch."""
    E, nb, g, me = cfg.total_epochs, cfg.batches_per_epoch, cfg.group_count, cfg.local_rank
    W0 = cfg.W_init if cfg.W_init > 0 else max(1, cfg.B_init // 4)
    B, W = cfg.B_init, W0
    cycling_epochs = [e for e in range(E) if phase_of(cfg, e) == CYCLING]
    last_cycling_step = (cycling_epochs[-1] + 1) * nb - 1 if cycling_epochs else -1

    plans: List[Dict[str, int]] = []
    arriving: Dict[int, Tuple[int, int]] = {}   # step -> (group, S)
    exchanges = 0                               # exchanges started: whose turn it is
    since_start = 0                             # cycling batches since the last exchange started
    best = None
    flat = 0
    for epoch in range(E):
        phase = phase_of(cfg, epoch)
        for b in range(nb):
            t = epoch * nb + b
            plan = {"step": t, "epoch": epoch, "batch": b, "phase": phase, "B": B, "W": W,
                    "actions": 0, "S": -1, "sync_group": -1, "merge_group": -1}
            if t in arriving:                   # copies sent S batches ago arrive now
                grp, S = arriving.pop(t)
                plan["merge_group"], plan["S"] = grp, S
                plan["actions"] |= MERGE if grp == me else RECV_BCAST
            if phase == CYCLING:
                since_start += 1
                if since_start == B:
                    since_start = 0
                    arrive = t + W
                    if arrive <= last_cycling_step and arrive not in arriving:
                        grp = exchanges % g
                        exchanges += 1
                        arriving[arrive] = (grp, W)
                        plan["sync_group"] = grp
                        if grp == me:
                            plan["actions"] |= SEND
            else:                               # blocking: average now, S = 0
                grp = exchanges % g
                exchanges += 1
                plan["sync_group"] = plan["merge_group"] = grp
                plan["S"] = 0
                plan["actions"] |= BLOCKING if grp == me else RECV_BCAST
            plans.append(plan)

        # the epoch's loss decides B and W for the next epoch
        if phase != CYCLING:
            continue
        loss = losses[epoch]
        if best is None or loss < best - cfg.plateau_rel_tol * abs(best):
            best, flat = loss, 0
            continue
        flat += 1
        if flat < cfg.patience:
            continue
        flat = 0
        if B == 1 and W == 1:
            newB, newW = cfg.B_init, W0
        else:
            newB, newW = max(1, B // 2), max(1, W // 2)
        if (newB, newW) != (B, W):
            since_start = 0
        B, W = newB, newW
    return plans
