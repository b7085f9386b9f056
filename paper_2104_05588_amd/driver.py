"""One GPU's DASO synchronisation, batch by batch (Section 3).

`DasoSync` asks the native schedule (daso_schedule_*) what the coming batch
does and runs the matching library calls on this GPU's flat buffers:

  * every batch: local gradient average over the g replicas and the SGD step;
  * DASO_ACT_SEND: the step's state is packed into the wire for a
    non-blocking exchange, which the caller posts;
  * DASO_ACT_MERGE: the copies sent S batches ago have arrived; they are merged
    with Eq. (1) and S = plan["S"], in the same pass as the step;
  * DASO_ACT_BLOCKING: the step's state is packed, the caller exchanges the
    wire within the group and hands the P copies (this GPU's own included) to
    blocking_average(), whose plain average (S = 0) becomes the state;
  * DASO_ACT_RECV_BCAST: the caller overwrites the parameters with the state
    its node's group member merged (the local update step).

With exchange="bf16" (the default) every exchange carries bf16 (Section 4:
DASO compresses to bfloat16).  With exchange="cast_blocking" only the blocking
exchanges are cast to bf16, while the non-blocking ones of the cycling phase
send the parameters uncast in fp32 (Section 3: casting would only hold back a
non-blocking send); self.wire is then the bf16 wire and self.wire_f32 the fp32
one, and the copies handed to step() must be of the type that was sent.

The exchanges themselves (the collectives) are the caller's: this module only
orders the kernel calls.  Every computation runs in the library's kernels.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import torch

from . import _lib as L


class DasoSync:
    def __init__(self, schedule: "L.Schedule", params: torch.Tensor, momentum: torch.Tensor,
                 bucket_spans: Sequence[Tuple[int, int]], lr: float, mu: float, weight_decay: float = 0.0,
                 stats: bool = False, exchange: str = "bf16"):
        if exchange not in ("bf16", "cast_blocking"):
            raise ValueError("exchange is 'bf16' or 'cast_blocking'")
        self.schedule = schedule
        self.params = params
        self.momentum = momentum
        self.spans = [(int(s), int(k)) for (s, k) in bucket_spans]
        self.lr, self.mu, self.wd = float(lr), float(mu), float(weight_decay)
        self.exchange = exchange
        n = params.numel()
        self.wire = torch.empty(n, dtype=torch.int16, device=params.device)
        self.wire_f32 = (torch.empty(n, dtype=torch.float32, device=params.device)
                         if exchange == "cast_blocking" else None)
        self.stats = L.new_stats(len(self.spans), device=params.device) if stats else None

    def next_plan(self) -> Optional[dict]:
        """The plan of the coming batch (None once training is over)."""
        return self.schedule.next_batch()

    def end_epoch(self, loss: float) -> None:
        self.schedule.end_epoch(loss)

    def _buckets(self, S: int) -> List[Tuple[int, int, int]]:
        return [(s, k, S) for (s, k) in self.spans]

    def step(self, plan: dict, grads: Sequence[torch.Tensor],
             arrived: Optional[Sequence[torch.Tensor]] = None) -> None:
        """This GPU's step for the batch described by `plan`: the local average of
        the g replica gradients and the SGD step, merged with the copies that
        arrived (required, and only allowed, with DASO_ACT_MERGE) and packed
        into self.wire when the plan sends or synchronises (blocking)."""
        acts = plan["actions"]
        merge = bool(acts & L.ACT_MERGE)
        if merge != (arrived is not None):
            raise ValueError("copies are passed exactly when the plan merges (DASO_ACT_MERGE)")
        stale = list(arrived) if merge else []
        S = plan["S"] if merge else 0
        uncast = self.exchange == "cast_blocking" and plan["phase"] == L.PHASE_CYCLING
        if uncast and any(c.dtype != torch.float32 for c in stale):
            raise ValueError("with exchange='cast_blocking' the cycling phase's copies are fp32")
        wire = None
        if acts & (L.ACT_SEND | L.ACT_BLOCKING):
            wire = self.wire_f32 if uncast else self.wire
        L.fused_sync_step(grads, self.params, self.momentum, stale, self._buckets(S), self.lr, self.mu, self.wd,
                          wire=wire, stats=self.stats)

    def fast_forward(self, batches: int, losses: Sequence[float]) -> None:
        """Resume a checkpointed run: bring this object's fresh controller to
        the point after `batches` batches.  The controller depends only on its
        configuration and the epoch losses, so replaying its plans, with the
        loss of every epoch completed within those batches, restores it.  The
        parameters, momentum and the copies still in flight are the caller's to
        restore."""
        nb = self.schedule.config.batches_per_epoch
        if int(batches) < 0:
            raise ValueError("batches must be >= 0")
        if len(losses) < int(batches) // nb:
            raise ValueError(f"{int(batches)} batches complete {int(batches) // nb} epochs, "
                             f"but only {len(losses)} epoch losses were given")
        for _ in range(int(batches)):
            plan = self.schedule.next_batch()
            if plan is None:
                raise ValueError("the schedule has fewer batches than that")
            if plan["batch"] == nb - 1:
                self.schedule.end_epoch(losses[plan["epoch"]])

    def blocking_average(self, copies: Sequence[torch.Tensor]) -> None:
        """Finish a blocking synchronisation: the parameters become the plain
        average (Eq. (1) with S = 0) of the group's P exchanged copies."""
        L.global_merge(self.params, list(copies), self._buckets(0))
