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
                 stats: bool = False):
        self.schedule = schedule
        self.params = params
        self.momentum = momentum
        self.spans = [(int(s), int(k)) for (s, k) in bucket_spans]
        self.lr, self.mu, self.wd = float(lr), float(mu), float(weight_decay)
        n = params.numel()
        self.wire = torch.empty(n, dtype=torch.int16, device=params.device)
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
        wire = self.wire if acts & (L.ACT_SEND | L.ACT_BLOCKING) else None
        L.fused_sync_step(grads, self.params, self.momentum, stale, self._buckets(S), self.lr, self.mu, self.wd,
                          wire=wire, stats=self.stats)

    def blocking_average(self, copies: Sequence[torch.Tensor]) -> None:
        """Finish a blocking synchronisation: the parameters become the plain
        average (Eq. (1) with S = 0) of the group's P exchanged copies."""
        L.global_merge(self.params, list(copies), self._buckets(0))
