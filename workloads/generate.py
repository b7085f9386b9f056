"""Seeded synthetic inputs for the DASO synchronisation step.

Value recipe (per workload):
  params   ~ N(0, 0.02)                          fp32
  grads    g independent streams ~ N(0, 1e-3)    fp32
  stale    P streams: bf16(params + N(0, sigma)) with sigma = 1e-4, or
           1e-4 * S_b per bucket for the larger workloads (fresher copies for
           small staleness); rounding to bf16 uses torch's own cast
  momentum 0 (an optimizer's first step)

Two generators serve the two sizes of test:
  * ``host_inputs`` / ``host_bucket_inputs``: numpy PCG64, seeded per
    (workload, stream kind, stream index, bucket), so one bucket can be produced
    without the others (bounded host memory for the big workloads);
  * ``device_inputs``: torch's device generator, for full-size runs where a host
    generator would be too slow; oracle checks then gather sampled elements.

Nothing in here computes any part of the DASO step itself.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from .recipes import Workload

SEED_BASE = 210405588
KIND_PARAMS, KIND_GRAD, KIND_STALE = 0, 1, 2

PARAM_SIGMA = 0.02
GRAD_SIGMA = 1e-3
STALE_SIGMA = 1e-4


def stale_sigma(w: Workload, S: int) -> float:
    return STALE_SIGMA * S if (w.stale_sigma_per_S and S > 0) else STALE_SIGMA


def _rng(w: Workload, kind: int, idx: int, bucket: int) -> np.random.Generator:
    ss = np.random.SeedSequence([SEED_BASE, w.index, kind, idx, bucket])
    return np.random.Generator(np.random.PCG64(ss))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of a float32 array, via torch's CPU cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def host_bucket_inputs(w: Workload, b: int) -> Dict[str, object]:
    """Inputs restricted to bucket ``b`` of workload ``w`` (numpy, host)."""
    bk = w.buckets[b]
    k = bk.numel
    x = _rng(w, KIND_PARAMS, 0, b).standard_normal(k, dtype=np.float32) * np.float32(PARAM_SIGMA)
    grads = [_rng(w, KIND_GRAD, r, b).standard_normal(k, dtype=np.float32) * np.float32(GRAD_SIGMA)
             for r in range(w.g)]
    sig = np.float32(stale_sigma(w, bk.S))
    stale = []
    for i in range(w.P):
        z = _rng(w, KIND_STALE, i, b).standard_normal(k, dtype=np.float32) * sig
        stale.append(to_bf16_bits(x + z))
    return {"params": x, "momentum": np.zeros(k, np.float32), "grads": grads, "stale": stale}


def host_inputs(w: Workload) -> Dict[str, object]:
    """Full flat inputs of workload ``w`` on the host (small and medium sizes)."""
    n = w.n
    x = np.empty(n, np.float32)
    grads = [np.empty(n, np.float32) for _ in range(w.g)]
    stale = [np.empty(n, np.uint16) for _ in range(w.P)]
    for b, bk in enumerate(w.buckets):
        sl = slice(bk.start, bk.start + bk.numel)
        part = host_bucket_inputs(w, b)
        x[sl] = part["params"]
        for r in range(w.g):
            grads[r][sl] = part["grads"][r]
        for i in range(w.P):
            stale[i][sl] = part["stale"][i]
    return {"params": x, "momentum": np.zeros(n, np.float32), "grads": grads, "stale": stale}


def device_inputs(w: Workload, device: str = "cuda", seed: Optional[int] = None) -> Dict[str, object]:
    """Full flat inputs generated on the device with torch's generator.

    Returns torch tensors: params/momentum fp32 [n], grads list of g fp32 [n],
    stale list of P int16 [n] holding bf16 bit patterns."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(SEED_BASE * 100 + w.index if seed is None else seed)
    n = w.n
    x = torch.randn(n, generator=gen, device=device, dtype=torch.float32) * PARAM_SIGMA
    grads: List[object] = []
    for _ in range(w.g):
        grads.append(torch.randn(n, generator=gen, device=device, dtype=torch.float32) * GRAD_SIGMA)
    sig = torch.empty(n, device=device, dtype=torch.float32)
    for bk in w.buckets:
        sig[bk.start:bk.start + bk.numel] = stale_sigma(w, bk.S)
    stale: List[object] = []
    for _ in range(w.P):
        z = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
        stale.append((x + z * sig).to(torch.bfloat16).view(torch.int16))
    del sig
    return {"params": x, "momentum": torch.zeros(n, device=device, dtype=torch.float32),
            "grads": grads, "stale": stale}
