"""Plain CPU oracle of the DASO parameter-synchronisation step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests, the smoke check and the CPU-baseline leg of the bench
use it.  It shares no code with the HIP kernels or the C ABI.

What it computes (arXiv 2104.05588), per parameter element j, with every
floating-point operation written out as one IEEE-754 binary32 operation
(round to nearest even, no fused multiply-add, subnormals kept), in a fixed
order so that a GPU implementation can reproduce the same bits:

  1. local synchronisation (Section 3, Figure 2): the gradients of the g
     node-local replicas are averaged and every replica takes the average:
         s = G_0 ; s = s + G_r for r = 1..g-1 ; gbar = s / g
  2. the node-local optimizer step (Section 3.1: a PyTorch optimizer such as
     SGD; Section 4: momentum 0.9, weight decay 1e-4), PyTorch SGD semantics
     with zero dampening and no Nesterov term:
         d  = gbar                     (wd == 0)
         d  = gbar + (wd * x)          (wd != 0)
         m' = (mu * m) + d
         xl = x - (lr * m')
  3. the staleness-weighted merge of Eq. (1) (Section 3; restated in the
     appendix's convergence proof) of the local state with the P exchanged
     model states that arrive S batches late:
         x' = (2S * xl + sum_{i=1..P} x_i) / (2S + P)
     computed as a = (2S) * xl ; a = a + x_i for i = 1..P ; x' = a / (2S + P);
     with P = 0 the merge is the identity.  S = 0 (blocking synchronisation)
     is the plain average: a = x_1 ; a = a + x_i for i = 2..P ; x' = a / P.
     The x_i arrive as bf16 and are widened exactly (bits << 16).
  4. buffer packaging for the exchange (Section 3: the send buffer holds a
     16-bit rendering of the parameters, widened again by the receiver;
     Section 4: DASO uses bfloat16): wire = bf16_rne(x').

The fp32 exchange (Section 3: without blocking, the cast would only hold back
the send, so the parameters go out uncast) keeps the same arithmetic with
binary32 copies: widen() is the identity and the wire is x' itself.

Readings taken where the paper is silent (each also listed in the design
notes of the repository): the local state entering Eq. (1) is the state after
this batch's optimizer step; S is per bucket; the momentum buffer is neither
merged nor exchanged; NaN packs to the quiet NaN 0x7FC0; the packed value is
the merged state (a flag selects the pre-merge local state instead).

Side outputs (not in the paper; defined for monitoring): per bucket, the sum
of gbar^2, the sum of (x' - xl)^2 (both in float64) and the number of
non-finite x'.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F32 = np.float32
QNAN_BF16 = np.uint16(0x7FC0)

PACK_PRE_MERGE = 1  # pack the post-step, pre-merge local state instead of x'


# ------------------------------------------------------------------ bf16
def bf16_rne(x) -> np.ndarray:
    """binary32 -> bfloat16 bit patterns, round to nearest, ties to even.

    bfloat16 keeps the top 16 bits of a binary32 value.  Adding 0x7FFF plus the
    lowest kept bit to the pattern and truncating rounds to nearest with ties to
    the even pattern; a carry out of the mantissa moves to the next binade and,
    from the largest finite value, to infinity, as IEEE-754 requires.  NaN maps
    to the quiet NaN 0x7FC0."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    kept_lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + kept_lsb) >> np.uint64(16)).astype(np.uint16)
    r[np.isnan(x)] = QNAN_BF16
    return r


def bf16_widen(h) -> np.ndarray:
    """bfloat16 bit patterns -> binary32, exact (the pattern becomes the top half)."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------- the steps
def local_avg(grads: Sequence[np.ndarray]) -> np.ndarray:
    """Local synchronisation (Section 3, Figure 2): mean of the g replica
    gradients, summed in replica order, then one division by g."""
    g = len(grads)
    if g < 1:
        raise ValueError("need at least one replica gradient")
    s = np.array(grads[0], dtype=np.float32, copy=True)
    for r in range(1, g):
        s = s + np.asarray(grads[r], dtype=np.float32)
    return s / F32(g)


def sgd_momentum(x: np.ndarray, m: np.ndarray, gbar: np.ndarray,
                 lr: float, mu: float, wd: float) -> Tuple[np.ndarray, np.ndarray]:
    """One node-local SGD step with momentum (Sections 3.1 and 4).

    Returns (xl, m').  Weight decay is the coupled L2 form added to the
    gradient; with wd == 0 it is skipped entirely."""
    x = np.asarray(x, dtype=np.float32)
    m = np.asarray(m, dtype=np.float32)
    d = np.asarray(gbar, dtype=np.float32)
    if wd != 0.0:
        d = d + (F32(wd) * x)
    m_new = (F32(mu) * m) + d
    xl = x - (F32(lr) * m_new)
    return xl, m_new


def _received(st: np.ndarray) -> np.ndarray:
    """An exchanged state as binary32: bf16 patterns (uint16) are widened
    exactly, binary32 copies (fp32 exchange) are taken as they are."""
    st = np.asarray(st)
    if st.dtype == np.float32:
        return st
    if st.dtype != np.uint16:
        raise TypeError("exchanged states are uint16 bf16 patterns or float32")
    return bf16_widen(st)


def merge_eq1(xl: np.ndarray, stale: Sequence[np.ndarray], S: int) -> np.ndarray:
    """Eq. (1): staleness-weighted average of the local state xl with the P
    exchanged states (bf16 bit patterns or fp32), local weight 2S, each copy
    weight 1.

    S = 0 is the blocking global synchronisation of the warm-up and cool-down
    phases (Section 3): the result is the plain average of the P exchanged
    states (this GPU's own state is one of them), so the local term is left
    out rather than multiplied by zero, and a non-finite local state does not
    reach the result."""
    if S < 0:
        raise ValueError("S must be >= 0")
    P = len(stale)
    xl = np.asarray(xl, dtype=np.float32)
    if P == 0:
        return xl.copy()
    if S == 0:
        a = np.array(_received(stale[0]), dtype=np.float32, copy=True)
        rest = stale[1:]
    else:
        a = F32(2 * S) * xl
        rest = stale
    for st in rest:
        a = a + _received(st)
    return a / F32(2 * S + P)


def _check_buckets(n: int, buckets: Sequence[Tuple[int, int, int]]) -> None:
    spans = sorted((int(s), int(k)) for (s, k, _) in buckets)
    pos = 0
    for s, k in spans:
        if s != pos or k < 0:
            raise ValueError("buckets must tile [0, n) without gaps or overlaps")
        pos = s + k
    if pos != n:
        raise ValueError("buckets must tile [0, n) without gaps or overlaps")
    for (_, _, S) in buckets:
        if int(S) < 0:
            raise ValueError("S must be >= 0")


# -------------------------------------------------- operations of the ABI
def pack_bf16(x: np.ndarray) -> np.ndarray:
    """Buffer packaging: the wire holds bf16_rne of every parameter."""
    return bf16_rne(x)


def _pack(x: np.ndarray, exchange: str) -> np.ndarray:
    if exchange == "bf16":
        return bf16_rne(x)
    if exchange == "f32":
        return np.array(x, dtype=np.float32, copy=True)
    raise ValueError("exchange is 'bf16' or 'f32'")


def global_merge(params: np.ndarray, stale: Sequence[np.ndarray],
                 buckets: Sequence[Tuple[int, int, int]],
                 pack: bool = False, exchange: str = "bf16") -> Tuple[np.ndarray, Optional[np.ndarray]]:
    """Eq. (1) applied bucket by bucket with each bucket's own S; optionally
    packs the merged parameters in the exchange type.  Returns (x', wire or None)."""
    x = np.asarray(params, dtype=np.float32)
    n = x.shape[0]
    _check_buckets(n, buckets)
    _check_exchange(stale, exchange)
    out = np.empty(n, np.float32)
    for (s, k, S) in buckets:
        sl = slice(int(s), int(s) + int(k))
        out[sl] = merge_eq1(x[sl], [st[sl] for st in stale], int(S))
    return out, (_pack(out, exchange) if pack else None)


def _check_exchange(stale: Sequence[np.ndarray], exchange: str) -> None:
    want = {"bf16": np.uint16, "f32": np.float32}.get(exchange)
    if want is None:
        raise ValueError("exchange is 'bf16' or 'f32'")
    for st in stale:
        if np.asarray(st).dtype != want:
            raise TypeError(f"{exchange} exchange takes {np.dtype(want).name} copies")


def fused_sync_step(grads: Sequence[np.ndarray], params: np.ndarray, momentum: np.ndarray,
                    stale: Sequence[np.ndarray], buckets: Sequence[Tuple[int, int, int]],
                    lr: float, mu: float, wd: float = 0.0, flags: int = 0,
                    exchange: str = "bf16") -> Dict[str, object]:
    """One DASO synchronisation step for one GPU's parameters: local gradient
    average, SGD-momentum step, Eq. (1) merge per bucket, pack for the exchange
    (bf16, or fp32 for the non-blocking path), and the per-bucket side outputs.
    Inputs are not modified."""
    x = np.asarray(params, dtype=np.float32)
    n = x.shape[0]
    _check_buckets(n, buckets)
    _check_exchange(stale, exchange)
    gbar = local_avg(grads)
    xl, m_new = sgd_momentum(x, momentum, gbar, lr, mu, wd)
    x_new = np.empty(n, np.float32)
    stats: List[Tuple[float, float, int]] = []
    for (s, k, S) in buckets:
        sl = slice(int(s), int(s) + int(k))
        x_new[sl] = merge_eq1(xl[sl], [st[sl] for st in stale], int(S))
        stats.append(bucket_stats(gbar[sl], xl[sl], x_new[sl]))
    wire = _pack(xl if (flags & PACK_PRE_MERGE) else x_new, exchange)
    return {"params": x_new, "momentum": m_new, "wire": wire, "grad_avg": gbar,
            "x_local": xl, "stats": stats}


def bucket_stats(gbar: np.ndarray, xl: np.ndarray, x_new: np.ndarray) -> Tuple[float, float, int]:
    """Side outputs of one bucket: (sum gbar^2, sum (x' - xl)^2, #non-finite x'),
    the sums taken in float64 from the binary32 values."""
    g64 = np.asarray(gbar, dtype=np.float64)
    dlt = np.asarray(x_new, dtype=np.float64) - np.asarray(xl, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        gsq = float(np.sum(g64 * g64))
        dsq = float(np.sum(dlt * dlt))
    nonfinite = int(np.count_nonzero(~np.isfinite(x_new)))
    return gsq, dsq, nonfinite
