"""Synthetic parameter-set recipes for the DASO synchronisation step.

The sync arithmetic never looks at data, only at the flattened parameter
vector of a network, so each workload is a list of tensor element counts
laid out densely in forward order, plus a bucket plan and the DASO knobs
(g node-local replicas, P exchanged copies, staleness S per bucket).

The networks are the ones the paper trains in its evaluation (Section 4:
ResNet-50 on ImageNet, a multi-scale attention segmentation network on
CityScapes), plus a smaller ResNet-18 and a GPT-2-medium-shaped stress case.
Only shapes are reproduced; no weights, no data.

Bucketing follows the "tensor fusion" / bucketing idea the paper names for
Horovod and DDP (Sections 2 and 4): tensors are walked from the last to the
first, and a bucket is closed as soon as it holds at least ``cap`` elements
(25 MiB of fp32 = 6,553,600 elements by default); whatever is left forms the
last bucket.  Bucket ``b`` is the b-th bucket of that walk, so bucket 0 sits at
the end of the flat buffer.

This module holds no DASO arithmetic: it only describes inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

BUCKET_CAP_ELEMS = 25 * 1024 * 1024 // 4  # 25 MiB of fp32


# ----------------------------------------------------------------- shapes
def _bn(c: int) -> List[int]:
    """BatchNorm affine parameters: weight and bias vectors."""
    return [c, c]


def resnet18_numels() -> List[int]:
    """torchvision-style ResNet-18 parameter tensors in forward order."""
    t = [64 * 3 * 7 * 7] + _bn(64)
    cin = 64
    for width, stride_block in ((64, False), (128, True), (256, True), (512, True)):
        for blk in range(2):
            first_in = cin if blk == 0 else width
            t += [width * first_in * 9] + _bn(width)
            t += [width * width * 9] + _bn(width)
            if blk == 0 and stride_block:
                t += [width * first_in] + _bn(width)
        cin = width
    t += [1000 * 512, 1000]
    return t


def resnet50_numels() -> List[int]:
    """torchvision-style ResNet-50 (bottleneck [3,4,6,3], expansion 4)."""
    t = [64 * 3 * 7 * 7] + _bn(64)
    cin = 64
    for width, nblocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        out = 4 * width
        for blk in range(nblocks):
            first_in = cin if blk == 0 else out
            t += [width * first_in] + _bn(width)
            t += [width * width * 9] + _bn(width)
            t += [out * width] + _bn(out)
            if blk == 0:
                t += [out * first_in] + _bn(out)
        cin = out
    t += [1000 * 2048, 1000]
    return t


# (kernel size, cin, cout, count) for the segmentation-shaped recipe.
_SEG_CONVS: Tuple[Tuple[int, int, int, int], ...] = (
    (3, 48, 48, 150), (3, 96, 96, 96), (3, 192, 192, 48), (3, 384, 384, 26),
    (1, 720, 512, 4),
    (1, 96, 48, 46), (1, 192, 48, 46), (1, 384, 48, 46),
    (1, 192, 96, 46), (1, 384, 96, 46), (1, 384, 192, 46),
)


def segnet_numels() -> List[int]:
    """Multi-scale-attention-style segmentation net: 600 convs, each followed by
    BatchNorm weight and bias, emitted round-robin over the conv kinds until every
    kind's count is used up (3x3 and 1x1 convs, 48..720 channels)."""
    left = [c for (_, _, _, c) in _SEG_CONVS]
    t: List[int] = []
    while any(left):
        for i, (k, cin, cout, _) in enumerate(_SEG_CONVS):
            if left[i]:
                left[i] -= 1
                t += [cout * cin * k * k] + _bn(cout)
    return t


def gpt_medium_numels(layers: int = 24, d: int = 1024, vocab: int = 50257,
                      ctx: int = 1024) -> List[int]:
    """GPT-2-medium-shaped transformer: embeddings, 24 blocks of LayerNorm,
    fused QKV, attention projection, 4d MLP (weights and biases), final LayerNorm."""
    t = [vocab * d, ctx * d]
    for _ in range(layers):
        t += [d, d]                       # ln1
        t += [3 * d * d, 3 * d]           # qkv
        t += [d * d, d]                   # attention out-projection
        t += [d, d]                       # ln2
        t += [4 * d * d, 4 * d]           # mlp fc
        t += [d * 4 * d, d]               # mlp projection
    t += [d, d]                           # ln_f
    return t


# ---------------------------------------------------------------- buckets
@dataclass(frozen=True)
class Bucket:
    """A contiguous element range [start, start+numel) with staleness S."""
    start: int
    numel: int
    S: int


def tensor_offsets(numels: Sequence[int]) -> List[int]:
    """Start element of each tensor in the dense forward-order flat layout."""
    off, acc = [], 0
    for n in numels:
        off.append(acc)
        acc += n
    return off


def plan_buckets(numels: Sequence[int], cap: int = BUCKET_CAP_ELEMS) -> List[Tuple[int, int]]:
    """(start, numel) of each bucket, in walk order (last tensor first).

    Tensors are taken from the end of the flat buffer towards its start; a
    bucket closes as soon as its element count reaches ``cap``."""
    offs = tensor_offsets(numels)
    out: List[Tuple[int, int]] = []
    end = sum(numels)
    size = 0
    for i in range(len(numels) - 1, -1, -1):
        size += numels[i]
        if size >= cap:
            out.append((offs[i], end - offs[i]))
            end = offs[i]
            size = 0
    if size:
        out.append((0, end))
    return out


# ---------------------------------------------------------------- configs
@dataclass(frozen=True)
class Workload:
    name: str
    index: int                      # position in the list below; feeds the seeds
    numels: Tuple[int, ...]
    g: int                          # node-local replicas whose grads are averaged
    P: int                          # exchanged stale copies merged by Eq. (1)
    S_cycle: Tuple[int, ...]        # S of bucket b is S_cycle[b % len(S_cycle)]
    stale_sigma_per_S: bool         # stale perturbation sigma = 1e-4 * S_b if True, else 1e-4
    lr: float = 0.1
    mu: float = 0.9
    wd: float = 0.0
    cap: int = BUCKET_CAP_ELEMS
    buckets: Tuple[Bucket, ...] = field(default=())

    @property
    def n(self) -> int:
        return int(sum(self.numels))


def _mk(name, index, numels, g, P, S_cycle, per_S, single_bucket=False) -> Workload:
    numels = tuple(int(x) for x in numels)
    if single_bucket:
        plan = [(0, sum(numels))]
    else:
        plan = plan_buckets(numels)
    bks = tuple(Bucket(s, k, S_cycle[b % len(S_cycle)]) for b, (s, k) in enumerate(plan))
    return Workload(name, index, numels, g, P, tuple(S_cycle), per_S, buckets=bks)


def all_workloads() -> List[Workload]:
    return [
        _mk("tiny", 0, [65536], 4, 2, (1,), False, single_bucket=True),
        _mk("resnet18", 1, resnet18_numels(), 4, 4, (2,), False),
        _mk("resnet50", 2, resnet50_numels(), 4, 8, (4,), True),
        _mk("segnet", 3, segnet_numels(), 4, 16, (4,), True),
        _mk("gpt_medium", 4, gpt_medium_numels(), 8, 32, (1, 2, 4, 8), True),
    ]


def workload(name: str) -> Workload:
    for w in all_workloads():
        if w.name == name:
            return w
    raise KeyError(name)


def custom_workload(n: int, g: int, P: int, buckets: Sequence[Tuple[int, int, int]],
                    name: str = "custom", index: int = 99, sigma_per_S: bool = True,
                    lr: float = 0.1, mu: float = 0.9, wd: float = 0.0) -> Workload:
    """An ad-hoc workload with explicit (start, numel, S) buckets covering [0, n)."""
    bks = tuple(Bucket(int(s), int(k), int(S)) for (s, k, S) in buckets)
    return Workload(name, index, (int(n),), g, P, tuple(b.S for b in bks) or (0,),
                    sigma_per_S, lr, mu, wd, buckets=bks)


def algorithmic_bytes_per_param(g: int, P: int) -> int:
    """Bytes the fused step must move per parameter, each stream counted once:
    g fp32 grads read, params and momentum read and written (fp32),
    P bf16 stale copies read, one bf16 wire element written."""
    return 4 * g + 4 + 4 + 2 * P + 4 + 4 + 2
