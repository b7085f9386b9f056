"""Thin ctypes binding of libdaso.so (declared in include/daso.h).

Argument marshalling only: tensors are checked for device, dtype, size and
contiguity, their device addresses and the current HIP stream cross the C ABI,
and every step of the computation runs in the library's kernels.  There is no
fallback: if the library is not built, or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdaso.so")

DASO_OK = 0
DASO_EINVAL = -1
DASO_EALIGN = -2
DASO_EALIAS = -3
DASO_EHIP = -4
DASO_ENOSPACE = -5
DASO_MAX_G = 64
DASO_MAX_P = 64
DASO_PACK_PRE_MERGE = 1
DASO_EXCHANGE_F32 = 2

EXPORTED = ("daso_local_avg", "daso_pack_bf16", "daso_global_merge", "daso_global_merge_f32",
            "daso_fused_sync_step", "daso_fused_sync_step_noalloc", "daso_fused_launch_config",
            "daso_plan_buckets", "daso_schedule_create", "daso_schedule_next",
            "daso_schedule_end_epoch", "daso_schedule_destroy", "daso_status_string", "daso_abi_version")
BUCKET_CAP_ELEMS = 25 * 1024 * 1024 // 4  # 25 MiB of fp32


class daso_bucket(ctypes.Structure):
    _fields_ = [("start", ctypes.c_int64), ("numel", ctypes.c_int64),
                ("S", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class daso_bucket_stats(ctypes.Structure):
    _fields_ = [("grad_sq", ctypes.c_double), ("delta_sq", ctypes.c_double),
                ("nonfinite", ctypes.c_uint64)]


class daso_sync_args(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("g", ctypes.c_int32), ("P", ctypes.c_int32),
        ("grads", ctypes.POINTER(ctypes.c_void_p)), ("stale", ctypes.POINTER(ctypes.c_void_p)),
        ("params", ctypes.c_void_p), ("momentum", ctypes.c_void_p),
        ("wire", ctypes.c_void_p), ("grad_avg", ctypes.c_void_p),
        ("buckets", ctypes.POINTER(daso_bucket)), ("nbuckets", ctypes.c_int32),
        ("lr", ctypes.c_float), ("mu", ctypes.c_float), ("weight_decay", ctypes.c_float),
        ("flags", ctypes.c_uint32), ("stats", ctypes.c_void_p),
        ("stale_f32", ctypes.POINTER(ctypes.c_void_p)), ("wire_f32", ctypes.c_void_p),
    ]


class daso_launch_config(ctypes.Structure):
    _fields_ = [("tile_elems", ctypes.c_int64), ("ntiles", ctypes.c_int64),
                ("xcd_run_tiles", ctypes.c_int32), ("lds_bytes", ctypes.c_int32)]


class DasoError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libdaso.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2104_05588_amd.build` "
                           "(there is no fallback implementation)")
    # torch is imported first so that its HIP runtime is the one the library binds to
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.daso_local_avg.argtypes = [ctypes.POINTER(vp), i32, vp, i64, vp]
    lib.daso_pack_bf16.argtypes = [vp, vp, i64, vp]
    lib.daso_global_merge.argtypes = [vp, ctypes.POINTER(vp), i32, ctypes.POINTER(daso_bucket), i32,
                                      vp, i64, vp]
    lib.daso_global_merge_f32.argtypes = lib.daso_global_merge.argtypes
    lib.daso_fused_sync_step.argtypes = [ctypes.POINTER(daso_sync_args), vp]
    lib.daso_fused_sync_step_noalloc.argtypes = [ctypes.POINTER(daso_sync_args), vp]
    lib.daso_fused_launch_config.argtypes = [ctypes.POINTER(daso_sync_args), ctypes.POINTER(daso_launch_config)]
    lib.daso_plan_buckets.argtypes = [ctypes.POINTER(i64), i32, i64, ctypes.POINTER(i32), i32,
                                      ctypes.POINTER(daso_bucket), i32]
    lib.daso_plan_buckets.restype = i32
    lib.daso_status_string.argtypes = [ctypes.c_int]
    lib.daso_status_string.restype = ctypes.c_char_p
    lib.daso_abi_version.argtypes = []
    for name in ("daso_local_avg", "daso_pack_bf16", "daso_global_merge", "daso_global_merge_f32",
                 "daso_fused_sync_step", "daso_fused_sync_step_noalloc", "daso_fused_launch_config",
                 "daso_abi_version"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().daso_status_string(int(status)).decode()


# ------------------------------------------------------------- marshalling
# torch's raw getter for the current stream's handle costs about 0.1 us per
# call against about 3 us for torch.cuda.current_stream(), which builds a
# Stream object; the public route serves a torch without it.
_current_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> ctypes.c_void_p:
    if stream is not None:
        return ctypes.c_void_p(stream.cuda_stream)
    if _current_raw_stream is not None:
        return ctypes.c_void_p(_current_raw_stream(torch.cuda.current_device()))
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor], dtypes: Tuple[torch.dtype, ...], n: int, what: str) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{what} is on {t.device}, not on the current device cuda:{torch.cuda.current_device()}")
    if t.dtype not in dtypes:
        raise ValueError(f"{what} must have dtype in {dtypes}, got {t.dtype}")
    if t.numel() != n or not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous with {n} elements")
    return t.data_ptr()


_F32 = (torch.float32,)
_BF16 = (torch.int16, torch.bfloat16, torch.uint16)


def _ptr_array(ts: Sequence[torch.Tensor], dtypes, n: int, what: str):
    arr = (ctypes.c_void_p * max(len(ts), 1))()
    for i, t in enumerate(ts):
        arr[i] = _ptr(t, dtypes, n, f"{what}[{i}]")
    return arr


def bucket_table(buckets: Sequence[Tuple[int, int, int]]):
    arr = (daso_bucket * max(len(buckets), 1))()
    for i, (s, k, S) in enumerate(buckets):
        arr[i].start, arr[i].numel, arr[i].S, arr[i].reserved = int(s), int(k), int(S), 0
    return arr


def plan_buckets(numels: Sequence[int], cap: int = BUCKET_CAP_ELEMS,
                 S_cycle: Sequence[int] = (1,)) -> List[Tuple[int, int, int]]:
    """Bucket plan of a flat buffer of tensors (see daso_plan_buckets):
    (start, numel, S) per bucket, in walk order (last tensor first)."""
    lib = load()
    nt = len(numels)
    arr = (ctypes.c_int64 * max(nt, 1))(*[int(k) for k in numels])
    cyc = (ctypes.c_int32 * max(len(S_cycle), 1))(*[int(S) for S in S_cycle])
    count = lib.daso_plan_buckets(arr, nt, int(cap), cyc, len(S_cycle), None, 0)
    _check(min(count, 0), "daso_plan_buckets")
    out = (daso_bucket * max(count, 1))()
    lib.daso_plan_buckets(arr, nt, int(cap), cyc, len(S_cycle), out, count)
    return [(out[i].start, out[i].numel, out[i].S) for i in range(count)]


def _check(rc: int, what: str) -> None:
    if rc != DASO_OK:
        raise DasoError(rc, what)


# --------------------------------------------------------------- the calls
def local_avg(grads: Sequence[torch.Tensor], out: torch.Tensor, stream=None) -> torch.Tensor:
    """out = mean of the replica gradients (local synchronisation)."""
    n = out.numel()
    arr = _ptr_array(grads, _F32, n, "grads")
    _check(load().daso_local_avg(arr, len(grads), _ptr(out, _F32, n, "out"), n, _stream_handle(stream)),
           "daso_local_avg")
    return out


def pack_bf16(src: torch.Tensor, wire: torch.Tensor, stream=None) -> torch.Tensor:
    """wire = bf16 round-to-nearest-even bit patterns of src."""
    n = src.numel()
    _check(load().daso_pack_bf16(_ptr(src, _F32, n, "src"), _ptr(wire, _BF16, n, "wire"), n,
                                 _stream_handle(stream)), "daso_pack_bf16")
    return wire


def _is_f32_exchange(stale: Sequence[torch.Tensor], wire: Optional[torch.Tensor]) -> bool:
    """fp32 copies (or, with none, an fp32 wire) select the fp32 exchange."""
    probe = stale[0] if len(stale) else wire
    return probe is not None and probe.dtype == torch.float32


def global_merge(params: torch.Tensor, stale: Sequence[torch.Tensor],
                 buckets: Sequence[Tuple[int, int, int]], wire: Optional[torch.Tensor] = None,
                 stream=None) -> torch.Tensor:
    """Eq. (1) merge of the exchanged copies into params, in place: bf16 copies
    (int16/bfloat16 tensors) use daso_global_merge, fp32 copies daso_global_merge_f32."""
    n = params.numel()
    f32 = _is_f32_exchange(stale, wire)
    xt = _F32 if f32 else _BF16
    arr = _ptr_array(stale, xt, n, "stale")
    bt = bucket_table(buckets)
    fn = load().daso_global_merge_f32 if f32 else load().daso_global_merge
    _check(fn(_ptr(params, _F32, n, "params"), arr, len(stale), bt, len(buckets), _ptr(wire, xt, n, "wire"), n,
              _stream_handle(stream)), "daso_global_merge_f32" if f32 else "daso_global_merge")
    return params


def new_stats(nbuckets: int, device="cuda") -> torch.Tensor:
    """Device buffer for per-bucket statistics: float64 [nbuckets, 3] whose third
    column holds the uint64 non-finite count (read it with decode_stats)."""
    return torch.zeros((nbuckets, 3), dtype=torch.float64, device=device)


def decode_stats(stats: torch.Tensor) -> List[Tuple[float, float, int]]:
    h = stats.detach().cpu()
    counts = h[:, 2].contiguous().view(torch.int64)
    return [(float(h[i, 0]), float(h[i, 1]), int(counts[i])) for i in range(h.shape[0])]


class FusedStep:
    """A prepared daso_fused_sync_step: argument checks and marshalling happen
    once here, so that each call costs one C call.  The tensors must stay alive
    (and keep their storage) while the object is used.  noalloc=True calls
    daso_fused_sync_step_noalloc instead (statistics scratch in the library's
    fixed device array: no allocation, DasoError with DASO_ENOSPACE beyond it)."""

    def __init__(self, grads: Sequence[torch.Tensor], params: torch.Tensor, momentum: torch.Tensor,
                 stale: Sequence[torch.Tensor], buckets: Sequence[Tuple[int, int, int]],
                 lr: float, mu: float, weight_decay: float = 0.0, wire: Optional[torch.Tensor] = None,
                 grad_avg: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None,
                 flags: int = 0, noalloc: bool = False):
        n = params.numel()
        self._keep = (list(grads), params, momentum, list(stale), wire, grad_avg, stats)
        f32 = _is_f32_exchange(stale, wire)
        xt = _F32 if f32 else _BF16
        self._grads = _ptr_array(grads, _F32, n, "grads")
        self._stale = _ptr_array(stale, xt, n, "stale")
        self._buckets = bucket_table(buckets)
        if stats is not None:
            if not stats.is_cuda or stats.dtype != torch.float64 or tuple(stats.shape) != (len(buckets), 3) \
                    or not stats.is_contiguous():
                raise ValueError("stats must be a contiguous float64 device tensor of shape [nbuckets, 3]")
            if stats.device.index != torch.cuda.current_device():
                raise ValueError(f"stats is on {stats.device}, not on the current device")
        self._device = torch.cuda.current_device()
        a = daso_sync_args()
        a.n, a.g, a.P = n, len(grads), len(stale)
        a.grads = self._grads
        if f32:
            a.stale_f32 = self._stale
            a.wire_f32 = _ptr(wire, xt, n, "wire")
            flags |= DASO_EXCHANGE_F32
        else:
            a.stale = self._stale
            a.wire = _ptr(wire, xt, n, "wire")
        a.params = _ptr(params, _F32, n, "params")
        a.momentum = _ptr(momentum, _F32, n, "momentum")
        a.grad_avg = _ptr(grad_avg, _F32, n, "grad_avg")
        a.buckets = self._buckets
        a.nbuckets = len(buckets)
        a.lr, a.mu, a.weight_decay = float(lr), float(mu), float(weight_decay)
        a.flags = int(flags)
        a.stats = stats.data_ptr() if stats is not None else None
        self.args = a
        self._byref = ctypes.byref(a)
        self._name = "daso_fused_sync_step_noalloc" if noalloc else "daso_fused_sync_step"
        self._fn = getattr(load(), self._name)

    def launch_config(self) -> dict:
        """The launch shape of this call (daso_fused_launch_config): elements per
        tile, tiles of the first launch, tiles per XCD run, LDS per workgroup."""
        c = daso_launch_config()
        _check(load().daso_fused_launch_config(self._byref, ctypes.byref(c)), "daso_fused_launch_config")
        return {f: getattr(c, f) for f, _ in daso_launch_config._fields_}

    def __call__(self, stream=None) -> None:
        if torch.cuda.current_device() != self._device:
            raise ValueError(f"prepared on cuda:{self._device}, called with cuda:{torch.cuda.current_device()} "
                             "current")
        _check(self._fn(self._byref, _stream_handle(stream)), self._name)


def fused_sync_step(grads, params, momentum, stale, buckets, lr, mu, weight_decay=0.0, wire=None,
                    grad_avg=None, stats=None, flags=0, stream=None, noalloc=False) -> None:
    """One DASO synchronisation step (see include/daso.h), in place on params
    and momentum; writes wire, grad_avg and stats when given.  noalloc=True
    uses daso_fused_sync_step_noalloc."""
    FusedStep(grads, params, momentum, stale, buckets, lr, mu, weight_decay, wire, grad_avg, stats,
              flags, noalloc)(stream)


# ------------------------------------------------- phase/schedule controller
class daso_schedule_config(ctypes.Structure):
    _fields_ = [("total_epochs", ctypes.c_int32), ("warmup_epochs", ctypes.c_int32),
                ("cooldown_epochs", ctypes.c_int32), ("batches_per_epoch", ctypes.c_int32),
                ("B_init", ctypes.c_int32), ("W_init", ctypes.c_int32), ("group_count", ctypes.c_int32),
                ("local_rank", ctypes.c_int32), ("patience", ctypes.c_int32),
                ("plateau_rel_tol", ctypes.c_double)]


class daso_batch_plan(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int64), ("epoch", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("phase", ctypes.c_int32), ("B", ctypes.c_int32), ("W", ctypes.c_int32),
                ("actions", ctypes.c_uint32), ("S", ctypes.c_int32), ("sync_group", ctypes.c_int32),
                ("merge_group", ctypes.c_int32)]


PHASE_WARMUP, PHASE_CYCLING, PHASE_COOLDOWN = 0, 1, 2
ACT_SEND, ACT_MERGE, ACT_BLOCKING, ACT_RECV_BCAST = 1, 2, 4, 8


def _schedule_fns():
    lib = load()
    if not getattr(lib, "_daso_schedule_typed", False):
        lib.daso_schedule_create.argtypes = [ctypes.POINTER(daso_schedule_config), ctypes.POINTER(ctypes.c_void_p)]
        lib.daso_schedule_create.restype = ctypes.c_int
        lib.daso_schedule_next.argtypes = [ctypes.c_void_p, ctypes.POINTER(daso_batch_plan)]
        lib.daso_schedule_next.restype = ctypes.c_int
        lib.daso_schedule_end_epoch.argtypes = [ctypes.c_void_p, ctypes.c_double]
        lib.daso_schedule_end_epoch.restype = ctypes.c_int
        lib.daso_schedule_destroy.argtypes = [ctypes.c_void_p]
        lib.daso_schedule_destroy.restype = None
        lib._daso_schedule_typed = True
    return lib


class Schedule:
    """DASO's phase and exchange schedule for one GPU (daso_schedule_* in daso.h).

    next_batch() returns the plan of the next batch as a dict (None once
    training is over); end_epoch(loss) reports each epoch's training loss."""

    def __init__(self, total_epochs: int, warmup_epochs: int, cooldown_epochs: int, batches_per_epoch: int,
                 B_init: int, W_init: int = 0, group_count: int = 1, local_rank: int = 0, patience: int = 1,
                 plateau_rel_tol: float = 0.0):
        self._lib = _schedule_fns()
        self.config = daso_schedule_config(total_epochs, warmup_epochs, cooldown_epochs, batches_per_epoch, B_init,
                                           W_init, group_count, local_rank, patience, float(plateau_rel_tol))
        h = ctypes.c_void_p()
        _check(self._lib.daso_schedule_create(ctypes.byref(self.config), ctypes.byref(h)), "daso_schedule_create")
        self._h = h
        self._plan = daso_batch_plan()

    def next_batch(self):
        rc = self._lib.daso_schedule_next(self._h, ctypes.byref(self._plan))
        if rc == 0:
            return None
        if rc < 0:
            raise DasoError(rc, "daso_schedule_next")
        p = self._plan
        return {f: getattr(p, f) for f, _ in daso_batch_plan._fields_}

    def end_epoch(self, loss: float) -> None:
        _check(self._lib.daso_schedule_end_epoch(self._h, float(loss)), "daso_schedule_end_epoch")

    def close(self) -> None:
        if self._h:
            self._lib.daso_schedule_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
