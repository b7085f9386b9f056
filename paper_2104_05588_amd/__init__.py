"""DASO parameter-synchronisation hot path for MI355X (gfx950).

The computation lives in libdaso.so (hand-written HIP kernels behind the C ABI
of include/daso.h); this package holds the build script and a ctypes binding
that only marshals arguments."""
from ._lib import (local_avg, pack_bf16, global_merge, fused_sync_step, FusedStep,  # noqa: F401
                   new_stats, decode_stats, bucket_table, plan_buckets, load, status_string, DasoError,
                   DASO_PACK_PRE_MERGE, DASO_EXCHANGE_F32, LIB_PATH, EXPORTED, Schedule,
                   PHASE_WARMUP, PHASE_CYCLING, PHASE_COOLDOWN, ACT_SEND, ACT_MERGE, ACT_BLOCKING,
                   ACT_RECV_BCAST)
from .driver import DasoSync  # noqa: F401,E402
