"""CPU oracle for the DASO synchronisation step: test infrastructure only.

Imported by the tests, the smoke check and the CPU-baseline leg of the bench;
never by the product package."""
from .daso_oracle import (bf16_rne, bf16_widen, local_avg, sgd_momentum, merge_eq1,  # noqa: F401
                          pack_bf16, global_merge, fused_sync_step, bucket_stats,
                          PACK_PRE_MERGE, QNAN_BF16)
