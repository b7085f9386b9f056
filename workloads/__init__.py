"""Synthetic DASO workloads: parameter-set recipes and seeded input generators.

Holds no part of the DASO arithmetic; both the oracle tests and the GPU path
take their inputs from here."""
from .recipes import (Bucket, Workload, all_workloads, workload, custom_workload,  # noqa: F401
                      plan_buckets, tensor_offsets, algorithmic_bytes_per_param,
                      BUCKET_CAP_ELEMS)
from .generate import host_inputs, host_bucket_inputs, device_inputs, to_bf16_bits  # noqa: F401
