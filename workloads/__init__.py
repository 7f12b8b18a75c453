"""Seeded synthetic decode-attention workloads (sizes, lengths, page pools).

Shared by the oracle's tests and by the GPU path's tests and bench; holds no
attention arithmetic."""
from .configs import CONFIGS, PAGE_SIZE, LengthModel, WorkloadConfig, get_config
from .generate import (Workload, custom_config, host_arrays, make_workload,
                       prefix_groups, to_page_format)
from .append import MIXES, DecodeRun, make_decode_run
