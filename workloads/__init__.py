"""Seeded synthetic workloads (sizes, distributions, block placement, N(0,1) bf16 tensors).

Shared by the oracle tests and the GPU tests; holds none of the attention arithmetic."""
from .configs import (ALL, BY_NAME, EXTRA, TINY, LLAMA3_8B_PREFILL, LLAMA3_8B_DECODE, MIXED_70B,
                      LONG_DOC_SHARED_PROMPT, LONG_PREFIX_FEW_TUPLES, WorkloadSpec, BatchSpec,
                      Dist, SEED_BASE, BLOCK_SIZE)
from .gen import (Case, BatchData, plan_case, fill_host, fill_device, make_case,
                  f32_to_bf16_bits, BF16_NAN)
