"""Seeded synthetic inputs for paged-KV attention.

This package is shared by the CPU oracle (``oracle/``) and the HIP path
(``paper_2608_23658_amd``). It holds no attention arithmetic: it draws
sequence lengths, block tables, queries and keys/values from seeded
generators and scatters the keys/values into the documented paged layout.
"""
from .configs import (  # noqa: F401
    DECODE_B256, MIXED_STEP, PREFILL_L32768, TINY_DECODE_F32, WORKLOADS, BatchSpec,
)
from .gen import (  # noqa: F401
    PagedBatch,
    layout_offsets,
    make_batch,
    make_batch_from_lens,
    nan_bits,
    storage_torch_dtype,
)
