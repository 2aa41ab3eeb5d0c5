"""Seeded synthetic inputs for paged-KV attention.

This package is shared by the CPU oracle (``oracle/``) and the HIP path
(``paper_2608_23658_amd``). It holds no attention arithmetic: it draws
sequence lengths, block tables, queries and keys/values from seeded
generators and scatters the keys/values into the documented paged layout.
"""
from .configs import CONFIGS, BatchSpec, config_spec  # noqa: F401
from .gen import (  # noqa: F401
    PagedBatch,
    layout_offsets,
    make_batch,
    make_batch_from_lens,
    nan_bits,
    storage_torch_dtype,
)
