"""CPU oracle (fp64). Test infrastructure: see ``oracle.paged_kv``."""
from .paged_kv import (  # noqa: F401
    attend,
    gather_kv,
    paged_attention,
    paged_attention_rows,
    paged_decode,
    storage_to_f64,
)
from .append import copy_blocks, kv_append  # noqa: F401
