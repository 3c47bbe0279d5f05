"""Seeded synthetic inputs for one mixed prefill+decode paged-attention step.

This package draws inputs only.  It holds none of the attention arithmetic:
it draws sequence lengths, block tables and N(0,1) values, rounds values to
bf16 where asked, and lays the pre-append KV pool out in the cache layout that
``include/mpa.h`` defines.  Both the CPU oracle and the HIP library read the
arrays it returns; neither of them is imported here.
"""

from .gen import (  # noqa: F401
    Batch,
    SeqSpec,
    HeadSpec,
    bf16_bits_from_f32,
    make_batch,
    k_cache_shape,
    v_cache_shape,
)
from .configs import CONFIGS, config_specs  # noqa: F401
