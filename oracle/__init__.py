"""CPU oracle (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg import this package.  The library never does, and nothing here imports the
library or its binding.
"""

from .ref import (  # noqa: F401
    append_reference,
    attention_reference,
    decode_raw,
    gather_kv,
    lse_merge,
    sequence_attention,
    softmax_attention,
)
