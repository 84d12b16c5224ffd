"""fp64 CPU reference for multi-cartridge prefix attention.

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the bench's
CPU-baseline leg to check and time the HIP library. The library never imports
it, and it shares no code with the library.
"""
from .attention import (  # noqa: F401
    backward,
    forward,
    head_backward,
    head_forward,
    key_grads,
    key_grads_many,
    packed_backward,
    packed_forward,
    packed_key_grads_many,
    packed_rows_forward_backward,
    paged_decode_forward,
    paged_keys,
    row_keys,
    rows_forward_backward,
    visible_mask,
)
from . import adam  # noqa: F401,E402
from . import pool  # noqa: F401,E402
