"""Seeded synthetic inputs for the mixed-batch attention step.

This package only draws numbers and lays them out in the paged-cache format
(block pool, block table, query rows). It holds none of the attention or
scheduling arithmetic, so both the CPU oracle and the HIP library can consume
exactly the same bytes. Floating-point tensors in reduced precision are stored
as their raw bit patterns (bf16 as uint16, fp8 as uint8) because numpy has no
such dtypes.
"""

from .attn_inputs import (  # noqa: F401
    AttnBatch,
    ParkCase,
    make_config,
    make_tiny_mixed,
    make_decode_8b,
    make_mixed_8b,
    make_long_context,
    make_decode_gqa8_fp8,
    make_prefill_8b,
    make_prefill_gqa8_fp8,
    make_batch_from_lengths,
    make_new_kv,
    poison_new_slots,
    round_to_bf16_bits,
    encode_e4m3fn_bits,
    BF16_NAN,
    FP8_NAN,
)
