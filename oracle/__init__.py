"""CPU oracle (test infrastructure only): plain float64 paged-KV attention written from the
definition.  Imported only by tests, the smoke check and the benchmark's CPU baseline."""
from .paged_attention import (  # noqa: F401
    PAGE, attention, attention_scalar_loops, attention_split, attention_unit, bf16_bits_to_f64,
    compare, f64_to_bf16_bits, gather_kv, kv_append, kv_pack, kv_unpack, merge_states, partial_state,
)
