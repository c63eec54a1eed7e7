"""MI355X (gfx950) paged-KV attention for multi-turn rollout: kv_append, prefill-append, decode,
colocated mixed batches and KV transfer pack/unpack between pools, as hand-written HIP kernels
behind a C ABI (include/pearl_attn.h).

The Python layer only marshals arguments (see ``binding``); it has no compute fallback."""
from .binding import (  # noqa: F401
    LIB_PATH, PearlError, abi_version, decode, decode_append, kv_append, kv_pack, kv_unpack, last_error, load, mixed,
    prefill_append, workspace_bytes,
)

__all__ = ["kv_append", "kv_pack", "kv_unpack", "prefill_append", "decode", "decode_append", "mixed", "workspace_bytes",
           "abi_version", "last_error", "load", "PearlError", "LIB_PATH"]
