"""CPU fp64 oracle — test infrastructure only (see paged_attention.py)."""
from .paged_attention import (PAGE, append, attend, attend_causal, decode, decode_seq, gather,
                              kv_head_of, new_pool, offload, prefill, prefill_seq, restore, widen_bf16)

__all__ = ["PAGE", "append", "attend", "attend_causal", "decode", "decode_seq", "gather", "kv_head_of",
           "new_pool", "offload", "prefill", "prefill_seq", "restore", "widen_bf16"]
