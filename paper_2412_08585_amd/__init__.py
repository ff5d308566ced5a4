"""MI355X (gfx950) TurboAttention hot path: FlashQ + SAS quantized attention.

The computation lives in libturboattn.so (hand-written HIP for gfx950 behind
the C ABI of include/turbo_attn.h); this package only marshals arguments.
"""
from .binding import (KVTail, PagedKVCache, TurboKVCacheStruct, TurboKVTailStruct, decode_auto_split,
                      decode_split, decode_workspace, lib, page_bytes, turbo_append_kv, turbo_attn_decode,
                      turbo_attn_decode_noalloc,
                      turbo_attn_decode_trace, turbo_attn_prefill, turbo_attn_prefill_q8,
                      turbo_attn_prefill_trace, turbo_head_priority, turbo_int2_heads,
                      turbo_qkv_project, turbo_quantize_kv, turbo_sas_softmax, turbo_tail_init)

__all__ = ["KVTail", "PagedKVCache", "TurboKVCacheStruct", "TurboKVTailStruct", "decode_auto_split",
           "decode_split",
           "decode_workspace", "lib", "page_bytes", "turbo_append_kv", "turbo_attn_decode",
           "turbo_attn_decode_noalloc",
           "turbo_attn_decode_trace", "turbo_attn_prefill", "turbo_attn_prefill_q8",
           "turbo_attn_prefill_trace", "turbo_head_priority", "turbo_int2_heads",
           "turbo_qkv_project", "turbo_quantize_kv", "turbo_sas_softmax", "turbo_tail_init"]
