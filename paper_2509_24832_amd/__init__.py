"""SemShareKV hot path for MI355X (gfx950): fuzzy token matching and KV reuse.

The compute lives in libsemshare.so (HIP kernels behind the C ABI of
include/semshare.h); ``semshare`` is its thin ctypes binding.
"""
from .semshare import (  # noqa: F401
    BF16, FP32, SemShareError, attention_mass, attention_plan, attention_plan_bytes, bank_similarity, declared_symbols, dynamic_recompute, gather_kv, gather_rows,
    last_error, load, lsh_encode, match, match_mfma,
    partial_prefill, partial_prefill_workspace_bytes, prefill_attention, prefill_attention_noalloc,
    prefill_attention_workspace_bytes,
    qkv_rope, qkv_rope_dev_ref, qkv_rope_workspace_bytes, retention, retention_layer, rope_embed, rope_lsh_encode, rope_table, rope_table_bytes, select_recompute, select_recompute_nested, version,
)
