"""The attention entry point that allocates nothing
(semshare_prefill_attention_noalloc: its work plan and partial results live
in the library's static device scratch) against semshare_prefill_attention
with a caller workspace: bit for bit the same output, on two calls in a row,
the second with a smaller input (the scratch keeps the first call's contents,
none of which the second may use)."""
import numpy as np
import pytest
import torch

import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import announce, dev, dev_i32

pytestmark = pytest.mark.gpu


def _case(n_tok, n_sel, hq, hkv, d, tag):
    cfg = CONFIGS[1]
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=tag)
    k, v = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=tag + 1)
    q = workloads.make_rows(cfg, n_sel, hq * d, tag=tag + 2).reshape(n_sel, hq, d)
    return dev(q, "bf16"), dev_i32(sel), dev(k[0], "bf16"), dev(v[0], "bf16")


def test_noalloc_attention_equals_workspace_attention_twice():
    for n_tok, n_sel, hq, hkv, d in ((5120, 1280, 32, 8, 128), (700, 200, 16, 4, 128)):
        announce(f"no-alloc attention n_tok={n_tok} n_sel={n_sel} hq={hq} hkv={hkv} d={d}")
        q, ps, k, v = _case(n_tok, n_sel, hq, hkv, d, tag=90 + n_sel % 7)
        want = ss.prefill_attention(q, ps, k, v, hkv)
        got = torch.full_like(want, 9.0)
        ss.prefill_attention_noalloc(q, ps, k, v, hkv, out=got)
        torch.cuda.synchronize()
        assert torch.equal(got, want)


def test_noalloc_attention_rejects_sizes_beyond_its_scratch():
    # 512 kv heads of head_dim 128: two partial-result slots per head, 64 MiB > 40 MiB
    n_tok, n_sel, hq, hkv, d = 64, 64, 512, 512, 128
    q = torch.zeros((n_sel, hq, d), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((n_tok, hkv, d), dtype=torch.bfloat16, device="cuda")
    ps = torch.arange(n_sel, dtype=torch.int32, device="cuda")
    out = torch.full_like(q, 9.0)
    with pytest.raises(ss.SemShareError) as e:
        ss.prefill_attention_noalloc(q, ps, k, k, hkv, out=out)
    assert e.value.status == ss.semshare.E_UNSUPPORTED and "scratch" in str(e.value)
    assert torch.all(out == 9.0)  # nothing was enqueued
