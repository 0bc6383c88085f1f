"""GPU parity at the long-context shape: target and reference prompts of
32768 tokens, Llama-3-8B attention layer (hidden 4096, 32 q / 8 kv heads,
head_dim 128, bf16), 128-bit LSH, recompute fraction 0.10 (3277 rows), causal
attention over the whole 32k assembled cache (Sections 4.2 and 4.3).

Each test runs the kernels in the launch configuration of the benchmark (the
split projection and attention calls with a shared RoPE table and attention
plan) and compares with the oracle: every recomputed K/V row and deviation,
output rows on a sample that includes the first and the last selected row,
both matchers bit for bit over 32768 x 32768 codes, and a two-layer gather
bit for bit.  Tolerances as in the other parity tests (attention max-abs
2e-2; projections within one bf16 spacing plus the worst-case fp32
dot-product error; deviation relative 1e-3)."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import (announce, bf16_ulp, check_cache_rows, dev, dev_codes, dev_i32, fp32_dot_error_bound, host,
                     rotated_pair_bound)

pytestmark = pytest.mark.gpu

CFG = CONFIGS[4]
T = CFG.n_tok


def test_long_context_partial_layer():
    hidden, hq, hkv, d = CFG.dim, CFG.n_q_heads, CFG.n_kv_heads, CFG.head_dim
    n_sel = CFG.n_sel(CFG.recompute_fracs[0])
    assert (T, n_sel) == (32768, 3277)
    x_sel = workloads.make_rows(CFG, n_sel, hidden, tag=300)
    w = workloads.make_weights(CFG, 0)
    k, v = workloads.make_cache(CFG, 1, T, tag=301)
    k, v = k[0], v[0]
    sel = workloads.make_sel_pos(CFG, T, n_sel, tag=302)
    announce(f"long context layer: n_tok={T} n_sel={n_sel} hidden={hidden}")
    kc, vc = dev(k, "bf16"), dev(v, "bf16")
    ps = dev_i32(sel)
    table = ss.rope_table(ps, T, d)
    plan = ss.attention_plan(ps, T, hq, hkv, d)
    q, sig = ss.qkv_rope(dev(x_sel, "bf16"), ps, dev(w.wq, "bf16"), dev(w.wk, "bf16"), dev(w.wv, "bf16"), kc, vc,
                         hq, hkv, want_deviation=True, rope_table=table)
    out = ss.prefill_attention(q, ps, kc, vc, hkv, plan=plan)
    out_g, sig_g, q_g = host(out).reshape(n_sel, -1), host(sig), host(q).reshape(n_sel, -1)
    kc_g, vc_g = host(kc), host(vc)

    _, kn, vn = orc.qkv_rows(x_sel, sel, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_q=False)
    kc_r = k.reshape(T, -1).astype(np.float64)
    vc_r = v.reshape(T, -1).astype(np.float64)
    sig_r = orc.deviation(kc_r, vc_r, sel, kn, vn)
    np.testing.assert_allclose(sig_g, sig_r, rtol=1e-3)
    kc_r[sel] = kn
    vc_r[sel] = vn
    check_cache_rows("bf16", kc_g, kc_r, k, sel, x_sel, w.wk, True)
    check_cache_rows("bf16", vc_g, vc_r, v, sel, x_sel, w.wv, False)
    del kc_g, vc_g

    rows = np.unique(np.concatenate([[0, n_sel - 1], np.random.default_rng(4).choice(n_sel, 46, replace=False)]))
    qr, _, _ = orc.qkv_rows(x_sel[rows], sel[rows], w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_kv=False)
    b = rotated_pair_bound(fp32_dot_error_bound(x_sel[rows], w.wq), d) + 1e-6 * np.abs(qr)
    assert np.all(np.abs(q_g[rows] - qr) <= bf16_ulp(qr) + b)
    out_r = orc.attention_rows(qr, sel[rows], kc_r, vc_r, hq, hkv, d, dtype="bf16")
    err = np.abs(out_g[rows] - out_r).max()
    assert err <= 2e-2, f"attention max-abs error {err}"


def test_long_context_match_bit_exact():
    """Codes of the long shape's token structure (windowed permutation, noise
    0.3, 20% fresh tokens; RoPE then 128-bit LSH by the oracle, at embedding
    width 256 so that the oracle encodes 2 x 32768 rows quickly): both
    matchers over 32768 x 32768 codes equal the oracle's brute-force scan."""
    pair = workloads.make_prompt_pair(CFG, dim=256)
    planes = workloads.make_planes(CFG, dim=256)
    ct = orc.lsh_encode(orc.rope_embed(pair.e_tgt, dtype="bf16"), planes)
    cr = orc.lsh_encode(orc.rope_embed(pair.e_ref, dtype="bf16"), planes)
    idx_r, dist_r = orc.match(ct, cr)
    tgt, ref = dev_codes(ct), dev_codes(cr)
    for name, fn in (("match", ss.match), ("match_mfma", ss.match_mfma)):
        announce(f"long context {name} {T} x {T}")
        idx, dist = fn(tgt, ref, want_dist=True)
        assert np.array_equal(idx.cpu().numpy(), idx_r), name
        assert np.array_equal(dist.cpu().numpy(), dist_r), name
    # the copied tokens mostly find their source (reported, not graded beyond a floor)
    copied = pair.pi >= 0
    assert (idx_r[copied] == pair.pi[copied]).mean() > 0.5


def test_long_context_gather_two_layers():
    """Two layers of a 32768-token cache gathered bit for bit, with and
    without the recomputed rows (3277, listed in ascending order) excepted."""
    L, hkv, d = 2, CFG.n_kv_heads, CFG.head_dim
    r = np.random.default_rng(5)
    ref_k = r.integers(0, 2 ** 16, size=(L, T, hkv, d), dtype=np.uint16)
    ref_v = r.integers(0, 2 ** 16, size=(L, T, hkv, d), dtype=np.uint16)
    idx = r.integers(0, T, size=T).astype(np.int32)
    sel = workloads.make_sel_pos(CFG, T, CFG.n_sel(0.10), tag=303)

    def bf(a):
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)

    announce(f"long context gather: L={L} n={T}")
    rk, rv, ix = bf(ref_k), bf(ref_v), dev_i32(idx)
    ok, ov = ss.gather_kv(rk, rv, ix)
    want_k, want_v = orc.gather_rows(ref_k, idx), orc.gather_rows(ref_v, idx)
    assert np.array_equal(ok.cpu().view(torch.int16).numpy().view(np.uint16), want_k)
    assert np.array_equal(ov.cpu().view(torch.int16).numpy().view(np.uint16), want_v)
    ek = torch.full_like(ok, 3.0)
    ev = torch.full_like(ov, 3.0)
    ss.gather_kv(rk, rv, ix, out_k=ek, out_v=ev, except_pos=dev_i32(sel))
    keep = np.ones(T, bool)
    keep[sel] = False
    for got_t, want in ((ek, want_k), (ev, want_v)):
        got = got_t.cpu().view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(got[:, keep], want[:, keep])
        assert np.all(got[:, sel] == np.uint16(0x4040))  # bf16 3.0, untouched
