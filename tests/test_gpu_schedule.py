"""GPU parity of the per-layer schedules (Section 4.3.3 recomputation,
Section 4.3.4 retention; Appendix A.5, A.6) against the oracle: a later
layer's recompute set drawn from the previous layer's, a later layer's kept
set and compaction plan (bit-exact), and a layer whose recomputed tokens
attend over its compacted cache, checked against the oracle's attention over
the kept positions of the full assembled cache (max-abs 2e-2, K/V rows within
the projection bound)."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import announce, check_cache_rows, dev, dev_i32, host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,m,ties", [(1, 1, False), (300, 100, True), (5120, 1280, False), (5120, 5120, True),
                                      (100000, 33333, True), (64, 0, False)])
def test_nested_selection_matches_oracle(n, m, ties):
    r = np.random.default_rng(n + m)
    cand = np.sort(r.choice(4 * n, n, replace=False)).astype(np.int32)
    sig = (r.integers(0, 5, n) if ties else r.exponential(size=n)).astype(np.float32)
    announce(f"nested selection n={n} m={m} ties={ties}")
    got = ss.select_recompute_nested(torch.from_numpy(sig).cuda(), dev_i32(cand), m)
    assert np.array_equal(got.cpu().numpy(), orc.select_recompute_nested(sig, cand, m))


@pytest.mark.parametrize("n_tok,n_retain,n_sel", [(1, 1, 1), (100, 40, 30), (5120, 3000, 1280), (5120, 0, 512),
                                                  (32768, 20000, 3277), (1 << 20, 700000, 100000)])
def test_retention_layer_matches_oracle(n_tok, n_retain, n_sel):
    r = np.random.default_rng(n_tok + n_retain)
    rank = r.permutation(n_tok).astype(np.int32)
    sel = np.sort(r.choice(n_tok, n_sel, replace=False)).astype(np.int32)
    idx = r.integers(0, n_tok, n_tok).astype(np.int32)
    announce(f"retention layer n_tok={n_tok} n_retain={n_retain} n_sel={n_sel}")
    kept, src, rows, nk = ss.retention_layer(dev_i32(rank), n_retain, dev_i32(sel), dev_i32(idx))
    k_r, s_r, rows_r = orc.retention_layer(rank, n_retain, sel, idx)
    nk = int(nk.cpu().numpy()[0])
    assert nk == k_r.size
    assert np.array_equal(kept.cpu().numpy()[:nk], k_r)
    assert np.array_equal(src.cpu().numpy()[:nk], s_r)
    assert np.array_equal(rows.cpu().numpy(), rows_r)


@pytest.mark.parametrize("n_tok,hidden,hq,hkv,n_retain,n_sel", [(1024, 512, 16, 4, 700, 200),
                                                                (5120, 1024, 32, 8, 4096, 1280)])
def test_layer_over_compacted_cache_matches_oracle(n_tok, hidden, hq, hkv, n_retain, n_sel):
    """The recomputed tokens of a layer whose cache keeps only the retained
    rows: compaction plan, gather of the kept rows from the reference cache
    through the match index, projection with the RoPE table of the tokens'
    positions written to their compacted rows, attention over the compacted
    cache with those rows as causal limits."""
    cfg, d = CONFIGS[1], 128
    r = np.random.default_rng(n_tok)
    x_sel = workloads.make_rows(cfg, n_sel, hidden, tag=400)
    w = workloads.make_weights(cfg, 3, hidden=hidden, n_q_heads=hq, n_kv_heads=hkv, head_dim=d)
    rk, rv = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=401)
    rk, rv = rk[0], rv[0]
    idx = r.integers(0, n_tok, n_tok).astype(np.int32)
    rank = r.permutation(n_tok).astype(np.int32)
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=402)
    announce(f"layer over compacted cache n_tok={n_tok} n_retain={n_retain} n_sel={n_sel}")
    ps = dev_i32(sel)
    kept, src, rows, nk_t = ss.retention_layer(dev_i32(rank), n_retain, ps, dev_i32(idx))
    nk = int(nk_t.cpu().numpy()[0])
    RK, RV = dev(rk, "bf16"), dev(rv, "bf16")
    kc = torch.empty((nk, hkv, d), dtype=torch.bfloat16, device="cuda")
    vc = torch.empty_like(kc)
    ss.gather_kv(RK[None], RV[None], src[:nk].contiguous(), out_k=kc[None], out_v=vc[None], except_pos=rows)
    table = ss.rope_table(ps, n_tok, d)
    q, _ = ss.qkv_rope(dev(x_sel, "bf16"), rows, dev(w.wq, "bf16"), dev(w.wk, "bf16"), dev(w.wv, "bf16"), kc, vc,
                       hq, hkv, rope_table=table)
    plan = ss.attention_plan(rows, nk, hq, hkv, d)
    out = ss.prefill_attention(q, rows, kc, vc, hkv, plan=plan)
    # oracle: the full assembled cache (every position's matched reference row, the recomputed rows
    # replaced), attention over the kept positions only
    k_r, _, rows_r = orc.retention_layer(rank, n_retain, sel, idx)
    assert nk == k_r.size and np.array_equal(rows.cpu().numpy(), rows_r)
    kfull = rk.reshape(n_tok, -1)[idx].astype(np.float64)
    vfull = rv.reshape(n_tok, -1)[idx].astype(np.float64)
    qr, kn, vn = orc.qkv_rows(x_sel, sel, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16")
    kfull[sel] = kn
    vfull[sel] = vn
    keep = np.zeros(n_tok, bool)
    keep[k_r] = True
    # the compacted cache: the kept rows of the full cache, in position order
    check_cache_rows("bf16", host(kc), kfull[k_r], kfull[k_r], rows_r, x_sel, w.wk, True)
    check_cache_rows("bf16", host(vc), vfull[k_r], vfull[k_r], rows_r, x_sel, w.wv, False)
    samp = np.unique(np.concatenate([[0, n_sel - 1], r.choice(n_sel, 30, replace=False)]))
    want = orc.attention_rows(qr[samp], sel[samp], kfull, vfull, hq, hkv, d, dtype="bf16", keep=keep)
    err = np.abs(host(out).reshape(n_sel, -1)[samp] - want).max()
    assert err <= 2e-2, f"attention max-abs error {err}"
    # evicting keys changes the result: the last rows over the full cache differ
    full = orc.attention_rows(qr[samp[-4:]], sel[samp[-4:]], kfull, vfull, hq, hkv, d, dtype="bf16")
    assert np.abs(full - want[-4:]).max() > 0.01
