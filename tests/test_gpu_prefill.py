"""GPU parity of semshare_partial_prefill (QKV projection + RoPE + deviation +
cache scatter + causal GQA attention) against the oracle, plus the method's
invariants: 100% recompute equals full prefill, every selected row is
overwritten before attention, identical prompts give zero deviation.

Tolerances: attention output max-abs <= 2e-2 (bf16) / 1e-4 (fp32).  A
recomputed cache element may differ from the oracle's by one spacing of the
storage dtype plus the worst-case fp32 dot-product error
gamma_K * sum_k |x_k||w_k| (summed over both members of a RoPE pair); rows not
selected must be untouched, bit for bit.  Deviation: relative error <= 1e-3
(bf16) / 1e-5 (fp32)."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import (announce, bf16_ulp, check_cache_rows, dev, dev_i32, fp32_dot_error_bound, host,
                     rotated_pair_bound)

pytestmark = pytest.mark.gpu

ATOL = {"bf16": 2e-2, "fp32": 1e-4}


def _case(cfg, n_tok, hidden, hq, hkv, d, n_sel, tag=0, cache_scale=1.0):
    x_all = workloads.make_rows(cfg, n_tok, hidden, tag=100 + tag)
    w = workloads.make_weights(cfg, tag, hidden=hidden, n_q_heads=hq, n_kv_heads=hkv, head_dim=d)
    k, v = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=tag, scale=cache_scale)
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=tag)
    return x_all, w, k[0], v[0], sel


def _run_gpu(cfg, x_sel, sel, w, k, v, hq, hkv, want_out=True, want_dev=True):
    dt = cfg.dtype
    kc, vc = dev(k, dt), dev(v, dt)
    out, sig = ss.partial_prefill(dev(x_sel, dt), dev_i32(sel), dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt), kc, vc,
                                  hq, hkv, want_out=want_out, want_deviation=want_dev)
    return (None if out is None else host(out).reshape(len(sel), -1), None if sig is None else host(sig),
            host(kc), host(vc))


def _check(cfg, got, ref, x_sel, sel, w, k0, v0):
    out_g, sig_g, kc_g, vc_g = got
    out_r, sig_r, kc_r, vc_r = ref
    dt = cfg.dtype
    if out_r is not None:
        err = np.abs(out_g - out_r).max()
        assert err <= ATOL[dt], f"attention max-abs error {err}"
    check_cache_rows(dt, kc_g, kc_r, k0, sel, x_sel, w.wk, True)
    check_cache_rows(dt, vc_g, vc_r, v0, sel, x_sel, w.wv, False)
    if sig_r is not None:
        np.testing.assert_allclose(sig_g, sig_r, rtol=1e-3 if dt == "bf16" else 1e-5, atol=1e-3)


@pytest.mark.parametrize("name,cid,n_tok,hidden,hq,hkv,d,n_sel", [
    ("tiny-fp32", 0, 512, 256, 4, 4, 64, 102),
    ("fp32-gqa", 0, 200, 128, 4, 2, 32, 50),
    # fp32 projection over several 64-row / 64-column tiles with ragged rows; the attention's tiled form
    # (at least 256 (16-row block, head) pairs) at each head_dim it is built for
    ("fp32-d128-tiles", 0, 2100, 512, 8, 2, 128, 600),
    ("fp32-d64-tiles", 0, 3000, 256, 16, 4, 64, 400),
    ("fp32-d32-tiles", 0, 1500, 128, 16, 16, 32, 300),
    ("bf16-gqa4-ragged-split", 1, 300, 256, 8, 2, 128, 75),
    ("bf16-d64", 1, 200, 256, 4, 2, 64, 60),
    ("bf16-mha", 1, 260, 256, 2, 2, 128, 130),
    ("bf16-gqa8", 1, 333, 256, 16, 2, 128, 90),
    ("llama3-8b-layer-1k", 1, 1024, 4096, 32, 8, 128, 256),
])
def test_partial_prefill_matches_oracle(name, cid, n_tok, hidden, hq, hkv, d, n_sel):
    cfg = CONFIGS[cid]
    x_all, w, k, v, sel = _case(cfg, n_tok, hidden, hq, hkv, d, n_sel)
    announce(f"partial_prefill {name}")
    got = _run_gpu(cfg, x_all[sel], sel, w, k, v, hq, hkv)
    ref = orc.partial_prefill(x_all[sel], sel, w.wq, w.wk, w.wv, k, v, hq, hkv, d, dtype=cfg.dtype,
                              want_sigma=True)
    _check(cfg, got, ref, x_all[sel], sel, w, k, v)


@pytest.mark.parametrize("cid,n_tok,hidden,hq,hkv,d", [(1, 300, 256, 8, 2, 128), (0, 128, 256, 4, 4, 64)])
def test_full_recompute_equals_oracle_full_prefill(cid, n_tok, hidden, hq, hkv, d):
    cfg = CONFIGS[cid]
    x_all, w, k, v, _ = _case(cfg, n_tok, hidden, hq, hkv, d, 1, tag=3, cache_scale=50.0)
    sel = np.arange(n_tok, dtype=np.int32)
    announce(f"full recompute cfg{cid} n_tok={n_tok}")
    got = _run_gpu(cfg, x_all, sel, w, k, v, hq, hkv)
    ref = orc.partial_prefill(x_all, sel, w.wq, w.wk, w.wv, np.zeros_like(k), np.zeros_like(v), hq, hkv, d,
                              dtype=cfg.dtype)
    _check(cfg, got[:1] + (None,) + got[2:], ref[:1] + (None,) + ref[2:], x_all, sel, w, k, v)
    # every row is overwritten before attention: garbage and zero caches agree bit for bit
    got0 = _run_gpu(cfg, x_all, sel, w, np.zeros_like(k), np.zeros_like(v), hq, hkv, want_dev=False)
    assert np.array_equal(got[0], got0[0])


def test_identical_prompt_zero_deviation_and_partial_equals_full():
    cfg = CONFIGS[1]
    n_tok, hidden, hq, hkv, d = 400, 256, 8, 2, 128
    x_all, w, _, _, _ = _case(cfg, n_tok, hidden, hq, hkv, d, 1, tag=4)
    allpos = np.arange(n_tok, dtype=np.int32)
    announce("identical prompt: own cache, then partial")
    dt = cfg.dtype
    kc = torch.zeros((n_tok, hkv, d), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    xa = dev(x_all, dt)
    wq, wk, wv = dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt)
    full, _ = ss.partial_prefill(xa, dev_i32(allpos), wq, wk, wv, kc, vc, hq, hkv)  # also builds the own cache
    sel = workloads.make_sel_pos(cfg, n_tok, 100, tag=4)
    part, sig = ss.partial_prefill(xa[torch.from_numpy(sel).long().cuda()].contiguous(), dev_i32(sel), wq, wk, wv,
                                   kc, vc, hq, hkv, want_deviation=True)
    assert not host(sig).any()  # recomputing a prompt's own rows reproduces them bit for bit
    # same rows, same cache: equal up to the split-KV summation order
    np.testing.assert_allclose(host(part), host(full)[sel], rtol=0, atol=1e-2)


def test_kv_only_mode_matches_oracle():
    cfg = CONFIGS[1]
    n_tok, hidden, hq, hkv, d = 256, 512, 8, 2, 128
    x_all, w, k, v, sel = _case(cfg, n_tok, hidden, hq, hkv, d, 256, tag=5)
    announce("kv-only mode")
    got = _run_gpu(cfg, x_all[sel], sel, w, k, v, hq, hkv, want_out=False, want_dev=False)
    assert got[0] is None
    ref = orc.partial_prefill(x_all[sel], sel, w.wq, w.wk, w.wv, k, v, hq, hkv, d, dtype="bf16", want_out=False)
    _check(cfg, got, ref, x_all[sel], sel, w, k, v)


def test_single_key_row_returns_value():
    # the row at position 0 attends only to itself
    cfg = CONFIGS[1]
    n_tok, hidden, hq, hkv, d = 64, 256, 8, 2, 128
    x_all, w, k, v, _ = _case(cfg, n_tok, hidden, hq, hkv, d, 1, tag=6)
    sel = np.array([0, 10, 63], dtype=np.int32)
    announce("single key row")
    out, _, _, vc = _run_gpu(cfg, x_all[sel], sel, w, k, v, hq, hkv, want_dev=False)
    G = hq // hkv
    for h in range(hq):
        g = h // G
        np.testing.assert_allclose(out[0, h * d:(h + 1) * d], vc[0, g], rtol=0, atol=2e-2)


def test_config2_layer_sampled_rows():
    """The 5k-token Llama-3-8B-shaped layer in the benchmark's launch
    configuration (n_sel = 1280), checked on sampled rows the oracle computes
    one by one."""
    cfg = CONFIGS[2]
    n_tok, hidden, hq, hkv, d = 5120, 4096, 32, 8, 128
    n_sel = cfg.n_sel(0.25)
    x_all, w, k, v, sel = _case(cfg, n_tok, hidden, hq, hkv, d, n_sel, tag=7)
    announce("config2 layer n_sel=1280")
    out_g, sig_g, kc_g, vc_g = _run_gpu(cfg, x_all[sel], sel, w, k, v, hq, hkv)
    # oracle: k/v of every selected row (they all enter the cache), q of sampled rows only
    _, kn, vn = orc.qkv_rows(x_all[sel], sel, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_q=False)
    kc_r = k.reshape(n_tok, -1).astype(np.float64).copy()
    vc_r = v.reshape(n_tok, -1).astype(np.float64).copy()
    sig_r = orc.deviation(kc_r, vc_r, sel, kn, vn)
    kc_r[sel] = kn
    vc_r[sel] = vn
    rows = np.unique(np.concatenate([[0, n_sel - 1], np.random.default_rng(7).choice(n_sel, 62, replace=False)]))
    q, _, _ = orc.qkv_rows(x_all[sel[rows]], sel[rows], w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_kv=False)
    out_r = orc.attention_rows(q, sel[rows], kc_r, vc_r, hq, hkv, d, dtype="bf16")
    assert np.abs(out_g[rows] - out_r).max() <= ATOL["bf16"]
    check_cache_rows("bf16", kc_g, kc_r, k, sel, x_all[sel], w.wk, True)
    check_cache_rows("bf16", vc_g, vc_r, v, sel, x_all[sel], w.wv, False)
    np.testing.assert_allclose(sig_g, sig_r, rtol=1e-3)


def test_split_calls_equal_partial_prefill():
    """semshare_qkv_rope followed by semshare_prefill_attention runs the same
    kernels as semshare_partial_prefill: identical outputs, caches and deviation."""
    cfg = CONFIGS[1]
    n_tok, hidden, hq, hkv, d = 700, 512, 16, 4, 128
    x_all, w, k, v, sel = _case(cfg, n_tok, hidden, hq, hkv, d, 200, tag=8)
    dt = cfg.dtype
    announce("split calls vs partial_prefill")
    xs, ps = dev(x_all[sel], dt), dev_i32(sel)
    wq, wk, wv = dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt)
    k1, v1, k2, v2 = dev(k, dt), dev(v, dt), dev(k, dt), dev(v, dt)
    out1, dev1 = ss.partial_prefill(xs, ps, wq, wk, wv, k1, v1, hq, hkv, want_deviation=True)
    q, dev2 = ss.qkv_rope(xs, ps, wq, wk, wv, k2, v2, hq, hkv, want_deviation=True)
    out2 = ss.prefill_attention(q, ps, k2, v2, hkv)
    for a, b in ((out1, out2), (dev1, dev2), (k1, k2), (v1, v2)):
        assert torch.equal(a, b)
    # and the q written by the projection step is the oracle's within the derived bound
    qr, _, _ = orc.qkv_rows(x_all[sel], sel, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_kv=False)
    b = rotated_pair_bound(fp32_dot_error_bound(x_all[sel], w.wq), d) + 1e-6 * np.abs(qr)
    assert np.all(np.abs(host(q).reshape(len(sel), -1) - qr) <= bf16_ulp(qr) + b)


@pytest.mark.parametrize("n_tok,hq,hkv,d,n_sel", [(700, 16, 4, 128, 200), (5120, 32, 8, 128, 1280),
                                                  (300, 8, 8, 64, 300)])
def test_planned_attention_equals_unplanned(n_tok, hq, hkv, d, n_sel):
    """One plan from semshare_attention_plan serves several layers' calls
    (different caches and queries, the same positions): each planned call is
    bit for bit the call that makes its own plan, and agrees with the oracle
    on sampled rows."""
    cfg = CONFIGS[1]
    announce(f"planned attention n_tok={n_tok} hq={hq} hkv={hkv} d={d} n_sel={n_sel}")
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=21)
    ps = dev_i32(sel)
    plan = ss.attention_plan(ps, n_tok, hq, hkv, d)
    assert plan.numel() == ss.attention_plan_bytes(n_sel, n_tok, hq, hkv, d) > 0
    for layer in range(2):
        k, v = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=30 + layer)
        q = workloads.make_rows(cfg, n_sel, hq * d, tag=40 + layer).reshape(n_sel, hq, d)
        qd, kd, vd = dev(q, "bf16"), dev(k[0], "bf16"), dev(v[0], "bf16")
        want = ss.prefill_attention(qd, ps, kd, vd, hkv)
        got = ss.prefill_attention(qd, ps, kd, vd, hkv, plan=plan)
        assert torch.equal(got, want)
        rows = np.unique(np.linspace(0, n_sel - 1, 6).astype(int))
        ref = orc.attention_rows(host(qd)[rows], sel[rows], host(kd), host(vd), hq, hkv, d, dtype="bf16")
        assert np.max(np.abs(host(got)[rows].reshape(len(rows), -1) - ref.reshape(len(rows), -1))) <= ATOL["bf16"]


def test_plan_for_other_sizes_is_not_used():
    """A plan made for other sizes is rejected on the device: the call writes nothing."""
    cfg = CONFIGS[1]
    n_tok, hq, hkv, d, n_sel = 700, 16, 4, 128, 200
    announce("plan size check")
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=22)
    ps = dev_i32(sel)
    other = ss.attention_plan(ps, n_tok + 64, hq, hkv, d)  # same buffer size, other n_tok
    assert other.numel() >= ss.attention_plan_bytes(n_sel, n_tok, hq, hkv, d)
    k, v = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=23)
    q = workloads.make_rows(cfg, n_sel, hq * d, tag=24).reshape(n_sel, hq, d)
    out = torch.full((n_sel, hq, d), 7.0, dtype=torch.bfloat16, device="cuda")
    ss.prefill_attention(dev(q, "bf16"), ps, dev(k[0], "bf16"), dev(v[0], "bf16"), hkv, out=out, plan=other)
    assert torch.all(out == 7.0)


@pytest.mark.parametrize("n_tok,hidden,hq,hkv,d,n_sel", [(700, 512, 16, 4, 128, 200), (300, 256, 8, 8, 64, 300),
                                                         (5120, 512, 32, 8, 128, 1280)])
def test_shared_rope_table_equals_own(n_tok, hidden, hq, hkv, d, n_sel):
    """One RoPE table from semshare_rope_table serves several layers'
    projections (different weights and caches, the same positions): each call
    with it is bit for bit the call that makes its own table (q, caches,
    deviation)."""
    cfg = CONFIGS[1]
    announce(f"shared rope table n_tok={n_tok} hidden={hidden} hq={hq} hkv={hkv} d={d} n_sel={n_sel}")
    dt = cfg.dtype
    sel = workloads.make_sel_pos(cfg, n_tok, n_sel, tag=51)
    ps = dev_i32(sel)
    table = ss.rope_table(ps, n_tok, d)
    assert table.numel() == ss.rope_table_bytes(n_sel, d) == n_sel * (d // 2) * 8
    for layer in range(2):
        x_all, w, k, v, _ = _case(cfg, n_tok, hidden, hq, hkv, d, n_sel, tag=60 + layer)
        xs = dev(x_all[sel], dt)
        wq, wk, wv = dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt)
        k1, v1, k2, v2 = dev(k, dt), dev(v, dt), dev(k, dt), dev(v, dt)
        q1, dev1 = ss.qkv_rope(xs, ps, wq, wk, wv, k1, v1, hq, hkv, want_deviation=True)
        q2, dev2 = ss.qkv_rope(xs, ps, wq, wk, wv, k2, v2, hq, hkv, want_deviation=True, rope_table=table)
        for a, b in ((q1, q2), (dev1, dev2), (k1, k2), (v1, v2)):
            assert torch.equal(a, b)
        # the same rows read in place from every row of x (no gathered copy)
        k3, v3 = dev(k, dt), dev(v, dt)
        q3, dev3 = ss.qkv_rope(dev(x_all, dt), ps, wq, wk, wv, k3, v3, hq, hkv, want_deviation=True,
                               rope_table=table, x_rows=ps)
        for a, b in ((q1, q3), (dev1, dev3), (k1, k3), (v1, v3)):
            assert torch.equal(a, b)


def test_projection_rows_read_in_place_clamped():
    """semshare_qkv_rope_tabled_rows with input rows in any order, repeated,
    and outside [0, n_x) (read as row 0 or row n_x - 1): equal, bit for bit,
    to gathering those rows first (700 x rows, 300 selected, hidden 512,
    16 q / 4 kv heads, head_dim 128)."""
    cfg = CONFIGS[1]
    n_tok, hidden, hq, hkv, d, n_sel = 700, 512, 16, 4, 128, 300
    announce("projection with rows read in place, clamped row indices")
    dt = cfg.dtype
    x_all, w, k, v, sel = _case(cfg, n_tok, hidden, hq, hkv, d, n_sel, tag=70)
    r = np.random.default_rng(70)
    rows = r.integers(-50, n_tok + 50, n_sel).astype(np.int32)
    rows[:3] = [-1, n_tok, n_tok + 7]
    ps, pr = dev_i32(sel), dev_i32(rows)
    table = ss.rope_table(ps, n_tok, d)
    wq, wk, wv = dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt)
    k1, v1, k2, v2 = dev(k, dt), dev(v, dt), dev(k, dt), dev(v, dt)
    xs = dev(x_all[np.clip(rows, 0, n_tok - 1)], dt)
    q1, dev1 = ss.qkv_rope(xs, ps, wq, wk, wv, k1, v1, hq, hkv, want_deviation=True, rope_table=table)
    q2, dev2 = ss.qkv_rope(dev(x_all, dt), ps, wq, wk, wv, k2, v2, hq, hkv, want_deviation=True, rope_table=table,
                           x_rows=pr)
    for a, b in ((q1, q2), (dev1, dev2), (k1, k2), (v1, v2)):
        assert torch.equal(a, b)


def test_attention_plan_over_1024_row_tiles():
    """More row tiles than the 1024 threads of the plan kernel (its passes
    loop over the row tiles in blocks of 1024): 36864 rows, 8 query heads per
    kv head (32 rows per row tile, 1152 row tiles per kv head).  The planned
    and unplanned calls agree bit for bit and sampled rows, first, middle and
    last, match the oracle."""
    cfg = CONFIGS[1]
    n_tok, hq, hkv, d = 36864, 32, 4, 64
    n_sel = n_tok
    announce(f"attention over 1152 row tiles n_tok={n_tok} hq={hq} hkv={hkv} d={d}")
    sel = np.arange(n_sel, dtype=np.int32)
    ps = dev_i32(sel)
    k, v = workloads.make_cache(cfg, 1, n_tok, n_kv_heads=hkv, head_dim=d, tag=71)
    q = workloads.make_rows(cfg, n_sel, hq * d, tag=72).reshape(n_sel, hq, d)
    qd, kd, vd = dev(q, "bf16"), dev(k[0], "bf16"), dev(v[0], "bf16")
    want = ss.prefill_attention(qd, ps, kd, vd, hkv)
    plan = ss.attention_plan(ps, n_tok, hq, hkv, d)
    got = ss.prefill_attention(qd, ps, kd, vd, hkv, plan=plan)
    assert torch.equal(got, want)
    rows = np.array([0, 1, 31, 32, 1023 * 32, 1024 * 32 + 5, n_sel // 2, n_sel - 33, n_sel - 1])
    ref = orc.attention_rows(host(qd)[rows], sel[rows], host(kd), host(vd), hq, hkv, d, dtype="bf16")
    assert np.max(np.abs(host(got)[rows].reshape(len(rows), -1) - ref.reshape(len(rows), -1))) <= ATOL["bf16"]


def test_config2_first_layer_full_recompute():
    """The benchmark's first layer in its launch configuration: all 5120 rows
    of the 5k-token Llama-3-8B-shaped layer recomputed (hidden 4096, 32 q /
    8 kv heads) by semshare_qkv_rope with the deviation of every row against
    the assembled cache rows it replaces, then semshare_prefill_attention over
    every row.  Every K/V row and every deviation is checked; output rows on a
    sample that includes the first and the last."""
    cfg = CONFIGS[2]
    n_tok, hidden, hq, hkv, d = 5120, 4096, 32, 8, 128
    x_all, w, k, v, _ = _case(cfg, n_tok, hidden, hq, hkv, d, 1, tag=9)
    allpos = np.arange(n_tok, dtype=np.int32)
    announce("config2 first layer: 5120 rows, hidden 4096")
    dt = cfg.dtype
    kc, vc = dev(k, dt), dev(v, dt)
    ps = dev_i32(allpos)
    q, sig = ss.qkv_rope(dev(x_all, dt), ps, dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt), kc, vc, hq, hkv,
                         want_deviation=True)
    out = ss.prefill_attention(q, ps, kc, vc, hkv)
    out_g, sig_g, kc_g, vc_g = host(out).reshape(n_tok, -1), host(sig), host(kc), host(vc)
    _, kn, vn = orc.qkv_rows(x_all, allpos, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_q=False)
    sig_r = orc.deviation(k.reshape(n_tok, -1), v.reshape(n_tok, -1), allpos, kn, vn)
    np.testing.assert_allclose(sig_g, sig_r, rtol=1e-3)
    check_cache_rows("bf16", kc_g, kn, k, allpos, x_all, w.wk, True)
    check_cache_rows("bf16", vc_g, vn, v, allpos, x_all, w.wv, False)
    rows = np.unique(np.concatenate([[0, 1, n_tok - 1], np.random.default_rng(9).choice(n_tok, 61, replace=False)]))
    qr, _, _ = orc.qkv_rows(x_all[rows], allpos[rows], w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_kv=False)
    out_r = orc.attention_rows(qr, allpos[rows], kn, vn, hq, hkv, d, dtype="bf16")
    err = np.abs(out_g[rows] - out_r).max()
    assert err <= ATOL["bf16"], f"attention max-abs error {err}"


@pytest.mark.parametrize("n_tok,n_ref,hidden,hq,hkv,d,n_sel", [(300, 280, 256, 8, 2, 128, 300),
                                                              (300, 280, 256, 8, 2, 128, 90),
                                                              (5120, 5120, 4096, 32, 8, 128, 5120)])
def test_first_layer_deviation_against_reference_rows(n_tok, n_ref, hidden, hq, hkv, d, n_sel):
    """semshare_qkv_rope_dev_ref gives bit for bit what semshare_gather_kv of
    the layer followed by semshare_qkv_rope with deviation gives: q, the
    recomputed cache rows, the deviation; rows not selected are untouched and
    an index outside the reference counts as a zero row."""
    cfg = CONFIGS[1]
    x_all, w, _, _, _ = _case(cfg, n_tok, hidden, hq, hkv, d, 1, tag=12)
    rk, rv = workloads.make_cache(cfg, 1, n_ref, n_kv_heads=hkv, head_dim=d, tag=13)
    idx = np.random.default_rng(14).integers(0, n_ref, n_tok).astype(np.int32)
    idx[3], idx[7] = -1, n_ref  # outside the reference: zero rows
    sel = np.arange(n_tok, dtype=np.int32) if n_sel == n_tok else workloads.make_sel_pos(cfg, n_tok, n_sel, tag=15)
    sel = np.unique(np.concatenate([sel, [3, 7]])).astype(np.int32)  # the two rows with no reference row
    announce(f"first-layer deviation against reference rows n_tok={n_tok} n_ref={n_ref} n_sel={len(sel)}")
    dt = "bf16"
    RK, RV, ix, ps = dev(rk[0], dt), dev(rv[0], dt), dev_i32(idx), dev_i32(sel)
    xs = dev(x_all[sel], dt)
    wq, wk, wv = dev(w.wq, dt), dev(w.wk, dt), dev(w.wv, dt)
    ka, va = ss.gather_kv(RK[None], RV[None], ix)
    qa, sa = ss.qkv_rope(xs, ps, wq, wk, wv, ka[0], va[0], hq, hkv, want_deviation=True)
    kb = torch.full((n_tok, hkv, d), 5.0, dtype=torch.bfloat16, device="cuda")
    vb = torch.full_like(kb, 5.0)
    qb, sb = ss.qkv_rope_dev_ref(xs, ps, wq, wk, wv, kb, vb, hq, hkv, RK, RV, ix)
    assert torch.equal(qa, qb) and torch.equal(sa, sb)
    keep = np.ones(n_tok, bool)
    keep[sel] = False
    for a_t, b_t in ((ka[0], kb), (va[0], vb)):
        a_h, b_h = host(a_t), host(b_t)
        assert np.array_equal(a_h[sel], b_h[sel])
        assert np.all(b_h[keep] == 5.0)
    if n_tok <= 1024:  # and the deviation against the oracle's gathered rows
        g_k = np.where((idx >= 0)[:, None] & (idx < n_ref)[:, None], rk[0].reshape(n_ref, -1)[np.clip(idx, 0, n_ref - 1)], 0)
        g_v = np.where((idx >= 0)[:, None] & (idx < n_ref)[:, None], rv[0].reshape(n_ref, -1)[np.clip(idx, 0, n_ref - 1)], 0)
        _, kn, vn = orc.qkv_rows(x_all[sel], sel, w.wq, w.wk, w.wv, hq, hkv, d, dtype="bf16", want_q=False)
        np.testing.assert_allclose(host(sb), orc.deviation(g_k, g_v, sel, kn, vn), rtol=1e-3)
