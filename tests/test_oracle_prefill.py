"""Pins of the oracle's partial prefill (Sections 4.2, 4.3.3), KV deviation
(Appendix A.4) and causal GQA attention: 100% recompute equals a library
full causal prefill, single-key and equal-key closed forms, GQA head mapping,
deviation closed forms, identical-prompt invariance.  CPU only."""
import numpy as np
import pytest
import torch

import workloads

HQ, HKV, D, HID = 4, 2, 16, 48


def _weights(seed, hid=HID, hq=HQ, hkv=HKV, d=D):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((hq * d, hid)) * 0.2, rng.standard_normal((hkv * d, hid)) * 0.2,
            rng.standard_normal((hkv * d, hid)) * 0.2)


def _library_full_prefill(orc, x, wq, wk, wv, hq, hkv, d, base=10000.0):
    """Full causal prefill from library pieces: numpy matmul for the
    projections, the (separately pinned) oracle RoPE per head, and torch's
    scaled_dot_product_attention in fp64 for causal GQA attention."""
    T = x.shape[0]
    q = (x @ wq.T).reshape(T, hq, d)
    k = (x @ wk.T).reshape(T, hkv, d)
    v = (x @ wv.T).reshape(T, hkv, d)
    q = np.stack([orc.rope_embed(q[:, h], base=base) for h in range(hq)], axis=1)
    k = np.stack([orc.rope_embed(k[:, h], base=base) for h in range(hkv)], axis=1)
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)
    return o[0].permute(1, 0, 2).reshape(T, hq * d).numpy(), k.reshape(T, -1), v.reshape(T, -1)


@pytest.mark.parametrize("hq,hkv", [(4, 2), (4, 4), (4, 1)])
def test_full_recompute_equals_library_causal_prefill(orc, hq, hkv):
    T = 37
    x = np.random.default_rng(1).standard_normal((T, HID))
    wq, wk, wv = _weights(2, hq=hq, hkv=hkv)
    garbage = np.random.default_rng(3).standard_normal((T, hkv * D)) * 1e3
    out, _, kc, vc = orc.partial_prefill(x, np.arange(T), wq, wk, wv, garbage, garbage.copy(),
                                         hq, hkv, D)
    ref_o, ref_k, ref_v = _library_full_prefill(orc, x, wq, wk, wv, hq, hkv, D)
    np.testing.assert_allclose(out, ref_o, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(kc, ref_k, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(vc, ref_v, rtol=1e-12, atol=1e-13)
    # every row is overwritten before attention: a zero cache gives the same result
    out0, _, _, _ = orc.partial_prefill(x, np.arange(T), wq, wk, wv, np.zeros_like(garbage),
                                        np.zeros_like(garbage), hq, hkv, D)
    assert np.array_equal(out, out0)


def test_partial_on_own_cache_equals_full_prefill_rows(orc):
    # identical prompts: the reused cache is the prompt's own, so any recompute
    # subset reproduces the full prefill on the recomputed rows
    T = 41
    x = np.random.default_rng(4).standard_normal((T, HID))
    wq, wk, wv = _weights(5)
    ref_o, ref_k, ref_v = _library_full_prefill(orc, x, wq, wk, wv, HQ, HKV, D)
    sel = np.array([0, 3, 4, 17, 40], dtype=np.int32)
    out, sig, _, _ = orc.partial_prefill(x[sel], sel, wq, wk, wv, ref_k, ref_v, HQ, HKV, D,
                                         want_sigma=True)
    np.testing.assert_allclose(out, ref_o[sel], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(sig, 0.0, atol=1e-11)


def test_single_key_returns_its_value(orc):
    T = 8
    x = np.random.default_rng(6).standard_normal((T, HID))
    wq, wk, wv = _weights(7)
    out, _, _, vc = orc.partial_prefill(x[:1], np.array([0], np.int32), wq, wk, wv,
                                        np.zeros((T, HKV * D)), np.zeros((T, HKV * D)), HQ, HKV, D)
    v0 = x[0] @ wv.T
    G = HQ // HKV
    for h in range(HQ):
        g = h // G
        np.testing.assert_allclose(out[0, h * D:(h + 1) * D], v0[g * D:(g + 1) * D], rtol=1e-13)


def test_equal_keys_average_values(orc):
    # Wk = 0 -> every key is 0 -> uniform softmax -> mean of V[0..p]
    T = 30
    rng = np.random.default_rng(8)
    x = rng.standard_normal((T, HID))
    wq, _, wv = _weights(9)
    wk = np.zeros((HKV * D, HID))
    kc = np.zeros((T, HKV * D))
    vc = rng.standard_normal((T, HKV * D))
    sel = np.array([2, 11, 29], dtype=np.int32)
    out, _, _, vc2 = orc.partial_prefill(x[sel], sel, wq, wk, wv, kc, vc, HQ, HKV, D)
    G = HQ // HKV
    for i, p in enumerate(sel):
        for h in range(HQ):
            g = h // G
            exp = vc2[:p + 1, g * D:(g + 1) * D].mean(axis=0)
            np.testing.assert_allclose(out[i, h * D:(h + 1) * D], exp, rtol=1e-12, atol=1e-14)


def test_gqa_equals_mha_with_repeated_kv(orc):
    T, G = 23, 4
    hq, hkv = 8, 2
    rng = np.random.default_rng(10)
    q = rng.standard_normal((T, hq * D))
    kc = rng.standard_normal((T, hkv * D))
    vc = rng.standard_normal((T, hkv * D))
    sel = np.arange(T, dtype=np.int32)
    gqa = orc.attention_rows(q, sel, kc, vc, hq, hkv, D)
    k_rep = np.repeat(kc.reshape(T, hkv, D), G, axis=1).reshape(T, hq * D)
    v_rep = np.repeat(vc.reshape(T, hkv, D), G, axis=1).reshape(T, hq * D)
    mha = orc.attention_rows(q, sel, k_rep, v_rep, hq, hq, D)
    np.testing.assert_allclose(gqa, mha, rtol=1e-13, atol=1e-15)


def test_attention_rows_subset_and_scale(orc):
    T = 19
    rng = np.random.default_rng(11)
    q = rng.standard_normal((T, HQ * D))
    kc, vc = rng.standard_normal((T, HKV * D)), rng.standard_normal((T, HKV * D))
    sel = np.arange(T, dtype=np.int32)
    full = orc.attention_rows(q, sel, kc, vc, HQ, HKV, D)
    part = orc.attention_rows(q, sel, kc, vc, HQ, HKV, D, rows=[0, 7, 18])
    assert np.array_equal(part[[0, 7, 18]], full[[0, 7, 18]]) and np.isnan(part[1]).all()
    np.testing.assert_array_equal(orc.attention_rows(q, sel, kc, vc, HQ, HKV, D, scale=1 / np.sqrt(D)), full)
    # doubling the scale equals doubling q
    np.testing.assert_allclose(orc.attention_rows(q, sel, kc, vc, HQ, HKV, D, scale=2 / np.sqrt(D)),
                               orc.attention_rows(2 * q, sel, kc, vc, HQ, HKV, D), rtol=1e-12)


def test_deviation_closed_form(orc):
    T = 12
    rng = np.random.default_rng(12)
    x = rng.standard_normal((T, HID))
    wq, wk, wv = _weights(13)
    _, _, kc, vc = orc.partial_prefill(x, np.arange(T), wq, wk, wv, np.zeros((T, HKV * D)),
                                       np.zeros((T, HKV * D)), HQ, HKV, D, want_out=False)
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[5, 3] += 0.75
    vc2[5, 0] -= 2.0
    vc2[9, 7] += 3.0
    kc2[9, 1] += 4.0
    sel = np.arange(T, dtype=np.int32)
    _, sig, _, _ = orc.partial_prefill(x, sel, wq, wk, wv, kc2, vc2, HQ, HKV, D, want_out=False,
                                       want_sigma=True)
    exp = np.zeros(T); exp[5] = 0.75 + 2.0; exp[9] = 3.0 + 4.0
    np.testing.assert_allclose(sig, exp, atol=1e-12)
    # a whole-row shift by delta in K gives sqrt(n) * |delta|
    kc3 = kc.copy(); kc3[2] += 0.5
    _, sig3, _, _ = orc.partial_prefill(x, sel, wq, wk, wv, kc3, vc, HQ, HKV, D, want_out=False,
                                        want_sigma=True)
    assert sig3[2] == pytest.approx(0.5 * np.sqrt(HKV * D), rel=1e-12)


def test_kv_only_mode_and_rounding(orc):
    T = 16
    x = workloads.round_bf16(np.random.default_rng(14).standard_normal((T, HID)).astype(np.float32))
    wq, wk, wv = (workloads.round_bf16(w.astype(np.float32)) for w in _weights(15))
    out, sig, kc, vc = orc.partial_prefill(x, np.arange(T), wq, wk, wv, np.zeros((T, HKV * D)),
                                           np.zeros((T, HKV * D)), HQ, HKV, D, dtype="bf16",
                                           want_out=False)
    assert out is None and sig is None
    _, _, kc64, vc64 = orc.partial_prefill(x, np.arange(T), wq, wk, wv, np.zeros((T, HKV * D)),
                                           np.zeros((T, HKV * D)), HQ, HKV, D, want_out=False)
    assert np.array_equal(kc, orc.round_to(kc64, "bf16")) and np.array_equal(vc, orc.round_to(vc64, "bf16"))


def test_qkv_rows_positions_enter_rope(orc):
    # the same input row at two positions gives rotated q/k: per-head inner
    # products of q(p1) and k(p2) depend only on p1 - p2
    x = np.random.default_rng(16).standard_normal((1, HID))
    wq, wk, wv = _weights(17)
    dots = []
    for p1, p2 in [(10, 4), (1006, 1000)]:
        q, _, _ = orc.qkv_rows(x, [p1], wq, wk, wv, HQ, HKV, D)
        _, k, v = orc.qkv_rows(x, [p2], wq, wk, wv, HQ, HKV, D)
        dots.append(q[0, :D] @ k[0, :D])
    assert dots[0] == pytest.approx(dots[1], rel=1e-9)
    _, _, v1 = orc.qkv_rows(x, [3], wq, wk, wv, HQ, HKV, D)
    np.testing.assert_allclose(v1[0], x[0] @ wv.T, rtol=1e-13)  # v carries no rotation
