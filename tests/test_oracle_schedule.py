"""Oracle pins for the per-layer schedules (Section 4.3.3 recomputation and
Section 4.3.4 retention; Appendix A.5 and A.6): attention over a cache that
keeps only some positions, a later layer's recompute set drawn from the
previous one's, and a later layer's kept set with its compaction.  CPU only."""
import numpy as np
import pytest
from scipy.special import softmax

import oracle as orc


def _qkv(r, n_tok, n_sel, hq, hkv, d):
    q = r.normal(size=(n_sel, hq * d))
    k = r.normal(size=(n_tok, hkv * d))
    v = r.normal(size=(n_tok, hkv * d))
    sel = np.sort(r.choice(n_tok, n_sel, replace=False)).astype(np.int32)
    return q, k, v, sel


def test_attention_keep_all_is_plain_attention():
    r = np.random.default_rng(0)
    q, k, v, sel = _qkv(r, 40, 9, 4, 2, 8)
    a = orc.attention_rows(q, sel, k, v, 4, 2, 8)
    b = orc.attention_rows(q, sel, k, v, 4, 2, 8, keep=np.ones(40, bool))
    assert np.array_equal(a, b)


def test_attention_keep_equals_masked_softmax_and_ignores_evicted_values():
    # a library softmax over the kept keys j <= p, head by head
    r = np.random.default_rng(1)
    n_tok, hq, hkv, d = 30, 4, 2, 8
    q, k, v, sel = _qkv(r, n_tok, 7, hq, hkv, d)
    keep = r.random(n_tok) < 0.6
    keep[sel] = True  # a query's own position is kept
    got = orc.attention_rows(q, sel, k, v, hq, hkv, d, keep=keep)
    G = hq // hkv
    for i, p in enumerate(sel):
        js = np.flatnonzero(keep[: p + 1])
        for h in range(hq):
            g = h // G
            s = k[js, g * d:(g + 1) * d] @ q[i, h * d:(h + 1) * d] / np.sqrt(d)
            want = softmax(s) @ v[js, g * d:(g + 1) * d]
            assert np.allclose(got[i, h * d:(h + 1) * d], want, rtol=0, atol=1e-12)
    # evicted rows may hold anything
    k2, v2 = k.copy(), v.copy()
    k2[~keep] = 1e3
    v2[~keep] = -7.0
    assert np.array_equal(orc.attention_rows(q, sel, k2, v2, hq, hkv, d, keep=keep), got)


def test_attention_keep_single_key_returns_its_value():
    r = np.random.default_rng(2)
    q, k, v, _ = _qkv(r, 20, 1, 2, 1, 8)
    keep = np.zeros(20, bool)
    keep[5] = True
    out = orc.attention_rows(q, np.array([12], np.int32), k, v, 2, 1, 8, keep=keep)
    assert np.array_equal(out[0, :8], v[5]) and np.array_equal(out[0, 8:], v[5])


def test_nested_selection_brute_force_and_ties():
    r = np.random.default_rng(3)
    for n, m in [(1, 1), (10, 3), (200, 57), (500, 500), (64, 0)]:
        cand = np.sort(r.choice(5 * n, n, replace=False)).astype(np.int32)
        sig = r.integers(0, 4, n).astype(np.float32)  # many ties
        got = orc.select_recompute_nested(sig, cand, m)
        order = sorted(range(n), key=lambda i: (-float(sig[i]), int(cand[i])))
        assert got.tolist() == sorted(int(cand[i]) for i in order[:m])
    with pytest.raises(ValueError):
        orc.select_recompute_nested(np.zeros(3, np.float32), np.arange(4), 1)


def test_retention_layer_worked_example():
    rank = np.array([3, 0, 5, 1, 4, 2], np.int64)  # ranking: positions 1, 3, 5, 0, 4, 2
    kept, src, rows = orc.retention_layer(rank, 3, [4], idx=np.array([9, 8, 7, 6, 5, 4]))
    assert kept.tolist() == [1, 3, 4, 5]           # ranks 0..2 plus the recomputed position 4
    assert src.tolist() == [8, 6, 5, 4]
    assert rows.tolist() == [2]
    kept0, src0, rows0 = orc.retention_layer(rank, 0, [])
    assert kept0.size == 0 and src0 is None and rows0.size == 0


@pytest.mark.parametrize("seed", range(4))
def test_retention_layer_invariants(seed):
    r = np.random.default_rng(10 + seed)
    n = int(r.integers(50, 400))
    rank = r.permutation(n)
    sel = np.sort(r.choice(n, int(r.integers(0, n // 3)), replace=False))
    retain = sorted(r.integers(0, n, 2))
    k_lo, _, rows_lo = orc.retention_layer(rank, retain[0], sel)
    k_hi, _, _ = orc.retention_layer(rank, retain[1], sel)
    assert set(sel) <= set(k_lo)                                   # never evicted
    assert set(k_lo) == set(np.flatnonzero(rank < retain[0])) | set(sel)
    assert set(k_lo) <= set(k_hi)                                  # nested for fewer kept
    assert np.array_equal(k_lo[rows_lo], sel) and np.all(np.diff(k_lo) > 0)
