"""Oracle pins for the average attention score per token, Attention Recovery
and the dynamic recompute set (Section 3 Insight 2 and its AR equation;
Section 4.3.3).  CPU only."""
import numpy as np
import pytest

import oracle as orc


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("T,hq,hkv", [(1, 2, 1), (9, 4, 2), (40, 4, 4)])
def test_mass_sums_to_one(T, hq, hkv):
    # every softmax row sums to 1, so the mean over heads and rows does too
    r = _rng(T)
    q, k = r.normal(size=(T, hq, 8)), r.normal(size=(T, hkv, 8))
    m = orc.attention_mass(q, k, hq, hkv, 8)
    assert m.shape == (T,) and abs(m.sum() - 1.0) < 1e-12 and (m > 0).all()


def test_mass_zero_queries_is_harmonic():
    # q = 0: row i spreads 1/(i+1) over keys 0..i, so mass_j = (H_T - H_j) / T
    T = 23
    k = _rng(1).normal(size=(T, 1, 16))
    m = orc.attention_mass(np.zeros((T, 2, 16)), k, 2, 1, 16)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    assert np.allclose(m, (H[T] - H[:T]) / T, rtol=0, atol=1e-15)


def test_mass_one_dominant_key_closed_form():
    # scores a against key 0 and 0 against every other key: P_i0 = e^a / (e^a + i)
    T, D, a = 17, 4, 3.0
    q = np.zeros((T, 1, D)); q[:, 0, 0] = 1.0
    k = np.zeros((T, 1, D)); k[0, 0, 0] = a * np.sqrt(D)
    m = orc.attention_mass(q, k, 1, 1, D)
    i = np.arange(T)
    assert abs(m[0] - np.mean(np.exp(a) / (np.exp(a) + i))) < 1e-14
    # every other key j gets 1 / (e^a + i) from each row i >= j
    for j in range(1, T):
        assert abs(m[j] - np.sum(1.0 / (np.exp(a) + i[j:])) / T) < 1e-14


def test_mass_gqa_equals_mha_with_repeated_kv():
    r = _rng(3)
    T, hq, hkv, D = 12, 4, 2, 8
    q, k = r.normal(size=(T, hq, D)), r.normal(size=(T, hkv, D))
    m_gqa = orc.attention_mass(q, k, hq, hkv, D)
    m_mha = orc.attention_mass(q, np.repeat(k, hq // hkv, axis=1), hq, hq, D)
    assert np.allclose(m_gqa, m_mha, rtol=0, atol=1e-15)


def test_attention_recovery_is_exact_below_any_fixed_point():
    # the top-k sum is compared with thres * total exactly: a difference of
    # 2^-60 (or one fp32 subnormal, 2^-149) decides, which neither fp64 sums
    # nor a 2^-40 fixed point can see
    q = np.float32(0.25)
    assert orc.attention_recovery(np.array([q, q, q, q], np.float32), 0.5)[0] == 2  # equality reaches
    for tiny in (2.0 ** -60, 2.0 ** -149):
        m = np.array([q, q, q, q, tiny], np.float32)
        assert float(m[4]) == tiny
        # total = 1 + tiny, half of it exceeds the top-2 sum 0.5 by tiny / 2
        assert orc.attention_recovery(m, 0.5)[0] == 3
    # thres 0.75 of [0.5, 0.25, 0.25 - 2^-30]: top-2 = 0.75 >= 0.75 (1 - 2^-32)
    m = np.array([0.5, 0.25, 0.25 - 2.0 ** -30], np.float32)
    assert orc.attention_recovery(m, 0.75)[0] == 2


@pytest.mark.parametrize("T,seed", [(57, 0), (5120, 1), (8192, 2)])
def test_attention_recovery_property_by_correctly_rounded_sums(T, seed):
    # AR is the first k whose top-k mass reaches thres of the total: checked with
    # math.fsum (correctly rounded) sums where the margin exceeds their rounding
    import math
    r = _rng(200 + seed)
    m = (r.exponential(size=T) / T).astype(np.float32)
    m = np.minimum(m, np.float32(1.0))
    ar, order = orc.attention_recovery(m, 0.55)
    vals = m.astype(np.float64)
    assert sorted(order.tolist()) == list(range(T))
    assert all(vals[order[i]] >= vals[order[i + 1]] for i in range(T - 1))
    total = math.fsum(vals)
    s_ar = math.fsum(vals[order[:ar]])
    s_prev = math.fsum(vals[order[:ar - 1]])
    eps = 4 * T * 2.0 ** -53 * total
    assert s_ar >= 0.55 * total - eps and s_prev < 0.55 * total + eps
    assert s_ar - 0.55 * total > -eps and (ar == 1 or 0.55 * total - s_prev > -eps)


def test_attention_recovery_rejects_masses_outside_unit_interval():
    for bad in ([0.5, -0.1], [1.5], [np.nan], [np.inf]):
        with pytest.raises(ValueError):
            orc.attention_recovery(np.array(bad, np.float32))


def test_attention_recovery_closed_forms():
    assert orc.attention_recovery(np.full(10, 0.1, np.float32), 0.55)[0] == 6  # ceil(0.55 * 10)
    assert orc.attention_recovery(np.full(201, 0.004, np.float32), 0.55)[0] == 111  # ceil(110.55)
    # thres is the exact value of its double: fl(0.55) exceeds 55/100, so 200
    # equal masses need 111 tokens (0.55 * 200 is 110 plus 8.9e-15)
    assert orc.attention_recovery(np.full(200, 0.005, np.float32), 0.55)[0] == 111
    assert orc.attention_recovery(np.full(200, 0.005, np.float32), 0.5)[0] == 100  # exact binary fraction
    one = np.full(50, 0.001, np.float32); one[31] = 0.9
    ar, order = orc.attention_recovery(one, 0.55)
    assert ar == 1 and order[0] == 31
    assert orc.attention_recovery(np.zeros(5, np.float32), 0.55)[0] == 1  # 0 >= 0 at once
    assert orc.attention_recovery(np.zeros(0, np.float32), 0.55)[0] == 0
    ties = np.array([0.2, 0.3, 0.2, 0.3], np.float32)
    assert orc.attention_recovery(ties, 0.55)[1].tolist() == [1, 3, 0, 2]  # lower position first on ties


def test_dynamic_recompute_counts_and_ties():
    n = 42
    m = np.full(n, 1.0 / n, np.float32)           # AR = ceil(0.55 * 42) = 24: positions 0..23 hot
    sig = np.ones(n, np.float32)                  # all equal: the lowest positions of each group
    ar, sel, n_hot = orc.dynamic_recompute(m, sig, 0.55, 0.5, 0.1)
    assert ar == 24 and n_hot == 12
    assert sel.tolist() == list(range(12)) + [24, 25]  # floor(0.1 * 18 + 1/2) = 2 cold
    # the deviation decides within each group
    sig2 = np.arange(n, dtype=np.float32)
    _, sel2, _ = orc.dynamic_recompute(m, sig2, 0.55, 0.5, 0.1)
    assert sel2.tolist() == list(range(12, 24)) + [40, 41]
    # w = 1 recomputes everything, w = 0 nothing
    assert orc.dynamic_recompute(m, sig2, 0.55, 1.0, 1.0)[1].tolist() == list(range(n))
    assert orc.dynamic_recompute(m, sig2, 0.55, 0.0, 0.0)[1].size == 0
    # an AR given by the caller replaces the computed one
    assert orc.dynamic_recompute(m, sig2, 0.55, 0.5, 0.1, ar=10)[0] == 10


def test_window_mass_last_row_is_its_softmax():
    # row_begin = T - 1: the mass is the last row's softmax averaged over heads
    r = _rng(7)
    T, hq, D = 11, 2, 8
    q, k = r.normal(size=(T, hq, D)), r.normal(size=(T, 1, D))
    m = orc.attention_mass(q, k, hq, 1, D, row_begin=T - 1)
    want = np.zeros(T)
    for h in range(hq):
        s = k[:, 0, :] @ q[T - 1, h, :] / np.sqrt(D)
        e = np.exp(s - s.max())
        want += e / e.sum()
    assert np.allclose(m, want / hq, rtol=0, atol=1e-15) and abs(m.sum() - 1) < 1e-12
    # the window average of every row is the full mass
    assert np.allclose(orc.attention_mass(q, k, hq, 1, D, row_begin=0), orc.attention_mass(q, k, hq, 1, D))


def test_retention_rules():
    n = 50
    m = np.full(n, 1.0 / n, np.float32)               # AR = 28 at 0.55: positions 0..27 hot
    ar, sel, _ = orc.dynamic_recompute(m, np.arange(n, dtype=np.float32))
    assert ar == 28
    score = np.arange(n, dtype=np.float32)[::-1].copy()  # lower positions score higher
    rank, kept, keep = orc.retention(m, score, ar, sel, 0.8)
    forced = set(range(28)) | set(sel.tolist())
    assert keep == 40                                   # floor(0.8 * 50 + 1/2)
    assert set(kept.tolist()) >= forced                 # never evicted
    assert sorted(rank[sorted(forced)].tolist()) == list(range(len(forced)))  # forced rank first
    rest = [j for j in range(n) if j not in forced]
    assert [j for j in np.argsort(rank) if j not in forced] == rest  # then by score (descending)
    assert kept.tolist() == sorted(np.argsort(rank)[:keep].tolist())
    # min_keep 1 keeps all; a large AR overrides min_keep; nested sets for fewer kept
    assert orc.retention(m, score, ar, sel, 1.0)[2] == n
    assert orc.retention(m, score, 45, [], 0.8)[2] == 45
    assert orc.retention(m, score, 45, sel, 0.8)[2] == 47  # 45 hot + the 2 cold recomputed: all kept
    assert set(np.argsort(rank)[:30].tolist()) <= set(kept.tolist())


def test_mass_columns_in_c_closed_forms():
    # the C statement of the same definition: q = 0 gives the harmonic form,
    # one dominant key gives e^a / (e^a + i) row by row, masses sum to 1
    T = 23
    k = _rng(11).normal(size=(T, 1, 16))
    m = orc.attention_mass_cols(np.zeros((T, 2, 16)), k, 2, 1, 16)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    assert np.allclose(m, (H[T] - H[:T]) / T, rtol=0, atol=1e-15)
    T, D, a = 17, 4, 3.0
    q = np.zeros((T, 1, D)); q[:, 0, 0] = 1.0
    k = np.zeros((T, 1, D)); k[0, 0, 0] = a * np.sqrt(D)
    m = orc.attention_mass_cols(q, k, 1, 1, D)
    i = np.arange(T)
    assert abs(m[0] - np.mean(np.exp(a) / (np.exp(a) + i))) < 1e-14
    assert all(abs(m[j] - np.sum(1.0 / (np.exp(a) + i[j:])) / T) < 1e-14 for j in range(1, T))
    r = _rng(12)
    q, k = r.normal(size=(30, 4, 8)), r.normal(size=(30, 2, 8))
    assert abs(orc.attention_mass_cols(q, k, 4, 2, 8).sum() - 1.0) < 1e-12


@pytest.mark.parametrize("T,hq,hkv,D,row_begin", [(9, 4, 2, 8, 0), (40, 4, 4, 16, 0), (33, 8, 2, 8, 20),
                                                  (64, 4, 1, 128, 63)])
def test_mass_columns_in_c_equal_the_matrix_form(T, hq, hkv, D, row_begin):
    r = _rng(T + D)
    q, k = r.normal(size=(T, hq, D)), r.normal(size=(T, hkv, D))
    full = orc.attention_mass(q, k, hq, hkv, D, row_begin=row_begin)
    assert np.allclose(orc.attention_mass_cols(q, k, hq, hkv, D, row_begin=row_begin), full, rtol=0, atol=1e-15)
    cols = np.array([T - 1, 0, T // 2])
    assert np.allclose(orc.attention_mass_cols(q, k, hq, hkv, D, row_begin=row_begin, cols=cols), full[cols],
                       rtol=0, atol=1e-15)
