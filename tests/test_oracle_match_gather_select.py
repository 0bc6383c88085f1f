"""Pins of the oracle's Hamming match (Section 4.3), KV gather (Section 4.3,
4.3.2), HD-token selection (Section 3 Insight 1, Section 4.2) and the
prompt-level similarity score (Appendix A.3) by brute force, library routines
and closed forms.  CPU only."""
import numpy as np
import pytest


def _py_match(tgt, ref):
    idx, dist = [], []
    for t in tgt:
        best, bj = None, -1
        for j, r in enumerate(ref):
            d = sum(bin(int(a) ^ int(b)).count("1") for a, b in zip(t, r))
            if best is None or d < best:
                best, bj = d, j
        idx.append(bj)
        dist.append(best)
    return np.array(idx), np.array(dist)


@pytest.mark.parametrize("n_words", [1, 2, 4])
def test_match_equals_brute_force(orc, n_words):
    rng = np.random.default_rng(n_words)
    tgt = rng.integers(0, 2**64, size=(37, n_words), dtype=np.uint64)
    ref = rng.integers(0, 2**64, size=(53, n_words), dtype=np.uint64)
    # plant near-duplicates and exact duplicates so ties occur
    ref[10] = tgt[3]
    ref[40] = tgt[3]
    one_bit = np.zeros(n_words, dtype=np.uint64)
    one_bit[0] = 1
    ref[7] = tgt[5] ^ one_bit
    ref[8] = tgt[5] ^ (one_bit << np.uint64(1))
    idx, dist = orc.match(tgt, ref)
    pi, pd = _py_match(tgt, ref)
    assert np.array_equal(idx, pi) and np.array_equal(dist, pd)
    assert idx[3] == 10 and dist[3] == 0 and idx[5] == 7 and dist[5] == 1


def test_match_small_codes_brute_force_exhaustive(orc):
    # every 6-bit pattern against every other, in the low bits of one word
    codes = np.arange(64, dtype=np.uint64)[:, None]
    ref = codes[::-1].copy()
    idx, dist = orc.match(codes, ref)
    pi, pd = _py_match(codes, ref)
    assert np.array_equal(idx, pi) and np.array_equal(dist, pd) and not dist.any()


def test_match_identical_prompts_self_match(orc):
    rng = np.random.default_rng(3)
    c = rng.integers(0, 2**64, size=(200, 2), dtype=np.uint64)
    idx, dist = orc.match(c, c)
    assert np.array_equal(idx, np.arange(200)) and not dist.any()


def test_match_ties_lowest_index(orc):
    ref = np.zeros((9, 2), dtype=np.uint64)
    tgt = np.array([[0, 0], [1, 0], [2**63, 2**63]], dtype=np.uint64)
    idx, dist = orc.match(tgt, ref)
    assert list(idx) == [0, 0, 0] and list(dist) == [0, 1, 2]


@pytest.mark.parametrize("n_words", [1, 2, 4])
def test_match_complement_distance_is_n_bits(orc, n_words):
    c = np.random.default_rng(4).integers(0, 2**64, size=(5, n_words), dtype=np.uint64)
    for t in range(5):
        _, dist = orc.match(c[t:t + 1], ~c[t:t + 1])
        assert dist[0] == 64 * n_words


def test_match_empty_target(orc):
    idx, dist = orc.match(np.zeros((0, 2), np.uint64), np.zeros((3, 2), np.uint64))
    assert idx.size == 0 and dist.size == 0


# -------------------------------------------------------------------- gather

def test_gather_equals_numpy_take(orc):
    rng = np.random.default_rng(5)
    src = rng.integers(0, 2**16, size=(3, 17, 4, 8), dtype=np.uint16)  # bf16 bit patterns
    idx = rng.integers(0, 17, size=29).astype(np.int32)
    got = orc.gather_rows(src, idx)
    assert got.dtype == src.dtype and np.array_equal(got, np.take(src, idx, axis=1))


def test_gather_identity_is_copy(orc):
    src = np.random.default_rng(6).standard_normal((2, 11, 3, 4)).astype(np.float32)
    assert np.array_equal(orc.gather_rows(src, np.arange(11, dtype=np.int32)), src)


def test_gather_rejects_out_of_range(orc):
    with pytest.raises(ValueError):
        orc.gather_rows(np.zeros((1, 4, 2), np.float32), np.array([0, 4], np.int32))


# -------------------------------------------------------------------- select

def test_select_matches_lexsort(orc):
    rng = np.random.default_rng(7)
    for n_tok, n_sel in [(100, 30), (257, 1), (64, 64), (50, 0)]:
        sigma = rng.integers(0, 20, size=n_tok).astype(np.float64)  # many ties
        got = orc.select_recompute(sigma, n_sel)
        order = np.lexsort((np.arange(n_tok), -sigma))  # by sigma desc, then position asc
        assert np.array_equal(got, np.sort(order[:n_sel]))


def test_select_all_equal_takes_first_positions(orc):
    assert list(orc.select_recompute(np.ones(10), 4)) == [0, 1, 2, 3]


def test_select_distinct_values(orc):
    sigma = np.array([0.5, 3.0, 0.1, 2.0, 7.0])
    assert list(orc.select_recompute(sigma, 3)) == [1, 3, 4]


# ---------------------------------------------------------------- similarity

def test_similarity_closed_forms(orc):
    assert orc.similarity(np.zeros(10, np.int32)) == 1.0
    assert orc.similarity(np.full(10, 30, np.int32)) == 0.0
    assert orc.similarity(np.full(10, 45, np.int32)) == 0.0
    assert orc.similarity(np.full(4, 15, np.int32)) == pytest.approx(0.5)
    assert orc.similarity(np.array([0, 6], np.int32)) == pytest.approx(0.9)


# ------------------------------------------------- reference retrieval (A.3)

def _py_bank(tgt, ref, offsets, dmin=0.0, dmax=30.0):
    """Brute force: per prompt, the sum of the target tokens' top-1 distances
    within it, and clip(1 - (mean - dmin) / (dmax - dmin), 0, 1)."""
    n_words = tgt.shape[1]
    sums, sims = [], []
    for b in range(len(offsets) - 1):
        prompt = ref[offsets[b]:offsets[b + 1]]
        total = 0
        for t in tgt:
            if len(prompt) == 0:
                total += 64 * n_words
                continue
            total += min(sum(bin(int(a) ^ int(c)).count("1") for a, c in zip(t, r)) for r in prompt)
        mean = total / len(tgt)
        sims.append(min(1.0, max(0.0, 1.0 - (mean - dmin) / (dmax - dmin))))
        sums.append(total)
    return np.array(sums), np.array(sims)


@pytest.mark.parametrize("n_words", [1, 2, 4])
def test_bank_similarity_equals_brute_force(orc, n_words):
    rng = np.random.default_rng(40 + n_words)
    tgt = rng.integers(0, 2**64, size=(23, n_words), dtype=np.uint64)
    lens = [7, 0, 19, 1, 11]
    ref = rng.integers(0, 2**64, size=(sum(lens), n_words), dtype=np.uint64)
    ref[30:33] = tgt[4:7] ^ np.uint64(3)  # prompt 2 holds near copies of three target tokens
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    dsum, sim = orc.bank_similarity(tgt, ref, offsets)
    ps, pm = _py_bank(tgt, ref, offsets)
    assert np.array_equal(dsum, ps)
    assert np.allclose(sim, pm, rtol=0, atol=1e-15)
    assert dsum[1] == len(tgt) * 64 * n_words  # the empty prompt: every distance the largest


def test_bank_similarity_closed_forms(orc):
    rng = np.random.default_rng(7)
    tgt = rng.integers(0, 2**64, size=(40, 2), dtype=np.uint64)
    other = rng.integers(0, 2**64, size=(40, 2), dtype=np.uint64)
    flip2 = tgt.copy()
    flip2[:, 0] ^= np.uint64(0b101)  # every token two bits away from its copy
    bank = np.concatenate([other, tgt[::-1], ~tgt, flip2])
    offsets = np.array([0, 40, 80, 120, 160], dtype=np.int64)
    dsum, sim = orc.bank_similarity(tgt, bank, offsets)
    assert dsum[1] == 0 and sim[1] == 1.0  # the same prompt in another order
    # the complemented prompt: each token's top-1 is 128 minus its largest distance to another token
    far = [max(sum(bin(int(a) ^ int(c)).count("1") for a, c in zip(t, r)) for r in tgt) for t in tgt]
    assert dsum[2] == sum(128 - f for f in far) and sim[2] == 0.0
    one, cmp1 = orc.bank_similarity(tgt[:1], ~tgt[:1], np.array([0, 1], dtype=np.int64))
    assert one[0] == 128 and cmp1[0] == 0.0  # a single token against its complement
    assert dsum[3] == 40 * 2 and sim[3] == pytest.approx(1.0 - 2.0 / 30.0)
    assert np.argmax(sim) == 1 and sim[0] < 0.8  # random codes sit far below the 0.8 gate
    # scale of the score: dmin/dmax are the paper's 0 and 30 by default
    d2, s2 = orc.bank_similarity(tgt, bank, offsets, dmin=0.0, dmax=60.0)
    assert np.array_equal(d2, dsum) and s2[3] == pytest.approx(1.0 - 2.0 / 60.0)
