"""GPU parity of the average attention score per token and of the dynamic
recompute set against the oracle (Section 3 Insight 2, Section 4.3.3)."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import announce, dev, host

pytestmark = pytest.mark.gpu


def _qk(cfg, T, hq, hkv, tag):
    q = orc.round_to(workloads.make_rows(cfg, T, hq * 128, tag=tag), "bf16").astype(np.float32)
    k = orc.round_to(workloads.make_rows(cfg, T, hkv * 128, tag=tag + 1), "bf16").astype(np.float32)
    return q.reshape(T, hq, 128), k.reshape(T, hkv, 128)


@pytest.mark.parametrize("T,hq,hkv", [(64, 4, 4), (300, 32, 8), (1024, 32, 8), (33, 8, 2)])
def test_attention_mass_matches_oracle(T, hq, hkv):
    cfg = CONFIGS[1]
    announce(f"attention mass T={T} hq={hq} hkv={hkv}")
    q, k = _qk(cfg, T, hq, hkv, tag=50 + T)
    m = host(ss.attention_mass(dev(q, "bf16"), dev(k, "bf16"), hq, hkv))
    ref = orc.attention_mass(q, k, hq, hkv, 128)
    # fp32 scores of exact bf16 products, exp2 within a few ulp, fp32 sums over <= T rows
    assert np.allclose(m, ref, rtol=1e-4, atol=1e-8), np.abs(m - ref).max()
    assert abs(m.astype(np.float64).sum() - 1.0) < 1e-4


def test_attention_mass_headline_shape_properties():
    # 5120 tokens, 32 / 8 heads: the masses sum to 1, and with q = 0 every row is
    # uniform over its keys, so mass_j = (H_T - H_j) / T exactly in exact arithmetic
    T, hq, hkv = 5120, 32, 8
    cfg = CONFIGS[2]
    announce("attention mass 5120 x 32/8")
    q, k = _qk(cfg, T, hq, hkv, tag=60)
    m = host(ss.attention_mass(dev(q, "bf16"), dev(k, "bf16"), hq, hkv)).astype(np.float64)
    assert abs(m.sum() - 1.0) < 1e-3 and (m > 0).all()
    mz = host(ss.attention_mass(torch.zeros(T, hq, 128, dtype=torch.bfloat16, device="cuda"), dev(k, "bf16"),
                                hq, hkv)).astype(np.float64)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, T + 1))])
    assert np.allclose(mz, (H[T] - H[:T]) / T, rtol=2e-4, atol=0)
    # every key column against the oracle's definition (plain C, fp64)
    ref = orc.attention_mass_cols(q, k, hq, hkv, 128)
    assert np.allclose(m, ref, rtol=1e-4, atol=1e-9), np.abs(m - ref).max()


def test_headline_mass_chain_into_selection_and_retention():
    """The GPU's own masses at 5120 tokens, 32 / 8 heads feed the GPU's
    dynamic recompute set and retention (window of the last 1 - AR/T rows);
    the oracle takes the same decisions on the same fp32 masses (floating
    point decides integers here, so both sides decide on the GPU's values),
    and the window masses match the oracle's definition."""
    T, hq, hkv = 5120, 32, 8
    cfg = CONFIGS[2]
    announce("mass chain 5120: masses -> recompute set -> retention window -> retention")
    q, k = _qk(cfg, T, hq, hkv, tag=64)
    qd, kd = dev(q, "bf16"), dev(k, "bf16")
    mass = ss.attention_mass(qd, kd, hq, hkv)
    sigma = torch.from_numpy(np.random.default_rng(65).exponential(size=T).astype(np.float32)).cuda()
    sel, counts = ss.dynamic_recompute(mass, sigma)
    m_h, s_h, c = host(mass).astype(np.float32), sigma.cpu().numpy(), counts.cpu().numpy()
    ar, ref_sel, n_hot = _oracle_dyn(m_h, s_h, int(c[0]))
    assert c[0] == ar and c[2] == n_hot and c[1] == len(ref_sel)
    assert np.array_equal(sel.cpu().numpy()[: c[1]], ref_sel)
    row_begin = min(T - 1, T - int(np.floor((1.0 - ar / T) * T + 0.5)))
    score = ss.attention_mass(qd, kd, hq, hkv, row_begin=row_begin)
    sc_h = host(score).astype(np.float32)
    cols = np.unique(np.concatenate([[0, T - 1], np.random.default_rng(66).choice(T, 254, replace=False)]))
    ref_sc = orc.attention_mass_cols(q, k, hq, hkv, 128, row_begin=row_begin, cols=cols)
    assert np.allclose(sc_h[cols], ref_sc, rtol=1e-4, atol=1e-9), np.abs(sc_h[cols] - ref_sc).max()
    rank, kept, n_kept = ss.retention(mass, score, sel, counts, 0.8)
    ref_rank, ref_kept, ref_keep = orc.retention(m_h, sc_h, ar, ref_sel, 0.8)
    nk = int(n_kept.cpu().numpy()[0])
    assert nk == ref_keep
    assert np.array_equal(rank.cpu().numpy()[:T], ref_rank)
    assert np.array_equal(kept.cpu().numpy()[:nk], ref_kept)


def _dyn_inputs(T, seed, ties):
    r = np.random.default_rng(seed)
    if ties:
        m = r.integers(1, 5, T).astype(np.float32) / np.float32(4 * T)
        s = r.integers(0, 3, T).astype(np.float32)
    else:
        m = (r.exponential(size=T) / T).astype(np.float32)
        s = r.exponential(size=T).astype(np.float32)
    return np.minimum(m, np.float32(1.0)), s


def _ar_valid(m32, ar_gpu, thres=0.55):
    """The kernel sums masses in 2^-40 fixed point and forms thres * total in
    fp64, so its AR can differ from the exact one only where the exact top-k
    sum S_k lies within eps = n 2^-40 + S 2^-53 of thres * S.  True when ar_gpu
    is the exact AR or such a neighbour: S_ar >= thres S - eps and
    S_(ar-1) <= thres S + eps."""
    from fractions import Fraction
    vals = [Fraction(float(v)) for v in np.asarray(m32, np.float32)]
    n = len(vals)
    order = sorted(range(n), key=lambda j: (-vals[j], j))
    total = sum(vals)
    eps = Fraction(n, 2 ** 40) + total / 2 ** 53
    goal = Fraction(thres) * total
    s_prev = sum(vals[j] for j in order[:ar_gpu - 1])
    s_ar = s_prev + vals[order[ar_gpu - 1]]
    return 1 <= ar_gpu <= n and s_ar >= goal - eps and (ar_gpu == 1 or s_prev <= goal + eps)


def _oracle_dyn(m, s, ar_gpu, **kw):
    """The oracle's recompute set; where the GPU's AR is a valid neighbour of
    the exact one (see _ar_valid), the oracle continues from the GPU's AR."""
    ar, sel, n_hot = orc.dynamic_recompute(m, s, **kw)
    if ar_gpu != ar:
        assert _ar_valid(m, ar_gpu, kw.get("thres", 0.55)), (ar_gpu, ar)
        ar, sel, n_hot = orc.dynamic_recompute(m, s, ar=ar_gpu, **kw)
    return ar, sel, n_hot


@pytest.mark.parametrize("T,seed,ties", [(1, 0, False), (7, 1, False), (100, 2, True), (1000, 3, False),
                                         (5120, 4, False), (5120, 5, True), (8192, 6, False)])
def test_dynamic_recompute_matches_oracle(T, seed, ties):
    announce(f"dynamic recompute T={T} ties={ties}")
    m, s = _dyn_inputs(T, seed, ties)
    sel, counts = ss.dynamic_recompute(torch.from_numpy(m).cuda(), torch.from_numpy(s).cuda())
    c = counts.cpu().numpy()
    ar, ref_sel, n_hot = _oracle_dyn(m, s, int(c[0]))
    assert c[0] == ar and c[2] == n_hot and c[1] == len(ref_sel)
    assert np.array_equal(sel.cpu().numpy()[: c[1]], ref_sel)


def test_dynamic_recompute_weights_and_empty():
    m, s = _dyn_inputs(500, 9, False)
    mt, st = torch.from_numpy(m).cuda(), torch.from_numpy(s).cuda()
    announce("dynamic recompute w = 1 / w = 0 / empty")
    sel, counts = ss.dynamic_recompute(mt, st, w_hot=1.0, w_cold=1.0)
    assert counts.cpu().numpy()[1] == 500 and np.array_equal(sel.cpu().numpy(), np.arange(500))
    _, counts = ss.dynamic_recompute(mt, st, w_hot=0.0, w_cold=0.0)
    assert counts.cpu().numpy()[1] == 0
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    _, counts = ss.dynamic_recompute(e, e)
    assert counts.cpu().numpy().tolist() == [0, 0, 0]


def test_dynamic_recompute_ar_within_the_fixed_point_band():
    # [1/4] * 4 + [2^-60] at thres 1/2: the exact AR is 3 (the total exceeds 1
    # by 2^-60), a 2^-40 fixed point sees 2; both are within the kernel's band
    m = np.array([0.25] * 4 + [2.0 ** -60], np.float32)
    s = np.arange(5, dtype=np.float32)
    announce("dynamic recompute: AR tie inside the fixed-point band")
    sel, counts = ss.dynamic_recompute(torch.from_numpy(m).cuda(), torch.from_numpy(s).cuda(), thres=0.5)
    c = counts.cpu().numpy()
    assert orc.attention_recovery(m, 0.5)[0] == 3
    assert c[0] in (2, 3) and _ar_valid(m, int(c[0]), 0.5)
    ar, ref_sel, n_hot = _oracle_dyn(m, s, int(c[0]), thres=0.5)
    assert c[1] == len(ref_sel) and np.array_equal(sel.cpu().numpy()[: c[1]], ref_sel)


@pytest.mark.parametrize("T,row_begin", [(300, 137), (1024, 900), (64, 63)])
def test_window_mass_matches_oracle(T, row_begin):
    cfg = CONFIGS[1]
    announce(f"window mass T={T} row_begin={row_begin}")
    q, k = _qk(cfg, T, 8, 2, tag=80 + T)
    m = host(ss.attention_mass(dev(q, "bf16"), dev(k, "bf16"), 8, 2, row_begin=row_begin))
    ref = orc.attention_mass(q, k, 8, 2, 128, row_begin=row_begin)
    assert np.allclose(m, ref, rtol=1e-4, atol=1e-8), np.abs(m - ref).max()


@pytest.mark.parametrize("T,seed,ties,min_keep", [(1, 0, False, 0.8), (50, 1, True, 0.8), (1000, 2, False, 0.8),
                                                  (5120, 3, False, 0.8), (5120, 4, True, 0.5), (8192, 5, False, 1.0)])
def test_retention_matches_oracle(T, seed, ties, min_keep):
    announce(f"retention T={T} ties={ties} min_keep={min_keep}")
    m, s = _dyn_inputs(T, seed, ties)
    score = _dyn_inputs(T, seed + 100, ties)[0]
    mt, st, sct = (torch.from_numpy(a).cuda() for a in (m, s, score))
    sel, counts = ss.dynamic_recompute(mt, st)          # the GPU's own selection feeds the GPU retention
    rank, kept, n_kept = ss.retention(mt, sct, sel, counts, min_keep)
    ar, ref_sel, _ = _oracle_dyn(m, s, int(counts.cpu().numpy()[0]))  # the oracle's selection feeds the oracle
    ref_rank, ref_kept, ref_keep = orc.retention(m, score, ar, ref_sel, min_keep)
    nk = int(n_kept.cpu().numpy()[0])
    assert nk == ref_keep
    assert np.array_equal(rank.cpu().numpy()[:T], ref_rank)
    assert np.array_equal(kept.cpu().numpy()[:nk], ref_kept)
