"""GPU parity of the average attention score per token and of the dynamic
recompute set against the oracle (Section 3 Insight 2, Section 4.3.3)."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import announce, dev, host, order_valid, recovery_valid, topk_valid

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
    """The masses of 5120 tokens, 32 / 8 heads, into the dynamic recompute set
    and retention, each side on its own values: the GPU's chain on its fp32
    masses, the oracle's on its fp64 masses (from the same q and K).  AR, the
    hot set, the recompute set, the ranking and the kept set must be equal, or,
    where floating point makes them differ, valid for the oracle's masses
    within the masses' tolerance (1e-4 relative + 1e-9)."""
    T, hq, hkv = 5120, 32, 8
    cfg = CONFIGS[2]
    announce("mass chain 5120: masses -> recompute set -> retention window -> retention")
    q, k = _qk(cfg, T, hq, hkv, tag=64)
    qd, kd = dev(q, "bf16"), dev(k, "bf16")
    mass = ss.attention_mass(qd, kd, hq, hkv)
    s_h = np.random.default_rng(65).exponential(size=T).astype(np.float32)
    sel, counts = ss.dynamic_recompute(mass, torch.from_numpy(s_h).cuda())
    m_g, c = host(mass), counts.cpu().numpy()
    m_r = orc.attention_mass_cols(q, k, hq, hkv, 128)
    tol = 1e-4 * m_r + 1e-9
    assert np.all(np.abs(m_g - m_r) <= tol)
    ar_r, order_r = orc.attention_recovery(m_r.astype(np.float32))
    ar_r2, sel_r, n_hot_r = orc.dynamic_recompute(m_r.astype(np.float32), s_h)
    # AR and the hot set: the GPU's order (by its masses) must be a valid order of the oracle's
    ar_g = int(c[0])
    order_g = np.array(sorted(range(T), key=lambda j: (-float(m_g[j]), j)))
    assert order_valid(m_r, order_g, tol)
    assert ar_g == ar_r or recovery_valid(m_r, order_g, ar_g, 0.55, float(tol.sum()))
    hot_g = np.zeros(T, bool)
    hot_g[order_g[:ar_g]] = True
    assert topk_valid(m_r, np.flatnonzero(hot_g), tol)
    sel_g = sel.cpu().numpy()[: c[1]]
    if ar_g == ar_r and np.array_equal(np.sort(order_g[:ar_g]), np.sort(order_r[:ar_r])):
        assert c[2] == n_hot_r and np.array_equal(sel_g, sel_r)  # same hot set: the same choice by deviation
    # the retention window (the last 1 - AR/T rows) and the ranking
    row_begin = min(T - 1, T - int(np.floor((1.0 - ar_g / T) * T + 0.5)))
    score = ss.attention_mass(qd, kd, hq, hkv, row_begin=row_begin)
    sc_g = host(score)
    sc_r = orc.attention_mass_cols(q, k, hq, hkv, 128, row_begin=row_begin)
    tol_s = 1e-4 * sc_r + 1e-9
    assert np.all(np.abs(sc_g - sc_r) <= tol_s), np.abs(sc_g - sc_r).max()
    rank, kept, n_kept = ss.retention(mass, score, sel, counts, 0.8)
    rank_g = rank.cpu().numpy()[:T]
    nk = int(n_kept.cpu().numpy()[0])
    forced = hot_g.copy()
    forced[sel_g] = True
    n_f = int(forced.sum())
    order_rank = np.argsort(rank_g)
    assert np.array_equal(order_rank[:n_f], np.flatnonzero(forced))  # never-evicted tokens first, by position
    assert order_valid(sc_r, order_rank[n_f:], tol_s)                  # then by window score
    assert nk == max(int(np.floor(max(0.8, ar_g / T) * T + 0.5)), n_f)
    assert np.array_equal(kept.cpu().numpy()[:nk], np.sort(order_rank[:nk]))


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
                                         (5120, 4, False), (5120, 5, True), (8192, 6, False), (8193, 7, False),
                                         (32768, 8, False), (32768, 9, True), (65536, 10, False)])
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


@pytest.mark.parametrize("T,hq,hkv,row_begin", [(300, 8, 2, 137), (5120, 32, 8, 4003), (1000, 32, 8, 999)])
def test_window_mass_reusing_normalisers(T, hq, hkv, row_begin):
    """The window pass that takes the row normalisers from the full pass's
    workspace equals the one that computes them (bit for bit: the same
    normaliser kernel wrote them) and the oracle's window average."""
    cfg = CONFIGS[1]
    announce(f"window mass reusing normalisers T={T} row_begin={row_begin}")
    q, k = _qk(cfg, T, hq, hkv, tag=90 + T)
    qd, kd = dev(q, "bf16"), dev(k, "bf16")
    ws = torch.empty(int(ss.semshare.load().semshare_attention_mass_workspace(T, hq)), dtype=torch.uint8,
                     device="cuda")
    ss.attention_mass(qd, kd, hq, hkv, workspace=ws)  # the full pass leaves the normalisers in ws
    reused = host(ss.attention_mass(qd, kd, hq, hkv, workspace=ws, row_begin=row_begin, reuse_normalisers=True))
    fresh = host(ss.attention_mass(qd, kd, hq, hkv, row_begin=row_begin))
    assert np.array_equal(reused, fresh)
    ref = orc.attention_mass_cols(q, k, hq, hkv, 128, row_begin=row_begin)
    assert np.allclose(reused, ref, rtol=1e-4, atol=1e-9), np.abs(reused - ref).max()


@pytest.mark.parametrize("T,seed,ties,min_keep", [(1, 0, False, 0.8), (50, 1, True, 0.8), (1000, 2, False, 0.8),
                                                  (5120, 3, False, 0.8), (5120, 4, True, 0.5), (8192, 5, False, 1.0),
                                                  (8193, 6, False, 0.8), (32768, 7, True, 0.8),
                                                  (65536, 8, False, 0.8)])
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
