"""The seeded input generators: determinism, storage-dtype values, and the
shape of the synthetic prompt pairs (windowed permutation, fresh fraction,
relative noise).  CPU only."""
import numpy as np

import workloads
from workloads import CONFIGS


def test_configs_shapes():
    c0, c2, c4 = CONFIGS[0], CONFIGS[2], CONFIGS[4]
    assert (c0.n_tok, c0.dim, c0.n_bits, c0.n_layers, c0.head_dim, c0.dtype) == (512, 256, 64, 2, 64, "fp32")
    assert c0.n_sel(0.2) == 102
    assert [c2.n_sel(f) for f in c2.recompute_fracs] == [512, 1280, 2560]
    assert c4.n_sel(0.1) == 3277 and CONFIGS[1].n_sel(0.25) == 256
    assert CONFIGS[3].n_words == 4 and c2.group == 4


def test_round_bf16_is_idempotent_and_nearest():
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    b = workloads.round_bf16(x)
    assert np.array_equal(workloads.round_bf16(b), b)
    assert not (b.view(np.uint32) & 0xFFFF).any()
    assert np.all(np.abs(b - x) <= np.abs(x) * 2.0 ** -8)


def test_prompt_pair_deterministic_and_structured():
    cfg = CONFIGS[0]
    a = workloads.make_prompt_pair(cfg)
    b = workloads.make_prompt_pair(cfg)
    assert np.array_equal(a.e_tgt, b.e_tgt) and np.array_equal(a.e_ref, b.e_ref)
    T = cfg.n_tok
    assert (a.pi == -1).sum() == round(cfg.fresh_frac * T)
    kept = np.nonzero(a.pi >= 0)[0]
    assert np.all(a.pi[kept] // 16 == kept // 16)  # shuffled only within windows of 16
    # relative noise: ||tgt - ref[pi]|| / ||ref[pi]|| is close to sigma
    rel = np.linalg.norm(a.e_tgt[kept] - a.e_ref[a.pi[kept]], axis=1) / np.linalg.norm(a.e_ref[a.pi[kept]], axis=1)
    assert abs(rel.mean() - cfg.noise_sigma) < 0.02


def test_bf16_config_values_are_bf16():
    cfg = CONFIGS[1]
    pair = workloads.make_prompt_pair(cfg, n_tok=64, dim=128)
    for arr in (pair.e_ref, pair.e_tgt, workloads.make_planes(cfg, dim=128),
                workloads.make_weights(cfg, 0, hidden=128, n_q_heads=4, n_kv_heads=1, head_dim=32).wq):
        assert not (arr.view(np.uint32) & 0xFFFF).any()


def test_planes_are_near_unit_norm():
    r = workloads.make_planes(CONFIGS[2])
    n = np.linalg.norm(r.astype(np.float64), axis=1)
    assert r.shape == (128, 4096) and abs(n.mean() - 1.0) < 0.01


def test_bank_layout():
    cfg = CONFIGS[3]
    bank = workloads.make_bank(cfg, n_tok=32, dim=64, n_refs=6)
    assert bank.e_refs.shape == (6 * 32, 64) and bank.e_tgt.shape == (32, 64)
    assert bank.sigmas == [0.2, 0.4, 0.6, 0.2, 0.4, 0.6]
    d0 = np.linalg.norm(bank.e_refs[:32] - bank.e_tgt, axis=1).mean()
    d2 = np.linalg.norm(bank.e_refs[64:96] - bank.e_tgt, axis=1).mean()
    assert d0 < d2


def test_sel_pos_sorted_unique_with_ends():
    p = workloads.make_sel_pos(CONFIGS[2], 5120, 1280)
    assert p.dtype == np.int32 and p[0] == 0 and p[-1] == 5119
    assert np.all(np.diff(p) > 0) and p.size == 1280
