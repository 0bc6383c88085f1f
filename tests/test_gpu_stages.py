"""GPU parity of the RoPE, LSH, match, gather and select kernels against the
oracle, each stage fed the oracle's (or the generator's) inputs.  Integer
results are compared bit for bit; floating-point results within the
tolerances derived in the design notes."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import (announce, bf16_ulp, bf16_ulp_distance, code_mismatch_ok, dev, dev_codes, dev_i32, host,
                     host_codes)

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------- RoPE

@pytest.mark.parametrize("cid,n_tok,dim,pos0", [
    (0, 512, 256, 0),          # tiny fp32 config
    (0, 37, 6, 3),             # ragged: width not a multiple of 8 (scalar path)
    (1, 1024, 4096, 0),        # one Llama-3-8B-shaped prompt
    (1, 64, 4096, 32700),      # positions near 32k: fp64 angle reduction matters
    (1, 5, 10, 0),             # tiny bf16, scalar path
])
def test_rope_embed_matches_oracle(cid, n_tok, dim, pos0):
    cfg = CONFIGS[cid]
    announce(f"rope cfg{cid} n_tok={n_tok} dim={dim} pos0={pos0}")
    x = workloads.make_rows(cfg, n_tok, dim, tag=1)
    y = host(ss.rope_embed(dev(x, cfg.dtype), pos0=pos0))
    # fp32 rotation error: sin/cos within ~1 ulp plus two roundings, <= 4e-7 (|x0| + |x1|)
    scale = np.abs(x[:, 0::2]).repeat(2, axis=1) + np.abs(x[:, 1::2]).repeat(2, axis=1)
    ref = orc.rope_embed(x, pos0=pos0, dtype=cfg.dtype)
    err = np.abs(y - ref)
    if cfg.dtype == "bf16":
        # both sides round once to bf16: at most one bf16 spacing apart beyond the fp32 error
        assert np.all(err <= bf16_ulp(ref) + 4e-7 * scale)
        assert (bf16_ulp_distance(y, ref) > 0).mean() < 1e-3
    else:
        assert np.all(err <= 4e-7 * scale + 1e-30)


def test_rope_embed_in_place_and_identity_at_zero():
    cfg = CONFIGS[1]
    x = workloads.make_rows(cfg, 16, 128, tag=2)
    t = dev(x, "bf16")
    announce("rope in place")
    ss.rope_embed(t, out=t, pos0=0)
    # row 0 sits at position 0: unchanged; others match the oracle
    y = host(t)
    assert np.array_equal(y[0], x[0])
    ref = orc.rope_embed(x, dtype="bf16")
    scale = np.abs(x[:, 0::2]).repeat(2, axis=1) + np.abs(x[:, 1::2]).repeat(2, axis=1)
    assert np.all(np.abs(y - ref) <= bf16_ulp(ref) + 4e-7 * scale)


# ----------------------------------------------------------------------- LSH

@pytest.mark.parametrize("cid,n_tok,dim,n_bits", [
    (0, 512, 256, 64),
    (0, 77, 132, 128),        # ragged rows, fp32 dim not a multiple of 64
    (1, 1024, 4096, 128),
    (1, 1000, 4096, 64),      # ragged (not a multiple of 32 rows)
    (3, 300, 4096, 256),      # bank code length
    (1, 33, 64, 128),         # single K chunk
])
def test_lsh_encode_matches_oracle(cid, n_tok, dim, n_bits):
    cfg = CONFIGS[cid]
    announce(f"lsh cfg{cid} n_tok={n_tok} dim={dim} n_bits={n_bits}")
    # fed the oracle's RoPE output, as the path does
    x = orc.rope_embed(workloads.make_rows(cfg, n_tok, dim, tag=3), dtype=cfg.dtype).astype(np.float32)
    planes = workloads.make_planes(cfg, n_bits=n_bits, dim=dim)
    codes = host_codes(ss.lsh_encode(dev(x, cfg.dtype), dev(planes, cfg.dtype)))
    ref = orc.lsh_encode(x, planes)
    proj = orc.lsh_project(x, planes)
    flips, outside = code_mismatch_ok(codes, ref, proj, x.astype(np.float64), planes.astype(np.float64))
    assert outside == 0, f"{flips} flips, {outside} outside the 1e-5 band"
    assert flips <= max(2, n_tok * n_bits // 20000)


@pytest.mark.parametrize("n_tok,dim,n_bits,pos0", [
    (1024, 4096, 128, 0),
    (1000, 4096, 64, 0),      # ragged last tile
    (777, 4096, 128, 100),    # positions from 100
    (3000, 512, 128, 0),      # 12 rows per workgroup
    (33, 128, 128, 32700),    # large angles
    (5, 64, 64, 0),           # one row per workgroup, one K chunk
    (256 * 33 + 7, 256, 128, 0),  # 33 rows wanted per workgroup: capped at 32
])
def test_rope_lsh_encode_matches_oracle(n_tok, dim, n_bits, pos0):
    # the fused pass against the oracle's RoPE (rounded to bf16, as stored) then LSH
    cfg = CONFIGS[1]
    announce(f"rope+lsh n_tok={n_tok} dim={dim} n_bits={n_bits} pos0={pos0}")
    x = workloads.make_rows(cfg, n_tok, dim, tag=7)
    planes = workloads.make_planes(cfg, n_bits=n_bits, dim=dim)
    codes = host_codes(ss.rope_lsh_encode(dev(x, "bf16"), dev(planes, "bf16"), pos0=pos0))
    xr = orc.rope_embed(x, pos0=pos0, dtype="bf16").astype(np.float32)
    ref = orc.lsh_encode(xr, planes)
    proj = orc.lsh_project(xr, planes)
    flips, outside = code_mismatch_ok(codes, ref, proj, xr.astype(np.float64), planes.astype(np.float64))
    assert outside == 0, f"{flips} flips, {outside} outside the 1e-5 band"
    assert flips <= max(2, n_tok * n_bits // 20000)


def test_rope_lsh_encode_equals_two_pass_path():
    # fused and unfused GPU paths on the 5120-token headline shape: codes agree
    # except for projections inside the flip band
    cfg = CONFIGS[2]
    announce("rope+lsh vs rope_embed + lsh_encode 5120 x 4096")
    x = dev(workloads.make_rows(cfg, 5120, 4096, tag=8), "bf16")
    planes = dev(workloads.make_planes(cfg, n_bits=128, dim=4096), "bf16")
    fused = host_codes(ss.rope_lsh_encode(x, planes))
    two = host_codes(ss.lsh_encode(ss.rope_embed(x), planes))
    diff = np.unpackbits((fused ^ two).view(np.uint8)).sum()
    assert diff <= 5120 * 128 // 20000


def test_lsh_zero_rows_give_zero_codes():
    cfg = CONFIGS[1]
    x = np.zeros((40, 128), np.float32)
    planes = workloads.make_planes(cfg, n_bits=128, dim=128)
    announce("lsh zero rows")
    assert not host_codes(ss.lsh_encode(dev(x, "bf16"), dev(planes, "bf16"))).any()


# --------------------------------------------------------------------- match
# Both matchers (XOR/popcount and the int8 matrix-core variant) share one
# contract and are held to the same bit-exact cases.
MATCHERS = {"xor": lambda *a, **k: ss.match(*a, **k), "mfma": lambda *a, **k: ss.match_mfma(*a, **k)}


@pytest.mark.parametrize("n_tgt,n_ref,n_words", [
    (512, 512, 1),
    (1024, 1024, 2),
    (1000, 777, 2),       # ragged both ways
    (130, 1, 2),          # single reference
    (5, 70000, 4),        # many splits, tiny target
    (4096, 4096, 4),
    (300, 2048, 3),
    (2000, 5000, 2),      # several splits with a ragged last block
])
@pytest.mark.parametrize("matcher", sorted(MATCHERS))
def test_match_matches_oracle(n_tgt, n_ref, n_words, matcher):
    cfg = CONFIGS[1]
    announce(f"match {matcher} n_tgt={n_tgt} n_ref={n_ref} W={n_words}")
    tgt = workloads.make_codes(cfg, n_tgt, n_words, tag=n_tgt)
    ref = workloads.make_codes(cfg, n_ref, n_words, tag=n_ref + 1)
    # plant exact and near matches plus duplicates so ties are exercised
    k = min(n_tgt, n_ref) // 3
    ref[:k] = tgt[:k]
    if n_ref > 2 * k + 1 and k:
        ref[k:2 * k] = tgt[:k]  # duplicates at higher indices: lowest index must win
    idx, dist = MATCHERS[matcher](dev_codes(tgt), dev_codes(ref))
    ri, rd = orc.match(tgt, ref)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), ri)
    assert np.array_equal(dist.cpu().numpy(), rd)


@pytest.mark.parametrize("matcher", sorted(MATCHERS))
def test_match_bank_shape(matcher):
    # one 4096-token target against 16 references of 4096 tokens (256-bit codes)
    cfg = CONFIGS[3]
    announce(f"match {matcher} bank 4096 x 65536 W=4")
    tgt = workloads.make_codes(cfg, 4096, 4, tag=11)
    ref = workloads.make_codes(cfg, 16 * 4096, 4, tag=12)
    ref[5 * 4096 + np.arange(0, 4096, 7)] = tgt[np.arange(0, 4096, 7)]
    idx, dist = MATCHERS[matcher](dev_codes(tgt), dev_codes(ref))
    ri, rd = orc.match(tgt, ref)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), ri) and np.array_equal(dist.cpu().numpy(), rd)


@pytest.mark.parametrize("matcher", sorted(MATCHERS))
def test_match_identical_prompts_self_match_and_no_dist(matcher):
    cfg = CONFIGS[2]
    c = workloads.make_codes(cfg, 5120, 2, tag=3)
    announce(f"match {matcher} identical 5120")
    idx, dist = MATCHERS[matcher](dev_codes(c), dev_codes(c), want_dist=False)
    assert dist is None
    assert np.array_equal(idx.cpu().numpy(), np.arange(5120))


@pytest.mark.parametrize("matcher", sorted(MATCHERS))
def test_match_complement_distance(matcher):
    cfg = CONFIGS[1]
    c = workloads.make_codes(cfg, 64, 2, tag=4)
    announce(f"match {matcher} complement")
    idx, dist = MATCHERS[matcher](dev_codes(c[:1]), dev_codes(~c[:1]))
    assert dist.cpu().numpy()[0] == 128 and idx.cpu().numpy()[0] == 0


@pytest.mark.parametrize("matcher", sorted(MATCHERS))
@pytest.mark.parametrize("n_words", [1, 2, 4])
def test_match_many_ties(matcher, n_words):
    # references drawn from 6 distinct codes: every target's nearest distance
    # is reached by hundreds of references, and the lowest index must win
    cfg = CONFIGS[1]
    announce(f"match {matcher} ties W={n_words}")
    pool = workloads.make_codes(cfg, 6, n_words, tag=20 + n_words)
    pick = np.random.default_rng(n_words).integers(0, 6, 3000)
    ref = pool[pick]
    tgt = workloads.make_codes(cfg, 700, n_words, tag=30 + n_words)
    tgt[:6] = pool  # exact hits too
    idx, dist = MATCHERS[matcher](dev_codes(tgt), dev_codes(ref))
    ri, rd = orc.match(tgt, ref)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), ri) and np.array_equal(dist.cpu().numpy(), rd)


@pytest.mark.parametrize("matcher", sorted(MATCHERS))
def test_match_all_references_equal(matcher):
    cfg = CONFIGS[1]
    announce(f"match {matcher} all references equal")
    one = workloads.make_codes(cfg, 1, 2, tag=40)
    ref = np.repeat(one, 1500, axis=0)
    tgt = workloads.make_codes(cfg, 257, 2, tag=41)
    idx, dist = MATCHERS[matcher](dev_codes(tgt), dev_codes(ref))
    _, rd = orc.match(tgt, ref)
    torch.cuda.synchronize()
    assert not idx.cpu().numpy().any() and np.array_equal(dist.cpu().numpy(), rd)


# -------------------------------------------------------------------- gather

@pytest.mark.parametrize("cid,L,n_ref,n_tgt", [(0, 2, 512, 512), (1, 3, 1024, 1000), (2, 2, 5120, 5120)])
def test_gather_kv_bitwise(cid, L, n_ref, n_tgt):
    cfg = CONFIGS[cid]
    announce(f"gather cfg{cid} L={L} n_ref={n_ref} n_tgt={n_tgt}")
    k, v = workloads.make_cache(cfg, L, n_ref, tag=cid)
    idx = np.random.default_rng(cid).integers(0, n_ref, n_tgt).astype(np.int32)
    ok, ov = ss.gather_kv(dev(k, cfg.dtype), dev(v, cfg.dtype), dev_i32(idx))
    assert np.array_equal(host(ok), orc.gather_rows(k, idx))
    assert np.array_equal(host(ov), orc.gather_rows(v, idx))


@pytest.mark.parametrize("n_except,repeats", [(0, False), (1, False), (250, False), (1000, False), (600, True)])
def test_gather_except_leaves_listed_rows(n_except, repeats):
    """The list is ascending, not necessarily strict: with repeats (600 draws
    with replacement) every listed row is still left alone exactly once."""
    cfg = CONFIGS[1]
    L, n_ref, n_tgt = 3, 777, 1000
    announce(f"gather except n_except={n_except} repeats={repeats}")
    k, v = workloads.make_cache(cfg, L, n_ref, tag=9)
    idx = np.random.default_rng(9).integers(0, n_ref, n_tgt).astype(np.int32)
    exc = np.sort(np.random.default_rng(10).choice(n_tgt, n_except, replace=repeats)).astype(np.int32)
    assert not repeats or len(np.unique(exc)) < n_except
    ok = torch.full((L, n_tgt) + k.shape[2:], 7.0, dtype=torch.bfloat16, device="cuda")
    ov = torch.full((L, n_tgt) + k.shape[2:], -3.0, dtype=torch.bfloat16, device="cuda")
    ss.gather_kv(dev(k, "bf16"), dev(v, "bf16"), dev_i32(idx), out_k=ok, out_v=ov, except_pos=dev_i32(exc))
    gk, gv = host(ok), host(ov)
    keep = np.ones(n_tgt, bool)
    keep[exc] = False
    assert np.array_equal(gk[:, keep], orc.gather_rows(k, idx)[:, keep])
    assert np.array_equal(gv[:, keep], orc.gather_rows(v, idx)[:, keep])
    assert (gk[:, ~keep] == 7.0).all() and (gv[:, ~keep] == -3.0).all()


def test_gather_identity_k_only_and_out_of_range():
    cfg = CONFIGS[1]
    k, _ = workloads.make_cache(cfg, 2, 64, tag=5)
    announce("gather identity / k-only / out of range")
    tk = dev(k, "bf16")
    ok, ov = ss.gather_kv(tk, None, dev_i32(np.arange(64)))
    assert ov is None and np.array_equal(host(ok), k)
    idx = np.array([0, -1, 63, 64, 1 << 30, 5], np.int32)
    ok, _ = ss.gather_kv(tk, None, dev_i32(idx))
    got = host(ok)
    for t, j in enumerate(idx):
        exp = k[:, j] if 0 <= j < 64 else np.zeros_like(k[:, 0])
        assert np.array_equal(got[:, t], exp)


def test_gather_rows_wide():
    cfg = CONFIGS[1]
    x = workloads.make_rows(cfg, 300, 4096, tag=6)  # 8 KB rows
    idx = np.random.default_rng(6).integers(0, 300, 111).astype(np.int32)
    announce("gather rows 8KB")
    assert np.array_equal(host(ss.gather_rows(dev(x, "bf16"), dev_i32(idx))), x[idx])


# -------------------------------------------------------------------- select

@pytest.mark.parametrize("n_tok,n_sel,levels", [
    (5120, 1280, 0), (5120, 512, 0), (5120, 2560, 7), (300, 300, 0), (300, 1, 3), (1000, 999, 2),
    (32768, 3277, 50), (17, 5, 1),
])
def test_select_recompute_matches_oracle(n_tok, n_sel, levels):
    rng = np.random.default_rng(n_tok + n_sel)
    if levels:
        sigma = rng.integers(0, levels, n_tok).astype(np.float32)  # many ties
    else:
        sigma = (rng.random(n_tok) * 50).astype(np.float32)
    announce(f"select n_tok={n_tok} n_sel={n_sel} levels={levels}")
    got = ss.select_recompute(torch.from_numpy(sigma).cuda(), n_sel).cpu().numpy()
    assert np.array_equal(got, orc.select_recompute(sigma, n_sel))


# ------------------------------------------------- reference retrieval (A.3)

def _flip(codes: np.ndarray, rate: float, seed: int) -> np.ndarray:
    """codes with each bit flipped with probability `rate` (seeded)."""
    rng = np.random.default_rng(seed)
    bits = rng.random((codes.shape[0], codes.shape[1], 64)) < rate
    mask = (bits.astype(np.uint64) << np.arange(64, dtype=np.uint64)).sum(axis=2, dtype=np.uint64)
    return codes ^ mask


@pytest.mark.gpu
@pytest.mark.parametrize("n_words", [1, 2, 4])
def test_bank_similarity_matches_oracle(n_words):
    """Sums of top-1 distances per prompt bit-exact and scores equal to the
    oracle's: prompts of 0, 1, 300, 700 (two LDS stages) and 1300 codes, a
    ragged target of 333 tokens, near copies planted at several flip rates."""
    cfg = CONFIGS[1]
    announce(f"bank similarity W={n_words}")
    tgt = workloads.make_codes(cfg, 333, n_words, tag=80 + n_words)
    lens = [300, 0, 700, 1, 1300]
    parts = [workloads.make_codes(cfg, n, n_words, tag=90 + i) if n else np.zeros((0, n_words), np.uint64)
             for i, n in enumerate(lens)]
    parts[2][:333] = _flip(tgt, 0.05, 1)   # a close prompt
    parts[4][500:833] = _flip(tgt, 0.15, 2)  # a farther one
    ref = np.concatenate(parts)
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    dsum, sim = ss.bank_similarity(dev_codes(tgt), dev_codes(ref), torch.from_numpy(offsets).cuda())
    rs, rm = orc.bank_similarity(tgt, ref, offsets)
    assert np.array_equal(dsum.cpu().numpy(), rs)
    assert np.allclose(sim.cpu().numpy(), rm, rtol=0, atol=1e-15)
    assert int(np.argmax(rm)) == 2


@pytest.mark.gpu
def test_bank_similarity_bank_shape_picks_the_closest_member():
    """One 4096-token target against a bank of 16 prompts of 4096 tokens at
    128 bits, member b holding the target with bits flipped at rate
    (0.02, 0.05, 0.1)[b % 3] (others random): the scores equal the oracle's
    and the closest member scores highest."""
    cfg = CONFIGS[3]
    announce("bank similarity 4096 x 16 x 4096 W=2")
    tgt = workloads.make_codes(cfg, 4096, 2, tag=13)
    members = []
    for b in range(16):
        m = workloads.make_codes(cfg, 4096, 2, tag=200 + b)
        if b in (3, 7, 11):
            m = _flip(tgt, (0.02, 0.05, 0.1)[(b // 4) % 3], 300 + b)[np.random.default_rng(b).permutation(4096)]
        members.append(m)
    ref = np.concatenate(members)
    offsets = (np.arange(17) * 4096).astype(np.int64)
    dsum, sim = ss.bank_similarity(dev_codes(tgt), dev_codes(ref), torch.from_numpy(offsets).cuda())
    rs, rm = orc.bank_similarity(tgt, ref, offsets)
    assert np.array_equal(dsum.cpu().numpy(), rs)
    assert np.allclose(sim.cpu().numpy(), rm, rtol=0, atol=1e-15)
    assert int(np.argmax(sim.cpu().numpy())) == 3


@pytest.mark.gpu
def test_bank_similarity_empty_target():
    cfg = CONFIGS[1]
    announce("bank similarity empty target")
    ref = workloads.make_codes(cfg, 10, 2, tag=5)
    dsum, sim = ss.bank_similarity(dev_codes(np.zeros((0, 2), np.uint64)), dev_codes(ref),
                                   torch.tensor([0, 4, 10], dtype=torch.int64, device="cuda"))
    assert dsum.cpu().tolist() == [0, 0] and sim.cpu().tolist() == [0.0, 0.0]
