"""Pins of the oracle's rounding, RoPE (Appendix A.1 Eq. 1) and sign-bit LSH
(Section 4.3, Appendix A.2) against closed forms, invariants and independent
library routines.  CPU only."""
import math
from fractions import Fraction

import numpy as np
import pytest

import workloads


# ------------------------------------------------------------------ rounding

def _bf16_exact(v: float) -> float:
    """Nearest bf16 of v by exact rational arithmetic (ties to even)."""
    if v == 0.0:
        return v
    f = Fraction(v)
    e = math.frexp(v)[1]
    sh = max(e - 8, -133)
    q = f / Fraction(2) ** sh
    lo = math.floor(q)
    rem = q - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    return math.ldexp(float(lo), sh)


def test_bf16_rounding_matches_exact_rational(orc):
    rng = np.random.default_rng(5)
    vals = list(rng.standard_normal(2000) * 10.0 ** rng.integers(-30, 30, 2000))
    # exact ties and near-ties at both parities, incl. ones a detour via fp32 gets wrong
    for a in (1.0, 1.0078125, 3.140625, -2.5, 1e-3):
        a = _bf16_exact(a)
        h = math.ldexp(1.0, math.frexp(a)[1] - 9)  # half an ulp of bf16 at a
        vals += [a + h, a - h, a + h + h * 2.0 ** -30, a + h - h * 2.0 ** -30, a + 3 * h]
    got = orc.round_to(np.array(vals), "bf16")
    exp = np.array([_bf16_exact(float(v)) for v in vals])
    assert np.array_equal(got, exp)


def test_bf16_rounding_matches_generator_rounding_on_fp32(orc):
    rng = np.random.default_rng(6)
    x = (rng.standard_normal(5000) * 100).astype(np.float32)
    assert np.array_equal(orc.round_to(x, "bf16"), workloads.round_bf16(x).astype(np.float64))


def test_fp32_rounding(orc):
    rng = np.random.default_rng(7)
    x = rng.standard_normal(1000)
    assert np.array_equal(orc.round_to(x, "fp32"), x.astype(np.float32).astype(np.float64))


# ---------------------------------------------------------------------- RoPE

def test_rope_position_zero_is_identity(orc):
    x = np.random.default_rng(1).standard_normal((1, 64))
    assert np.array_equal(orc.rope_embed(x, pos0=0), x)
    xb = workloads.round_bf16(x.astype(np.float32))
    assert np.array_equal(orc.rope_embed(xb, pos0=0, dtype="bf16"), xb)


@pytest.mark.parametrize("m", [1, 7, 1000, 32767])
def test_rope_known_angles(orc, m):
    # d = 8, base 1e4: theta_k = 1e4^(-2k/8) = 1, 0.1, 0.01, 0.001
    thetas = [1.0, 0.1, 0.01, 0.001]
    for k, th in enumerate(thetas):
        for which in (0, 1):
            x = np.zeros((m + 1, 8))
            x[m, 2 * k + which] = 1.0
            y = orc.rope_embed(x, pos0=0)[m]
            a = m * th
            exp = np.zeros(8)
            if which == 0:
                exp[2 * k], exp[2 * k + 1] = math.cos(a), math.sin(a)
            else:
                exp[2 * k], exp[2 * k + 1] = -math.sin(a), math.cos(a)
            np.testing.assert_allclose(y, exp, rtol=0, atol=1e-12)


def test_rope_pos0_offset(orc):
    x = np.random.default_rng(2).standard_normal((10, 16))
    full = orc.rope_embed(np.vstack([np.zeros((5, 16)), x]), pos0=0)[5:]
    np.testing.assert_allclose(orc.rope_embed(x, pos0=5), full, rtol=0, atol=0)


def test_rope_preserves_pair_norms(orc):
    x = np.random.default_rng(3).standard_normal((300, 128))
    y = orc.rope_embed(x, pos0=12345)
    nx = x[:, 0::2] ** 2 + x[:, 1::2] ** 2
    ny = y[:, 0::2] ** 2 + y[:, 1::2] ** 2
    np.testing.assert_allclose(ny, nx, rtol=1e-12)


def test_rope_inner_product_depends_on_offset_only(orc):
    rng = np.random.default_rng(4)
    d = 32
    a, b = rng.standard_normal(d), rng.standard_normal(d)
    dots = []
    for m, n in [(5, 2), (105, 102), (3003, 3000)]:
        T = max(m, n) + 1
        xa = np.zeros((T, d)); xa[m] = a
        xb = np.zeros((T, d)); xb[n] = b
        dots.append(orc.rope_embed(xa)[m] @ orc.rope_embed(xb)[n])
    np.testing.assert_allclose(dots, dots[0], rtol=1e-9)
    # and the offset changes it
    T = 11
    xa = np.zeros((T, d)); xa[10] = a
    xb = np.zeros((T, d)); xb[2] = b
    assert abs(orc.rope_embed(xa)[10] @ orc.rope_embed(xb)[2] - dots[0]) > 1e-3


def test_rope_interleaved_pairs_not_half_split(orc):
    # a half-split pairing would move energy from element 0 into element d/2
    x = np.zeros((4, 16)); x[3, 0] = 1.0
    y = orc.rope_embed(x)[3]
    assert y[8] == 0.0 and abs(y[1] - math.sin(3.0)) < 1e-15


def test_rope_rounds_once_to_storage(orc):
    x = workloads.round_bf16(np.random.default_rng(8).standard_normal((64, 32)).astype(np.float32))
    y64 = orc.rope_embed(x, pos0=100, dtype="f64")
    assert np.array_equal(orc.rope_embed(x, pos0=100, dtype="bf16"), orc.round_to(y64, "bf16"))
    assert np.array_equal(orc.rope_embed(x, pos0=100, dtype="fp32"), orc.round_to(y64, "fp32"))


# ----------------------------------------------------------------------- LSH

def _py_code(bits):
    words = []
    for w in range(len(bits) // 64):
        words.append(sum(1 << j for j in range(64) if bits[64 * w + j]))
    return words


@pytest.mark.parametrize("n_bits", [64, 128, 256])
def test_lsh_identity_planes_give_sign_bits_lsb_first(orc, n_bits):
    rng = np.random.default_rng(n_bits)
    x = rng.standard_normal((5, n_bits))
    x[0, 3] = 0.0  # exactly zero projection -> bit 0
    planes = np.eye(n_bits)
    codes = orc.lsh_encode(x, planes)
    for t in range(5):
        exp = _py_code([x[t, j] > 0 for j in range(n_bits)])
        assert [int(c) for c in codes[t]] == exp


def test_lsh_projection_equals_matmul(orc):
    rng = np.random.default_rng(9)
    x, r = rng.standard_normal((40, 96)), rng.standard_normal((128, 96))
    np.testing.assert_allclose(orc.lsh_project(x, r), x @ r.T, rtol=1e-12, atol=1e-12)


def test_lsh_zero_vector_is_all_zero_code(orc):
    r = np.random.default_rng(10).standard_normal((128, 32))
    assert not orc.lsh_encode(np.zeros((3, 32)), r).any()


def test_lsh_scale_invariance_and_negation(orc):
    rng = np.random.default_rng(11)
    x, r = rng.standard_normal((50, 64)), rng.standard_normal((256, 64))
    c = orc.lsh_encode(x, r)
    for alpha in (0.25, 3.0, 1e6):
        assert np.array_equal(orc.lsh_encode(alpha * x, r), c)
    assert np.array_equal(orc.lsh_encode(-x, r), ~c)


def test_lsh_charikar_angle_law(orc):
    # P[bit differs] = angle(x, y) / pi for Gaussian hyperplanes
    rng = np.random.default_rng(12)
    d, nb = 48, 4096
    r = rng.standard_normal((nb, d))
    for phi in (math.pi / 6, math.pi / 3, math.pi / 2, 2 * math.pi / 3):
        u = rng.standard_normal(d); u /= np.linalg.norm(u)
        w = rng.standard_normal(d); w -= (w @ u) * u; w /= np.linalg.norm(w)
        v = math.cos(phi) * u + math.sin(phi) * w
        cu, cv = orc.lsh_encode(u[None], r), orc.lsh_encode(v[None], r)
        ham = sum(bin(int(a) ^ int(b)).count("1") for a, b in zip(cu[0], cv[0]))
        p = phi / math.pi
        assert abs(ham / nb - p) < 5 * math.sqrt(p * (1 - p) / nb)
