"""Pins for the oracle's RoPE re-encode (§4.1, Eq. (1)) and its rounding.

R(t) is the RoFormer rotation on pairs of the head dimension. The pairing
(j, j + d/2), frequencies theta_j = base^(-2j/d) and the sign of the rotation
are pinned against a second formulation (complex multiplication), against the
HuggingFace Qwen3 helper the paper's caches come from, and by the identities
the paper relies on (relative position, norm preservation, composition)."""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle


def test_theta0_is_one_and_first_pair_closed_form():
    d = 64
    th = oracle.rope_inv_freq(d, 1e4)
    assert th[0] == 1.0
    assert abs(th[-1] - 1e4 ** (-(d - 2) / d)) <= 1e-16
    for s in (1, 7, 300):
        e0 = np.zeros(d)
        e0[0] = 1.0
        c, sn = oracle.rope_angles(s, d, 1e4)
        y = oracle.rotate_pairs(e0, c, sn)
        assert y[0] == math.cos(s) and y[d // 2] == math.sin(s)
        assert np.count_nonzero(y) == 2


def test_matches_complex_multiplication():
    rng = np.random.default_rng(0)
    d = 128
    x = rng.standard_normal((5, d))
    for s in (0, 1, 513, 260_000):
        c, sn = oracle.rope_angles(s, d, 1e6)
        y = oracle.rotate_pairs(x, c, sn)
        theta = 1e6 ** (-np.arange(0, d, 2) / d)
        z = (x[:, : d // 2] + 1j * x[:, d // 2:]) * np.exp(1j * s * theta)
        # theta_j from numpy's array pow may differ from the scalar pow by an ulp,
        # which the angle s * theta_j amplifies by s
        tol = 1e-13 + s * 4e-16 * np.abs(x).max()
        assert np.allclose(y[:, : d // 2], z.real, rtol=0, atol=tol)
        assert np.allclose(y[:, d // 2:], z.imag, rtol=0, atol=tol)


def test_matches_huggingface_qwen3_convention():
    torch = pytest.importorskip("torch")
    mq = pytest.importorskip("transformers.models.qwen3.modeling_qwen3")
    rng = np.random.default_rng(1)
    d, base = 64, 1e4
    k = torch.from_numpy(rng.standard_normal((1, 2, 3, d)))
    for s in (1, 17, 90):
        c, sn = oracle.rope_angles(s, d, base)
        cos = torch.from_numpy(np.concatenate([c, c]))[None, None, :].expand(1, 3, d)
        sin = torch.from_numpy(np.concatenate([sn, sn]))[None, None, :].expand(1, 3, d)
        _, k_hf = mq.apply_rotary_pos_emb(k, k, cos, sin)
        y = oracle.rotate_pairs(k.numpy(), c, sn)
        assert np.allclose(k_hf.numpy(), y, rtol=0, atol=1e-14)
    # HF's default frequencies (fp32) agree with theta_j = base^(-2j/d)
    inv = 1.0 / (base ** (torch.arange(0, d, 2, dtype=torch.int64).float() / d))
    assert np.allclose(inv.double().numpy(), oracle.rope_inv_freq(d, base), rtol=1e-6, atol=0)


def test_relative_position_identity():
    """<R(a) q, R(b) k> = <q, R(b - a) k>: attention sees only the displacement."""
    rng = np.random.default_rng(2)
    d = 64
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    for a, b in ((3, 10), (100, 37), (0, 5000)):
        qa = oracle.rotate_pairs(q, *oracle.rope_angles(a, d, 1e4))
        kb = oracle.rotate_pairs(k, *oracle.rope_angles(b, d, 1e4))
        kd = oracle.rotate_pairs(k, *oracle.rope_angles(b - a, d, 1e4))
        assert abs(qa @ kb - q @ kd) <= 1e-11 * (np.linalg.norm(q) * np.linalg.norm(k))


def test_norm_preservation_composition_inverse():
    rng = np.random.default_rng(3)
    d = 128
    x = rng.standard_normal((4, d))
    ra = oracle.rope_angles(700, d, 1e6)
    rb = oracle.rope_angles(4000, d, 1e6)
    rab = oracle.rope_angles(4700, d, 1e6)
    rneg = oracle.rope_angles(-700, d, 1e6)
    ya = oracle.rotate_pairs(x, *ra)
    pair_norm = lambda v: np.hypot(v[..., : d // 2], v[..., d // 2:])
    assert np.allclose(pair_norm(ya), pair_norm(x), rtol=1e-14, atol=0)
    assert np.allclose(oracle.rotate_pairs(ya, *rb), oracle.rotate_pairs(x, *rab), rtol=0, atol=1e-12)
    assert np.allclose(oracle.rotate_pairs(ya, *rneg), x, rtol=0, atol=1e-13)


def test_interleaved_style_pairs_adjacent_elements():
    d = 8
    x = np.arange(1.0, d + 1)
    c, sn = oracle.rope_angles(3, d, 1e4)
    y = oracle.rotate_pairs(x, c, sn, style="interleaved")
    for j in range(d // 2):
        z = (x[2 * j] + 1j * x[2 * j + 1]) * complex(c[j], sn[j])
        assert abs(y[2 * j] - z.real) < 1e-14 and abs(y[2 * j + 1] - z.imag) < 1e-14


# ----------------------------------------------------------------- rounding to bf16

def _bf16_value(bits):
    return float(oracle.bf16_bits_to_f64(np.array([bits], np.uint16))[0])


def _exact_rne_bf16(y: float) -> int:
    """Brute force: among all finite bf16 values pick the nearest to y exactly
    (rational arithmetic), ties to the even bit pattern; beyond the last
    midpoint the result is infinity."""
    if math.isnan(y):
        return 0x7FC0
    sign = 0x8000 if math.copysign(1.0, y) < 0 else 0
    a = abs(y)
    if math.isinf(a):
        return sign | 0x7F80
    fa = Fraction(a)
    lo, hi = 0, 0x7F7F
    while lo < hi:                                  # largest pattern with value <= a
        mid = (lo + hi + 1) // 2
        if Fraction(_bf16_value(mid)) <= fa:
            lo = mid
        else:
            hi = mid - 1
    below = lo
    if Fraction(_bf16_value(below)) == fa:
        return sign | below
    if below == 0x7F7F:
        top = Fraction(_bf16_value(0x7F7F))
        half_ulp = Fraction(2) ** (127 - 8)
        return sign | (0x7F80 if fa >= top + half_ulp else 0x7F7F)
    above = below + 1
    db = fa - Fraction(_bf16_value(below))
    da = Fraction(_bf16_value(above)) - fa
    if db < da or (db == da and below % 2 == 0):
        return sign | below
    return sign | above


def test_bf16_rounding_against_exact_rationals():
    rng = np.random.default_rng(4)
    vals = list(rng.standard_normal(300) * np.exp2(rng.integers(-140, 128, 300)))
    vals += list(rng.standard_normal(200))
    vals += [3.3895e38, 3.3961e38, 3.39e38, 1e39, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135,
             2.0 ** -126, 2.0 ** -127 * 1.00390625, -0.0, 0.0, 1.0 + 2.0 ** -8,
             1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -30, float("inf"), -float("inf")]
    y = np.array(vals, np.float64)
    got = oracle.f64_to_bf16_bits(y)
    for v, g in zip(vals, got):
        assert int(g) == _exact_rne_bf16(float(v)), (v, hex(int(g)))


def test_bf16_rounding_is_single_step():
    # 1 + 2^-8 + 2^-30 lies just above a bf16 midpoint: the correct result is
    # 1 + 2^-7; rounding through fp32 first lands on the midpoint and then on 1.
    y = np.array([1.0 + 2.0 ** -8 + 2.0 ** -30])
    assert int(oracle.f64_to_bf16_bits(y)[0]) == 0x3F81
    assert int(oracle.f64_to_bf16_bits(np.array([1.0 + 2.0 ** -8]))[0]) == 0x3F80     # tie -> even
    assert int(oracle.f64_to_bf16_bits(np.array([float("nan")]))[0]) == 0x7FC0
    # the render's rounding entry point takes the same single step
    assert int(oracle.round_to_dtype(y, "bfloat16")[0]) == 0x3F81
    rng = np.random.default_rng(6)
    v = rng.standard_normal(20000) * (1.0 + 2.0 ** -30)
    assert np.array_equal(oracle.round_to_dtype(v, "bfloat16"), oracle.f64_to_bf16_bits(v))


def test_bf16_rounding_agrees_with_torch_on_fp32_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x32 = (rng.standard_normal(5000) * np.exp2(rng.integers(-30, 30, 5000))).astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.f64_to_bf16_bits(x32.astype(np.float64)), ref)


def test_fp32_rounding_is_ieee():
    y = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 1.0 + 2.0 ** -24 + 2.0 ** -50])
    got = oracle.round_to_dtype(y, "float32")
    assert got[0] == np.float32(1.0) and got[1] == np.float32(1.0 + 2.0 ** -22)
    assert got[2] == np.float32(1.0 + 2.0 ** -23)
