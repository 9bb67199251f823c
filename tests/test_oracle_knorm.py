"""Pins for the oracle's score: mean K-norm rho of Eq. (3) / Alg. 1 over the
routing layer's last T* rows, and its fixed-order sum S = rho * H * T*."""

import math

import numpy as np
import pytest

import oracle
from helpers import copy_fragment, rand_fragment


def test_pairwise_tree_shape_closed_form():
    # (x0 + x1) + (x2 + x3) with x = [2^53, 1, 1, -2^53]: 2^53 + 1 rounds to 2^53
    # (tie to even) and 1 - 2^53 is exact, so the tree gives 1; a left-to-right
    # sum gives 0 and the exact sum is 2.
    x = np.array([2.0 ** 53, 1.0, 1.0, -(2.0 ** 53)])
    assert oracle.pairwise_sum(x) == 1.0
    # zero padding to the next power of two leaves an exact integer sum unchanged
    for n in (1, 2, 3, 5, 7, 64, 100, 1000):
        v = np.arange(1, n + 1, dtype=np.float64)
        assert oracle.pairwise_sum(v) == n * (n + 1) / 2


def test_pairwise_sum_close_to_exact_sum():
    rng = np.random.default_rng(0)
    for n in (3, 17, 128, 4095):
        v = rng.standard_normal(n)
        assert abs(oracle.pairwise_sum(v) - math.fsum(v)) <= 1e-13 * np.abs(v).sum()


def _frag_from_k(K, dtype="float32"):
    V = np.zeros_like(K)
    return oracle.Fragment(dtype, [(K, V)])


def test_key_closed_form_power_of_two_rows():
    # every entry +-2^k in a row of d = 64 gives a row norm of exactly 2^k * 8
    rng = np.random.default_rng(1)
    H, T, d = 3, 10, 64
    k = rng.integers(-4, 5, size=(H, T))
    signs = rng.choice([-1.0, 1.0], size=(H, T, d))
    K = (signs * (2.0 ** k)[..., None]).astype(np.float32)[None]
    f = _frag_from_k(K)
    assert oracle.fragment_key(f, 0, T) == float(np.sum(8.0 * 2.0 ** k))
    # tail of 4 rows: only rows T-4.. count
    assert oracle.fragment_key(f, 0, 4) == float(np.sum(8.0 * 2.0 ** k[:, -4:]))


def test_key_one_hot_rows_give_rho_one():
    H, T, d = 2, 7, 16
    K = np.zeros((1, H, T, d), np.float32)
    for h in range(H):
        for t in range(T):
            K[0, h, t, (3 * h + t) % d] = -1.0 if t % 2 else 1.0
    f = _frag_from_k(K)
    assert oracle.mean_knorm(f, 0, T) == 1.0
    assert oracle.fragment_key(f, 0, T) == H * T


def test_key_matches_library_norm():
    """rho is the mean over heads and tail rows of the per-row L2 norm (numpy.linalg.norm)."""
    rng = np.random.default_rng(2)
    f = rand_fragment(rng, L=3, H=4, T=50, d=64, k_scale=1.7)
    for layer in range(3):
        for tail in (1, 13, 50):
            x = f.layers[layer][0][0, :, -tail:, :].astype(np.float64)
            want = np.linalg.norm(x, axis=-1).mean()
            got = oracle.mean_knorm(f, layer, tail)
            assert abs(got - want) <= 1e-13 * want


def test_key_bf16_exact_upcast():
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F80, 0x8000], np.uint16)
    v = oracle.bf16_bits_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 2.0 ** -133 and np.isinf(v[3])
    assert v[4] == 0.0 and np.signbit(v[4])
    rng = np.random.default_rng(3)
    f = rand_fragment(rng, L=1, H=2, T=9, d=32, dtype="bfloat16")
    x = oracle.bf16_bits_to_f64(f.layers[0][0])[0]
    want = np.linalg.norm(x, axis=-1).mean()
    assert abs(oracle.mean_knorm(f, 0, 9) - want) <= 1e-13 * want


def test_key_is_tail_aligned_and_routing_layer_only():
    rng = np.random.default_rng(4)
    f = rand_fragment(rng, L=3, H=2, T=20, d=32)
    base = oracle.fragment_key(f, 1, 8)
    g = copy_fragment(f)
    g.layers[1][0][0, :, :12, :] *= 3.0                    # rows before T - T*
    g.layers[0][0][...] *= 5.0                             # another layer
    g.layers[1][1][...] *= 7.0                             # V of the routing layer
    assert oracle.fragment_key(g, 1, 8) == base
    g.layers[1][0][0, 1, 12, 5] += 1.0                     # first tail row
    assert oracle.fragment_key(g, 1, 8) != base


def test_key_invariant_under_rope_rotation():
    """R(s) is orthogonal on every pair, so row norms (hence rho) are unchanged."""
    rng = np.random.default_rng(5)
    H, T, d = 2, 33, 64
    x = rng.standard_normal((H, T, d))
    c, sn = oracle.rope_angles(12345, d, 1e6)
    y = oracle.rotate_pairs(x, c, sn)

    def key64(a):
        return oracle.pairwise_sum(np.sqrt(oracle.pairwise_sum(a * a)).reshape(-1))

    assert abs(key64(y) - key64(x)) <= 1e-12 * key64(x)


def test_key_rejects_bad_tail():
    rng = np.random.default_rng(6)
    f = rand_fragment(rng, T=5)
    with pytest.raises(ValueError):
        oracle.fragment_key(f, 0, 0)
    with pytest.raises(ValueError):
        oracle.fragment_key(f, 0, 6)
