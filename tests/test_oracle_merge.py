"""Pins for the oracle's order, render and set operations (§4.2-§4.5, Alg. 1-2,
App. A, §5.9 Table 10)."""

import itertools

import numpy as np
import pytest

import oracle
from helpers import cache_bytes, copy_fragment, rand_fragment


def _frags_with_scales(rng, scales, T=6, L=2, H=2, d=16, dtype="float32"):
    return [rand_fragment(rng, L=L, H=H, T=T, d=d, dtype=dtype, k_scale=s) for s in scales]


# ------------------------------------------------------------------ App. A

def test_app_a_permutation_invariance_and_lengths(golden):
    g = golden("app_a_byte_crdt.json")
    rng = np.random.default_rng(0)
    T = g["positions_per_thinker"]
    total = 0
    for N in (2, 3, 4, 5):
        frags = _frags_with_scales(rng, [1.0 + 0.5 * j for j in range(N)], T=T)
        ref = cache_bytes(oracle.canonical_merge(frags, 1, 1e4)["cache"])
        count = 0
        for perm in itertools.permutations(range(N)):
            out = oracle.canonical_merge([frags[p] for p in perm], 1, 1e4)["cache"]
            assert cache_bytes(out) == ref
            count += 1
        assert count == g["permutations_per_N"][str(N)]
        total += count
        if str(N) in g["rendered_length_per_N"]:
            assert all(K.shape[2] == g["rendered_length_per_N"][str(N)] for K, _ in
                       oracle.canonical_merge(frags, 1, 1e4)["cache"])
    assert total == g["permutations_total"]
    assert sum(len(list(itertools.permutations(range(N)))) for N in (2, 3, 4)) == \
        g["extra_permutations_N2_to_4"]


def test_descending_score_places_densest_first():
    rng = np.random.default_rng(1)
    frags = _frags_with_scales(rng, [0.5, 3.0, 1.0, 2.0], T=20)
    res = oracle.canonical_merge(frags, 0, 1e4)
    assert res["order"] == [1, 3, 2, 0]
    assert res["offsets"] == [0, 20, 40, 60]
    keys = res["keys"]
    assert all(keys[a] > keys[b] for a, b in zip(res["order"], res["order"][1:]))


def test_equal_scores_fall_to_descending_digest():
    rng = np.random.default_rng(2)
    for trial in range(12):                               # independent pairs: no lucky agreement
        a = rand_fragment(rng, T=9)
        b = copy_fragment(a)
        for l in range(b.L):                              # same K, fresh V: equal score, new Id
            b.layers[l] = (b.layers[l][0],
                           rng.standard_normal(b.layers[l][1].shape).astype(np.float32))
        ida, idb = oracle.fragment_id(a), oracle.fragment_id(b)
        assert ida != idb
        res = oracle.canonical_merge([a, b], 0, 1e4)
        assert res["keys"][0] == res["keys"][1]
        first = 0 if ida > idb else 1                     # bytes compare as big-endian unsigned
        assert res["order"][0] == first
        assert cache_bytes(oracle.canonical_merge([b, a], 0, 1e4)["cache"]) == \
            cache_bytes(res["cache"])


def test_two_input_reduction():
    """With two caches the N-ary path equals the direct two-input rule: A goes
    first iff (rho_A, h_A) > (rho_B, h_B)."""
    rng = np.random.default_rng(3)
    for trial in range(6):
        A, B = _frags_with_scales(rng, rng.uniform(0.5, 2.0, 2), T=int(rng.integers(3, 12)))
        tail = min(A.T, B.T)
        ra, rb = oracle.mean_knorm(A, 1, tail), oracle.mean_knorm(B, 1, tail)
        ha, hb = oracle.fragment_id(A), oracle.fragment_id(B)
        first, second = (A, B) if (ra, ha) > (rb, hb) else (B, A)
        direct = oracle.render_in_order([first, second], 1e4)
        assert cache_bytes(direct) == cache_bytes(oracle.canonical_merge([B, A], 1, 1e4)["cache"])


# ------------------------------------------------------------------ Eq. (1)-(2)

def test_render_layout_v_exact_k_slot0_exact():
    rng = np.random.default_rng(4)
    frags = [rand_fragment(rng, T=t, k_scale=s, dtype="bfloat16") for t, s in ((5, 1.0), (8, 2.0), (3, 0.5))]
    res = oracle.canonical_merge(frags, 1, 1e4)
    order, offs = res["order"], res["offsets"]
    assert offs == oracle.offsets_of([frags[i].T for i in order])
    for l, (K, V) in enumerate(res["cache"]):
        assert K.shape == (1, 2, 16, 16) and V.shape == K.shape
        for i, s in zip(order, offs):
            t = frags[i].T
            assert np.array_equal(V[:, :, s:s + t], frags[i].layers[l][1])
        first = frags[order[0]]
        assert np.array_equal(K[:, :, :first.T], first.layers[l][0])


def test_render_equals_one_long_sequence():
    """§4.2: R(s) shifts a fragment's positions 0..T-1 to s..s+T-1. Fragments
    whose keys were rotated at their local positions render into the keys one
    sequence would hold at global positions (rotation written here as complex
    multiplication, independent of the oracle's rotation)."""
    rng = np.random.default_rng(5)
    d, base, H = 32, 1e4, 2
    theta = base ** (-np.arange(0, d, 2) / d)

    def rot(raw, pos):                                     # raw [H, T, d], pos [T]
        z = (raw[..., : d // 2] + 1j * raw[..., d // 2:]) * np.exp(1j * pos[None, :, None] * theta)
        return np.concatenate([z.real, z.imag], axis=-1)

    raws, frags = [], []
    for t, s in ((7, 1.0), (11, 2.0), (4, 1.5)):
        raw = rng.standard_normal((H, t, d)) * s
        K = rot(raw, np.arange(t)).astype(np.float32)[None]
        raws.append(raw)
        frags.append(oracle.Fragment("float32", [(K, np.zeros_like(K))]))
    res = oracle.canonical_merge(frags, 0, base)
    K = res["cache"][0][0][0].astype(np.float64)
    for i, s in zip(res["order"], res["offsets"]):
        t = frags[i].T
        want = rot(raws[i], s + np.arange(t))
        assert np.allclose(K[:, s:s + t], want, rtol=0, atol=4e-7 * np.abs(want).max())


def test_single_fragment_renders_as_byte_copy():
    rng = np.random.default_rng(6)
    f = rand_fragment(rng, T=13, dtype="bfloat16")
    s = oracle.FragmentSet()
    s.ingest(f)
    assert cache_bytes(s.render(1, 1e6)["cache"]) == cache_bytes(f.layers)


def test_mixed_shapes_rejected():
    rng = np.random.default_rng(7)
    with pytest.raises(ValueError):
        oracle.canonical_merge([rand_fragment(rng, d=16), rand_fragment(rng, d=32)], 0, 1e4)
    with pytest.raises(ValueError):
        oracle.canonical_merge([rand_fragment(rng, L=2), rand_fragment(rng, L=3)], 0, 1e4)


# ------------------------------------------------------------------ Alg. 2 state

def _set_of(frags):
    s = oracle.FragmentSet()
    for f in frags:
        s.ingest(f)
    return s


def test_union_laws_on_ids_and_rendered_bytes():
    rng = np.random.default_rng(8)
    pool = _frags_with_scales(rng, [0.7, 1.1, 1.6, 2.3, 3.0], T=6)
    for trial in range(5):
        pick = lambda: [pool[i] for i in rng.choice(5, size=rng.integers(1, 5), replace=False)]
        A, B, C = _set_of(pick()), _set_of(pick()), _set_of(pick())
        r = lambda S: cache_bytes(S.render(1, 1e4)["cache"])
        assert A.merge(B).ids() == B.merge(A).ids()                              # commutative
        assert r(A.merge(B)) == r(B.merge(A))
        assert A.merge(B).merge(C).ids() == A.merge(B.merge(C)).ids()            # associative
        assert r(A.merge(B).merge(C)) == r(A.merge(B.merge(C)))
        assert A.merge(A).ids() == A.ids() and r(A.merge(A)) == r(A)             # idempotent
        assert A.merge(A.merge(B)).ids() == A.merge(B).ids()                     # absorbing
        assert A.ids() <= A.merge(B).ids()                                       # inflationary


def test_dedupe_partition_equals_byte_equality():
    rng = np.random.default_rng(9)
    base = _frags_with_scales(rng, [1.0, 1.3, 1.9], T=5)
    deliveries = [copy_fragment(base[i]) for i in (0, 1, 0, 2, 2, 2, 1)]
    ids = [oracle.fragment_id(f) for f in deliveries]
    raw = [b"".join(k + v for k, v in cache_bytes(f.layers)) for f in deliveries]
    for i in range(len(deliveries)):
        for j in range(len(deliveries)):
            assert (ids[i] == ids[j]) == (raw[i] == raw[j])
    res = oracle.render_deliveries(deliveries, 1, 1e4)
    assert res["n_unique"] == 3
    assert res["T_out"] == 15
    assert sorted(res["order"]) == [0, 1, 3]                 # first arrival of each Id kept
    assert cache_bytes(res["cache"]) == cache_bytes(oracle.canonical_merge(base, 1, 1e4)["cache"])


def test_table10_redelivery(golden):
    g = golden("table10_redelivery.json")
    rng = np.random.default_rng(10)
    A = rand_fragment(rng, L=2, H=1, T=150, d=16, k_scale=2.0)
    B = rand_fragment(rng, L=2, H=1, T=158, d=16, k_scale=1.0)
    ref = None
    for R, naive_len, crdt_len in zip(g["R"], g["naive_length"], g["crdt_length"]):
        deliveries = [copy_fragment(f) for f in [A, B] * R]
        rng.shuffle(deliveries)
        naive = oracle.render_multiset_naive(deliveries, 1, 1e6)
        assert naive[0][0].shape[2] == naive_len
        S = _set_of(deliveries)
        out = S.render(1, 1e6)["cache"]
        assert out[0][0].shape[2] == crdt_len
        assert len(S) == g["set_size"]
        ref = ref or cache_bytes(out)
        assert cache_bytes(out) == ref


def test_rendered_operator_is_not_idempotent_but_the_set_is():
    """§4.4: the copy of B inside CM(A, B) is RoPE-shifted, so re-merging B
    does not absorb it; the set of unshifted fragments does."""
    rng = np.random.default_rng(11)
    A, B = _frags_with_scales(rng, [2.0, 1.0], T=6)
    ab = oracle.canonical_merge([A, B], 1, 1e4)
    merged_frag = oracle.Fragment("float32", list(ab["cache"]))
    again = oracle.canonical_merge([merged_frag, B], 1, 1e4)["cache"]
    assert again[0][0].shape[2] == 18 != ab["cache"][0][0].shape[2]
    assert oracle.fragment_id(merged_frag) not in {oracle.fragment_id(A), oracle.fragment_id(B)}
    S = _set_of([A, B])
    S.ingest(copy_fragment(B))
    assert len(S) == 2
    assert cache_bytes(S.render(1, 1e4)["cache"]) == cache_bytes(ab["cache"])
