"""The seeded workload recipes and generator (shared input source for the
oracle and the HIP path)."""

import itertools

import numpy as np
import pytest
import torch

import oracle
import synth


def test_recipe_shapes():
    t = synth.tiny()
    assert (t.L, t.H, t.d, t.dtype, t.lengths, t.k_scale, t.routing_layer) == \
        (2, 2, 64, "float32", (16, 24), (1.0, 1.5), 1)
    n2 = synth.qwen3_17b_n2()
    assert (n2.L, n2.H, n2.d, n2.dtype, n2.lengths, n2.routing_layer, n2.rope_base) == \
        (28, 8, 128, "bfloat16", (512, 768), 14, 1e6)
    n5 = synth.qwen3_17b_n5()
    assert n5.n_distinct == 5 and all(256 <= x <= 2048 for x in n5.lengths)
    counts = [n5.deliveries.count(i) for i in range(5)]
    assert all(1 <= c <= 3 for c in counts) and sum(counts) == n5.n_deliveries
    n4 = synth.qwen3_4b_n4()
    assert (n4.L, n4.routing_layer, n4.lengths) == (36, 18, (4096,) * 4)
    assert n4.render_bytes == 4_831_838_208
    big = synth.qwen3_4b_large()
    assert big.n_distinct == 31 and big.n_deliveries == 32
    assert 250_000 <= big.merged_tokens <= 270_000
    assert all(2048 <= x <= 16384 for x in big.lengths)
    dup = [i for i in range(31) if big.deliveries.count(i) == 2]
    assert len(dup) == 1 and sorted(set(big.deliveries)) == list(range(31))
    (a, b), = big.shared_k
    assert big.lengths[a] == big.lengths[b]


def test_recipes_are_seeded():
    assert synth.qwen3_4b_large(42) == synth.qwen3_4b_large(42)
    assert synth.qwen3_17b_n5(42) != synth.qwen3_17b_n5(7)


def test_draws_are_reproducible_and_independent():
    w = synth.custom(L=2, H=2, d=64, lengths=(20, 30), dtype="bfloat16")
    a = synth.draw_tensor(w, 0, 1, "k")
    assert torch.equal(a, synth.draw_tensor(w, 0, 1, "k"))
    assert not torch.equal(a, synth.draw_tensor(w, 0, 0, "k"))
    frags = synth.make_fragments(w)
    assert torch.equal(frags[0][1][0], a)
    assert frags[1][0][0].shape == (1, 2, 30, 64) and frags[1][0][0].dtype == torch.bfloat16


def test_deliveries_copy_rather_than_alias():
    w = synth.custom(lengths=(8, 9), deliveries=(0, 1, 0))
    frags = synth.make_fragments(w)
    dl = synth.make_deliveries(w, frags)
    assert dl[0] is frags[0] and dl[2] is not frags[0]
    assert all(torch.equal(x, y) for (x, _), (y, _) in zip(dl[0], dl[2]))
    assert dl[2][0][0].data_ptr() != dl[0][0][0].data_ptr()


def test_shared_k_pair_has_equal_k_and_distinct_v():
    w = synth.custom(lengths=(10, 10, 12), shared_k=((0, 1),))
    f = synth.make_fragments(w)
    for l in range(w.L):
        assert torch.equal(f[0][l][0], f[1][l][0])
        assert not torch.equal(f[0][l][1], f[1][l][1])


def _routing_keys(w):
    t_star = min(w.lengths)
    keys = []
    for i in range(w.n_distinct):
        K = synth.tensor_to_numpy(synth.draw_tensor(w, i, w.routing_layer, "k"))
        frag = oracle.Fragment(w.dtype, [(K, np.zeros_like(K))])
        keys.append(oracle.fragment_key(frag, 0, t_star))
    return keys


@pytest.mark.parametrize("name", ["tiny", "qwen3-1.7b-n2", "qwen3-1.7b-n5", "qwen3-4b-n4"])
def test_score_gaps_at_least_1e3_relative(name):
    w = synth.workload(name)
    keys = _routing_keys(w)
    for a, b in itertools.combinations(range(len(keys)), 2):
        assert abs(keys[a] - keys[b]) >= 1e-3 * max(keys[a], keys[b]), (a, b)


@pytest.mark.slow
def test_large_workload_score_gaps_and_designed_tie():
    w = synth.qwen3_4b_large()
    keys = _routing_keys(w)
    (sa, sb), = w.shared_k
    assert keys[sa] == keys[sb]
    for a, b in itertools.combinations(range(len(keys)), 2):
        if {a, b} != {sa, sb}:
            assert abs(keys[a] - keys[b]) >= 1e-3 * max(keys[a], keys[b]), (a, b)
