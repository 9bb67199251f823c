"""bench.py's CPU baseline runs the oracle's functions on a thread pool (tensor
roots and (layer, slot) renders as tasks); the composition must give exactly
the oracle's own render of the same fragments, and the record must state the
threads used, the host's allowance, the CPU model and the sample's bytes."""

import numpy as np
import torch

import bench
import oracle
import synth


def _sample(name, k):
    w = synth.workload(name, 3)
    frags = synth.make_fragments(w, device=torch.device("cpu"))
    idx = sorted(range(w.n_distinct), key=lambda i: w.lengths[i])[:k]
    return w, frags, [oracle.Fragment(*synth.to_numpy_cache(frags[i])) for i in idx]


def test_threaded_oracle_path_equals_the_oracle_render():
    w, _, sample = _sample("tiny", 5)
    ref = oracle.render_deliveries(sample, w.routing_layer, w.rope_base)
    for workers in (1, 4):
        out = bench._oracle_path(sample, w, workers)
        assert len(out) == w.L
        for (K, V), (Kr, Vr) in zip(out, ref["cache"]):
            assert np.array_equal(K, Kr) and np.array_equal(V, Vr)


def test_cpu_baseline_record():
    w, frags, _ = _sample("tiny", 5)
    rec = bench.cpu_baseline(w, frags)
    assert rec["kind"] == "oracle" and rec["unit"] == "GB/s"
    assert 1 <= rec["cores"] <= min(16, rec["cores_allowed"])
    assert rec["value"] == rec["value_all"] > 0 and rec["value_1thread"] > 0
    shortest = sorted(range(w.n_distinct), key=lambda i: w.lengths[i])[:5]
    assert rec["sample_bytes"] == 2 * sum(w.fragment_bytes(i) for i in shortest)
    assert isinstance(rec["model"], str) and rec["model"]
