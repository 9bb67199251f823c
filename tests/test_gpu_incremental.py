"""GPU: incremental render (MergedCache / cm_render_merge_range). After every
ingest the merged cache, re-rendered only from the first slot whose fragment
changed, equals the full render of the set bit for bit; the full render itself
is checked against the oracle elsewhere, and the final set here is checked
against the oracle too."""

import random

import numpy as np
import pytest
import torch

import synth
import paper_2607_01308_amd as cm
from gpu_util import check_render, log

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    yield
    torch.cuda.synchronize()


def _same(cache_a, cache_b):
    return all(torch.equal(Ka, Kb) and torch.equal(Va, Vb)
               for (Ka, Va), (Kb, Vb) in zip(cache_a, cache_b))


@pytest.mark.parametrize("dtype,d,capacity", [("bfloat16", 128, 0), ("bfloat16", 128, 4000),
                                              ("float32", 64, 0)])
def test_incremental_equals_full_render(dtype, d, capacity):
    lengths = (300, 517, 45, 129, 1000, 64, 260)
    w = synth.custom("incr", dtype=dtype, d=d, H=2, L=3, lengths=lengths, routing_layer=1)
    frags = synth.make_fragments(w, device="cuda")
    order = list(range(len(frags)))
    random.Random(5).shuffle(order)
    S = cm.LatentFragmentSet()
    mc = cm.MergedCache(S, w.routing_layer, w.rope_base, capacity=capacity)
    suffix_only = 0
    for step, i in enumerate(order):
        S.ingest(frags[i])
        got = mc.update()
        full = S.render(w.routing_layer, w.rope_base)
        torch.cuda.synchronize()
        log(f"[incr] {dtype} step {step}: +fragment {i} (T={lengths[i]}), rendered from slot "
            f"{mc.last_first_slot}, {mc.last_rows} of {mc.T_out} rows, T_cap {mc.T_cap}")
        assert mc.T_out == full.T_out
        assert _same(got, full.cache), f"step {step}"
        suffix_only += mc.last_first_slot > 0
        # re-delivering a member changes nothing and renders nothing
        S.ingest(tuple((K.clone(), V.clone()) for K, V in frags[i]))
        mc.update()
        assert mc.last_rows == 0
    assert suffix_only > 0                     # some inserts re-rendered a suffix only
    dl = [frags[i] for i in order]
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    check_render(res, dl, dtype, w.routing_layer, w.rope_base)
    assert _same(mc.cache, res.cache)
