"""GPU: the whole path captured into a HIP graph (cm_render_deliveries_graph,
RenderGraph). Every replay is compared with the eager call's result (plan,
Ids, scores, merged cache, bit for bit), with the program's own eager work and
synchronisations between the replays; after new contents are written into the
same fragment tensors, a replay equals the eager render of the new contents.
The eager path is checked against the oracle in the parity tests."""

import numpy as np
import pytest
import torch

import synth
import paper_2607_01308_amd as cm
from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    yield
    torch.cuda.synchronize()


def _same(res, ref):
    assert np.array_equal(res.plan, ref.plan)
    assert torch.equal(res.digests_dev, ref.digests_dev)
    assert torch.equal(res.keys_dev, ref.keys_dev)
    assert torch.equal(res.merged, ref.merged)


CASES = [
    dict(name="graph-bf16", dtype="bfloat16", d=128, H=2, L=3, lengths=(300, 517, 45, 300),
         deliveries=(0, 1, 2, 3, 1), shared_k=((0, 3),), style="half"),
    dict(name="graph-tiny", dtype="float32", d=64, H=2, L=2, lengths=(16, 24), style="half"),
    dict(name="graph-il", dtype="bfloat16", d=64, H=3, L=2, lengths=(33, 70, 1), style="interleaved"),
]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_graph_replays_equal_the_eager_call(case):
    kw = {k: v for k, v in case.items() if k not in ("style",)}
    w = synth.custom(routing_layer=1, rope_base=1e4, seed=7, **kw)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    style = case["style"]
    ref = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style=style)
    ref.plan
    torch.cuda.synchronize()
    log(f"[graph] {case['name']}")
    g = cm.RenderGraph(dl, w.routing_layer, w.rope_base, style=style)
    try:
        for r in range(3):
            res = g.replay()
            torch.cuda.synchronize()
            _same(res, ref)
            # eager work of the program between replays, on the same stream
            other = cm.render_deliveries(dl[::-1], w.routing_layer, w.rope_base, style=style)
            assert torch.equal(other.merged, ref.merged)        # the order does not matter
            torch.cuda.synchronize()
        # new contents written into the same tensors: the replay reads them
        w2 = synth.custom(routing_layer=1, rope_base=1e4, seed=19, **kw)
        dl2 = synth.make_deliveries(w2, synth.make_fragments(w2, device="cuda"))
        for c, c2 in zip(dl, dl2):
            for (K, V), (K2, V2) in zip(c, c2):
                K.copy_(K2)
                V.copy_(V2)
        ref2 = cm.render_deliveries(dl2, w.routing_layer, w.rope_base, style=style)
        ref2.plan
        torch.cuda.synchronize()
        res = g.replay()
        torch.cuda.synchronize()
        _same(res, ref2)
        assert not torch.equal(ref2.digests_dev, ref.digests_dev)
    finally:
        g.close()
