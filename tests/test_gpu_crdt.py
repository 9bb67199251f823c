"""GPU: the set semantics of Alg. 2 on the product path (LatentFragmentSet,
its Ids from the library's hash kernels, its render from cm_render_set).

Replicas that ingest overlapping parts of the deliveries, in different orders
and groupings, merge to the same set and render the same bytes (commutative,
associative, idempotent union; absorbed re-deliveries); a delivery that was
dropped and later retried leaves the replica equal to one that never lost it;
a single flipped byte makes a new Id, so the damaged copy is not absorbed and
renders as a fragment of its own. The reference render is checked against the
oracle."""

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


def _workload():
    w = synth.custom("crdt", dtype="bfloat16", d=128, H=2, L=3, lengths=(120, 300, 47, 210, 9),
                     deliveries=(0, 1, 2, 3, 4, 1, 3, 0), routing_layer=1, rope_base=1e4)
    return w, synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))


def _set(caches):
    S = cm.LatentFragmentSet()
    S.ingest_many(caches)
    return S


def test_replicas_converge_under_any_grouping():
    w, dl = _workload()
    full = _set(dl)
    ref = full.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    check_render(ref, [dl[i] for i in range(5)], w.dtype, w.routing_layer, w.rope_base)
    rng = np.random.default_rng(3)
    parts = [[dl[i] for i in (0, 1, 5)], [dl[i] for i in (1, 2, 3, 6)], [dl[i] for i in (4, 7, 3)]]
    A, B, C = (_set([p[i] for i in rng.permutation(len(p))]) for p in parts)
    log("[crdt] three replicas")
    for merged in (A.merge(B).merge(C), A.merge(B.merge(C)), C.merge(A).merge(B),
                   B.merge(C).merge(A).merge(A), A.merge(A).merge(B).merge(C)):
        assert merged.ids() == full.ids()
        out = merged.render(w.routing_layer, w.rope_base)
        torch.cuda.synchronize()
        assert np.array_equal(out.plan[:4], ref.plan[:4])
        assert torch.equal(out.merged, ref.merged)


def test_dropped_then_retried_delivery():
    w, dl = _workload()
    full = _set(dl).render(w.routing_layer, w.rope_base)
    R = _set([c for i, c in enumerate(dl) if i != 2])       # fragment 2's only delivery lost
    partial = R.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert partial.T_out == full.T_out - w.lengths[2]
    R.ingest(dl[2])                                          # retried
    again = R.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert torch.equal(again.merged, full.merged)


def test_one_flipped_byte_is_a_new_fragment():
    w, dl = _workload()
    S = _set(dl)
    before = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    bad = tuple((K.clone(), V.clone()) for K, V in dl[3])
    raw = bad[2][1].view(torch.uint8).view(-1)               # V of layer 2: not in the score
    raw[12345] ^= 0x01
    new_id = S.ingest(bad)
    assert new_id not in before.digests and len(S) == len(set(before.digests)) + 1
    after = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert after.T_out == before.T_out + w.lengths[3]
    # the damaged copy has fragment 3's score; the tie falls to the Ids
    check_render(after, [dl[i] for i in range(5)] + [bad], w.dtype, w.routing_layer,
                 w.rope_base)
