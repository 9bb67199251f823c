"""GPU: the render over paged storage (cm_paged_tables + cm_paged_render). The
merged cache read back through its K and V block tables equals the dense render
of the same fragments bit for bit (the dense render is checked against the
oracle elsewhere; one case here is checked against the oracle directly), reused
pages are the fragments' own, and no page outside the fresh list changes."""

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


CASES = [
    dict(dtype="bfloat16", d=128, B=16, lengths=(64, 128, 32, 256)),      # every slot page-aligned
    dict(dtype="bfloat16", d=128, B=16, lengths=(300, 517, 45, 129)),     # ragged
    dict(dtype="float32", d=64, B=16, lengths=(70, 33, 129)),
    dict(dtype="bfloat16", d=64, B=8, lengths=(41, 16, 90)),              # 1 KiB pages
    dict(dtype="bfloat16", d=128, B=64, lengths=(200, 64, 7)),            # 16 KiB pages
    dict(dtype="bfloat16", d=32, B=32, lengths=(99, 64, 1)),              # 64-byte rows
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c['dtype']}-d{c['d']}-B{c['B']}" for c in CASES])
@pytest.mark.parametrize("style", ["half", "interleaved"])
def test_paged_render_equals_dense_render(case, style):
    w = synth.custom("paged", dtype=case["dtype"], d=case["d"], H=2, L=3, lengths=case["lengths"],
                     routing_layer=1, rope_base=1e4)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    dense = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style=style)
    torch.cuda.synchronize()
    pool, lengths, page_lists, free = synth.make_paged(dl, case["B"], spare_pages=64, seed=3)
    before = pool.clone()
    pset = cm.PagedSet(pool, lengths, page_lists)
    log(f"[paged] {case} style={style}")
    pr = cm.render_paged(pset, dense.plan, free, w.rope_base, style=style)
    torch.cuda.synchronize()
    K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
    V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
    assert torch.equal(K, dense.merged[:, 0]) and torch.equal(V, dense.merged[:, 1])
    written = {(c & 1, int((pr.v_table if c & 1 else pr.k_table)[c >> 1])) for c in pr.fresh}
    frag_pages = {q for pages in page_lists for q in pages}
    assert all(p not in frag_pages for _, p in written)
    for kv in (0, 1):
        keep = [q for q in range(pool.shape[2]) if (kv, q) not in written]
        idx = torch.tensor(keep, device="cuda")
        assert torch.equal(pool[:, kv, idx], before[:, kv, idx])      # nothing else changed
    if all(T % case["B"] == 0 for T in case["lengths"]):
        # aligned slots: every V page and slot 0's K pages are the fragments' own
        assert pr.reused_pages == len(pr.v_table) + dense.lengths[0] // case["B"]


def test_paged_render_against_oracle():
    w = synth.custom("paged-oracle", dtype="bfloat16", d=128, H=2, L=2, lengths=(48, 77, 16),
                     routing_layer=1)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    dense = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    check_render(dense, dl, w.dtype, w.routing_layer, w.rope_base)
    pool, lengths, page_lists, free = synth.make_paged(dl, 16, spare_pages=32, seed=1)
    pr = cm.render_paged(cm.PagedSet(pool, lengths, page_lists), dense.plan, free, w.rope_base)
    torch.cuda.synchronize()
    K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
    V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
    paged = dense.merged.clone()
    paged[:, 0], paged[:, 1] = K, V
    dense.merged.copy_(paged)                 # the cache views now show the paged result
    check_render(dense, dl, w.dtype, w.routing_layer, w.rope_base)
