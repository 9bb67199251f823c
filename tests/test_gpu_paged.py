"""GPU: the render over paged storage (cm_paged_tables + cm_paged_render). The
merged cache read back through its K and V block tables equals the dense render
of the same fragments bit for bit (the dense render is checked against the
oracle elsewhere; one case here is checked against the oracle directly), reused
pages are the fragments' own, and no page outside the fresh list changes. The
fused paged render + hash (cm_paged_render_hash) leaves the pool exactly as the
paged render does and writes the dense form's Ids. Steps 1-5 on fragments that
live only in the pool (cm_paged_order, then the fused kernel or the paged render
beside the paged hash) are checked against the oracle: Ids, scores, plan and
merged cache."""

import numpy as np
import pytest
import torch

import synth
import paper_2607_01308_amd as cm
from paper_2607_01308_amd import _cabi as C
from gpu_util import (check_render, k_close, k_stats, log, oracle_ids, oracle_keys,
                      oracle_layers, oracle_plan)

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


@pytest.mark.parametrize("case", CASES, ids=[f"{c['dtype']}-d{c['d']}-B{c['B']}" for c in CASES])
@pytest.mark.parametrize("style", ["half", "interleaved"])
def test_paged_render_hash_equals_render_plus_hash(case, style):
    """cm_paged_render_hash with the tables of cm_paged_tables leaves the pool
    byte for byte as cm_paged_render does (fresh pages written, every other
    page, reused ones included, untouched) and writes the Ids of the slot
    deliveries selected with 0, equal to the dense path's, leaving the others'
    digests as they were."""
    w = synth.custom("paged-fused", dtype=case["dtype"], d=case["d"], H=2, L=3,
                     lengths=case["lengths"], routing_layer=1, rope_base=1e4)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    dense = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style=style)
    torch.cuda.synchronize()
    ids = dense.digests_dev.cpu().numpy().copy()
    pool, lengths, page_lists, free = synth.make_paged(dl, case["B"], spare_pages=64, seed=3)
    before = pool.clone()
    pset = cm.PagedSet(pool, lengths, page_lists)
    log(f"[paged-fused] {case} style={style}")
    pr = cm.render_paged(pset, dense.plan, free, w.rope_base, style=style)
    torch.cuda.synchronize()
    ref = pool.clone()
    pool.copy_(before)
    n = len(lengths)
    select = torch.tensor([k % 2 for k in range(n)], dtype=torch.uint8, device="cuda")
    digests = torch.full((n, 32), 0xAB, dtype=torch.uint8, device="cuda")
    ws = torch.empty(cm.paged_workspace_size(pset), dtype=torch.uint8, device="cuda")
    plan_dev = torch.from_numpy(dense.plan).cuda()
    kd = torch.from_numpy(pr.k_table).cuda()
    vd = torch.from_numpy(pr.v_table).cuda()
    cm.paged_render_hash(pset, plan_dev, dense.plan, w.rope_base, style, pr.k_table, pr.v_table,
                         kd, vd, select, digests, ws)
    torch.cuda.synchronize()
    assert torch.equal(pool, ref)
    got = digests.cpu().numpy()
    for k in range(n):
        if k % 2 == 0:
            assert bytes(got[k]) == bytes(ids[k]), f"Id of delivery {k}"
        else:
            assert (got[k] == 0xAB).all(), f"digest {k} was not selected and must stay"


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


SET_CASES = [
    # duplicate delivery and an equal-score pair (shared K), ragged lengths
    dict(dtype="bfloat16", d=128, B=16, H=2, L=3, lengths=(300, 517, 45, 300),
         deliveries=(0, 1, 2, 3, 1), shared_k=((0, 3),)),
    dict(dtype="float32", d=64, B=16, H=3, L=2, lengths=(70, 33, 129, 2),
         deliveries=(2, 0, 1, 3, 2, 2)),
    dict(dtype="bfloat16", d=32, B=32, H=2, L=2, lengths=(99, 64, 1, 200)),     # 64-byte rows, T=1
    dict(dtype="bfloat16", d=256, B=8, H=4, L=2, lengths=(1030, 77, 513)),     # 512-byte rows
    dict(dtype="float32", d=256, B=16, H=1, L=2, lengths=(257, 4096)),         # 1 KiB rows, 16 KiB pages
    dict(dtype="bfloat16", d=128, B=16, H=2, L=2, lengths=(1,)),               # one token: all pages kept
    dict(dtype="float32", d=32, B=32, H=1, L=2, lengths=(3,),
         deliveries=(0, 0, 0)),                                               # one fragment, three times
]


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "overlapped"])
@pytest.mark.parametrize("case", SET_CASES,
                         ids=[f"{c['dtype']}-d{c['d']}-B{c['B']}-n{len(c.get('deliveries', c['lengths']))}"
                              for c in SET_CASES])
def test_paged_set_steps_1_to_5_against_oracle(case, fused):
    """render_paged_set on a pool holding every delivery (copies on pages of
    their own): the Ids are the dense form's content addresses, the scores and
    the plan are the oracle's, and the merged cache read back through the block
    tables is the oracle's render; with the render and the remaining Ids in one
    kernel (cm_paged_render_hash) and with the paged render and the paged hash
    beside it. The fragments' dense tensors serve only to fill the pool and to
    compute the oracle's answer; they are dropped before the paged path runs."""
    w = synth.custom("paged-set", dtype=case["dtype"], d=case["d"], H=case["H"], L=case["L"],
                     lengths=case["lengths"], deliveries=case.get("deliveries"),
                     shared_k=case.get("shared_k", ()), routing_layer=1, rope_base=1e4)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    tail = min(w.lengths)
    ids = oracle_ids(dl, w.dtype)
    keys = oracle_keys(dl, w.dtype, w.routing_layer, tail)
    plan = oracle_plan(dl, ids, keys)
    ref = oracle_layers(dl, w.dtype, plan["order"], w.rope_base, range(w.L))
    # room for every merged block of K and V to be fresh
    spare = 2 * (sum(w.lengths) // case["B"] + len(w.lengths) + 1)
    pool, lengths, page_lists, free = synth.make_paged(dl, case["B"], spare_pages=spare, seed=5)
    del dl
    torch.cuda.synchronize()
    log(f"[paged-set] {case} fused={fused}")
    pset = cm.PagedSet(pool, lengths, page_lists)
    pr = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free, fused=fused)
    torch.cuda.synchronize()
    # the tables (built on the device by the one-call path) follow cm_paged_tables' rule
    kt, vt, fresh = cm.paged_tables(pset, pr.plan, free)
    assert np.array_equal(pr.k_table, kt) and np.array_equal(pr.v_table, vt)
    assert np.array_equal(pr.fresh, fresh)
    assert [bytes(x) for x in pr.digests_dev.cpu().numpy()] == ids
    assert list(pr.keys_dev.cpu().numpy()) == keys
    n = len(ids)
    p = pr.plan
    assert p[2] == plan["n_unique"] and p[3] == plan["T_out"] == pr.T_out
    assert list(p[4:4 + plan["n_unique"]]) == plan["order"]
    assert list(p[4 + n:4 + n + plan["n_unique"]]) == plan["offsets"]
    assert list(p[4 + 3 * n:4 + 4 * n]) == plan["slot_of_delivery"]
    K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
    V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
    worst = 0
    for l in range(w.L):
        gK, gV = synth.tensor_to_numpy(K[l]), synth.tensor_to_numpy(V[l])
        rK, rV = ref[l]
        assert np.array_equal(gV, rV), f"V of layer {l} differs"
        ok, _ = k_close(gK, rK, w.dtype)
        worst = max(worst, k_stats(gK, rK, w.dtype)[0])
        assert ok, f"K of layer {l} outside tolerance"
    log(f"  paged set: {n} deliveries, {plan['n_unique']} slots, T_out {pr.T_out}, "
        f"K largest distance {worst} ulp")


def test_paged_deliveries_with_too_few_free_pages():
    """The one-call paged path builds its block tables on the device; a free list
    shorter than the render needs is reported through the plan (CM_EINVAL, with
    the number of pages needed) when the result is read, and no page of the pool
    is written."""
    w = synth.custom("paged-short", dtype="bfloat16", d=128, H=2, L=2, lengths=(300, 517, 45),
                     routing_layer=1, rope_base=1e4)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    pool, lengths, page_lists, free = synth.make_paged(dl, 16, spare_pages=64, seed=2)
    del dl
    before = pool.clone()
    pset = cm.PagedSet(pool, lengths, page_lists)
    log("[paged-short]")
    pr = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free[:5], fused=True)
    torch.cuda.synchronize()
    with pytest.raises(cm.CmError) as e:
        pr.k_table
    assert e.value.status == C.CM_EINVAL and "free list" in str(e.value)
    assert torch.equal(pool, before)
    # with room for every merged block it renders
    pr = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free, fused=True)
    assert pr.T_out == sum(lengths) and len(pr.fresh) > 5
