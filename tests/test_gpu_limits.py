"""GPU: the path at the limits of its arguments, against the oracle.

* The most deliveries one call takes (CM_MAX_FRAGMENTS = 1024): 700 distinct
  fragments of 1 to 48 tokens (so T* = 1), 324 re-deliveries drawn at random
  and 40 pairs with equal K (ties broken by the digest); every layer is
  compared with the oracle, and the serial pipeline and the render of the
  ingested set equal the fused one. The same deliveries on pages of 8 tokens,
  through the one-call paged path, equal the dense render.
* A page pool whose slices pass 4 GiB, with pages on both sides: the paged
  paths equal the dense render.
* The most layers a fragment can have (2 L H <= 65535: L = 32767 at H = 1):
  the Id's message is 32768 blocks, 2048 chunks folded in the Id kernel's 32
  groups of 64; digests, keys and order against the oracle, and the first,
  middle and last layers.
* A tensor past 2 GiB: one layer of 8 heads x 1.2M tokens (2.46 GB for each of
  K and V) next to a 3-token fragment that sorts first, so the long one is
  rotated at offset 3. Keys, Ids, order, and the first, middle and last rows
  of every head are checked against the oracle; V and the short fragment's K
  are compared with the inputs on the device; the render of the ingested set
  equals the fused render."""

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_01308_amd as cm
from paper_2607_01308_amd import _cabi as C
from oracle import cmerge_oracle as om
from gpu_util import check_render, k_close, log, oracle_ids, oracle_keys, oracle_plan

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    yield
    torch.cuda.synchronize()


def _max_fragments_workload():
    rng = np.random.default_rng(2024)
    n = 700
    lengths = rng.integers(1, 49, size=n)
    lengths[:3] = (1, 1, 48)
    perm = rng.permutation(np.arange(3, n))
    pairs = [(int(perm[2 * k]), int(perm[2 * k + 1])) for k in range(40)]
    for a, b in pairs:
        lengths[b] = lengths[a]
    extra = rng.choice(n, size=C.CM_MAX_FRAGMENTS - n, replace=True)
    deliveries = list(range(n)) + [int(i) for i in extra]
    deliveries = [int(x) for x in rng.permutation(deliveries)]
    return synth.custom("max-n", dtype="bfloat16", d=64, H=1, L=2, lengths=lengths,
                        deliveries=deliveries, shared_k=pairs, routing_layer=1, seed=5)


def test_max_fragments_per_call():
    w = _max_fragments_workload()
    assert w.n_deliveries == C.CM_MAX_FRAGMENTS and min(w.lengths) == 1
    frags = synth.make_fragments(w, device="cuda")
    dl = synth.make_deliveries(w, frags)
    log(f"[limits] {w.n_deliveries} deliveries, {w.n_distinct} distinct, T_out {sum(w.lengths)}")
    ids = oracle_ids(dl, w.dtype)
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, ids_ref=ids)
    assert res.n_unique == w.n_distinct
    ties = sum(1 for a, b in w.shared_k
               if abs(res.slot_of_delivery[w.deliveries.index(a)]
                      - res.slot_of_delivery[w.deliveries.index(b)]) == 1)
    assert ties == len(w.shared_k)                 # every equal-K pair sits side by side
    serial = cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="serial")
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    from_set = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert torch.equal(serial.merged, res.merged) and torch.equal(from_set.merged, res.merged)


def test_max_fragments_on_pages():
    """The same 1024 deliveries stored only on 1 KiB pages (8 tokens each),
    through the one-call paged path: 700 slots and about 2,100 merged blocks for
    the device-built block tables. Ids, scores and plan equal the dense path's
    (checked against the oracle above), the tables follow cm_paged_tables' rule,
    and the merged cache read back through them equals the dense render."""
    w = _max_fragments_workload()
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    B = 8
    spare = 2 * (sum(w.lengths) // B + len(w.lengths) + 1)
    pool, lengths, page_lists, free = synth.make_paged(dl, B, spare_pages=spare, seed=7)
    del dl
    pset = cm.PagedSet(pool, lengths, page_lists)
    log(f"[limits-paged] {w.n_deliveries} deliveries on pages of {B} tokens")
    pr = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free, fused=True)
    torch.cuda.synchronize()
    assert np.array_equal(pr.plan, res.plan)
    assert torch.equal(pr.digests_dev, res.digests_dev)
    assert torch.equal(pr.keys_dev, res.keys_dev)
    kt, vt, fresh = cm.paged_tables(pset, pr.plan, free)
    assert np.array_equal(pr.k_table, kt) and np.array_equal(pr.v_table, vt)
    assert np.array_equal(pr.fresh, fresh)
    K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
    V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
    assert torch.equal(K, res.merged[:, 0]) and torch.equal(V, res.merged[:, 1])


def test_paged_pool_past_4gib():
    """A pool whose (layer, K/V) slice holds 4.6 GB (140,000 pages of 16 bf16
    rows of 8 heads x 128), so fragment and fresh pages sit past 4 GiB: the
    one-call paged path (32-bit pool rows, 64-bit byte offsets) and the
    two-stream form equal the dense render."""
    w = synth.custom("big-pool", dtype="bfloat16", d=128, H=8, L=1, lengths=(3000, 1000, 7),
                     routing_layer=0, seed=11)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    need = sum((T + 15) // 16 for T in w.lengths)
    P = 140_000
    pool, lengths, page_lists, free = synth.make_paged(dl, 16, spare_pages=P - need, seed=3)
    assert pool.shape[2] == P and pool[0, 0].numel() * pool.element_size() > 4 * 2**30
    assert max(max(p) for p in page_lists) >= 2**32 // (8 * 16 * 128 * 2)   # past 4 GiB
    log(f"[limits-pool] {pool.numel() * pool.element_size() / 1e9:.1f} GB pool")
    pset = cm.PagedSet(pool, lengths, page_lists)
    for fused in (True, False):
        pr = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free[::-1], fused=fused)
        torch.cuda.synchronize()
        assert np.array_equal(pr.plan, res.plan)
        assert torch.equal(pr.digests_dev, res.digests_dev)
        assert max(pr.k_table.max(), pr.v_table.max()) >= 2**32 // (8 * 16 * 128 * 2)
        K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
        V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
        assert torch.equal(K, res.merged[:, 0]) and torch.equal(V, res.merged[:, 1])


def test_most_layers_per_fragment():
    w = synth.custom("max-L", dtype="float32", d=16, H=1, L=32767, lengths=(2, 3),
                     deliveries=(0, 1, 0), routing_layer=32766)
    frags = synth.make_fragments(w, device="cuda")
    dl = synth.make_deliveries(w, frags)
    log(f"[limits] L={w.L}: {w.n_deliveries} deliveries of {2 * w.L} tensors")
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, layers=[0, 1, 16383, 32766])
    assert res.n_unique == 2 and res.T_out == 5


def test_tensor_larger_than_2gib():
    T = 1_200_000
    w = synth.custom("big", dtype="bfloat16", d=128, H=8, L=1, lengths=(T, 3),
                     k_scale=(0.5, 2.0), routing_layer=0, seed=9)
    assert w.H * T * w.d * 2 > 2 ** 31
    frags = synth.make_fragments(w, device="cuda")
    dl = synth.make_deliveries(w, frags)
    log(f"[limits] one layer, {T} tokens: {w.H * T * w.d * 2 / 2 ** 30:.2f} GiB per tensor")
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    keys = oracle_keys(dl, w.dtype, w.routing_layer, 3)
    assert [float(k) for k in res.keys] == keys
    log("[limits] oracle Ids")
    ids = [om.fragment_id(oracle.Fragment(*synth.to_numpy_cache(c))) for c in dl]
    assert res.digests == ids
    plan = oracle_plan(dl, ids, keys)
    assert res.order == plan["order"] == [1, 0] and res.offsets == [0, 3] and res.T_out == T + 3

    K, V = res.cache[0]
    assert torch.equal(K[:, :, :3], dl[1][0][0]) and torch.equal(V[:, :, :3], dl[1][0][1])
    assert torch.equal(V[:, :, 3:], dl[0][0][1])
    rows = [0, 1, T // 2, T - 2, T - 1]
    g = synth.tensor_to_numpy(K.index_select(2, torch.tensor([3 + r for r in rows], device="cuda")))
    src = synth.tensor_to_numpy(dl[0][0][0].index_select(2, torch.tensor(rows, device="cuda")))
    c, sn = oracle.rope_angles(3, w.d, w.rope_base)
    want = oracle.round_to_dtype(oracle.rotate_pairs(om.to_f64(src, w.dtype), c, sn), w.dtype)
    ok, same = k_close(g, want, w.dtype)
    assert ok and same >= 0.99, f"sampled K rows: identical {same}"

    merged = res.merged
    del res
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    r2 = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert torch.equal(r2.merged, merged)
    log("[limits] done")
