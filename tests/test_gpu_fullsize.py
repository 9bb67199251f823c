"""GPU: the Qwen3-4B-shaped large workload at full size (32 deliveries, 31
distinct, 264,181 merged tokens, 78 GB of render traffic), run as the benchmark
runs it: the fused pipeline over the deliveries (steps 1-5), then the render of
the ingested set (steps 2-5, Ids from Ingest).

The oracle cannot render 78 GB within a test, so it checks what it can compute
piece by piece, from the generator's tensors:
  * every delivery's key (the routing-layer tail), bit for bit;
  * every delivery's Id (39 GB hashed by the oracle's BLAKE3, one tensor per
    task in a thread pool over the host's cores), bit for bit;
  * dedupe, the order and the offsets from those keys and Ids;
  * the routing layer in full, and in every layer the first, middle and last
    row of every slot;
and, over the whole output: V of every slot and layer and K of the slot at
offset 0 are the input bytes (compared on the device), and the render of the
ingested set equals the fused render bit for bit."""

import concurrent.futures as cf
import os

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_01308_amd as cm
from oracle import cmerge_oracle as om
from gpu_util import k_close, k_stats, log, oracle_keys, oracle_layers, oracle_plan

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    yield
    torch.cuda.synchronize()


def _oracle_ids(deliveries, dtype):
    """Oracle Id of every delivery: the 2L tensor roots of each, one tensor per
    task on a pool of the host's cores (the oracle's BLAKE3 runs in C outside
    the interpreter lock), then the header-and-roots hash of each delivery."""
    tasks = [(j, l, kv) for j, cache in enumerate(deliveries) for l in range(len(cache))
             for kv in (0, 1)]
    workers = min(16, len(os.sched_getaffinity(0)))
    with cf.ThreadPoolExecutor(workers) as ex:
        roots = list(ex.map(
            lambda t: om.tensor_root(synth.tensor_to_numpy(deliveries[t[0]][t[1]][t[2]])), tasks))
    ids, k = [], 0
    for cache in deliveries:
        L = len(cache)
        _, H, T, d = cache[0][0].shape
        ids.append(om.fragment_id_from_roots(om.fragment_header(dtype, L, H, T, d),
                                             roots[k:k + 2 * L]))
        k += 2 * L
    return ids


@pytest.mark.timeout(900)
def test_qwen3_4b_large_full_size():
    w = synth.workload("qwen3-4b-large")
    log(f"[fullsize] generating {w.name}: {w.n_deliveries} deliveries, {w.merged_tokens} tokens")
    frags = synth.make_fragments(w, device="cuda")
    dl = synth.make_deliveries(w, frags)
    batch = cm.FragmentBatch(dl)
    torch.cuda.synchronize()
    log("[fullsize] fused pipeline")
    res = cm.render_deliveries(batch, w.routing_layer, w.rope_base)
    torch.cuda.synchronize()

    tail = min(w.lengths)
    assert res.tail_len == tail
    log("[fullsize] oracle keys")
    keys = oracle_keys(dl, w.dtype, w.routing_layer, tail)
    assert [float(k) for k in res.keys] == keys               # fp64, bit for bit

    log("[fullsize] oracle Ids of every delivery")
    ids = _oracle_ids(dl, w.dtype)
    assert res.digests == ids
    groups = {}
    for i, k in enumerate(keys):
        groups.setdefault(k, []).append(i)
    colliding = sorted(i for g in groups.values() if len(g) > 1 for i in g)
    first = {i: w.deliveries.index(i) for i in set(w.deliveries)}
    dup = [j for j, i in enumerate(w.deliveries) if w.deliveries.count(i) > 1]
    a, b = w.shared_k[0]
    assert colliding == sorted(dup + [first[a], first[b]])   # the workload's copy and tie
    assert len(set(ids)) == w.n_distinct
    plan = oracle_plan(dl, ids, keys)
    assert res.n_unique == plan["n_unique"] == w.n_distinct
    assert res.order == plan["order"]
    assert res.offsets == plan["offsets"]
    assert res.lengths == plan["lengths"]
    assert res.T_out == plan["T_out"] == w.merged_tokens
    assert res.slot_of_delivery == plan["slot_of_delivery"]

    order, offs, lens = plan["order"], plan["offsets"], plan["lengths"]
    log("[fullsize] V of every slot and layer, K at offset 0, on the device")
    for l in range(w.L):
        Kout, Vout = res.cache[l]
        for s, i in enumerate(order):
            K, V = dl[i][l]
            assert torch.equal(Vout[:, :, offs[s]:offs[s] + lens[s]], V), f"V layer {l} slot {s}"
            if offs[s] == 0:
                assert torch.equal(Kout[:, :, :lens[s]], K), f"K layer {l} slot {s}"

    log(f"[fullsize] oracle render of layer {w.routing_layer} in full")
    ref = oracle_layers(dl, w.dtype, order, w.rope_base, [w.routing_layer])[w.routing_layer]
    gK = synth.tensor_to_numpy(res.cache[w.routing_layer][0])
    gV = synth.tensor_to_numpy(res.cache[w.routing_layer][1])
    assert np.array_equal(gV, ref[1])
    ok, same = k_close(gK, ref[0], w.dtype)
    ulp, _ = k_stats(gK, ref[0], w.dtype)
    log(f"[fullsize] layer {w.routing_layer}: {same:.6f} of K elements bit-identical, "
        f"largest distance {ulp} ulp")
    assert ok and same >= 0.999, f"layer {w.routing_layer}: K identical {same}"
    del ref, gK, gV

    log("[fullsize] first, middle and last row of every slot in every layer")
    rows = [t for s in range(len(order)) for t in (0, lens[s] // 2, lens[s] - 1)]
    out_rows = torch.tensor([offs[s] + t for s in range(len(order)) for t in (0, lens[s] // 2, lens[s] - 1)],
                            device="cuda")
    for l in range(w.L):
        g = synth.tensor_to_numpy(res.cache[l][0].index_select(2, out_rows))
        for s, i in enumerate(order):
            src = synth.tensor_to_numpy(dl[i][l][0].index_select(
                2, torch.tensor(rows[3 * s:3 * s + 3], device="cuda")))
            if offs[s] == 0:
                want = src
            else:
                c, sn = oracle.rope_angles(offs[s], w.d, w.rope_base)
                want = oracle.round_to_dtype(oracle.rotate_pairs(om.to_f64(src, w.dtype), c, sn),
                                             w.dtype)
            ok, _ = k_close(g[:, :, 3 * s:3 * s + 3], want, w.dtype)
            assert ok, f"K layer {l} slot {s}"

    log("[fullsize] render of the ingested set")
    merged = res.merged
    del res
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    assert len(S) == w.n_distinct
    r2 = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    assert r2.T_out == w.merged_tokens
    assert torch.equal(r2.merged, merged)
    log("[fullsize] done")
