"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Digests, scores, dedupe, order, offsets and V are compared bit for bit; K
element by element within 2^-7 (bf16) or 1e-5 (fp32) relative to
max(|ref|, smallest normal), and the bit-identical fraction is asserted too.
Inputs come from the seeded generator, never from the HIP path."""

import itertools

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_01308_amd as cm
from gpu_util import (check_render, gpu_deliveries, k_close, log, oracle_ids, oracle_keys,
                      oracle_plan)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    yield
    torch.cuda.synchronize()


def _run(w, deliveries, style="half"):
    log(f"[render] {w.name} n={len(deliveries)} L={w.L} H={w.H} d={w.d} {w.dtype}")
    res = cm.render_deliveries(deliveries, w.routing_layer, w.rope_base, style=style)
    torch.cuda.synchronize()
    return res


def test_tiny_workload():
    w = synth.tiny()
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    frac = check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)
    assert res.T_out == 40 and res.n_unique == 2
    log(f"tiny: K bit-identical fraction {frac:.6f}")


SHAPES = [
    dict(name="bf16-d128-ragged", dtype="bfloat16", d=128, H=2, L=3, lengths=(300, 517, 1000),
         deliveries=(0, 1, 2, 1, 0)),
    dict(name="fp32-d64", dtype="float32", d=64, H=3, L=2, lengths=(129, 64, 7), deliveries=(2, 0, 1)),
    dict(name="bf16-d32-row64B", dtype="bfloat16", d=32, H=4, L=2, lengths=(33, 100)),
    dict(name="bf16-d512-row1KiB", dtype="bfloat16", d=512, H=1, L=2, lengths=(40, 77, 5)),
    dict(name="fp32-d16-row64B", dtype="float32", d=16, H=2, L=2, lengths=(5, 3, 11)),
    dict(name="fp32-d256-row1KiB", dtype="float32", d=256, H=2, L=2, lengths=(70, 31)),
    dict(name="bf16-T1", dtype="bfloat16", d=128, H=8, L=2, lengths=(1, 1, 2)),
]


@pytest.mark.parametrize("spec", SHAPES, ids=[s["name"] for s in SHAPES])
def test_shapes_tiles_and_ragged_tails(spec):
    spec = dict(spec)
    name = spec.pop("name")
    w = synth.custom(name, routing_layer=1, rope_base=1e6, **spec)
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    frac = check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)
    log(f"{name}: unique={res.n_unique} T_out={res.T_out} K identical {frac:.6f}")


def test_interleaved_rope_style():
    w = synth.custom("interleaved", dtype="bfloat16", d=64, H=2, L=2, lengths=(200, 90),
                     routing_layer=0, rope_base=1e4)
    _, dl = gpu_deliveries(w)
    res = _run(w, dl, style="interleaved")
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, style="interleaved")


def test_multi_level_hash_trees():
    # 500, 1004 and 8 BLAKE3 chunks per tensor (full stripes plus a rest of 52, 44
    # and 8 chunks): odd counts carried up at several levels
    w = synth.custom("tree", dtype="bfloat16", d=128, H=2, L=2, lengths=(1000, 2008, 16))
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    assert res.digests == oracle_ids(dl, w.dtype)


@pytest.mark.parametrize("style", ["half", "interleaved"])
@pytest.mark.parametrize("dtype,d,lengths", [
    # 512 bytes per token: 32 tokens are 16 chunks (hashed by quads), 33 are 17
    # (one lane per chunk), 127 just under one stripe; every tensor shorter than
    # a stripe selects the short-tensor variant of the fused kernel
    ("bfloat16", 128, (32, 33, 127, 1)),
    ("float32", 64, (1, 16, 17, 63)),
    # one tensor of exactly one stripe: the other variant, same short stripes
    ("bfloat16", 128, (32, 128, 5)),
])
def test_short_tensor_stripes(dtype, d, lengths, style):
    w = synth.custom("short", dtype=dtype, d=d, H=2, L=2, lengths=lengths, routing_layer=1,
                     deliveries=tuple(range(len(lengths))) + (0,))
    _, dl = gpu_deliveries(w)
    res = _run(w, dl, style=style)
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, style=style)


@pytest.mark.parametrize("L", [15, 16, 255, 256, 1100])
def test_fragment_id_message_lengths(L):
    # The Id hashes L + 1 blocks: one chunk up to L = 15, at most 16 chunks (one
    # quad of lanes per chunk) up to L = 255, one lane per chunk past that, and
    # groups of 64 chunks past L = 1023. Tensors of one chunk, so the Ids come
    # from the Id kernel alone.
    w = synth.custom(f"id-L{L}", dtype="float32", d=16, H=1, L=L, lengths=(3, 5, 3),
                     deliveries=(0, 1, 2, 0), routing_layer=L // 2)
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)
    assert res.n_unique == 3


def test_single_fragment_and_all_duplicates():
    w = synth.custom("one", dtype="bfloat16", d=128, H=2, L=2, lengths=(77,), deliveries=(0, 0, 0, 0))
    frags, dl = gpu_deliveries(w)
    res = _run(w, dl)
    assert res.n_unique == 1 and res.T_out == 77 and res.slot_of_delivery == [0, 0, 0, 0]
    assert res.order == [0]
    for l in range(w.L):
        assert torch.equal(res.cache[l][0], frags[0][l][0])
        assert torch.equal(res.cache[l][1], frags[0][l][1])
    assert len(set(res.digests)) == 1


def test_equal_scores_fall_to_digest():
    w = synth.custom("tie", dtype="bfloat16", d=128, H=2, L=2, lengths=(64, 64, 40),
                     shared_k=((0, 1),), routing_layer=0)
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    k = res.keys
    assert k[0] == k[1]
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)
    d0, d1 = res.digests[0], res.digests[1]
    s0, s1 = res.slot_of_delivery[0], res.slot_of_delivery[1]
    assert (s0 < s1) == (d0 > d1)


def test_rerun_and_permutations_byte_identical():
    w = synth.custom("perm", dtype="bfloat16", d=128, H=2, L=2, lengths=(90, 130, 40, 75))
    frags, _ = gpu_deliveries(w)
    ref = cm.render_deliveries(frags, w.routing_layer, w.rope_base)
    again = cm.render_deliveries(frags, w.routing_layer, w.rope_base)
    assert torch.equal(ref.merged, again.merged)
    count = 0
    for perm in itertools.permutations(range(4)):
        out = cm.render_deliveries([frags[p] for p in perm], w.routing_layer, w.rope_base)
        assert torch.equal(out.merged, ref.merged)
        count += 1
    assert count == 24


def test_nonfinite_score_is_an_error():
    w = synth.custom("nan", dtype="bfloat16", d=128, H=2, L=2, lengths=(20, 30), routing_layer=1)
    frags, _ = gpu_deliveries(w)
    frags[1][1][0][0, 1, 25, 3] = float("nan")       # inside the routing layer's tail
    for pipe in cm.PIPELINES:            # fused: raised when the result is first used
        with pytest.raises(cm.CmError) as e:
            cm.render_deliveries(frags, w.routing_layer, w.rope_base, pipeline=pipe).T_out
        assert e.value.status == -4
    frags2, _ = gpu_deliveries(w)
    frags2[1][1][0][0, 1, 3, 3] = float("inf")        # before the tail (T* = 20 -> rows 10..29)
    frags2[0][0][0][0, 0, 5, 7] = float("nan")        # another layer
    res = cm.render_deliveries(frags2, w.routing_layer, w.rope_base)
    check_render(res, frags2, w.dtype, w.routing_layer, w.rope_base)


def test_nonfinite_score_in_a_set_render_and_incremental_cache():
    """A NaN in the routing layer's tail of a set member: the set render and the
    incremental cache report CM_ENONFINITE (-4) and hand out no cache; the
    order kernel writes an empty plan for it; a later valid set renders."""
    w = synth.custom("nan-set", dtype="bfloat16", d=128, H=2, L=2, lengths=(20, 30, 24),
                     routing_layer=1)
    frags, _ = gpu_deliveries(w)
    fs = cm.LatentFragmentSet()
    fs.ingest_many(frags)
    mc = cm.MergedCache(fs, w.routing_layer, w.rope_base)
    mc.update()
    cap, before = mc.T_cap, [x.clone() for kv in mc.cache for x in kv]
    bad = [tuple((K.clone(), V.clone()) for K, V in f) for f in frags]
    bad[2][1][0][0, 0, 23, 5] = float("nan")      # routing layer, last row (inside T* = 20)
    fs_bad = cm.LatentFragmentSet()
    fs_bad.ingest_many(bad)
    res = fs_bad.render(w.routing_layer, w.rope_base)
    with pytest.raises(cm.CmError) as e:
        res.cache
    assert e.value.status == -4
    with pytest.raises(cm.CmError) as e:
        res.merged
    assert e.value.status == -4
    plan = res.plan_dev.cpu().numpy()
    n = len(bad)
    assert plan[0] == -4 and plan[2] == 0 and plan[3] == 0
    assert (plan[4:4 + 4 * n] == -1).all()
    # the incremental cache of a set that gains the bad fragment is left as it was
    fs.ingest(bad[2])                              # a new Id (different bytes)
    with pytest.raises(cm.CmError) as e:
        mc.update()
    assert e.value.status == -4
    assert mc.T_cap == cap
    after = [x for kv in mc.cache for x in kv]
    assert all(torch.equal(a, b) for a, b in zip(before, after))
    # a valid set still renders, as the deliveries' render (checked against the oracle)
    ok = cm.LatentFragmentSet()
    ok.ingest_many(frags)
    a = ok.render(w.routing_layer, w.rope_base)
    b = cm.render_deliveries(frags, w.routing_layer, w.rope_base)
    check_render(b, frags, w.dtype, w.routing_layer, w.rope_base)
    assert torch.equal(a.merged, b.merged)


def test_render_equals_one_long_sequence():
    """Fragments keyed at local positions (rotation done here by complex
    multiplication in fp64) render into one long sequence's keys (§4.2)."""
    rng = np.random.default_rng(0)
    H, d, base = 2, 64, 1e4
    theta = base ** (-np.arange(0, d, 2) / d)

    def rot(raw, pos):
        z = (raw[..., : d // 2] + 1j * raw[..., d // 2:]) * np.exp(1j * pos[None, :, None] * theta)
        return np.concatenate([z.real, z.imag], axis=-1)

    raws, caches = [], []
    for T, s in ((300, 1.0), (170, 2.0), (45, 1.4)):
        raw = rng.standard_normal((H, T, d)) * s
        K = torch.from_numpy(rot(raw, np.arange(T)).astype(np.float32))[None].cuda()
        raws.append(raw)
        caches.append(((K, torch.zeros_like(K)),))
    res = cm.render_deliveries(caches, 0, base)
    out = res.cache[0][0][0].cpu().numpy().astype(np.float64)
    for i, off in zip(res.order, res.offsets):
        T = raws[i].shape[1]
        want = rot(raws[i], off + np.arange(T))
        assert np.allclose(out[:, off:off + T], want, rtol=0, atol=4e-7 * np.abs(want).max())


def test_latent_fragment_set_matches_delivery_render():
    w = synth.custom("set", dtype="bfloat16", d=128, H=2, L=2, lengths=(50, 80, 33),
                     deliveries=(1, 0, 1, 2, 2))
    frags, dl = gpu_deliveries(w)
    S = cm.LatentFragmentSet()
    S.ingest_many(dl[:2])
    T = cm.LatentFragmentSet()
    T.ingest_many(dl[2:])
    U = S.merge(T)
    assert len(U) == 3 and U.ids() == T.merge(S).ids()
    assert U.merge(U).ids() == U.ids()
    a = U.render(w.routing_layer, w.rope_base)
    b = cm.render_deliveries(dl, w.routing_layer, w.rope_base)
    assert torch.equal(a.merged, b.merged)
    assert set(U.ids()) == set(oracle_ids([frags[i] for i in range(3)], w.dtype))


def test_long_tail_scores_fold_in_the_order_kernels():
    """Scores whose row tree leaves more partial sums than one workgroup folds
    (3 fragments x 2048 partials): one tree launch, then the fold inside the
    order kernel (set render) or the key-mask kernel (whole path). Keys equal the
    oracle's bit for bit; the set render equals the serial pipeline, whose
    scores take the full tree of launches."""
    w = synth.custom("long-tail", dtype="bfloat16", d=64, H=8, L=1,
                     lengths=(40000, 40003, 40001), routing_layer=0)
    frags, dl = gpu_deliveries(w)
    tail = min(w.lengths)
    want = oracle_keys(dl, w.dtype, 0, tail)
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    a = S.render(w.routing_layer, w.rope_base)
    b = cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="serial")
    c = cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="fused")
    torch.cuda.synchronize()
    assert torch.equal(a.merged, b.merged) and torch.equal(c.merged, b.merged)
    assert list(b.keys_dev.cpu().numpy()) == want
    assert list(c.keys_dev.cpu().numpy()) == want
    # the set's keys follow its members' order (by Id), not the deliveries'
    ids = oracle_ids(dl, w.dtype)
    by_id = dict(zip(ids, want))
    assert list(a.keys_dev.cpu().numpy()) == [by_id[bytes(x)] for x in a.digests_dev.cpu().numpy()]


def test_render_set_rejects_members_with_one_id():
    """cm_render_set on a table that lists one fragment twice: the dedupe
    absorbs the copy, the plan's T_out falls short of the caller's, the plan
    says CM_ESHAPE and nothing is rendered."""
    w = synth.custom("set-dup", dtype="bfloat16", d=128, H=2, L=2, lengths=(40, 24),
                     deliveries=(0, 1, 0), routing_layer=1)
    _, dl = gpu_deliveries(w)
    batch = cm.FragmentBatch(dl)
    ws = torch.empty(max(cm.workspace_size(batch), 256), dtype=torch.uint8, device="cuda")
    digests = torch.empty((batch.n, 32), dtype=torch.uint8, device="cuda")
    cm.fragment_hash(batch, digests, ws)
    keys = torch.empty(batch.n, dtype=torch.float64, device="cuda")
    plan = torch.full((cm.plan_elems(batch.n),), 7, dtype=torch.int64, device="cuda")
    T_out = int(sum(batch.lengths))
    out = torch.zeros((batch.L, 2, 1, batch.H, T_out, batch.d), dtype=batch.torch_dtype,
                      device="cuda")
    cm.render_set(batch, digests, w.routing_layer, min(batch.lengths), w.rope_base, "half", keys,
                  plan, out, T_out, ws)
    torch.cuda.synchronize()
    p = plan.cpu().numpy()
    assert p[0] == -2 and p[2] == 2 and p[3] == 64
    assert not bool(out.any())


@pytest.mark.parametrize("dtype,d,style", [("bfloat16", 128, "interleaved"),
                                           ("float32", 64, "half"),
                                           ("float32", 256, "interleaved"),
                                           ("bfloat16", 32, "half")])
def test_set_render_styles_and_row_sizes(dtype, d, style):
    """cm_render_set (scores, order and unit tables in one launch, then the
    unit render) for each pairing and several row sizes: the same cache as the
    deliveries' render, which is checked against the oracle."""
    w = synth.custom("set-style", dtype=dtype, d=d, H=3, L=2, lengths=(130, 61, 200, 7),
                     deliveries=(2, 0, 1, 3, 0), routing_layer=1, rope_base=1e4)
    _, dl = gpu_deliveries(w)
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    a = S.render(w.routing_layer, w.rope_base, style=style)
    b = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style=style, pipeline="serial")
    torch.cuda.synchronize()
    check_render(b, dl, w.dtype, w.routing_layer, w.rope_base, style=style)
    assert a.T_out == b.T_out and torch.equal(a.merged, b.merged)


def test_compact_releases_the_fused_buffer():
    """A fused result over re-deliveries holds an output buffer sized for every
    delivery; compact() moves the merged cache into one of exactly T_out rows,
    with the same bytes, and drops the larger buffer."""
    w = synth.custom("compact", dtype="bfloat16", d=128, H=2, L=2, lengths=(64, 40),
                     deliveries=(0, 1, 0, 0, 1), routing_layer=1)
    _, dl = gpu_deliveries(w)
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="fused")
    before = res.merged.clone()
    big = res.merged.untyped_storage().nbytes()
    res.compact()
    torch.cuda.synchronize()
    assert torch.equal(res.merged, before) and res.T_out == 104
    assert res.merged.untyped_storage().nbytes() == before.numel() * before.element_size() < big
    assert all(torch.equal(k, res.merged[l, 0]) for l, (k, _) in enumerate(res.cache))
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)


def test_timing_api_counts_launches():
    w = synth.custom("timing", lengths=(64, 32))
    _, dl = gpu_deliveries(w)
    cm.timing_reset()
    cm.timing_enable(True)
    try:
        cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="fused")
        cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="serial")
        torch.cuda.synchronize()
        # (the fragments' Ids come from the tree's top launch: hash_final runs
        # only for sets whose tensors are single chunks)
        for k in ("hash_leaf", "hash_parent", "knorm_rows", "order", "key_mask",
                  "render_prep", "render", "render_hash"):
            ms, n = cm.timing_query(k)
            assert n >= 1 and ms > 0.0, k
    finally:
        cm.timing_enable(False)
        cm.timing_reset()


def test_binding_rejects_bad_tensors():
    K = torch.zeros((1, 2, 8, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        cm.FragmentBatch([((K.transpose(2, 3).contiguous().transpose(2, 3), K),)])
    with pytest.raises(ValueError):
        cm.FragmentBatch([((K, K),), ((K, K), (K, K))])
    with pytest.raises(TypeError):
        cm.FragmentBatch([((K.half(), K.half()),)])


# ---------------------------------------------------------------- workload sizes

def test_qwen3_17b_n2_full():
    w = synth.qwen3_17b_n2()
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    frac = check_render(res, dl, w.dtype, w.routing_layer, w.rope_base)
    log(f"qwen3-1.7b-n2: K bit-identical fraction {frac:.7f}")


def test_qwen3_17b_n5_all_permutations_and_redelivery():
    w = synth.qwen3_17b_n5()
    frags, dl = gpu_deliveries(w)
    res = _run(w, dl)
    frac = check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, layers=(0, 14, 27))
    log(f"qwen3-1.7b-n5: oracle parity on layers 0/14/27, K identical {frac:.7f}")
    assert res.n_unique == 5 and res.T_out == sum(w.lengths)
    copies = {i: tuple((K.clone(), V.clone()) for K, V in frags[i]) for i in range(5)}
    redelivered = [i for i in range(5) for _ in range(w.deliveries.count(i) - 1)]
    rng = np.random.default_rng(11)
    count = 0
    for perm in itertools.permutations(range(5)):
        lst = [frags[p] for p in perm]
        for i in redelivered:                               # re-deliveries at random places
            lst.insert(int(rng.integers(0, len(lst) + 1)), copies[i])
        out = cm.render_deliveries(lst, w.routing_layer, w.rope_base)
        assert out.n_unique == 5 and torch.equal(out.merged, res.merged)
        count += 1
    assert count == 120
    log("qwen3-1.7b-n5: 120 permutations with shuffled re-deliveries byte-identical")


def test_qwen3_4b_n4_sampled_layers():
    w = synth.qwen3_4b_n4()
    _, dl = gpu_deliveries(w)
    res = _run(w, dl)
    frac = check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, layers=(0, 18, 35))
    log(f"qwen3-4b-n4: K identical {frac:.7f}")


# ---------------------------------------------------------------- overlapped pipeline

def _keys_and_mask(batch, w):
    ws = torch.empty(max(cm.workspace_size(batch), 256), dtype=torch.uint8, device="cuda")
    keys = torch.empty(batch.n, dtype=torch.float64, device="cuda")
    mask = torch.empty(batch.n, dtype=torch.uint8, device="cuda")
    cm.fragment_knorm(batch, w.routing_layer, min(batch.lengths), keys, ws)
    cm.equal_key_mask(batch, keys, mask)
    torch.cuda.synchronize()
    return ws, keys, mask


def test_equal_key_mask_marks_copies_and_ties():
    w = synth.custom("mask", dtype="bfloat16", d=128, H=2, L=2, lengths=(64, 64, 40, 70),
                     shared_k=((0, 1),), deliveries=(0, 1, 2, 3, 2), routing_layer=0)
    _, dl = gpu_deliveries(w)
    batch = cm.FragmentBatch(dl)
    _, keys, mask = _keys_and_mask(batch, w)
    assert mask.cpu().tolist() == [1, 1, 1, 0, 1]


def test_hash_select_writes_only_selected_digests():
    w = synth.custom("sel", dtype="bfloat16", d=128, H=2, L=2, lengths=(300, 64, 129))
    _, dl = gpu_deliveries(w)
    batch = cm.FragmentBatch(dl)
    ws = torch.empty(max(cm.workspace_size(batch), 256), dtype=torch.uint8, device="cuda")
    sel = torch.tensor([0, 1, 0], dtype=torch.uint8, device="cuda")
    dig = torch.full((3, 32), 0xAB, dtype=torch.uint8, device="cuda")
    cm.fragment_hash_select(batch, sel, 1, dig, ws)
    torch.cuda.synchronize()
    ref = oracle_ids(dl, w.dtype)
    got = [bytes(r) for r in dig.cpu().numpy()]
    assert got[1] == ref[1] and got[0] == bytes([0xAB]) * 32 and got[2] == bytes([0xAB]) * 32
    cm.fragment_hash_select(batch, sel, 0, dig, ws)
    torch.cuda.synchronize()
    assert [bytes(r) for r in dig.cpu().numpy()] == ref


def test_order_reads_only_colliding_digests():
    w = synth.custom("ordsel", dtype="bfloat16", d=128, H=2, L=2, lengths=(64, 64, 40, 70),
                     shared_k=((0, 1),), deliveries=(2, 0, 1, 3, 2))
    _, dl = gpu_deliveries(w)
    batch = cm.FragmentBatch(dl)
    ws, keys, mask = _keys_and_mask(batch, w)
    dig = torch.empty((batch.n, 32), dtype=torch.uint8, device="cuda")
    cm.fragment_hash(batch, dig, ws)
    plan_a = torch.empty(cm.plan_elems(batch.n), dtype=torch.int64, device="cuda")
    cm.canonical_order(batch, keys, dig, plan_a)
    noisy = dig.clone()
    rnd = torch.randint(0, 256, noisy.shape, dtype=torch.uint8, device="cuda")
    noisy[mask == 0] = rnd[mask == 0]
    plan_b = torch.empty_like(plan_a)
    cm.canonical_order(batch, keys, noisy, plan_b)
    torch.cuda.synchronize()
    assert torch.equal(plan_a, plan_b)


PIPE_SHAPES = [
    dict(dtype="bfloat16", d=128, H=4, L=3, lengths=(700, 700, 300, 1200), shared_k=((0, 1),),
         deliveries=(3, 0, 2, 1, 0)),
    dict(dtype="bfloat16", d=64, H=3, L=2, lengths=(3000, 77, 1)),       # multi-stripe, tiny T
    dict(dtype="float32", d=64, H=2, L=2, lengths=(130, 4100, 9)),
    dict(dtype="bfloat16", d=32, H=4, L=2, lengths=(513, 40), deliveries=(1, 0, 1)),  # 64 B rows
    dict(dtype="bfloat16", d=512, H=1, L=2, lengths=(300, 257)),         # 1 KiB rows
    dict(dtype="float32", d=16, H=2, L=2, lengths=(70, 33)),             # 64 B rows, fp32
    dict(dtype="bfloat16", d=256, H=2, L=2, lengths=(520, 61, 3)),       # partner 16 lanes away
    dict(dtype="float32", d=32, H=3, L=2, lengths=(300, 17)),            # partner 4 lanes away
    dict(dtype="float32", d=128, H=2, L=2, lengths=(140, 1025)),         # partner 16 lanes away
    # every tensor one chunk (no parent levels), with a re-delivery whose Id is
    # computed before the order
    dict(dtype="float32", d=16, H=2, L=2, lengths=(5, 3, 8), deliveries=(0, 1, 2, 1)),
    # a tree of one parent level (the tail launch alone)
    dict(dtype="bfloat16", d=64, H=1, L=3, lengths=(9, 16, 2), deliveries=(2, 0, 1, 0)),
]


@pytest.mark.parametrize("spec", PIPE_SHAPES, ids=[f"pipe{i}" for i in range(len(PIPE_SHAPES))])
def test_pipelines_agree_and_match_oracle(spec):
    w = synth.custom("pipes", routing_layer=1, **spec)
    _, dl = gpu_deliveries(w)
    outs = {p: cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline=p)
            for p in cm.PIPELINES}
    torch.cuda.synchronize()
    ref = outs["serial"]
    for p, r in outs.items():
        assert torch.equal(r.merged, ref.merged), p
        assert r.digests == ref.digests, p
        assert list(r.plan) == list(ref.plan), p
    check_render(outs["fused"], dl, w.dtype, w.routing_layer, w.rope_base)


@pytest.mark.parametrize("dtype", ["bfloat16", "float32"])
def test_fused_interleaved_style(dtype):
    w = synth.custom("fused-il", dtype=dtype, d=128, H=2, L=2, lengths=(600, 333),
                     routing_layer=0, rope_base=1e4)
    _, dl = gpu_deliveries(w)
    a = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style="interleaved", pipeline="fused")
    b = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style="interleaved", pipeline="serial")
    torch.cuda.synchronize()
    assert torch.equal(a.merged, b.merged) and a.digests == b.digests
    check_render(a, dl, w.dtype, w.routing_layer, w.rope_base, style="interleaved")


def test_devplan_render_equals_host_checked_render_and_rejects_bad_plans():
    """cm_render_merge_devplan renders the device plan exactly like
    cm_render_merge; a plan that fails the device check moves no byte and
    reports CM_ESHAPE in its status entry, unless its status already reports an
    error (a non-finite score, CM_ENONFINITE), which it keeps."""
    w = synth.custom("devplan", dtype="bfloat16", d=128, H=2, L=2, lengths=(300, 129, 77),
                     routing_layer=1)
    _, dl = gpu_deliveries(w)
    ref = cm.render_deliveries(dl, w.routing_layer, w.rope_base, pipeline="serial")
    torch.cuda.synchronize()
    batch = cm.FragmentBatch(dl)
    ws = torch.empty(max(cm.workspace_size(batch), 256), dtype=torch.uint8, device="cuda")
    plan = torch.from_numpy(ref.plan.copy()).to("cuda")
    out = torch.zeros_like(ref.merged)
    cm.render_merge_devplan(batch, plan, w.rope_base, "half", out, ref.T_out, ws)
    torch.cuda.synchronize()
    assert torch.equal(out, ref.merged)
    assert int(plan[0]) == 0
    n = batch.n
    for what, mutate in (("offset", lambda p: p.__setitem__(4 + n + 1, p[4 + n + 1] + 1)),
                         ("length", lambda p: p.__setitem__(4 + 2 * n, p[4 + 2 * n] - 1)),
                         ("delivery", lambda p: p.__setitem__(4, 7)),
                         ("status", lambda p: p.__setitem__(0, -4))):
        bad = ref.plan.copy()
        mutate(bad)
        log(f"[devplan] corrupted {what}")
        plan = torch.from_numpy(bad).to("cuda")
        out = torch.full_like(ref.merged, 3)
        cm.render_merge_devplan(batch, plan, w.rope_base, "half", out, ref.T_out, ws)
        torch.cuda.synchronize()
        assert int(plan[0]) == (-4 if what == "status" else -2), what
        assert bool((out == 3).all()), what
    plan = torch.from_numpy(ref.plan.copy()).to("cuda")
    shape = list(ref.merged.shape)
    shape[4] -= 1                                                  # T_out one short
    out = torch.full(shape, 3, dtype=ref.merged.dtype, device="cuda")
    cm.render_merge_devplan(batch, plan, w.rope_base, "half", out, ref.T_out - 1, ws)
    torch.cuda.synchronize()
    assert int(plan[0]) == -2 and bool((out == 3).all())


def test_results_on_two_streams_and_read_late():
    """Fused calls on two caller streams, each result read only after later calls
    were enqueued: every call keeps its own scratch and buffers, so each result
    equals the same render made alone (and the oracle's plan)."""
    w1 = synth.custom("streams-a", dtype="bfloat16", d=128, H=2, L=2, lengths=(300, 517, 128),
                      deliveries=(0, 1, 2, 1), routing_layer=1)
    w2 = synth.custom("streams-b", dtype="bfloat16", d=128, H=2, L=3, lengths=(200, 90),
                      seed=11, routing_layer=2)
    f1, dl1 = gpu_deliveries(w1)
    f2, dl2 = gpu_deliveries(w2)
    ref1 = _run(w1, dl1)
    ref2 = _run(w2, dl2)
    check_render(ref1, dl1, w1.dtype, w1.routing_layer, w1.rope_base)
    check_render(ref2, dl2, w2.dtype, w2.routing_layer, w2.rope_base)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    pending = []
    for rep in range(3):
        log(f"[streams] round {rep}")
        pending.append((ref1, cm.render_deliveries(dl1, w1.routing_layer, w1.rope_base, stream=sa)))
        pending.append((ref2, cm.render_deliveries(dl2, w2.routing_layer, w2.rope_base, stream=sb)))
    for ref, res in reversed(pending):
        assert res.T_out == ref.T_out
        assert np.array_equal(res.plan, ref.plan)
        assert res.digests == ref.digests
        assert torch.equal(res.merged, ref.merged)


def test_eight_streams_of_independent_merges():
    """Eight different sets merged at once, one per caller stream, three rounds
    issued before any result is read: each result equals that set's render made
    alone, which the oracle checks for two of them."""
    ws, dls, refs = [], [], []
    for k in range(8):
        w = synth.custom(f"streams8-{k}", dtype=["bfloat16", "float32"][k % 2], d=64 * (1 + k % 2),
                         H=1 + k % 3, L=2, lengths=(17 + 31 * k, 40 + 7 * k, 3 + k),
                         deliveries=(0, 1, 2, k % 3), routing_layer=k % 2, seed=40 + k)
        _, dl = gpu_deliveries(w)
        ws.append(w)
        dls.append(dl)
        refs.append(_run(w, dl))
    for k in (0, 5):
        check_render(refs[k], dls[k], ws[k].dtype, ws[k].routing_layer, ws[k].rope_base)
    streams = [torch.cuda.Stream() for _ in range(8)]
    torch.cuda.synchronize()
    pending = []
    for rep in range(3):
        for k, st in enumerate(streams):
            pending.append((refs[k], cm.render_deliveries(dls[k], ws[k].routing_layer,
                                                          ws[k].rope_base, stream=st)))
    log(f"[streams8] {len(pending)} merges issued")
    for ref, res in pending:
        assert np.array_equal(res.plan, ref.plan)
        assert res.digests == ref.digests
        assert torch.equal(res.merged, ref.merged)
