"""cm_render_deliveries_noalloc, called through the C ABI, against
cm_render_deliveries with a caller workspace: the same keys, key mask, Ids, plan
and merged cache, byte for byte (both run the same kernels; only where the
scratch lives differs). Two calls in a row share the library's fixed scratch,
the second on a smaller set, so what the first left there must not leak into
the second; each set's Ids are also checked against the oracle's."""

import pytest
import torch

import paper_2607_01308_amd as cm
import synth
from paper_2607_01308_amd import _cabi as C
from paper_2607_01308_amd import binding

from gpu_util import gpu_deliveries, log, oracle_ids

pytestmark = pytest.mark.gpu

# a larger set (duplicate delivery, an equal-score pair, ragged lengths, bf16
# d=128 rows of 256 B) and then a smaller one (fp32, rows of 256 B)
FIRST = dict(name="noalloc-a", dtype="bfloat16", d=128, H=4, L=3,
             lengths=(700, 700, 300, 1213), shared_k=((0, 1),), deliveries=(0, 1, 2, 3, 2),
             routing_layer=1)
SECOND = dict(name="noalloc-b", dtype="float32", d=64, H=2, L=2, lengths=(77, 129, 5),
              deliveries=(1, 0, 2, 1), routing_layer=0)


def _outputs(batch, T_cap):
    dev = batch.device
    return dict(keys=torch.full((batch.n,), float("nan"), dtype=torch.float64, device=dev),
                mask=torch.full((batch.n,), 7, dtype=torch.uint8, device=dev),
                digests=torch.zeros((batch.n, 32), dtype=torch.uint8, device=dev),
                plan=torch.full((cm.plan_elems(batch.n),), -9, dtype=torch.int64, device=dev),
                out=torch.zeros(batch.L * 2 * batch.H * T_cap * batch.d, dtype=batch.torch_dtype,
                                device=dev))


def _run(batch, w, noalloc):
    T_cap = int(sum(batch.lengths))
    o = _outputs(batch, T_cap)
    tail = min(batch.lengths)
    if noalloc:
        binding.render_deliveries_noalloc(batch, w.routing_layer, tail, w.rope_base, "half",
                                          o["keys"], o["mask"], o["digests"], o["plan"],
                                          o["out"], T_cap)
    else:
        ws = torch.empty(max(cm.workspace_size(batch), 256), dtype=torch.uint8,
                         device=batch.device)
        binding.render_deliveries_async(batch, w.routing_layer, tail, w.rope_base, "half",
                                        o["keys"], o["mask"], o["digests"], o["plan"], o["out"],
                                        T_cap, ws)
    torch.cuda.synchronize()
    return o


def _same(a, b):
    plan = a["plan"].cpu().numpy()
    assert plan[C.PLAN_STATUS] == 0
    T_out = int(plan[C.PLAN_TOUT])
    for k in ("keys", "mask", "digests", "plan"):
        assert torch.equal(a[k], b[k]), k
    return plan, T_out


def test_noalloc_equals_workspace_call_twice_second_smaller():
    sets = []
    for spec in (FIRST, SECOND):
        w = synth.custom(**spec)
        _, dl = gpu_deliveries(w)
        batch = cm.FragmentBatch(dl)
        assert cm.workspace_size(batch) <= C.NOALLOC_SCRATCH_BYTES
        sets.append((w, dl, batch))
    # the two no-allocation calls back to back, then the references
    got = []
    for w, _, batch in sets:
        log(f"[noalloc] {w.name}: lengths {w.lengths} deliveries {w.deliveries} {w.dtype}")
        got.append(_run(batch, w, noalloc=True))
    for (w, dl, batch), g in zip(sets, got):
        ref = _run(batch, w, noalloc=False)
        _, T_out = _same(g, ref)
        rows = batch.L * 2 * batch.H * T_out * batch.d
        assert torch.equal(g["out"][:rows], ref["out"][:rows])
        # the Ids against the oracle's, from the generator's tensors
        assert [bytes(r) for r in g["digests"].cpu().numpy()] == oracle_ids(dl, w.dtype)
        assert T_out == sum(w.lengths[i] for i in sorted(set(w.deliveries)))
        log(f"[noalloc] {w.name}: T_out {T_out}, {rows} elements identical")


def test_noalloc_rejects_a_set_beyond_its_scratch():
    """The size check runs on the host before anything is enqueued: the outputs
    (allocated at full size all the same) stay untouched. Two bf16 fragments of
    8 heads x 200,000 rows x 128: 1.6 GB, whose workspace is about 77 MB."""
    w = synth.custom("noalloc-big", dtype="bfloat16", d=128, H=8, L=1, lengths=(200000, 200000),
                     routing_layer=0)
    _, dl = gpu_deliveries(w)
    batch = cm.FragmentBatch(dl)
    assert cm.workspace_size(batch) > C.NOALLOC_SCRATCH_BYTES
    T_cap = int(sum(batch.lengths))
    o = _outputs(batch, T_cap)
    with pytest.raises(cm.CmError) as e:
        binding.render_deliveries_noalloc(batch, 0, 1, w.rope_base, "half", o["keys"], o["mask"],
                                          o["digests"], o["plan"], o["out"], T_cap)
    assert e.value.status == C.CM_EWORKSPACE
    torch.cuda.synchronize()
    assert int(o["plan"][0]) == -9 and bool(torch.isnan(o["keys"]).all())
    assert not bool(o["out"].any())
