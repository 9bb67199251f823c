"""GPU: seeded random workloads across the supported shapes, against the oracle.

Each case draws a dtype, a row size (64 B to 1 KiB), heads, layers, the routing
layer, 1-6 distinct fragments of 1-600 tokens (some page- or chunk-aligned),
re-deliveries, pairs with equal K (ties broken by the digest), the RoPE pairing
and base, and a page size. The whole path is compared with the oracle on every
layer (digests, scores, plan and V bit for bit, K within the dtype's
tolerance); the render of the ingested set and steps 1-5 on the same deliveries
stored on pages (one call, device-built block tables) must equal it."""

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


def _draw(seed):
    rng = np.random.default_rng(1000 + seed)
    dtype = ["bfloat16", "float32"][rng.integers(2)]
    esize = 2 if dtype == "bfloat16" else 4
    d = int(rng.choice([x for x in (16, 32, 64, 128, 256, 512) if 64 <= x * esize <= 1024]))
    H, L = int(rng.integers(1, 5)), int(rng.integers(2, 5))
    n = int(rng.integers(1, 7))
    lengths = []
    for _ in range(n):
        kind = rng.integers(4)
        lengths.append(int(rng.integers(1, 8)) if kind == 0 else
                       int(16 * rng.integers(1, 20)) if kind == 1 else int(rng.integers(1, 601)))
    shared = []
    if n >= 2 and rng.random() < 0.5:
        a, b = (int(x) for x in rng.choice(n, 2, replace=False))
        lengths[b] = lengths[a]
        shared.append((a, b))
    deliveries = [i for i in range(n) for _ in range(int(rng.integers(1, 4)))]
    deliveries = [int(x) for x in rng.permutation(deliveries)]
    rb = d * esize
    B = int(rng.choice([b for b in (1, 2, 4, 8, 16, 32, 64, 128, 256) if 1024 <= b * rb <= 16384]))
    return dict(dtype=dtype, d=d, H=H, L=L, lengths=tuple(lengths), deliveries=tuple(deliveries),
                shared_k=tuple(shared), routing_layer=int(rng.integers(L)),
                rope_base=float(rng.choice([1e4, 1e6])),
                style=["half", "interleaved"][rng.integers(2)], B=B, seed=seed)


CASES = [_draw(s) for s in range(64)]


@pytest.mark.parametrize("case", CASES, ids=[f"r{c['seed']}" for c in CASES])
def test_random_workload_against_oracle(case):
    w = synth.custom(f"random{case['seed']}", dtype=case["dtype"], d=case["d"], H=case["H"],
                     L=case["L"], lengths=case["lengths"], deliveries=case["deliveries"],
                     shared_k=case["shared_k"], routing_layer=case["routing_layer"],
                     rope_base=case["rope_base"], seed=case["seed"] + 7)
    dl = synth.make_deliveries(w, synth.make_fragments(w, device="cuda"))
    style = case["style"]
    log(f"[random] {case}")
    res = cm.render_deliveries(dl, w.routing_layer, w.rope_base, style=style)
    torch.cuda.synchronize()
    check_render(res, dl, w.dtype, w.routing_layer, w.rope_base, style=style, min_identical=0.99)
    # the render of the ingested set
    S = cm.LatentFragmentSet()
    S.ingest_many(dl)
    assert torch.equal(S.render(w.routing_layer, w.rope_base, style=style).merged, res.merged)
    # the same deliveries on pages, steps 1-5 in one call
    B = case["B"]
    spare = 2 * (sum(len_ for len_ in (c[0][0].shape[2] for c in dl)) // B + len(dl) + 1)
    pool, lengths, page_lists, free = synth.make_paged(dl, B, spare_pages=spare, seed=case["seed"])
    pr = cm.render_paged_set(cm.PagedSet(pool, lengths, page_lists), w.routing_layer,
                             w.rope_base, free, style=style)
    torch.cuda.synchronize()
    assert np.array_equal(pr.plan, res.plan)
    assert torch.equal(pr.digests_dev, res.digests_dev)
    K = synth.gather_paged(pool, pr.k_table, pr.T_out)[:, 0]
    V = synth.gather_paged(pool, pr.v_table, pr.T_out)[:, 1]
    assert torch.equal(K, res.merged[:, 0]) and torch.equal(V, res.merged[:, 1])
