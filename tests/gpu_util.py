"""Helpers for the GPU parity tests: run the HIP path and build the oracle's
answer from the generator's tensors (never from the HIP path's outputs)."""

from __future__ import annotations

import sys
from typing import Dict, Iterable, List, Optional, Sequence

import numpy as np
import torch

import oracle
import synth
from oracle import cmerge_oracle as om


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def k_close(gpu: np.ndarray, ref: np.ndarray, dtype: str):
    """|g - r| <= tol * max(|r|, smallest normal): tol 2^-7 (bf16), 1e-5 (fp32).
    Returns (all within tolerance, fraction bit-identical)."""
    if dtype == "bfloat16":
        g, r = oracle.bf16_bits_to_f64(gpu), oracle.bf16_bits_to_f64(ref)
        tol, tiny = 2.0 ** -7, 2.0 ** -126
    else:
        g, r = gpu.astype(np.float64), ref.astype(np.float64)
        tol, tiny = 1e-5, float(np.finfo(np.float32).tiny)
    both_nan = np.isnan(g) & np.isnan(r)
    with np.errstate(invalid="ignore"):
        ok = (g == r) | both_nan | (np.abs(g - r) <= tol * np.maximum(np.abs(r), tiny))
    return bool(ok.all()), float(np.mean(gpu.view(np.uint8) == ref.view(np.uint8)))


def oracle_ids(deliveries: Sequence, dtype: str) -> List[bytes]:
    """Oracle Id of each delivery, streaming one tensor at a time to the host."""
    ids = []
    for cache in deliveries:
        L = len(cache)
        _, H, T, d = cache[0][0].shape
        roots = []
        for K, V in cache:
            for x in (K, V):
                roots.append(om.tensor_root(synth.tensor_to_numpy(x)))
        ids.append(om.fragment_id_from_roots(om.fragment_header(dtype, L, H, T, d), roots))
    return ids


def oracle_keys(deliveries: Sequence, dtype: str, layer: int, tail: int) -> List[float]:
    out = []
    for cache in deliveries:
        K = synth.tensor_to_numpy(cache[layer][0])
        f = oracle.Fragment(dtype, [(K, np.zeros_like(K))])
        out.append(oracle.fragment_key(f, 0, tail))
    return out


def oracle_plan(deliveries: Sequence, ids: List[bytes], keys: List[float]):
    """Dedupe (first arrival kept), canonical order, offsets."""
    first: Dict[bytes, int] = {}
    for i, fid in enumerate(ids):
        first.setdefault(fid, i)
    kept = sorted(first.values())
    order_local = oracle.canonical_order([keys[i] for i in kept], [ids[i] for i in kept])
    order = [kept[j] for j in order_local]
    lengths = [deliveries[i][0][0].shape[2] for i in order]
    slot_of_id = {ids[i]: s for s, i in enumerate(order)}
    return {
        "order": order,
        "lengths": lengths,
        "offsets": oracle.offsets_of(lengths),
        "n_unique": len(kept),
        "T_out": int(sum(lengths)),
        "slot_of_delivery": [slot_of_id[f] for f in ids],
    }


def oracle_layers(deliveries: Sequence, dtype: str, order: List[int], rope_base: float,
                  layers: Iterable[int], style: str = "half"):
    """Oracle render (Eq. (1)-(2)) of the chosen layers, in the given slot order."""
    out = {}
    for l in layers:
        frags = []
        for i in order:
            K, V = deliveries[i][l]
            frags.append(oracle.Fragment(dtype, [(synth.tensor_to_numpy(K), synth.tensor_to_numpy(V))]))
        out[l] = oracle.render_in_order(frags, rope_base, style)[0]
    return out


def check_render(res, deliveries: Sequence, dtype: str, routing_layer: int, rope_base: float,
                 layers: Optional[Iterable[int]] = None, ids_ref: Optional[List[bytes]] = None,
                 min_identical: float = 0.999, style: str = "half"):
    """Full comparison of a GPU RenderResult with the oracle (all layers unless
    `layers` is given). Returns the fraction of K bytes identical."""
    L = len(deliveries[0])
    tail = min(c[0][0].shape[2] for c in deliveries)
    assert res.tail_len == tail
    ids = ids_ref if ids_ref is not None else oracle_ids(deliveries, dtype)
    assert res.digests == ids, "digests differ from the oracle"
    keys = oracle_keys(deliveries, dtype, routing_layer, tail)
    gk = res.keys
    for i, k in enumerate(keys):
        assert gk[i] == k, f"score of delivery {i}: gpu {gk[i]!r} oracle {k!r}"
    plan = oracle_plan(deliveries, ids, keys)
    assert res.n_unique == plan["n_unique"]
    assert res.order == plan["order"]
    assert res.offsets == plan["offsets"]
    assert res.lengths == plan["lengths"]
    assert res.T_out == plan["T_out"]
    assert res.slot_of_delivery == plan["slot_of_delivery"]
    layers = list(range(L)) if layers is None else list(layers)
    ref = oracle_layers(deliveries, dtype, plan["order"], rope_base, layers, style)
    same_total = []
    for l in layers:
        gK = synth.tensor_to_numpy(res.cache[l][0])
        gV = synth.tensor_to_numpy(res.cache[l][1])
        rK, rV = ref[l]
        assert gK.shape == rK.shape and gV.shape == rV.shape
        assert np.array_equal(gV, rV), f"V of layer {l} differs"
        ok, same = k_close(gK, rK, dtype)
        assert ok, f"K of layer {l} outside tolerance"
        same_total.append(same)
    frac = float(np.mean(same_total))
    assert frac >= min_identical, f"only {frac:.6f} of K bytes identical"
    return frac


def gpu_deliveries(w, device="cuda"):
    frags = synth.make_fragments(w, device=device)
    return frags, synth.make_deliveries(w, frags)
