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


def _ordered(bits: np.ndarray, sign: int) -> np.ndarray:
    """Sign-magnitude float bit patterns as integers in the order of the values
    (adjacent representable values differ by 1; +0 and -0 both map to 0)."""
    b = bits.astype(np.int64)
    return np.where(b & sign, -(b & (sign - 1)), b)


def k_stats(gpu: np.ndarray, ref: np.ndarray, dtype: str):
    """(largest distance in units in the last place of the storage type,
    fraction of elements bit-identical) between two K arrays (bf16 as uint16
    bits, or fp32). NaN against NaN counts as distance 0."""
    if dtype == "bfloat16":
        g, r, sign = gpu.view(np.uint16), ref.view(np.uint16), 0x8000
        nan_g, nan_r = (g & 0x7FFF) > 0x7F80, (r & 0x7FFF) > 0x7F80
    else:
        g, r, sign = gpu.view(np.uint32), ref.view(np.uint32), 0x80000000
        nan_g, nan_r = (g & 0x7FFFFFFF) > 0x7F800000, (r & 0x7FFFFFFF) > 0x7F800000
    dist = np.abs(_ordered(g, sign) - _ordered(r, sign))
    dist = np.where(nan_g & nan_r, 0, np.where(nan_g | nan_r, np.iinfo(np.int64).max, dist))
    return int(dist.max()) if dist.size else 0, float(np.mean(g == r)) if g.size else 1.0


def k_close(gpu: np.ndarray, ref: np.ndarray, dtype: str):
    """K within the stated bound: |g - r| <= tol * max(|r|, smallest normal) with
    tol 2^-7 (bf16), 1e-5 (fp32), and no element more than one unit in the last
    place of the storage type away. Both sides compute each element in fp64 with
    one rounding to the storage type; they differ only in the fused multiply-add
    and in the last fp64 bit of cos/sin, so two results can land on the two
    sides of a rounding boundary, one unit apart, and no further (the inputs are
    random, so a cancellation that would amplify fp64 differences has
    probability far below the test sizes). Returns (all within both bounds,
    fraction of elements bit-identical)."""
    if dtype == "bfloat16":
        g, r = oracle.bf16_bits_to_f64(gpu), oracle.bf16_bits_to_f64(ref)
        tol, tiny = 2.0 ** -7, 2.0 ** -126
    else:
        g, r = gpu.astype(np.float64), ref.astype(np.float64)
        tol, tiny = 1e-5, float(np.finfo(np.float32).tiny)
    both_nan = np.isnan(g) & np.isnan(r)
    with np.errstate(invalid="ignore"):
        ok = (g == r) | both_nan | (np.abs(g - r) <= tol * np.maximum(np.abs(r), tiny))
    ulp, same = k_stats(gpu, ref, dtype)
    return bool(ok.all()) and ulp <= 1, same


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
    `layers` is given). Returns the fraction of K elements bit-identical."""
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
    same_total, worst = [], 0
    for l in layers:
        gK = synth.tensor_to_numpy(res.cache[l][0])
        gV = synth.tensor_to_numpy(res.cache[l][1])
        rK, rV = ref[l]
        assert gK.shape == rK.shape and gV.shape == rV.shape
        assert np.array_equal(gV, rV), f"V of layer {l} differs"
        ok, same = k_close(gK, rK, dtype)
        ulp, _ = k_stats(gK, rK, dtype)
        assert ok, f"K of layer {l} outside tolerance (largest distance {ulp} ulp)"
        same_total.append(same)
        worst = max(worst, ulp)
    frac = float(np.mean(same_total))
    log(f"  K against the oracle: {frac:.6f} of elements bit-identical, largest distance "
        f"{worst} ulp")
    assert frac >= min_identical, f"only {frac:.6f} of K elements identical"
    return frac


def gpu_deliveries(w, device="cuda"):
    frags = synth.make_fragments(w, device=device)
    return frags, synth.make_deliveries(w, frags)
