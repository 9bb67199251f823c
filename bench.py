"""Benchmark: the CanonicalMerge render of a LatentFragmentSet on one MI355X.

One step = the whole path over one batch of deliveries (steps 1-5): scores,
the Id of every delivery whose score collides with another's, dedupe
+ canonical order + offsets, one small device-to-host plan copy, output
allocation, then the fused kernel that renders the merged cache and computes
the remaining Ids from the same loads. Inputs are resident in HBM before timing
starts. A workload smaller than 1 GiB of deliveries (four times the 256 MiB
Infinity Cache) is replicated and successive steps take successive copies, so
its reads come from HBM; `step_ms_p10_p50_p90` gives the spread of the timed
steps (HIP events between steps).

value = merged-cache bytes read + written per step (2 x the bytes of the
distinct fragments) / step time, in GB/s; merges_per_s = 1 / step time.
`render_set` is the same render over the already-ingested set (steps 2-5, Ids
computed at ingest), the path whose bytes are all HBM streaming.

Prints one JSON line. `roofline` is for the kernel with the largest share of
the step, measured with per-kernel HIP events on the launch stream over the
timed steps: the fused hash+render kernel against the VALU issue rate (its
algorithmic operations: 672 per hashed 64-byte block, 4 per rotated K
element). `roofline_render` gives the render kernel of `render_set` against
HBM bandwidth. `cpu_baseline` times the CPU oracle on a bounded sample of the
same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0                 # MI355X HBM3E
VALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12  # 256 CUs x 64 lanes x 2.4 GHz: one 32-bit or fp64 op
B3_OPS_PER_BLOCK = 672                 # BLAKE3: 7 rounds x 8 G x 12 VALU ops (add3, add, xor, alignbit)
ROT_OPS_PER_ELEM = 4                   # widen, fp64 product, fp64 FMA, narrow
OTHER_WORKLOADS = ("qwen3-4b-n4", "qwen3-1.7b-n5", "qwen3-1.7b-n2", "tiny")
MALL_BYTES = 256 << 20                 # MI355X Infinity Cache: inputs smaller than 4x this are
ROTATE_TARGET = 4 * MALL_BYTES         # replicated and the steps cycle through the copies

# source files each timed kernel is built from: a traffic summary is only used
# while these are unchanged
KERNEL_SOURCES = {
    "render_hash": ["render_hash.hip", "fused_geometry.h", "rotate.h", "blake3.h", "blake3_quad.h",
                    "chunk_ops.h", "stream_ops.h", "internal.h"],
    "render": ["render.hip", "render_geometry.h", "render_tables.h", "rotate.h", "stream_ops.h",
               "internal.h"],
}


def kernel_source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2607_01308_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _traffic(kernel: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it was
    taken on the current kernel sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha256_16") != kernel_source_hash(kernel):
        return None
    return t.get("hbm_bytes_per_launch")


def fused_work(w, r, mask):
    """Algorithmic work of one fused launch: VALU ops (hash of every slot whose
    Id it computes, rotation of every K element at a non-zero offset) and the
    bytes it must move."""
    tok = w.L * w.H * w.d                       # elements per token per tensor kind
    esize = 2 if w.dtype == "bfloat16" else 4
    hashed_blocks = sum(2 * tok * T * esize // 64 for i, T in zip(r.order, r.lengths)
                        if int(mask[i]) == 0)
    rotated = sum(tok * T for off, T in zip(r.offsets, r.lengths) if off != 0)
    return B3_OPS_PER_BLOCK * hashed_blocks + ROT_OPS_PER_ELEM * rotated, hashed_blocks * 64, rotated


def delivered_bytes(w):
    """Bytes of every delivery (duplicates counted): what the naive render moves each way."""
    return w.delivery_bytes


def percentiles(ms):
    """p10, p50, p90 of per-step times (nearest rank)."""
    v = sorted(ms)
    return [round(v[min(len(v) - 1, int(q * len(v)))], 4) for q in (0.1, 0.5, 0.9)]


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_path(sample, w, workers):
    """The oracle's functions over the sample: the Id of every fragment (one
    tensor root per task), the keys, the order and offsets, then the render of
    every (layer, slot) (K rotated and rounded, V copied) into the layer's
    merged arrays; tasks run on `workers` threads (numpy and the C BLAKE3 run
    outside the interpreter lock)."""
    import concurrent.futures as cf

    import numpy as np
    from oracle import cmerge_oracle as om

    with cf.ThreadPoolExecutor(workers) as ex:
        roots = list(ex.map(lambda t: om.tensor_root(np.ascontiguousarray(sample[t[0]].layers[t[1]][t[2]])),
                            [(i, l, kv) for i in range(len(sample)) for l in range(w.L)
                             for kv in (0, 1)]))
        ids = []
        for i, f in enumerate(sample):
            ids.append(om.fragment_id_from_roots(om.fragment_header(f.dtype, f.L, f.H, f.T, f.d),
                                                 roots[2 * w.L * i:2 * w.L * (i + 1)]))
        tail = min(f.T for f in sample)
        keys = [om.fragment_key(f, w.routing_layer, tail) for f in sample]
        order = om.canonical_order(keys, ids)
        offs = om.offsets_of([sample[i].T for i in order])
        T_out = sum(f.T for f in sample)
        out = [(np.empty((1, w.H, T_out, w.d), sample[0].layers[0][0].dtype),
                np.empty((1, w.H, T_out, w.d), sample[0].layers[0][0].dtype)) for _ in range(w.L)]

        def unit(t):
            l, k = t
            f, off = sample[order[k]], offs[k]
            K, V = f.layers[l]
            if off == 0:
                out[l][0][:, :, :f.T] = K
            else:
                c, sn = om.rope_angles(off, w.d, w.rope_base)
                out[l][0][:, :, off:off + f.T] = om.round_to_dtype(
                    om.rotate_pairs(om.to_f64(K, f.dtype), c, sn), f.dtype)
            out[l][1][:, :, off:off + f.T] = V

        list(ex.map(unit, [(l, k) for l in range(w.L) for k in range(len(order))]))
    return out


def cpu_baseline(w, frags):
    """The oracle, unchanged, over the five shortest distinct fragments of the
    workload, on the cores the process may use (a thread pool over (layer,
    fragment) tasks, at most 16 threads: a GPU host's share per GPU) and on one
    thread."""
    import numpy as np
    import oracle
    import synth
    idx = sorted(range(w.n_distinct), key=lambda i: w.lengths[i])[:5]
    sample = [oracle.Fragment(*synth.to_numpy_cache(frags[i])) for i in idx]
    nbytes = 2 * sum(w.fragment_bytes(i) for i in idx)
    allowed = len(os.sched_getaffinity(0))
    cores = min(allowed, 16)
    t0 = time.perf_counter()
    _oracle_path(sample, w, cores)
    dt_all = time.perf_counter() - t0
    t0 = time.perf_counter()
    _oracle_path(sample, w, 1)
    dt_one = time.perf_counter() - t0
    return {
        "value": round(nbytes / dt_all / 1e9, 4),
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "value_all": round(nbytes / dt_all / 1e9, 4),
        "value_1thread": round(nbytes / dt_one / 1e9, 4),
        "cores_allowed": allowed,
        "model": _cpu_model(),
        "numpy": np.__version__,
        "python": sys.version.split()[0],
        "sample_bytes": nbytes,
        "sample": f"full path (Id of every fragment, score, order, render) over the 5 shortest "
                  f"distinct fragments (T={[w.lengths[i] for i in idx]}, {nbytes / 1e9:.2f} GB "
                  f"read+write): {dt_all:.1f} s on {cores} threads (tensor roots and (layer, "
                  f"slot) renders as tasks), {dt_one:.1f} s on one; numpy + the oracle's C BLAKE3",
    }


def time_steps(step_fn, steps, warmup, kernel_timing=True):
    """Mean ms per step (host clock around `steps` steps bracketed by device
    synchronisation), p10/p50/p90 of per-step HIP event times, and the library's
    per-kernel totals over the timed steps (kernel_timing; the library then
    records an event pair around every launch, which costs a few microseconds
    per launch: negligible for the large workload, not for the small ones)."""
    import torch
    import paper_2607_01308_amd as cm

    for _ in range(warmup):
        r = step_fn(0)
        del r
    torch.cuda.synchronize()
    cm.timing_reset()
    cm.timing_enable(kernel_timing)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(steps):
        r = step_fn(i)
        ev[i + 1].record()
        del r
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cm.timing_enable(False)
    pct = percentiles([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
    kernels = {}
    for k in cm.KERNELS:
        ms, n = cm.timing_query(k)
        if n:
            kernels[k] = {"total_ms": ms, "launches": n, "avg_ms": ms / n}
    cm.timing_reset()
    return (t1 - t0) / steps * 1e3, pct, kernels


def replicas(w, deliveries):
    """Copies of a workload's deliveries so that successive steps read different
    inputs: a workload under four times the Infinity Cache would otherwise be
    served from it."""
    n_copies = max(1, min(32, -(-ROTATE_TARGET // w.delivery_bytes)))
    return [deliveries] + [[tuple((K.clone(), V.clone()) for K, V in c) for c in deliveries]
                           for _ in range(n_copies - 1)]


def other_workload(name, seed, steps, warmup, dev):
    """Whole path (steps 1-5) and render of the ingested set (steps 2-5) of one
    more workload."""
    import torch
    import synth
    import paper_2607_01308_amd as cm

    w = synth.workload(name, seed)
    frags = synth.make_fragments(w, device=dev)
    copies = replicas(w, synth.make_deliveries(w, frags))
    batches = [cm.FragmentBatch(c) for c in copies]
    n = len(batches)
    sets = []
    for c in copies:
        sets.append(cm.LatentFragmentSet())
        sets[-1].ingest_many(c)
    whole = lambda i: cm.render_deliveries(batches[i % n], w.routing_layer, w.rope_base)
    render = lambda i: sets[i % n].render(w.routing_layer, w.rope_base)
    # the step times without per-launch events, then the same steps again for the
    # per-kernel breakdown (event-timed, so each kernel's figure includes its
    # launch latency)
    ms, pct, _ = time_steps(whole, steps, warmup, kernel_timing=False)
    ms_set, pct_set, _ = time_steps(render, steps, warmup, kernel_timing=False)
    _, _, kern = time_steps(whole, steps, 0)
    _, _, kern_set = time_steps(render, steps, 0)
    # the whole path captured into a HIP graph per input copy, replayed: one
    # launch per step instead of one per kernel
    graphs = [cm.RenderGraph(bt, w.routing_layer, w.rope_base) for bt in batches]
    replay = lambda i: graphs[i % n].replay()
    ms_g, pct_g, _ = time_steps(replay, steps, warmup, kernel_timing=False)
    rg, re_ = graphs[0].replay(), whole(0)
    graph_equal = bool(torch.equal(rg.merged, re_.merged) and torch.equal(rg.digests_dev,
                                                                          re_.digests_dev))
    del rg, re_
    for g in graphs:
        g.close()
    del graphs
    # independent merges at once, each on a stream of its own (default priority)
    # and its own input copy: a small merge's dependent kernels leave most of the
    # chip idle, concurrent ones fill it
    n_streams = min(8, n)
    conc_ms, conc_equal = None, None
    if n_streams >= 2:
        streams = [torch.cuda.Stream(device=dev) for _ in range(n_streams)]

        def conc_step(i):
            return [cm.render_deliveries(batches[(i * n_streams + j) % n], w.routing_layer,
                                         w.rope_base, stream=st) for j, st in enumerate(streams)]

        for i in range(warmup):
            conc_step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            r = conc_step(i)
            del r
        torch.cuda.synchronize()
        conc_ms = (time.perf_counter() - t0) / steps * 1e3
        got = conc_step(0)
        torch.cuda.synchronize()
        conc_equal = all(torch.equal(g.merged, whole(j).merged) for j, g in enumerate(got))
        del got, streams
    b = w.render_bytes
    out = {
        "render_bytes": b, "deliveries": w.n_deliveries, "distinct": w.n_distinct,
        "merged_tokens": w.merged_tokens, "input_copies": n,
        "whole_path": {"ms": round(ms, 4), "ms_p10_p50_p90": pct,
                       "GBps": round(b / (ms / 1e3) / 1e9, 1),
                       "pct_hbm_peak": round(100 * b / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 2),
                       "merges_per_s": round(1e3 / ms, 1),
                       "launches_per_step": round(sum(v["launches"] for v in kern.values()) / steps, 1),
                       "kernels_ms": {k: round(v["total_ms"] / steps, 4) for k, v in kern.items()}},
        "whole_path_graph": {"ms": round(ms_g, 4), "ms_p10_p50_p90": pct_g,
                             "GBps": round(b / (ms_g / 1e3) / 1e9, 1),
                             "pct_hbm_peak": round(100 * b / (ms_g / 1e3) / 1e9 / HBM_PEAK_GBPS, 2),
                             "merges_per_s": round(1e3 / ms_g, 1), "equals_eager": graph_equal,
                             "what": "the whole path captured into a HIP graph per input copy "
                                     "(RenderGraph), replayed: one launch per step"},
        "whole_path_concurrent": None if conc_ms is None else {
            "streams": n_streams, "ms_per_round": round(conc_ms, 4),
            "merges_per_s": round(n_streams * 1e3 / conc_ms, 1),
            "GBps": round(n_streams * b / (conc_ms / 1e3) / 1e9, 1),
            "equals_single_stream": conc_equal,
            "what": "independent merges of different input copies, one per stream, issued "
                    "together; a round is one merge on every stream"},
        "render_set": {"ms": round(ms_set, 4), "ms_p10_p50_p90": pct_set,
                       "GBps": round(b / (ms_set / 1e3) / 1e9, 1),
                       "pct_hbm_peak": round(100 * b / (ms_set / 1e3) / 1e9 / HBM_PEAK_GBPS, 2),
                       "merges_per_s": round(1e3 / ms_set, 1),
                       "launches_per_step": round(sum(v["launches"] for v in kern_set.values())
                                                  / steps, 1),
                       "kernels_ms": {k: round(v["total_ms"] / steps, 4)
                                      for k, v in kern_set.items()}},
    }
    del sets, batches, copies, frags
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen3-4b-large")
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the whole-path and set-render figures of the four smaller workloads")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain streaming kernel (torch.neg over 2 GiB of bf16), whose "
                         "known read/write bytes scale rocprofv3's FETCH_SIZE/WRITE_SIZE counters")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the render is a "
              "single-GPU path and no multi-GPU figure is produced", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    import paper_2607_01308_amd as cm

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        src = torch.ones(1 << 30, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print("[bench] calibration copy: 3 x torch.neg over 2 GiB in, 2 GiB out",
              file=sys.stderr, flush=True)
        del src, dst
    w = synth.workload(args.workload, args.seed)
    print(f"[bench] generating {w.name}: {w.n_deliveries} deliveries, {w.n_distinct} distinct, "
          f"{w.merged_tokens} merged tokens", file=sys.stderr, flush=True)
    frags = synth.make_fragments(w, device=dev)
    deliveries = synth.make_deliveries(w, frags)
    batch = cm.FragmentBatch(deliveries)
    # a workload that would sit in the Infinity Cache is replicated, each step
    # taking the next copy, so every step reads its inputs from HBM
    copies = replicas(w, deliveries)
    n_copies = len(copies)
    batches = [batch] + [cm.FragmentBatch(c) for c in copies[1:]]
    torch.cuda.synchronize()

    ms_step, step_pct, per_kernel = time_steps(
        lambda i: cm.render_deliveries(batches[i % n_copies], w.routing_layer, w.rope_base),
        args.steps, args.warmup)
    print("[bench] whole path timed", file=sys.stderr, flush=True)

    # steps 2-5 on the ingested set (ids already computed at Ingest, Alg. 2)
    sets = []
    for c in copies:
        sets.append(cm.LatentFragmentSet())
        sets[-1].ingest_many(c)
    S = sets[0]
    ms_render_set, set_pct, set_kernels = time_steps(
        lambda i: sets[i % n_copies].render(w.routing_layer, w.rope_base), args.steps, 2)

    # the paper's baselines over the same render: the naive multiset re-render
    # (§5.9, every delivery its own operand) and BagMerge in delivery order (§4.2)
    def timed(fn):
        for i in range(2):
            r = fn(batches[i % n_copies])
            del r
        torch.cuda.synchronize()
        ta = time.perf_counter()
        for i in range(args.steps):
            r = fn(batches[i % n_copies])
            T = r.T_out
            del r
        torch.cuda.synchronize()
        return (time.perf_counter() - ta) / args.steps * 1e3, T

    multiset_bytes = 2 * delivered_bytes(w)
    ms_naive, T_naive = timed(lambda b: cm.render_multiset(b, w.routing_layer, w.rope_base))
    order = list(range(batch.n))
    ms_bag, T_bag = timed(lambda b: cm.bag_merge(b, order, w.rope_base))
    baselines = {
        "naive_multiset": {"ms": round(ms_naive, 4), "T_out": T_naive,
                           "GBps": round(multiset_bytes / (ms_naive / 1e3) / 1e9, 1),
                           "what": "steps 1-5 without dedupe: hash, score, multiset order, render "
                                   "of every delivery (fused)"},
        "bag_merge_default": {"ms": round(ms_bag, 4), "T_out": T_bag,
                              "GBps": round(multiset_bytes / (ms_bag / 1e3) / 1e9, 1),
                              "pct_hbm_peak": round(100 * multiset_bytes / (ms_bag / 1e3) / 1e9
                                                    / HBM_PEAK_GBPS, 2),
                              "what": "render of every delivery in delivery order (plan on the host)"},
    }

    # incremental render: a set missing one fragment X of middle rank is
    # rendered into a buffer with room for all; ingesting X then re-renders only
    # the slots from X's rank on (timed), and is compared with the full render
    full = S.render(w.routing_layer, w.rope_base)
    torch.cuda.synchronize()
    distinct = list(S._items.values())
    mid = full.order[len(full.order) // 2]
    x_cache = distinct[mid]
    S_without = cm.LatentFragmentSet()
    S_without.ingest_many([c for k, c in enumerate(distinct) if k != mid])
    S_with = S_without.merge(cm.LatentFragmentSet())
    S_with.ingest(x_cache)
    mc = cm.MergedCache(S_without, w.routing_layer, w.rope_base, capacity=full.T_out)
    mc.update()
    incr_ms = []
    for _ in range(args.steps):
        mc.fset = S_with
        torch.cuda.synchronize()
        ta = time.perf_counter()
        mc.update()
        torch.cuda.synchronize()
        incr_ms.append((time.perf_counter() - ta) * 1e3)
        rows, first = mc.last_rows, mc.last_first_slot
        mc.fset = S_without
        mc.update()
    mc.fset = S_with
    mc.update()
    torch.cuda.synchronize()
    incr_equal = all(torch.equal(a, b) and torch.equal(c, e)
                     for (a, c), (b, e) in zip(mc.cache, full.cache))
    token_bytes = 2 * w.L * w.H * w.d * (2 if w.dtype == "bfloat16" else 4)
    incr_bytes = 2 * rows * token_bytes
    ms_incr = sorted(incr_ms)[len(incr_ms) // 2]
    del mc, full

    # paged render (§4.5): the distinct fragments on pages of 16 tokens; block
    # tables reuse every whole fragment page they can, the kernel writes the rest
    del S_with, S_without, sets[1:], batches[1:], copies[1:]
    torch.cuda.empty_cache()
    res_set = S.render(w.routing_layer, w.rope_base)
    set_plan = res_set.plan.copy()
    del res_set
    torch.cuda.empty_cache()
    B = 16
    pool, lengths, page_lists, free = synth.make_paged(distinct, B, spare_pages=2 * (
        (w.merged_tokens + B - 1) // B + len(distinct)), seed=args.seed)
    pset = cm.PagedSet(pool, lengths, page_lists)
    for _ in range(2):
        pr = cm.render_paged(pset, set_plan, free, w.rope_base)
    torch.cuda.synchronize()
    cm.timing_reset()
    cm.timing_enable(True)
    tp = time.perf_counter()
    for _ in range(args.steps):
        pr = cm.render_paged(pset, set_plan, free, w.rope_base)
    torch.cuda.synchronize()
    ms_paged = (time.perf_counter() - tp) / args.steps * 1e3
    cm.timing_enable(False)
    k_ms, k_n = cm.timing_query("paged")
    cm.timing_reset()
    # steps 1-5 on the pool alone: scores, the colliding deliveries' Ids and the
    # order on the device, the plan to the host, block tables, then the render of
    # the merged rows no fragment page holds with the other Ids from the same
    # loads (fused, cm_paged_render_hash); and, beside it, the earlier two-kernel
    # form: the paged render with the other Ids hashed beside it on a second
    # stream (every fragment byte read twice)
    def paged_set_steps(fused):
        for _ in range(2):
            ps = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free, fused=fused)
        torch.cuda.synchronize()
        cm.timing_reset()
        cm.timing_enable(True)
        tp = time.perf_counter()
        for _ in range(args.steps):
            ps = cm.render_paged_set(pset, w.routing_layer, w.rope_base, free, fused=fused)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - tp) / args.steps * 1e3
        cm.timing_enable(False)
        kernels = {}
        for k in cm.KERNELS:
            kms, kn = cm.timing_query(k)
            if kn:
                kernels[k] = round(kms / args.steps, 4)
        cm.timing_reset()
        return ms, kernels, ps

    ms_paged_set, paged_set_kernels, ps = paged_set_steps(True)
    paged_set_equal = bool(np.array_equal(ps.plan, set_plan))
    fused_ids = ps.digests_dev.cpu().numpy()
    del ps
    ms_paged_two, paged_two_kernels, ps = paged_set_steps(False)
    paged_two_equal = bool(np.array_equal(ps.plan, set_plan)) and bool(
        np.array_equal(ps.digests_dev.cpu().numpy(), fused_ids))
    del ps
    page_bytes = w.L * w.H * B * w.d * (2 if w.dtype == "bfloat16" else 4)
    paged_bytes = 2 * len(pr.fresh) * page_bytes
    paged = {"ms": round(ms_paged, 4), "kernel_ms": round(k_ms / max(k_n, 1), 4),
             "block_tokens": B, "merged_blocks": len(pr.k_table), "pages_written": len(pr.fresh),
             "pages_reused": pr.reused_pages, "bytes": paged_bytes,
             "bytes_vs_dense": round(paged_bytes / w.render_bytes, 4),
             "kernel_GBps": round(paged_bytes / (k_ms / max(k_n, 1) / 1e3) / 1e9, 1),
             "what": "block tables (host) + table upload + paged render kernel per step",
             "set_steps_1_to_5": {"ms": round(ms_paged_set, 4), "kernels_ms": paged_set_kernels,
                                  "plan_equals_dense_set_plan": paged_set_equal,
                                  "what": "cm_paged_order (scores, colliding Ids, order) + plan to "
                                          "host + block tables + cm_paged_render_hash (render and "
                                          "the other Ids from one read), fragments only in the "
                                          "pool"},
             "set_steps_1_to_5_two_kernels": {
                 "ms": round(ms_paged_two, 4), "kernels_ms": paged_two_kernels,
                 "plan_and_ids_equal_fused": paged_two_equal,
                 "what": "as set_steps_1_to_5 with cm_paged_render and cm_paged_hash_select on "
                         "a second stream in place of the fused kernel"}}
    del pool, pset, pr
    torch.cuda.empty_cache()

    render_bytes = w.render_bytes
    value = render_bytes / (ms_step / 1e3) / 1e9

    # dominant kernel of the step and its roofline
    dom = max(per_kernel, key=lambda k: per_kernel[k]["total_ms"])
    delivered = w.delivery_bytes
    rooflines = {}
    if "render_hash" in per_kernel:
        r = cm.render_deliveries(batch, w.routing_layer, w.rope_base)
        keys = torch.empty(batch.n, dtype=torch.float64, device=dev)
        mask = torch.empty(batch.n, dtype=torch.uint8, device=dev)
        ws = torch.empty(cm.workspace_size(batch), dtype=torch.uint8, device=dev)
        cm.fragment_knorm(batch, w.routing_layer, r.tail_len, keys, ws)
        cm.equal_key_mask(batch, keys, mask)
        ops, hashed_bytes, rotated = fused_work(w, r, mask.cpu().numpy())
        del r, ws
        pk = per_kernel["render_hash"]
        avg = pk["total_ms"] / pk["launches"] / 1e3
        ach = ops / avg / 1e12
        rooflines["render_hash"] = {
            "bound": "alu", "achieved": round(ach, 3), "peak": round(VALU_PEAK_TOPS, 3),
            "unit": "Tops/s", "frac": round(ach / VALU_PEAK_TOPS, 4),
            "traffic": _traffic("render_hash", w.name),
            "ops_per_launch": ops, "hashed_bytes": hashed_bytes, "rotated_elements": rotated,
            "avg_ms": round(avg * 1e3, 4), "hbm_GBps": round(render_bytes / avg / 1e9, 1)}
        # the fused paged kernel does the same work (same plan, same deliveries
        # hashed, same elements rotated) on the pool
        pms = paged.get("set_steps_1_to_5", {}).get("kernels_ms", {}).get("paged_hash_render")
        if pms:
            achp = ops / (pms / 1e3) / 1e12
            paged["set_steps_1_to_5"]["roofline"] = {
                "kernel": "paged_hash_render", "bound": "alu", "achieved": round(achp, 3),
                "peak": round(VALU_PEAK_TOPS, 3), "unit": "Tops/s",
                "frac": round(achp / VALU_PEAK_TOPS, 4), "ops_per_launch": ops, "avg_ms": pms}
    if "render" in set_kernels:
        pk = set_kernels["render"]
        avg = pk["total_ms"] / pk["launches"] / 1e3
        ach = render_bytes / avg / 1e9
        rooflines["render"] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                               "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                               "traffic": _traffic("render", w.name),
                               "bytes_per_launch": render_bytes, "avg_ms": round(avg * 1e3, 4)}
    out = {
        "metric": "merged-cache render GB/s (read+write) and % of MI355X HBM peak; merges/s",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_ms_p10_p50_p90": step_pct,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic of the path: BLAKE3 in 32-bit integers, scores and the
        # rotation in fp64; the cache elements it moves are element_dtype
        "dtype": "u32+f64",
        "element_dtype": "bf16" if w.dtype == "bfloat16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "deliveries": w.n_deliveries, "distinct": w.n_distinct,
                   "merged_tokens": w.merged_tokens, "layers": w.L, "kv_heads": w.H,
                   "head_dim": w.d, "routing_layer": w.routing_layer, "rope_base": w.rope_base,
                   "render_bytes": render_bytes, "delivery_bytes": delivered,
                   "input_copies": n_copies, "parallelism": "single GPU"},
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "merges_per_s": round(1e3 / ms_step, 3),
        # the dominant kernel; where that is not one of the two render kernels (a set
        # whose deliveries are mostly re-deliveries hashes most bytes before the
        # order), the fused kernel's figure
        "roofline": (dict(rooflines[dom], kernel=dom) if dom in rooflines else
                     dict(rooflines["render_hash"], kernel="render_hash",
                          dominant_kernel=dom) if "render_hash" in rooflines else None),
        "roofline_render": rooflines.get("render"),
        "kernels_ms_per_step": {k: round(v["total_ms"] / args.steps, 4) for k, v in per_kernel.items()},
        "render_set": {"ms": round(ms_render_set, 4), "ms_p10_p50_p90": set_pct,
                       "GBps": round(render_bytes / (ms_render_set / 1e3) / 1e9, 1),
                       "pct_hbm_peak": round(100 * render_bytes / (ms_render_set / 1e3) / 1e9
                                             / HBM_PEAK_GBPS, 2),
                       "merges_per_s": round(1e3 / ms_render_set, 3),
                       "kernels_ms": {k: round(v["total_ms"] / args.steps, 4)
                                      for k, v in set_kernels.items()}},
        "baselines": baselines,
        "paged": paged,
        "incremental": {"ms": round(ms_incr, 4), "first_slot": first, "slots": len(distinct),
                        "rows_rendered": rows, "T_out": w.merged_tokens,
                        "bytes": incr_bytes, "GBps": round(incr_bytes / (ms_incr / 1e3) / 1e9, 1),
                        "equals_full_render": incr_equal,
                        "what": "ingest one fragment of middle rank into a rendered set: knorm, "
                                "order, plan copy, render of the slots from its rank (median of "
                                "the timed steps)"},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, frags)
    if not args.no_other_workloads:
        del frags, deliveries, batch, batches, copies, sets, S, distinct
        torch.cuda.empty_cache()
        out["workloads"] = {}
        for name in OTHER_WORKLOADS:
            if name == w.name:
                continue
            print(f"[bench] workload {name}", file=sys.stderr, flush=True)
            # many short steps: a step of tens of microseconds needs hundreds for a
            # mean that the first step's host latency does not move
            out["workloads"][name] = other_workload(name, args.seed, max(args.steps, 200),
                                                    args.warmup, dev)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
