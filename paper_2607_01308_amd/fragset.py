"""LatentFragmentSet (Alg. 2) and the render path on one GPU.

render_deliveries runs the whole path over a list of deliveries: scores
(cm_fragment_knorm), the Id of every delivery whose score collides
with another's (cm_equal_key_mask + cm_fragment_hash_select: only those decide
dedupe and ties), dedupe + canonical order + offsets (cm_canonical_order), then
the rotate-and-concatenate render fused with the Ids of every other delivery
(cm_render_merge_hash), so each byte is read once. By default one library call
(cm_render_deliveries) enqueues all of it with the plan kept on the device and
the output sized for the sum of the delivery lengths; pipeline="overlap" and
pipeline="serial" bring the plan to the host before the render, which runs
beside (overlap: cm_render_merge next to the remaining Ids on a second stream)
or after (serial) the remaining Ids. LatentFragmentSet keeps the state of
Alg. 2 (a set keyed by Id) and renders it with the ids computed at Ingest.

Every call enqueues its work on one stream (the `stream` argument, else the
current stream) and allocates its buffers there. Scratch memory is cached per
(device, stream), so calls on different streams never share it."""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Union

import numpy as np
import torch

from . import _cabi as C
from .binding import (FragmentBatch, bag_plan, canonical_order, equal_key_mask, fragment_hash,
                      fragment_hash_select, fragment_knorm, multiset_order, plan_elems,
                      paged_render, paged_tables, paged_workspace_size, render_merge,
                      render_deliveries_async, render_merge_devplan, render_merge_hash,
                      render_merge_range, render_set, workspace_size, paged_order,
                      paged_hash_select, paged_render_hash, paged_deliveries,
                      render_deliveries_graph, graph_launch, graph_destroy)
from .binding import PagedSet

_WS: Dict[tuple, torch.Tensor] = {}
_SIDE: Dict[torch.device, torch.cuda.Stream] = {}


def _workspace(batch: FragmentBatch, stream: torch.cuda.Stream) -> torch.Tensor:
    """Scratch for the calls enqueued on `stream`, cached per (device, stream) and
    allocated on that stream, so that work on one stream never races with work on
    another over it, and a buffer replaced by a larger one is only reused by
    work ordered after what was enqueued with it."""
    need = max(workspace_size(batch), 256)
    key = (batch.device, stream.cuda_stream)
    ws = _WS.get(key)
    if ws is None or ws.numel() < need:
        with torch.cuda.stream(stream):
            ws = torch.empty(need, dtype=torch.uint8, device=batch.device)
        _WS[key] = ws
    return ws


def _main_stream(device: torch.device, stream) -> torch.cuda.Stream:
    return stream if stream is not None else torch.cuda.current_stream(device)


def _side_stream(device: torch.device) -> torch.cuda.Stream:
    st = _SIDE.get(device)
    if st is None:
        st = torch.cuda.Stream(device=device)  # default priority
        _SIDE[device] = st
    return st


_PINNED: Dict[tuple, torch.Tensor] = {}


def release_workspace() -> None:
    _WS.clear()
    _PINNED.clear()


def _plan_to_host(plan_dev: torch.Tensor, stream) -> np.ndarray:
    """Host copy of a plan through a cached pinned buffer (an asynchronous copy
    on the stream, then a wait for that stream only)."""
    key = (plan_dev.device, plan_dev.numel())
    buf = _PINNED.get(key)
    if buf is None:
        buf = torch.empty(plan_dev.numel(), dtype=torch.int64, pin_memory=True)
        _PINNED[key] = buf
    st = stream if stream is not None else torch.cuda.current_stream(plan_dev.device)
    with torch.cuda.stream(st):
        buf.copy_(plan_dev, non_blocking=True)
    st.synchronize()
    return buf.numpy().copy()


class RenderResult:
    """Result of a render: the merged cache (per layer (K, V), each [1, H, T_out, d],
    views of one [L, 2, 1, H, T_out, d] buffer), per-delivery digests and keys,
    and the plan (layout in include/cmerge.h).

    A result of the fused pipeline is returned before the device has finished:
    its plan travels to pinned host memory behind an event, and the first use of
    the plan, T_out, `merged` or `cache` waits for it. A render whose plan was
    checked on the device (LatentFragmentSet.render) brings the plan to the host
    on the first use of `merged` or `cache`. Either way a plan whose status is an
    error raises then, so a cache that was not rendered is never handed out."""

    def __init__(self, cache=None, merged=None, digests_dev=None, keys_dev=None,
                 plan_host: Optional[np.ndarray] = None, tail_len: int = 0,
                 plan_dev: Optional[torch.Tensor] = None, pending=None):
        self._cache = cache
        self._merged = merged
        self.digests_dev = digests_dev      # [n, 32] uint8, per delivery
        self.keys_dev = keys_dev            # [n] float64 S_i, per delivery
        self.plan_host = plan_host          # host copy of the plan
        self.tail_len = tail_len
        self.plan_dev = plan_dev
        self._pending = pending             # (event, pinned plan copy, output buffer, shape, where)

    @property
    def plan(self) -> np.ndarray:
        """The plan on the host (copied from the device on first use when the
        render did not need it; a rejected plan raises)."""
        if self.plan_host is None:
            if self._pending is not None:
                event, pinned, _, _, where = self._pending
                event.synchronize()
                plan = pinned.numpy().copy()
                _check_plan(plan, where)
            else:
                plan = self.plan_dev.to("cpu").numpy()
                status = int(plan[C.PLAN_STATUS])
                if status == C.CM_ENONFINITE:
                    raise C.CmError(status, "cm_canonical_order",
                                    "a score is NaN or infinite; nothing was rendered")
                if status != C.CM_OK:
                    raise C.CmError(status, "cm_render_merge_devplan",
                                    "the plan failed its device check")
            self.plan_host = plan
        return self.plan_host

    @property
    def merged(self) -> torch.Tensor:
        if self._merged is None:
            _, _, out, (L, H, d), _ = self._pending
            T_out = self.T_out
            self._merged = out[:L * 2 * H * T_out * d].view(L, 2, 1, H, T_out, d)
        elif self.plan_host is None:
            self.plan          # a plan checked on the device: raises if it was rejected
        return self._merged

    @property
    def cache(self) -> tuple:
        if self._cache is None:
            m = self.merged
            self._cache = tuple((m[l, 0], m[l, 1]) for l in range(m.shape[0]))
        elif self.plan_host is None:
            self.plan
        return self._cache

    @property
    def n_unique(self) -> int:
        return int(self.plan[C.PLAN_NUNIQUE])

    @property
    def T_out(self) -> int:
        return int(self.plan[C.PLAN_TOUT])

    @property
    def order(self) -> List[int]:
        n = int(self.plan[C.PLAN_N])
        return [int(x) for x in self.plan[C.PLAN_HEADER:C.PLAN_HEADER + self.n_unique]][:n]

    @property
    def offsets(self) -> List[int]:
        n = int(self.plan[C.PLAN_N])
        b = C.PLAN_HEADER + n
        return [int(x) for x in self.plan[b:b + self.n_unique]]

    @property
    def lengths(self) -> List[int]:
        n = int(self.plan[C.PLAN_N])
        b = C.PLAN_HEADER + 2 * n
        return [int(x) for x in self.plan[b:b + self.n_unique]]

    @property
    def slot_of_delivery(self) -> List[int]:
        n = int(self.plan[C.PLAN_N])
        b = C.PLAN_HEADER + 3 * n
        return [int(x) for x in self.plan[b:b + n]]

    def compact(self) -> "RenderResult":
        """Move the merged cache into a buffer of exactly T_out rows and release
        the larger one. A fused result's output buffer holds the sum of all
        delivery lengths (the bound the device has before the dedupe), so with
        many re-deliveries most of it is unused; this costs one copy of the
        merged cache on the current stream. Other results are already exact."""
        if self._pending is not None:
            merged = self.merged.clone()
            self._merged, self._cache, self._pending = merged, None, None
        return self

    def _wait(self) -> None:
        """Host wait for the work of a fused result (the copies below run on the
        current stream, which need not be the one the result was computed on)."""
        if self._pending is not None:
            self._pending[0].synchronize()

    @property
    def digests(self) -> List[bytes]:
        self._wait()
        return [bytes(r) for r in self.digests_dev.cpu().numpy()]

    @property
    def keys(self) -> np.ndarray:
        self._wait()
        return self.keys_dev.cpu().numpy()


def _check_plan(plan_host: np.ndarray, where: str) -> None:
    status = int(plan_host[C.PLAN_STATUS])
    if status != C.CM_OK:
        raise C.CmError(status, where, "plan status is not CM_OK "
                        "(a score is NaN or infinite)" if status == C.CM_ENONFINITE else "")


def _render_plan(batch: FragmentBatch, plan_dev: torch.Tensor, plan_host: np.ndarray,
                 rope_base: float, style: str, ws: torch.Tensor, stream, hash_select=None,
                 digests=None):
    _check_plan(plan_host, "cm_canonical_order")
    T_out = int(plan_host[C.PLAN_TOUT])
    merged = torch.empty((batch.L, 2, 1, batch.H, T_out, batch.d), dtype=batch.torch_dtype,
                         device=batch.device)
    if hash_select is None:
        render_merge(batch, plan_dev, plan_host, rope_base, style, merged, T_out, ws, stream)
    else:
        render_merge_hash(batch, plan_dev, plan_host, rope_base, style, hash_select, digests,
                          merged, T_out, ws, stream)
    return merged


PIPELINES = ("fused", "overlap", "serial")


def render_deliveries(deliveries: Union[FragmentBatch, Sequence], routing_layer: int,
                      rope_base: float, style: str = "half", stream=None,
                      pipeline: str = "fused") -> RenderResult:
    """The whole path over a list of deliveries (duplicates allowed).

    fused (default): one library call enqueues every step (scores, the Ids of
    deliveries whose keys collide, dedupe and order, then the render fused with
    the remaining Ids), the plan staying on the device; the output is allocated
    for the sum of the delivery lengths and the call returns without waiting (the
    result waits for the plan on first use; a non-finite score raises then).
    overlap / serial: the plan comes to the host before the render, which then
    runs beside (overlap) or after (serial) the remaining Ids, and the output is
    exactly the merged cache: the choice when re-deliveries make the sum of the
    delivery lengths much larger than the merged cache."""
    if pipeline not in PIPELINES:
        raise ValueError(f"pipeline must be one of {PIPELINES}")
    batch = deliveries if isinstance(deliveries, FragmentBatch) else FragmentBatch(deliveries)
    dev = batch.device
    main = _main_stream(dev, stream)
    with torch.cuda.stream(main):
        ws = _workspace(batch, main)
        digests = torch.empty((batch.n, 32), dtype=torch.uint8, device=dev)
        keys = torch.empty(batch.n, dtype=torch.float64, device=dev)
        mask = torch.empty(batch.n, dtype=torch.uint8, device=dev)
        plan_dev = torch.empty(plan_elems(batch.n), dtype=torch.int64, device=dev)
        tail = min(batch.lengths)
        if pipeline == "fused":
            T_cap = int(sum(batch.lengths))
            out = torch.empty(batch.L * 2 * batch.H * T_cap * batch.d, dtype=batch.torch_dtype,
                              device=dev)
            render_deliveries_async(batch, routing_layer, tail, rope_base, style, keys, mask,
                                    digests, plan_dev, out, T_cap, ws, main)
            # the plan follows the render to pinned host memory; nothing waits for it here
            pinned = torch.empty(plan_dev.numel(), dtype=torch.int64, pin_memory=True)
            pinned.copy_(plan_dev, non_blocking=True)
            done = torch.cuda.Event()
            done.record(main)
            return RenderResult(digests_dev=digests, keys_dev=keys, tail_len=tail,
                                plan_dev=plan_dev,
                                pending=(done, pinned, out, (batch.L, batch.H, batch.d),
                                         "cm_render_deliveries"))
        fragment_knorm(batch, routing_layer, tail, keys, ws, main)
        equal_key_mask(batch, keys, mask, main)
        fragment_hash_select(batch, mask, 1, digests, ws, main)   # the digests the order reads
        side_done = None
        if pipeline == "overlap":
            ready = torch.cuda.Event()
            ready.record(main)
            side = _side_stream(dev)
            side.wait_event(ready)
            fragment_hash_select(batch, mask, 0, digests, _workspace(batch, side), side)
            side_done = torch.cuda.Event()
            side_done.record(side)
        else:
            fragment_hash_select(batch, mask, 0, digests, ws, main)
        canonical_order(batch, keys, digests, plan_dev, main)
        plan_host = _plan_to_host(plan_dev, main)
        try:
            merged = _render_plan(batch, plan_dev, plan_host, rope_base, style, ws, main)
        finally:
            if side_done is not None:
                main.wait_event(side_done)
    return RenderResult(merged=merged, digests_dev=digests, keys_dev=keys,
                        plan_host=plan_host, tail_len=tail, plan_dev=plan_dev)


def render_multiset(deliveries: Union[FragmentBatch, Sequence], routing_layer: int,
                    rope_base: float, style: str = "half", stream=None) -> RenderResult:
    """The naive re-render of §5.9: every delivery is its own operand (no
    Ingest dedupe), in canonical order; copies sit next to each other, so R
    deliveries of each fragment give a cache R times as long (Table 10's
    foil). Digests as in render_deliveries (fused into the render)."""
    batch = deliveries if isinstance(deliveries, FragmentBatch) else FragmentBatch(deliveries)
    dev = batch.device
    main = _main_stream(dev, stream)
    with torch.cuda.stream(main):
        ws = _workspace(batch, main)
        digests = torch.empty((batch.n, 32), dtype=torch.uint8, device=dev)
        keys = torch.empty(batch.n, dtype=torch.float64, device=dev)
        mask = torch.empty(batch.n, dtype=torch.uint8, device=dev)
        plan_dev = torch.empty(plan_elems(batch.n), dtype=torch.int64, device=dev)
        tail = min(batch.lengths)
        fragment_knorm(batch, routing_layer, tail, keys, ws, main)
        equal_key_mask(batch, keys, mask, main)
        fragment_hash_select(batch, mask, 1, digests, ws, main)   # the digests the order reads
        multiset_order(batch, keys, digests, plan_dev, main)
        plan_host = _plan_to_host(plan_dev, main)
        merged = _render_plan(batch, plan_dev, plan_host, rope_base, style, ws, main,
                                     hash_select=mask, digests=digests)
    return RenderResult(merged=merged, digests_dev=digests, keys_dev=keys,
                        plan_host=plan_host, tail_len=tail, plan_dev=plan_dev)


def bag_merge(deliveries: Union[FragmentBatch, Sequence], order: Sequence[int],
              rope_base: float, style: str = "half", stream=None) -> RenderResult:
    """BagMerge (Eq. (1)-(2)) with a caller-supplied order, e.g. the paper's
    default (delivery order) and swap baselines: slot k renders delivery
    order[k]; no scores, no Ids, no dedupe (digests and keys stay empty)."""
    batch = deliveries if isinstance(deliveries, FragmentBatch) else FragmentBatch(deliveries)
    dev = batch.device
    main = _main_stream(dev, stream)
    plan_host = bag_plan(batch, order)
    with torch.cuda.stream(main):
        ws = _workspace(batch, main)
        plan_dev = torch.from_numpy(plan_host).to(dev, non_blocking=False)
        merged = _render_plan(batch, plan_dev, plan_host, rope_base, style, ws, main)
    empty = torch.empty(0, dtype=torch.uint8, device=dev)
    return RenderResult(merged=merged, digests_dev=empty,
                        keys_dev=torch.empty(0, dtype=torch.float64, device=dev),
                        plan_host=plan_host, tail_len=0, plan_dev=plan_dev)


def fragment_ids(caches: Sequence, stream=None) -> List[bytes]:
    """Id of Alg. 2 for each cache (one batched launch)."""
    batch = FragmentBatch(caches)
    main = _main_stream(batch.device, stream)
    with torch.cuda.stream(main):
        ws = _workspace(batch, main)
        digests = torch.empty((batch.n, 32), dtype=torch.uint8, device=batch.device)
        fragment_hash(batch, digests, ws, main)
        host = digests.cpu().numpy()       # a copy on `main`, ordered after the hash
    return [bytes(r) for r in host]


class LatentFragmentSet:
    """State of Alg. 2: fragments keyed by their content address. Ingest and
    Merge are set union (a byte-identical re-delivery is absorbed); Render is
    CanonicalMerge over the set, a pure function of the set."""

    def __init__(self, items: Optional[Dict[bytes, tuple]] = None):
        self._items: Dict[bytes, tuple] = dict(items or {})
        self._desc = None          # (FragmentBatch, device Id array) of the current members

    def ingest(self, cache) -> bytes:
        return self.ingest_many([cache])[0]

    def ingest_many(self, caches: Sequence) -> List[bytes]:
        ids = fragment_ids(caches)
        for fid, cache in zip(ids, caches):
            if fid not in self._items:
                self._items[fid] = cache
                self._desc = None
        return ids

    def _description(self):
        """The members as the C ABI sees them: fragment table and their Ids on the
        device; rebuilt only when the membership changes."""
        if self._desc is None:
            ids = list(self._items.keys())
            batch = FragmentBatch([self._items[k] for k in ids])
            digests = torch.tensor(np.frombuffer(b"".join(ids), dtype=np.uint8).reshape(-1, 32),
                                   device=batch.device)
            self._desc = (batch, digests)
        return self._desc

    def merge(self, other: "LatentFragmentSet") -> "LatentFragmentSet":
        out = dict(self._items)
        for k, v in other._items.items():
            out.setdefault(k, v)
        return LatentFragmentSet(out)

    def ids(self) -> frozenset:
        return frozenset(self._items)

    def __len__(self) -> int:
        return len(self._items)

    def render(self, routing_layer: int, rope_base: float, style: str = "half",
               stream=None) -> RenderResult:
        if not self._items:
            raise ValueError("cannot render an empty set")
        batch, digests = self._description()
        dev = batch.device
        main = _main_stream(dev, stream)
        with torch.cuda.stream(main):
            ws = _workspace(batch, main)
            digests.record_stream(main)      # the set may drop this array while main still reads it
            keys = torch.empty(batch.n, dtype=torch.float64, device=dev)
            plan_dev = torch.empty(plan_elems(batch.n), dtype=torch.int64, device=dev)
            tail = min(batch.lengths)
            # the members are distinct, so T_out is the sum of their lengths and the
            # plan stays on the device: scores, order and render in one call
            T_out = int(sum(batch.lengths))
            merged = torch.empty((batch.L, 2, 1, batch.H, T_out, batch.d),
                                 dtype=batch.torch_dtype, device=dev)
            render_set(batch, digests, routing_layer, tail, rope_base, style, keys, plan_dev,
                       merged, T_out, ws, main)
        # the per-layer views are made on first use of `cache` (tens of microseconds
        # of host time for a deep model, which would otherwise pace a render loop)
        return RenderResult(merged=merged, digests_dev=digests, keys_dev=keys, plan_host=None,
                            tail_len=tail, plan_dev=plan_dev)


class MergedCache:
    """The render of a LatentFragmentSet kept up to date as the set grows
    (Render of Alg. 2 without re-rendering every fragment each time).

    The merged cache lives in one buffer [L][2][1][H][T_cap][d]; `cache` are
    the [1, H, T_out, d] views of its first T_out rows. update() computes the
    set's plan and re-renders only the slots from the first one whose fragment
    differs from the previous render: inserting a fragment at rank r leaves the
    slots before r with the same fragments and offsets, hence the same bytes,
    so the result equals the full render of the set bit for bit. When T_out
    outgrows T_cap the buffer grows by `growth` and everything is rendered."""

    def __init__(self, fset: LatentFragmentSet, routing_layer: int, rope_base: float,
                 style: str = "half", capacity: int = 0, growth: float = 1.5):
        self.fset = fset
        self.routing_layer, self.rope_base, self.style = routing_layer, rope_base, style
        self.capacity, self.growth = int(capacity), float(growth)
        self.buffer: Optional[torch.Tensor] = None
        self.slot_ids: List[bytes] = []
        self.T_out = 0
        self.last_first_slot = 0        # first slot rendered by the last update
        self.last_rows = 0              # rows per row block rendered by the last update

    @property
    def T_cap(self) -> int:
        return 0 if self.buffer is None else int(self.buffer.shape[4])

    @property
    def cache(self) -> tuple:
        b = self.buffer
        return tuple((b[l, 0, :, :, :self.T_out], b[l, 1, :, :, :self.T_out])
                     for l in range(b.shape[0]))

    def update(self, stream=None) -> tuple:
        batch, digests = self.fset._description()
        ids = list(self.fset._items.keys())
        dev = batch.device
        main = _main_stream(dev, stream)
        with torch.cuda.stream(main):
            ws = _workspace(batch, main)
            digests.record_stream(main)
            keys = torch.empty(batch.n, dtype=torch.float64, device=dev)
            plan_dev = torch.empty(plan_elems(batch.n), dtype=torch.int64, device=dev)
            fragment_knorm(batch, self.routing_layer, min(batch.lengths), keys, ws, main)
            canonical_order(batch, keys, digests, plan_dev, main)
            plan = _plan_to_host(plan_dev, main)
        _check_plan(plan, "cm_canonical_order")     # before the plan is used or the buffer grows
        n, n_u, T_out = int(plan[C.PLAN_N]), int(plan[C.PLAN_NUNIQUE]), int(plan[C.PLAN_TOUT])
        slot_ids = [ids[int(plan[C.PLAN_HEADER + s])] for s in range(n_u)]
        if self.buffer is None or T_out > self.T_cap:
            T_cap = max(T_out, self.capacity, int(self.T_cap * self.growth))
            with torch.cuda.stream(main):
                self.buffer = torch.empty((batch.L, 2, 1, batch.H, T_cap, batch.d),
                                          dtype=batch.torch_dtype, device=dev)
            first = 0
        else:
            first = 0
            while first < min(n_u, len(self.slot_ids)) and slot_ids[first] == self.slot_ids[first]:
                first += 1
        if first < n_u:
            self.buffer.record_stream(main)
            render_merge_range(batch, plan_dev, plan, self.rope_base, self.style, first,
                               self.buffer, self.T_cap, ws, main)
        self.last_first_slot = first
        self.last_rows = T_out - (int(plan[C.PLAN_HEADER + n + first]) if first < n_u else T_out)
        self.slot_ids, self.T_out = slot_ids, T_out
        return self.cache


class RenderGraph:
    """Steps 1-5 of one batch of deliveries captured into a HIP graph
    (cm_render_deliveries_graph) over buffers this object owns: replay()
    enqueues every kernel of the whole path with one launch, for callers that
    merge sets of the same shape again and again and are bound by kernel
    launches (small sets run the path's kernels in tens of microseconds). Each
    replay reads the fragment tensors as they are then: write new contents into
    the same tensors in place to merge new data. The result of a replay is
    valid until the next replay, which writes the same buffers."""

    def __init__(self, deliveries: Union[FragmentBatch, Sequence], routing_layer: int,
                 rope_base: float, style: str = "half"):
        self.batch = (deliveries if isinstance(deliveries, FragmentBatch)
                      else FragmentBatch(deliveries))
        b = self.batch
        dev = b.device
        self.ws = torch.empty(max(workspace_size(b), 256), dtype=torch.uint8, device=dev)
        self.digests = torch.empty((b.n, 32), dtype=torch.uint8, device=dev)
        self.keys = torch.empty(b.n, dtype=torch.float64, device=dev)
        self.mask = torch.empty(b.n, dtype=torch.uint8, device=dev)
        self.plan_dev = torch.empty(plan_elems(b.n), dtype=torch.int64, device=dev)
        self.tail = min(b.lengths)
        self.T_cap = int(sum(b.lengths))
        self.out = torch.empty(b.L * 2 * b.H * self.T_cap * b.d, dtype=b.torch_dtype, device=dev)
        self._handle = None
        torch.cuda.synchronize(dev)           # the buffers exist before the graph refers to them
        self._handle = render_deliveries_graph(b, routing_layer, self.tail, rope_base, style,
                                               self.keys, self.mask, self.digests,
                                               self.plan_dev, self.out, self.T_cap, self.ws)

    def replay(self, stream=None) -> RenderResult:
        if self._handle is None:
            raise RuntimeError("the graph was closed")
        b = self.batch
        main = _main_stream(b.device, stream)
        with torch.cuda.stream(main):
            graph_launch(self._handle, b, main)
            pinned = torch.empty(self.plan_dev.numel(), dtype=torch.int64, pin_memory=True)
            pinned.copy_(self.plan_dev, non_blocking=True)
            done = torch.cuda.Event()
            done.record(main)
        return RenderResult(digests_dev=self.digests, keys_dev=self.keys, tail_len=self.tail,
                            plan_dev=self.plan_dev,
                            pending=(done, pinned, self.out, (b.L, b.H, b.d),
                                     "cm_render_deliveries_graph"))

    def close(self) -> None:
        """Free the graph (its buffers go with this object)."""
        if self._handle is not None:
            handle, self._handle = self._handle, None
            graph_destroy(handle)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PagedRender:
    """Block tables of a paged render (page id of each merged block of B rows,
    K and V; the fresh pages written, as codes 2j + kv, K first, by page id;
    T_out) and, for render_paged_set, the plan, Ids and scores it computed. A
    render enqueued with nothing waiting for the host (render_paged_set's fused
    path) fills the host fields on their first use, which waits for its copies;
    a plan it rejected (a score that is not finite, a free list too short)
    raises there."""

    def __init__(self, k_table=None, v_table=None, fresh=None, T_out=None, plan=None,
                 digests_dev=None, keys_dev=None, pending=None):
        self._k_table, self._v_table, self._fresh = k_table, v_table, fresh
        self._T_out, self._plan = T_out, plan
        self.digests_dev = digests_dev      # render_paged_set: [n, 32] Ids
        self.keys_dev = keys_dev            # render_paged_set: [n] scores S_i
        self._pending = pending             # (event, pinned copy, plan length, capacity, B,
                                            #  fragment pages)

    def _finish(self) -> None:
        if self._pending is None:
            return
        event, pinned, pe, cap, B, frag_pages = self._pending
        event.synchronize()
        buf = pinned.numpy()
        plan = buf[:pe].copy()
        if int(plan[C.PLAN_STATUS]) == C.CM_EINVAL:
            raise C.CmError(C.CM_EINVAL, "cm_paged_deliveries",
                            f"the free list is shorter than the render needs ({int(buf[pe])} "
                            "pages); nothing was rendered")
        _check_plan(plan, "cm_paged_deliveries")
        T_out = int(plan[C.PLAN_TOUT])
        nbo = (T_out + B - 1) // B
        tabs = buf[pe + 1:].view(np.int32)
        kt, vt = tabs[:nbo].copy(), tabs[cap:cap + nbo].copy()
        # every page that is not a fragment page came from the free list
        kf = np.nonzero(~np.isin(kt, frag_pages))[0]
        vf = np.nonzero(~np.isin(vt, frag_pages))[0]
        fresh = np.concatenate([2 * kf[np.argsort(kt[kf], kind="stable")],
                                2 * vf[np.argsort(vt[vf], kind="stable")] + 1]).astype(np.int32)
        self._k_table, self._v_table, self._fresh = kt, vt, fresh
        self._T_out, self._plan, self._pending = T_out, plan, None

    @property
    def k_table(self) -> np.ndarray:
        self._finish()
        return self._k_table

    @property
    def v_table(self) -> np.ndarray:
        self._finish()
        return self._v_table

    @property
    def fresh(self) -> np.ndarray:
        self._finish()
        return self._fresh

    @property
    def T_out(self) -> int:
        self._finish()
        return self._T_out

    @property
    def plan(self) -> Optional[np.ndarray]:
        self._finish()
        return self._plan

    @property
    def reused_pages(self) -> int:
        return 2 * len(self.k_table) - len(self.fresh)


def render_paged(pset: PagedSet, plan_host: np.ndarray, free_pages, rope_base: float,
                 style: str = "half", stream=None) -> PagedRender:
    """Steps 4-5 over paged storage (§4.5): block tables that reuse every
    fragment page a merged block equals (V of page-aligned slots, K only at
    offset 0), and a render of the other pages into free_pages. plan_host: a
    plan whose slots index pset's fragments (e.g. RenderResult.plan of the same
    fragments in dense form, or bag_plan)."""
    kt, vt, fresh = paged_tables(pset, plan_host, free_pages)
    dev = pset.device
    main = stream if stream is not None else torch.cuda.current_stream(dev)
    with torch.cuda.stream(main):
        ws = torch.empty(max(paged_workspace_size(pset), 256), dtype=torch.uint8, device=dev)
        plan_dev = torch.from_numpy(np.ascontiguousarray(plan_host, dtype=np.int64)).to(dev)
        kd, vd = torch.from_numpy(kt).to(dev), torch.from_numpy(vt).to(dev)
        fd = torch.from_numpy(fresh).to(dev)
        paged_render(pset, plan_dev, plan_host, rope_base, style, kd, vd, fd, ws, main)
    return PagedRender(k_table=kt, v_table=vt, fresh=fresh,
                       T_out=int(plan_host[C.PLAN_TOUT]))


def paged_fused_fits(pset: PagedSet) -> bool:
    """Whether cm_paged_render_hash takes this pool: it names a pool row of one
    (layer, K/V) slice with 32 bits, so P * H * B must not exceed 2^32 - 1."""
    return pset.P * pset.H * pset.B <= 0xFFFFFFFF


def render_paged_set(pset: PagedSet, routing_layer: int, rope_base: float, free_pages,
                     style: str = "half", stream=None, fused: Optional[bool] = None,
                     hash_workgroups_per_cu: int = 1) -> PagedRender:
    """Steps 1-5 on fragments that live only in the pool (§4.5).

    fused (the default when the pool fits its 32-bit row index): one call,
    cm_paged_deliveries, with nothing waiting for the host: scores, the Ids the
    order reads (deliveries whose key equals another's), dedupe, order and
    offsets, the merged block tables built on the device from free_pages, then
    the render of every merged row that no fragment page holds already with the
    remaining Ids (the content address of each fragment's dense form) from the
    same loads. The plan and tables reach the host on first use of the result.

    fused=False: cm_paged_order, the plan to the host, the block tables there,
    cm_paged_render, and the remaining Ids beside it on a second stream with
    hash_workgroups_per_cu chunk workgroups per CU (each byte read twice).

    No dense copy of any fragment is made; the result's digests wait for all of
    its work."""
    if fused is None:
        fused = paged_fused_fits(pset)
    dev = pset.device
    main = stream if stream is not None else torch.cuda.current_stream(dev)
    with torch.cuda.stream(main):
        need = max(paged_workspace_size(pset), 256)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        keys = torch.empty(pset.n, dtype=torch.float64, device=dev)
        mask = torch.empty(pset.n, dtype=torch.uint8, device=dev)
        digests = torch.empty((pset.n, 32), dtype=torch.uint8, device=dev)
        pe = plan_elems(pset.n)
        if fused:
            # plan, pages taken and both tables in one buffer, copied back once
            cap = (sum(pset.lengths) + pset.B - 1) // pset.B
            out = torch.empty(pe + 1 + cap, dtype=torch.int64, device=dev)
            tabs = out[pe + 1:].view(torch.int32)
            free_host = np.ascontiguousarray(np.asarray(free_pages, dtype=np.int32))
            staged = torch.empty(max(free_host.size, 1), dtype=torch.int32, pin_memory=True)
            staged[:free_host.size].copy_(torch.from_numpy(free_host))
            free_dev = staged.to(dev, non_blocking=True)
            paged_deliveries(pset, routing_layer, min(pset.lengths), rope_base, style, free_host,
                             free_dev, keys, mask, digests, out[:pe], tabs[:cap],
                             tabs[cap:2 * cap], out[pe:pe + 1], ws, main)
            pinned = torch.empty(out.numel(), dtype=torch.int64, pin_memory=True)
            pinned.copy_(out, non_blocking=True)
            done = torch.cuda.Event()
            done.record(main)
            return PagedRender(digests_dev=digests, keys_dev=keys,
                               pending=(done, pinned, pe, cap, pset.B, pset.blocks_host))
        plan_dev = torch.empty(pe, dtype=torch.int64, device=dev)
        paged_order(pset, routing_layer, min(pset.lengths), keys, mask, digests, plan_dev, ws, main)
        ready = torch.cuda.Event()
        ready.record(main)
        side = _side_stream(dev)
        side.wait_event(ready)
        with torch.cuda.stream(side):
            ws_side = torch.empty(need, dtype=torch.uint8, device=dev)
        paged_hash_select(pset, mask, 0, digests, ws_side, hash_workgroups_per_cu, side)
        for t in (mask, digests, ws_side):
            t.record_stream(side)
        side_done = torch.cuda.Event()
        side_done.record(side)
        plan_host = _plan_to_host(plan_dev, main)
        try:
            _check_plan(plan_host, "cm_paged_order")
            kt, vt, fresh = paged_tables(pset, plan_host, free_pages)
            kd, vd = torch.from_numpy(kt).to(dev), torch.from_numpy(vt).to(dev)
            fd = torch.from_numpy(fresh).to(dev)
            paged_render(pset, plan_dev, plan_host, rope_base, style, kd, vd, fd, ws, main)
        finally:
            main.wait_event(side_done)       # the digests are complete once main is
    return PagedRender(k_table=kt, v_table=vt, fresh=fresh, T_out=int(plan_host[C.PLAN_TOUT]),
                       plan=plan_host, digests_dev=digests, keys_dev=keys)
