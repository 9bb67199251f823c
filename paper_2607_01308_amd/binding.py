"""Python binding of the C ABI (include/cmerge.h), one function per entry point
with the same name. Argument marshalling only: every step runs in the HIP
kernels of libcmerge.so; torch provides device memory and streams."""

from __future__ import annotations

import ctypes
from typing import Sequence

import numpy as np
import torch

from . import _cabi as C

_DTYPES = {torch.bfloat16: C.CM_BF16, torch.float32: C.CM_F32}
_STYLES = {"half": C.CM_ROPE_HALF, "interleaved": C.CM_ROPE_INTERLEAVED}


def _ptr(t: torch.Tensor) -> ctypes.c_void_p:
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, owner) -> ctypes.c_void_p:
    """The stream a call enqueues on (the current one if None). The owner's device
    tables are marked as in use on it: the library's kernels read them after the
    call returns, so the caching allocator must not hand their memory to another
    tensor before the work enqueued there has finished, whichever stream they were
    allocated on."""
    s = stream if stream is not None else torch.cuda.current_stream(owner.device)
    for t in owner.device_tables:
        t.record_stream(s)
    return ctypes.c_void_p(s.cuda_stream)


class FragmentBatch:
    """A list of fragments (legacy KV caches on one GPU) described for the C ABI:
    host and device copies of the table {T_i, addr(K_i^0), addr(V_i^0), ...}.
    Holds references to the tensors so their addresses stay valid."""

    def __init__(self, caches: Sequence, device=None):
        if len(caches) == 0:
            raise ValueError("a fragment set needs at least one fragment")
        first_k = caches[0][0][0]
        self.L = len(caches[0])
        _, self.H, _, self.d = first_k.shape
        self.torch_dtype = first_k.dtype
        if self.torch_dtype not in _DTYPES:
            raise TypeError(f"unsupported dtype {self.torch_dtype} (bfloat16 or float32)")
        self.device = torch.device(device) if device is not None else first_k.device
        if self.device.type != "cuda":
            raise ValueError("fragments must live on a GPU")
        rows = []
        for i, cache in enumerate(caches):
            if len(cache) != self.L:
                raise ValueError(f"fragment {i} has {len(cache)} layers, expected {self.L}")
            T = cache[0][0].shape[2]
            row = [T]
            for l, (K, V) in enumerate(cache):
                for x in (K, V):
                    if (x.dim() != 4 or x.shape[0] != 1 or x.shape[1] != self.H or x.shape[2] != T
                            or x.shape[3] != self.d):
                        raise ValueError(f"fragment {i} layer {l}: shape {tuple(x.shape)} is not "
                                         f"[1, {self.H}, {T}, {self.d}]")
                    if x.dtype != self.torch_dtype or x.device != self.device:
                        raise ValueError(f"fragment {i} layer {l}: dtype/device differ from the set")
                    if not x.is_contiguous():
                        raise ValueError(f"fragment {i} layer {l}: tensor is not contiguous")
                    row.append(x.data_ptr())
            rows.append(row)
        self.caches = list(caches)
        self.table_host = np.ascontiguousarray(np.array(rows, dtype=np.int64))
        self.table_dev = torch.from_numpy(self.table_host).to(self.device)
        self.device_tables = (self.table_dev,)
        self.lengths = [int(r[0]) for r in rows]
        self.struct = C.CmFragset(
            n=len(caches), L=self.L, H=self.H, d=self.d, dtype=_DTYPES[self.torch_dtype],
            reserved=0, table_host=self.table_host.ctypes.data, table_dev=self.table_dev.data_ptr())

    @property
    def n(self) -> int:
        return len(self.caches)

    @property
    def elem_bytes(self) -> int:
        return 2 if self.torch_dtype == torch.bfloat16 else 4

    def fragment_bytes(self, i: int) -> int:
        return 2 * self.L * self.H * self.lengths[i] * self.d * self.elem_bytes


def workspace_size(batch: FragmentBatch) -> int:
    out = ctypes.c_size_t(0)
    C.check(C.lib().cm_workspace_size(ctypes.byref(batch.struct), ctypes.byref(out)),
            "cm_workspace_size")
    return int(out.value)


def fragment_hash(batch: FragmentBatch, digests: torch.Tensor, workspace: torch.Tensor,
                  stream=None) -> None:
    C.check(C.lib().cm_fragment_hash(ctypes.byref(batch.struct), _ptr(digests), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(),
                                     _stream(stream, batch)), "cm_fragment_hash")


def fragment_hash_select(batch: FragmentBatch, select: torch.Tensor, value: int,
                         digests: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    C.check(C.lib().cm_fragment_hash_select(ctypes.byref(batch.struct), _ptr(select), int(value),
                                            _ptr(digests), _ptr(workspace),
                                            workspace.numel() * workspace.element_size(),
                                            _stream(stream, batch)), "cm_fragment_hash_select")


def equal_key_mask(batch: FragmentBatch, keys: torch.Tensor, mask: torch.Tensor, stream=None) -> None:
    C.check(C.lib().cm_equal_key_mask(ctypes.byref(batch.struct), _ptr(keys), _ptr(mask),
                                      _stream(stream, batch)), "cm_equal_key_mask")


def fragment_knorm(batch: FragmentBatch, routing_layer: int, tail_len: int, keys: torch.Tensor,
                   workspace: torch.Tensor, stream=None) -> None:
    C.check(C.lib().cm_fragment_knorm(ctypes.byref(batch.struct), routing_layer, tail_len,
                                      _ptr(keys), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(),
                                      _stream(stream, batch)), "cm_fragment_knorm")


def canonical_order(batch: FragmentBatch, keys: torch.Tensor, digests: torch.Tensor,
                    plan: torch.Tensor, stream=None) -> None:
    C.check(C.lib().cm_canonical_order(ctypes.byref(batch.struct), _ptr(keys), _ptr(digests),
                                       _ptr(plan), _stream(stream, batch)),
            "cm_canonical_order")


def multiset_order(batch: FragmentBatch, keys: torch.Tensor, digests: torch.Tensor,
                   plan: torch.Tensor, stream=None) -> None:
    C.check(C.lib().cm_multiset_order(ctypes.byref(batch.struct), _ptr(keys), _ptr(digests),
                                      _ptr(plan), _stream(stream, batch)),
            "cm_multiset_order")


def bag_plan(batch: FragmentBatch, order) -> np.ndarray:
    """Host plan of BagMerge with the given order (delivery indices per slot)."""
    order = np.ascontiguousarray(np.asarray(order, dtype=np.int32))
    plan = np.empty(plan_elems(batch.n), dtype=np.int64)
    C.check(C.lib().cm_bag_plan(ctypes.byref(batch.struct),
                                order.ctypes.data_as(ctypes.c_void_p), int(order.size),
                                plan.ctypes.data_as(ctypes.c_void_p)), "cm_bag_plan")
    return plan


def render_merge(batch: FragmentBatch, plan_dev: torch.Tensor, plan_host: np.ndarray,
                 rope_base: float, style: str, out: torch.Tensor, T_out: int,
                 workspace: torch.Tensor, stream=None) -> None:
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_merge(ctypes.byref(batch.struct), _ptr(plan_dev),
                                    plan_host.ctypes.data_as(ctypes.c_void_p), ctypes.byref(rope),
                                    _ptr(out), T_out, _ptr(workspace),
                                    workspace.numel() * workspace.element_size(),
                                    _stream(stream, batch)), "cm_render_merge")


def render_merge_range(batch: FragmentBatch, plan_dev: torch.Tensor, plan_host: np.ndarray,
                       rope_base: float, style: str, first_slot: int, out: torch.Tensor,
                       T_cap: int, workspace: torch.Tensor, stream=None) -> None:
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_merge_range(ctypes.byref(batch.struct), _ptr(plan_dev),
                                          plan_host.ctypes.data_as(ctypes.c_void_p),
                                          ctypes.byref(rope), int(first_slot), _ptr(out), T_cap,
                                          _ptr(workspace),
                                          workspace.numel() * workspace.element_size(),
                                          _stream(stream, batch)), "cm_render_merge_range")


def render_merge_devplan(batch: FragmentBatch, plan_dev: torch.Tensor, rope_base: float,
                         style: str, out: torch.Tensor, T_out: int, workspace: torch.Tensor,
                         stream=None) -> None:
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_merge_devplan(ctypes.byref(batch.struct), _ptr(plan_dev),
                                            ctypes.byref(rope), _ptr(out), T_out, _ptr(workspace),
                                            workspace.numel() * workspace.element_size(),
                                            _stream(stream, batch)),
            "cm_render_merge_devplan")


def render_merge_hash(batch: FragmentBatch, plan_dev: torch.Tensor, plan_host: np.ndarray,
                      rope_base: float, style: str, select: torch.Tensor, digests: torch.Tensor,
                      out: torch.Tensor, T_out: int, workspace: torch.Tensor, stream=None) -> None:
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_merge_hash(ctypes.byref(batch.struct), _ptr(plan_dev),
                                         plan_host.ctypes.data_as(ctypes.c_void_p),
                                         ctypes.byref(rope), _ptr(select), _ptr(digests),
                                         _ptr(out), T_out, _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _stream(stream, batch)), "cm_render_merge_hash")


def render_deliveries_async(batch: FragmentBatch, routing_layer: int, tail_len: int,
                            rope_base: float, style: str, keys: torch.Tensor, mask: torch.Tensor,
                            digests: torch.Tensor, plan_dev: torch.Tensor, out: torch.Tensor,
                            T_cap: int, workspace: torch.Tensor, stream=None) -> None:
    """cm_render_deliveries: steps 1-5 enqueued in one call; nothing waits for the
    host. out holds [L, 2, 1, H, T_cap, d]; the cache of the plan's T_out rows is
    written to its first L * 2 * H * T_out * d elements."""
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_deliveries(ctypes.byref(batch.struct), routing_layer, tail_len,
                                         ctypes.byref(rope), _ptr(keys), _ptr(mask),
                                         _ptr(digests), _ptr(plan_dev), _ptr(out), T_cap,
                                         _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _stream(stream, batch)), "cm_render_deliveries")


def render_deliveries_graph(batch: FragmentBatch, routing_layer: int, tail_len: int,
                            rope_base: float, style: str, keys: torch.Tensor, mask: torch.Tensor,
                            digests: torch.Tensor, plan_dev: torch.Tensor, out: torch.Tensor,
                            T_cap: int, workspace: torch.Tensor) -> ctypes.c_void_p:
    """cm_render_deliveries_graph: the call of render_deliveries_async captured
    into a HIP graph over these buffers (nothing is enqueued); returns the
    handle for graph_launch / graph_destroy."""
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    handle = ctypes.c_void_p(0)
    C.check(C.lib().cm_render_deliveries_graph(ctypes.byref(batch.struct), routing_layer,
                                               tail_len, ctypes.byref(rope), _ptr(keys),
                                               _ptr(mask), _ptr(digests), _ptr(plan_dev),
                                               _ptr(out), T_cap, _ptr(workspace),
                                               workspace.numel() * workspace.element_size(),
                                               ctypes.byref(handle)),
            "cm_render_deliveries_graph")
    return handle


def graph_launch(handle: ctypes.c_void_p, owner, stream=None) -> None:
    """cm_graph_launch: every kernel of the captured call, one launch on `stream`
    (owner: the batch whose device tables the kernels read, marked as in use
    there)."""
    if not handle:
        raise ValueError("graph handle is NULL")
    C.check(C.lib().cm_graph_launch(handle, _stream(stream, owner)), "cm_graph_launch")


def graph_destroy(handle: ctypes.c_void_p) -> None:
    """cm_graph_destroy."""
    C.check(C.lib().cm_graph_destroy(handle), "cm_graph_destroy")


def render_set(batch: FragmentBatch, digests: torch.Tensor, routing_layer: int, tail_len: int,
               rope_base: float, style: str, keys: torch.Tensor, plan_dev: torch.Tensor,
               out: torch.Tensor, T_out: int, workspace: torch.Tensor, stream=None) -> None:
    """cm_render_set: steps 2-5 for a set of distinct fragments whose Ids are
    known, in one call; the plan's status tells whether it was rendered."""
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_set(ctypes.byref(batch.struct), _ptr(digests), routing_layer,
                                  tail_len, ctypes.byref(rope), _ptr(keys), _ptr(plan_dev),
                                  _ptr(out), T_out, _ptr(workspace),
                                  workspace.numel() * workspace.element_size(),
                                  _stream(stream, batch)), "cm_render_set")


def render_deliveries_noalloc(batch: FragmentBatch, routing_layer: int, tail_len: int,
                              rope_base: float, style: str, keys: torch.Tensor,
                              mask: torch.Tensor, digests: torch.Tensor, plan_dev: torch.Tensor,
                              out: torch.Tensor, T_cap: int, stream=None) -> None:
    """cm_render_deliveries_noalloc: as render_deliveries_async with the library's
    fixed per-GPU scratch in place of a workspace (nothing is allocated; calls on
    one GPU must be ordered)."""
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_render_deliveries_noalloc(ctypes.byref(batch.struct), routing_layer,
                                                 tail_len, ctypes.byref(rope), _ptr(keys),
                                                 _ptr(mask), _ptr(digests), _ptr(plan_dev),
                                                 _ptr(out), T_cap, _stream(stream, batch)),
            "cm_render_deliveries_noalloc")


def plan_elems(n: int) -> int:
    return int(C.lib().cm_plan_elems(n))


def timing_enable(on: bool) -> None:
    C.check(C.lib().cm_timing_enable(1 if on else 0), "cm_timing_enable")


def timing_reset() -> None:
    C.check(C.lib().cm_timing_reset(), "cm_timing_reset")


def timing_query(kernel: str):
    ms = ctypes.c_double(0.0)
    cnt = ctypes.c_int64(0)
    C.check(C.lib().cm_timing_query(kernel.encode(), ctypes.byref(ms), ctypes.byref(cnt)),
            "cm_timing_query")
    return float(ms.value), int(cnt.value)


KERNELS = ("hash_prep", "hash_leaf", "hash_parent", "hash_final", "knorm_rows", "knorm_tree",
           "order", "key_mask", "render_prep", "render", "render_hash", "paged",
           "paged_hash_render")


class PagedSet:
    """Fragments in a paged pool (see cm_pagedset): pool [L, 2, P, H, B, d],
    fragment i = its length and its ceil(T_i / B) page ids."""

    def __init__(self, pool: torch.Tensor, lengths: Sequence[int], page_lists: Sequence):
        if pool.dim() != 6 or pool.shape[1] != 2 or not pool.is_contiguous():
            raise ValueError("pool must be a contiguous [L, 2, P, H, B, d] tensor")
        if pool.dtype not in _DTYPES:
            raise TypeError(f"unsupported dtype {pool.dtype}")
        self.pool = pool
        self.L, _, self.P, self.H, self.B, self.d = pool.shape
        self.torch_dtype = pool.dtype
        self.device = pool.device
        self.lengths = [int(t) for t in lengths]
        rows, blocks = [], []
        for T, pages in zip(self.lengths, page_lists):
            rows.append([T, len(blocks)])
            blocks.extend(int(q) for q in pages)
        self.table_host = np.ascontiguousarray(np.array(rows, dtype=np.int64))
        self.blocks_host = np.ascontiguousarray(np.array(blocks, dtype=np.int32))
        self.table_dev = torch.from_numpy(self.table_host).to(self.device)
        self.blocks_dev = torch.from_numpy(self.blocks_host).to(self.device)
        self.device_tables = (self.table_dev, self.blocks_dev)
        self.struct = C.CmPagedset(
            n=len(self.lengths), L=self.L, H=self.H, d=self.d, dtype=_DTYPES[self.torch_dtype],
            block=self.B, pages=self.P, pool_dev=pool.data_ptr(),
            table_host=self.table_host.ctypes.data, table_dev=self.table_dev.data_ptr(),
            blocks_host=self.blocks_host.ctypes.data, blocks_dev=self.blocks_dev.data_ptr(),
            n_blocks=len(blocks))

    @property
    def n(self) -> int:
        return len(self.lengths)


def paged_workspace_size(pset: PagedSet) -> int:
    out = ctypes.c_size_t(0)
    C.check(C.lib().cm_paged_workspace_size(ctypes.byref(pset.struct), ctypes.byref(out)),
            "cm_paged_workspace_size")
    return int(out.value)


def paged_order(pset: PagedSet, routing_layer: int, tail_len: int, keys: torch.Tensor,
                mask: torch.Tensor, digests: torch.Tensor, plan_dev: torch.Tensor,
                workspace: torch.Tensor, stream=None) -> None:
    """cm_paged_order: scores, the equal-key mask, the Ids the order reads and the
    plan of fragments that live in the pool."""
    C.check(C.lib().cm_paged_order(ctypes.byref(pset.struct), routing_layer, tail_len,
                                   _ptr(keys), _ptr(mask), _ptr(digests), _ptr(plan_dev),
                                   _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _stream(stream, pset)), "cm_paged_order")


def paged_deliveries(pset: PagedSet, routing_layer: int, tail_len: int, rope_base: float,
                     style: str, free_host: np.ndarray, free_dev: torch.Tensor,
                     keys: torch.Tensor, mask: torch.Tensor, digests: torch.Tensor,
                     plan_dev: torch.Tensor, k_table: torch.Tensor, v_table: torch.Tensor,
                     n_fresh: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    """cm_paged_deliveries: steps 1-5 over the pool in one call (scores, the
    colliding Ids, the plan, the block tables on the device, the render with the
    other Ids), nothing waiting for the host. free_host and free_dev: the same
    free page ids (host, for the check; device, for the tables)."""
    fh = np.ascontiguousarray(free_host, dtype=np.int32)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_paged_deliveries(ctypes.byref(pset.struct), routing_layer, tail_len,
                                        ctypes.byref(rope), fh.ctypes.data_as(ctypes.c_void_p),
                                        _ptr(free_dev), int(fh.size), _ptr(keys), _ptr(mask),
                                        _ptr(digests), _ptr(plan_dev), _ptr(k_table),
                                        _ptr(v_table), _ptr(n_fresh), _ptr(workspace),
                                        workspace.numel() * workspace.element_size(),
                                        _stream(stream, pset)), "cm_paged_deliveries")


def paged_hash_select(pset: PagedSet, select: torch.Tensor, value: int, digests: torch.Tensor,
                      workspace: torch.Tensor, workgroups_per_cu: int = 0, stream=None) -> None:
    """cm_paged_hash_select: the Ids of the paged fragments i with select[i] == value."""
    C.check(C.lib().cm_paged_hash_select(ctypes.byref(pset.struct), _ptr(select), value,
                                         _ptr(digests), workgroups_per_cu, _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _stream(stream, pset)), "cm_paged_hash_select")


def paged_render_hash(pset: PagedSet, plan_dev: torch.Tensor, plan_host: np.ndarray,
                      rope_base: float, style: str, k_table_host: np.ndarray,
                      v_table_host: np.ndarray, k_table: torch.Tensor, v_table: torch.Tensor,
                      select: torch.Tensor, digests: torch.Tensor, workspace: torch.Tensor,
                      stream=None) -> None:
    """cm_paged_render_hash: the merged cache into the pages of the block tables
    (host arrays for the check, device copies for the kernel) and, from the same
    loads, the Ids of the slot deliveries i with select[i] == 0."""
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    kh = np.ascontiguousarray(k_table_host, dtype=np.int32)
    vh = np.ascontiguousarray(v_table_host, dtype=np.int32)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_paged_render_hash(ctypes.byref(pset.struct), _ptr(plan_dev),
                                         plan_host.ctypes.data_as(ctypes.c_void_p),
                                         ctypes.byref(rope),
                                         kh.ctypes.data_as(ctypes.c_void_p),
                                         vh.ctypes.data_as(ctypes.c_void_p), _ptr(k_table),
                                         _ptr(v_table), _ptr(select), _ptr(digests),
                                         _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _stream(stream, pset)), "cm_paged_render_hash")


def paged_tables(pset: PagedSet, plan_host: np.ndarray, free_pages):
    """Block tables of the merged cache (host): K table, V table, fresh codes 2j + kv."""
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    free = np.ascontiguousarray(np.asarray(free_pages, dtype=np.int32))
    nbo = (int(plan_host[C.PLAN_TOUT]) + pset.B - 1) // pset.B
    kt = np.empty(nbo, dtype=np.int32)
    vt = np.empty(nbo, dtype=np.int32)
    fresh = np.empty(2 * nbo, dtype=np.int32)
    count = ctypes.c_int64(0)
    C.check(C.lib().cm_paged_tables(ctypes.byref(pset.struct),
                                    plan_host.ctypes.data_as(ctypes.c_void_p),
                                    free.ctypes.data_as(ctypes.c_void_p), int(free.size),
                                    kt.ctypes.data_as(ctypes.c_void_p),
                                    vt.ctypes.data_as(ctypes.c_void_p),
                                    fresh.ctypes.data_as(ctypes.c_void_p), ctypes.byref(count)),
            "cm_paged_tables")
    return kt, vt, fresh[:count.value].copy()


def paged_render(pset: PagedSet, plan_dev: torch.Tensor, plan_host: np.ndarray, rope_base: float,
                 style: str, k_table: torch.Tensor, v_table: torch.Tensor, fresh: torch.Tensor,
                 workspace: torch.Tensor, stream=None) -> None:
    plan_host = np.ascontiguousarray(plan_host, dtype=np.int64)
    rope = C.CmRope(base=float(rope_base), style=_STYLES[style], reserved=0)
    C.check(C.lib().cm_paged_render(ctypes.byref(pset.struct), _ptr(plan_dev),
                                    plan_host.ctypes.data_as(ctypes.c_void_p), ctypes.byref(rope),
                                    _ptr(k_table), _ptr(v_table), _ptr(fresh), int(fresh.numel()),
                                    _ptr(workspace), workspace.numel() * workspace.element_size(),
                                    _stream(stream, pset)), "cm_paged_render")
