"""Stream bookkeeping of the binding, on the CPU with stand-ins for the
library and for device tensors.

The kernels read a set's device tables (the fragment table; for a paged set
also the page list) after the binding call has returned. Every call must
therefore mark each of those tables as in use on the stream it enqueues on
(record_stream), or the caching allocator may give their memory to another
tensor while the kernels still read it: a kernel then reads garbage tensor
addresses, the memory fault seen once on the GPU before this rule was in
place. Scratch memory must be cached per (device, stream), so calls on two
streams never share it."""

import ctypes
import contextlib
import inspect

import numpy as np
import pytest
import torch

import paper_2607_01308_amd as cm
from paper_2607_01308_amd import _cabi, binding, fragset


class FakeStream:
    def __init__(self, handle):
        self.cuda_stream = handle


class FakeTable:
    """A device table: remembers every stream it was marked on."""

    def __init__(self):
        self.streams = []

    def record_stream(self, s):
        self.streams.append(s)

    def data_ptr(self):
        return 0x1000


class FakeTensor:
    def data_ptr(self):
        return 0x2000

    def numel(self):
        return 256

    def element_size(self):
        return 1


class FakeLib:
    """Every entry point returns CM_OK and records which stream it was given."""

    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def f(*args):
            self.calls.append((name, args[-1] if args else None))
            return 0
        return f


def _owner(n_tables):
    o = type("Owner", (), {})()
    o.device = torch.device("cpu")
    o.device_tables = tuple(FakeTable() for _ in range(n_tables))
    o.struct = _cabi.CmFragset() if n_tables == 1 else _cabi.CmPagedset()
    o.n = 2
    return o


@pytest.fixture
def fake_lib(monkeypatch):
    lib = FakeLib()
    monkeypatch.setattr(_cabi, "lib", lambda: lib)
    return lib


# every binding function that enqueues device work, with arguments of stand-ins
T = FakeTensor()
PLAN = np.zeros(4 + 4 * 2, dtype=np.int64)
CALLS = {
    "fragment_hash": lambda b, s: binding.fragment_hash(b, T, T, s),
    "fragment_hash_select": lambda b, s: binding.fragment_hash_select(b, T, 1, T, T, s),
    "equal_key_mask": lambda b, s: binding.equal_key_mask(b, T, T, s),
    "fragment_knorm": lambda b, s: binding.fragment_knorm(b, 0, 1, T, T, s),
    "canonical_order": lambda b, s: binding.canonical_order(b, T, T, T, s),
    "multiset_order": lambda b, s: binding.multiset_order(b, T, T, T, s),
    "render_merge": lambda b, s: binding.render_merge(b, T, PLAN, 1e4, "half", T, 1, T, s),
    "render_merge_range": lambda b, s: binding.render_merge_range(b, T, PLAN, 1e4, "half", 0, T,
                                                                  1, T, s),
    "render_merge_devplan": lambda b, s: binding.render_merge_devplan(b, T, 1e4, "half", T, 1,
                                                                      T, s),
    "render_merge_hash": lambda b, s: binding.render_merge_hash(b, T, PLAN, 1e4, "half", T, T, T,
                                                                1, T, s),
    "render_deliveries_async": lambda b, s: binding.render_deliveries_async(
        b, 0, 1, 1e4, "half", T, T, T, T, T, 1, T, s),
    "render_deliveries_noalloc": lambda b, s: binding.render_deliveries_noalloc(
        b, 0, 1, 1e4, "half", T, T, T, T, T, 1, s),
    "render_set": lambda b, s: binding.render_set(b, T, 0, 1, 1e4, "half", T, T, T, 1, T, s),
}


def test_every_enqueuing_call_is_covered():
    """The list above names every binding function that takes a stream (paged
    render is checked separately below)."""
    takes_stream = {name for name, f in inspect.getmembers(binding, inspect.isfunction)
                    if "stream" in inspect.signature(f).parameters and not name.startswith("_")}
    assert takes_stream == set(CALLS) | {"paged_render", "paged_order", "paged_hash_select",
                                         "paged_render_hash", "paged_deliveries", "graph_launch"}


@pytest.mark.parametrize("name", sorted(CALLS))
def test_call_marks_its_tables_on_its_stream(fake_lib, name):
    batch = _owner(1)
    s1, s2 = FakeStream(11), FakeStream(22)
    CALLS[name](batch, s1)
    CALLS[name](batch, s2)
    assert batch.device_tables[0].streams == [s1, s2]
    # and the library was handed exactly that stream
    assert [c[1].value for c in fake_lib.calls] == [11, 22]


def test_paged_render_marks_both_tables(fake_lib):
    pset = _owner(2)
    s = FakeStream(33)
    binding.paged_render(pset, T, PLAN, 1e4, "half", T, T, T, T, s)
    assert [t.streams for t in pset.device_tables] == [[s], [s]]
    assert fake_lib.calls[-1][1].value == 33


def test_paged_render_hash_marks_both_tables(fake_lib):
    pset = _owner(2)
    s = FakeStream(34)
    tab = np.zeros(3, dtype=np.int32)
    binding.paged_render_hash(pset, T, PLAN, 1e4, "half", tab, tab, T, T, T, T, T, s)
    assert [t.streams for t in pset.device_tables] == [[s], [s]]
    assert fake_lib.calls[-1][0] == "cm_paged_render_hash"
    assert fake_lib.calls[-1][1].value == 34


def test_paged_deliveries_marks_both_tables(fake_lib):
    pset = _owner(2)
    s = FakeStream(35)
    free = np.zeros(4, dtype=np.int32)
    binding.paged_deliveries(pset, 0, 1, 1e4, "half", free, T, T, T, T, T, T, T, T, T, s)
    assert [t.streams for t in pset.device_tables] == [[s], [s]]
    assert fake_lib.calls[-1][0] == "cm_paged_deliveries"
    assert fake_lib.calls[-1][1].value == 35


def test_graph_launch_marks_the_batch_tables(fake_lib):
    """A graph's kernels read the batch's device table at every launch."""
    batch = _owner(1)
    s = FakeStream(36)
    binding.graph_launch(ctypes.c_void_p(0x1234), batch, s)
    assert batch.device_tables[0].streams == [s]
    assert fake_lib.calls[-1][0] == "cm_graph_launch" and fake_lib.calls[-1][1].value == 36
    with pytest.raises(ValueError):
        binding.graph_launch(ctypes.c_void_p(0), batch, s)


def test_paged_order_marks_both_tables(fake_lib):
    pset = _owner(2)
    s = FakeStream(44)
    binding.paged_order(pset, 0, 1, T, T, T, T, T, s)
    assert [t.streams for t in pset.device_tables] == [[s], [s]]
    assert fake_lib.calls[-1][1].value == 44
    s2 = FakeStream(45)
    binding.paged_hash_select(pset, T, 0, T, T, 2, s2)
    assert [t.streams for t in pset.device_tables] == [[s, s2], [s, s2]]
    assert fake_lib.calls[-1][1].value == 45


def test_scratch_is_cached_per_stream(monkeypatch):
    """fragset._workspace: one buffer per (device, stream), allocated on that
    stream; a stream's buffer is reused by later calls on it and replaced only
    when a larger one is needed."""
    made = []

    def fake_empty(n, dtype=None, device=None):
        t = torch.zeros(n, dtype=dtype)
        made.append(t)
        return t

    entered = []

    @contextlib.contextmanager
    def fake_stream_ctx(s):
        entered.append(s)
        yield

    need = {"v": 1000}
    monkeypatch.setattr(fragset, "workspace_size", lambda b: need["v"])
    monkeypatch.setattr(fragset.torch, "empty", fake_empty)
    monkeypatch.setattr(fragset.torch.cuda, "stream", fake_stream_ctx)
    fragset.release_workspace()
    batch = type("B", (), {"device": torch.device("cpu")})()
    a, b = FakeStream(1), FakeStream(2)
    wa = fragset._workspace(batch, a)
    wb = fragset._workspace(batch, b)
    assert wa is not wb and entered == [a, b]
    assert fragset._workspace(batch, a) is wa and fragset._workspace(batch, b) is wb
    need["v"] = 5000
    wa2 = fragset._workspace(batch, a)
    assert wa2 is not wa and wa2.numel() == 5000 and entered[-1] is a
    assert fragset._workspace(batch, b) is not wb           # grown on b as well, on b
    assert entered[-1] is b
    fragset.release_workspace()
