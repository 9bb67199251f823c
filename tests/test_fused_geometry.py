"""The address maps of the fused hash + render kernel and of the unit render,
walked on the CPU.

tests/native/hostcheck.hip compiles the kernel's own address arithmetic
(csrc/fused_geometry.h) for the host and walks every (slot, stripe, lane) of a
launch: each lane must read whole 64-byte blocks and whole rows inside its
tensor, the lanes' rows must partition the tensor, each row must land at merged
row h * T_out + off + t of Eq. (1)-(2)'s concatenation (its head h and position
t in slot order), and every merged row must be written exactly once. Shapes:
every row size the library takes (64 B to 1 KiB), fragments shorter than a
chunk, than a stripe, or of one token, heads that end inside a chunk, and the
slot lengths of the Qwen3-4B large workload. The unit render (one wave per 4 KiB
of the merged cache) is walked the same way (csrc/render_geometry.h): every
piece's slot holds its row, every source byte lies in that slot's tensor for
every head, and the pieces cover the rendered rows once, for whole renders and
for the range renders of the incremental cache."""

import ctypes
import os

import numpy as np
import pytest

import synth

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "libcm_hostcheck.so")


@pytest.fixture(scope="module")
def hc():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} missing: run __graft_entry__.build()")
    L = ctypes.CDLL(LIB)
    L.hc_fused_check.restype = ctypes.c_int64
    L.hc_unit_check.restype = ctypes.c_int64
    L.hc_unit_check.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                ctypes.c_int32, ctypes.c_int64, ctypes.c_int64]
    L.hc_fused_check.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                 ctypes.c_int32, ctypes.c_int64]
    return L


def _check(hc, lengths, H, rb):
    T = np.asarray(lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(T)[:-1]]).astype(np.int64)
    return hc.hc_fused_check(len(T), T.ctypes.data, off.ctypes.data, H, rb, int(T.sum()))


@pytest.mark.parametrize("rb", [64, 128, 256, 512, 1024])
@pytest.mark.parametrize("H,lengths", [
    (1, [1]),
    (2, [16, 24]),                       # Tiny
    (3, [1, 7, 5, 33]),                  # heads end inside chunks
    (8, [512, 768]),                     # 1.7B-N2
    (8, [4096, 1, 2047, 300]),
    (5, [257, 129, 65, 3]),
    (1, [70000]),                        # many stripes in one head
])
def test_fused_map_is_a_bijection_onto_the_merged_rows(hc, rb, H, lengths):
    assert _check(hc, lengths, H, rb) == 0


def test_fused_map_of_the_large_workload(hc):
    w = synth.workload("qwen3-4b-large")
    assert _check(hc, list(w.lengths), w.H, w.d * w.elem_bytes) == 0


def test_walker_finds_overlapping_slots(hc):
    """A layout the kernel does not produce is reported: two slots at the same
    offset write the same merged rows and leave others unwritten."""
    T = np.array([40, 40], dtype=np.int64)
    off = np.array([0, 0], dtype=np.int64)
    assert hc.hc_fused_check(2, T.ctypes.data, off.ctypes.data, 2, 256, 80) > 0


def _unit(hc, lengths, H, rb, first_slot=0):
    T = np.asarray(lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(T)[:-1]]).astype(np.int64)
    return hc.hc_unit_check(len(T), T.ctypes.data, off.ctypes.data, H, rb, int(off[first_slot]),
                            int(T.sum()))


@pytest.mark.parametrize("rb", [64, 128, 256, 512, 1024])
@pytest.mark.parametrize("H,lengths", [
    (1, [1]),
    (2, [16, 24]),
    (3, [1, 7, 5, 33]),
    (8, [512, 768]),
    (5, [257, 129, 65, 3, 1, 1, 2]),
])
def test_unit_map_covers_the_merged_rows_once(hc, rb, H, lengths):
    assert _unit(hc, lengths, H, rb) == 0
    assert _unit(hc, lengths, H, rb, first_slot=len(lengths) - 1) == 0   # a range render


def test_unit_map_of_the_large_workload(hc):
    w = synth.workload("qwen3-4b-large")
    rb = w.d * w.elem_bytes
    assert _unit(hc, list(w.lengths), w.H, rb) == 0
    assert _unit(hc, list(w.lengths), w.H, rb, first_slot=15) == 0


def test_unit_walker_finds_a_gap(hc):
    """Offsets that skip rows leave merged rows unwritten: reported."""
    T = np.array([10, 10], dtype=np.int64)
    off = np.array([0, 12], dtype=np.int64)
    assert hc.hc_unit_check(2, T.ctypes.data, off.ctypes.data, 2, 256, 0, 22) > 0


def _paged_layout(lengths, order, B, H, rb, spare_pages=None, seed=0):
    """Fragments on shuffled pages of a pool, the plan of `order`, and the merged
    K and V block tables from the library's own cm_paged_tables (host code)."""
    from paper_2607_01308_amd import _cabi as C
    rng = np.random.default_rng(seed)
    need = [(T + B - 1) // B for T in lengths]
    T_out = sum(lengths[i] for i in order)
    P = sum(need) + (2 * ((T_out + B - 1) // B) if spare_pages is None else spare_pages)
    perm = rng.permutation(P).astype(np.int32)
    first = np.concatenate([[0], np.cumsum(need)[:-1]]).astype(np.int64)
    blocks = np.ascontiguousarray(perm[:sum(need)])
    free = np.ascontiguousarray(perm[sum(need):])
    table = np.array([[T, f] for T, f in zip(lengths, first)], dtype=np.int64)
    n = len(lengths)
    plan = np.full(4 + 4 * n, -1, dtype=np.int64)
    plan[0], plan[1], plan[2], plan[3] = 0, n, len(order), T_out
    off = 0
    for s, i in enumerate(order):
        plan[4 + s], plan[4 + n + s], plan[4 + 2 * n + s] = i, off, lengths[i]
        off += lengths[i]
    dtype, d = (C.CM_BF16, rb // 2) if rb // 2 >= 32 else (C.CM_F32, rb // 4)
    ps = C.CmPagedset(n=n, L=1, H=H, d=d, dtype=dtype, block=B, pages=P, pool_dev=0x100000,
                      table_host=table.ctypes.data, table_dev=0x10000,
                      blocks_host=blocks.ctypes.data, blocks_dev=0x20000, n_blocks=len(blocks))
    nbo = (T_out + B - 1) // B
    kt, vt, fresh = (np.empty(nbo, np.int32), np.empty(nbo, np.int32),
                     np.empty(2 * nbo, np.int32))
    cnt = ctypes.c_int64(0)
    st = C.lib().cm_paged_tables(ctypes.byref(ps), plan.ctypes.data_as(ctypes.c_void_p),
                                 free.ctypes.data_as(ctypes.c_void_p), int(free.size),
                                 kt.ctypes.data_as(ctypes.c_void_p),
                                 vt.ctypes.data_as(ctypes.c_void_p),
                                 fresh.ctypes.data_as(ctypes.c_void_p), ctypes.byref(cnt))
    assert st == C.CM_OK, C.lib().cm_last_error()
    T = np.array([lengths[i] for i in order], dtype=np.int64)
    offs = np.array([plan[4 + n + s] for s in range(len(order))], dtype=np.int64)
    firsts = np.array([first[i] for i in order], dtype=np.int64)
    return dict(T=T, off=offs, first=firsts, blocks=blocks, P=P, T_out=T_out, kt=kt, vt=vt)


def _paged_check(hc, lay, H, rb, B, tab):
    tab = np.ascontiguousarray(tab, dtype=np.int32)
    return hc.hc_paged_fused_check(len(lay["T"]), lay["T"].ctypes.data, lay["off"].ctypes.data,
                                   lay["first"].ctypes.data, lay["blocks"].ctypes.data,
                                   len(lay["blocks"]), H, rb, int(B).bit_length() - 1, lay["P"],
                                   tab.ctypes.data, lay["T_out"])


@pytest.fixture(scope="module")
def hcp(hc):
    hc.hc_paged_fused_check.restype = ctypes.c_int64
    hc.hc_paged_fused_check.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64]
    return hc


@pytest.mark.parametrize("rb", [64, 128, 256, 512, 1024])
@pytest.mark.parametrize("small_pages", [False, True])
@pytest.mark.parametrize("H,lengths,order", [
    (2, [32, 48, 16], [1, 0, 2]),           # every slot page-aligned: V pages kept
    (2, [30, 50, 7, 64], [2, 0, 3, 1]),     # ragged: rows of a page from two slots
    (3, [1, 1, 3, 17], [3, 0, 2, 1]),       # one-row fragments, heads ending in chunks
    (5, [257, 129, 65, 3], [0, 1, 2, 3]),
    (1, [4000, 33], [1, 0]),                # many stripes in one head
])
def test_paged_fused_map(hcp, rb, small_pages, H, lengths, order):
    """The paged fused kernel's rows (fused_geometry.h): every read from the
    right fragment page, every write into the merged table's page at the right
    row and never into a fragment page, rows skipped only in the page they
    already occupy, every merged row of both tables accounted for once; pages of
    1 KiB (the fewest rows the library takes) and of 16 rows."""
    B = 1024 // rb if small_pages else 16
    lay = _paged_layout(lengths, order, B, H, rb)
    for tab in (lay["kt"], lay["vt"]):
        assert _paged_check(hcp, lay, H, rb, B, tab) == 0


def test_paged_fused_map_of_the_large_workload(hcp):
    w = synth.workload("qwen3-4b-large")
    lengths = [int(t) for t in w.lengths]
    order = list(np.random.default_rng(5).permutation(len(lengths)))
    rb = w.d * w.elem_bytes
    lay = _paged_layout(lengths, order, 16, w.H, rb)
    for tab in (lay["kt"], lay["vt"]):
        assert _paged_check(hcp, lay, w.H, rb, 16, tab) == 0


def test_paged_walker_finds_a_shared_page(hcp):
    """Two merged blocks on one fresh page write the same pool rows: reported."""
    lay = _paged_layout([30, 50], [1, 0], 16, 2, 256)
    kt = lay["kt"].copy()
    kt[2] = kt[1]
    assert _paged_check(hcp, lay, 2, 256, 16, kt) > 0
