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
