"""The library's BLAKE2s compression code, compiled for the host by the test
harness tests/native/hostcheck.hip, against Python's hashlib (RFC 7693) with
the tree parameters the GPU path uses; and the compiler's single-step
fp64 -> bf16 conversion used by the render kernel, against the oracle."""

import ctypes
import hashlib
import os

import numpy as np
import pytest

import oracle

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "libcm_hostcheck.so")


@pytest.fixture(scope="module")
def hc():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} missing: run __graft_entry__.build()")
    L = ctypes.CDLL(LIB)
    L.hc_blake2s_tree_node.argtypes = [ctypes.c_char_p, ctypes.c_uint64, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_int, ctypes.c_char_p]
    L.hc_blake2s_sequential.argtypes = [ctypes.c_char_p, ctypes.c_uint64, ctypes.c_char_p]
    L.hc_f64_to_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    return L


def _node(hc, data, off, depth, last):
    out = ctypes.create_string_buffer(32)
    assert hc.hc_blake2s_tree_node(data, len(data), off, depth, int(last), out) == 0
    return out.raw


@pytest.mark.parametrize("length", [64, 128, 1024, 4032, 4096])
def test_tree_node_matches_hashlib(hc, length):
    rng = np.random.default_rng(length)
    data = rng.integers(0, 256, size=length, dtype=np.uint8).tobytes()
    for off, depth, last in ((0, 0, False), (5, 0, True), (2 ** 40 + 3, 7, False), (1, 200, True)):
        want = hashlib.blake2s(data, digest_size=32, fanout=2, depth=255, leaf_size=4096,
                               node_offset=off, node_depth=depth, inner_size=32,
                               last_node=last).digest()
        assert _node(hc, data, off, depth, last) == want


def test_sequential_matches_hashlib(hc):
    rng = np.random.default_rng(9)
    for nblocks in (1, 2, 37):
        data = rng.integers(0, 256, size=64 * nblocks, dtype=np.uint8).tobytes()
        out = ctypes.create_string_buffer(32)
        assert hc.hc_blake2s_sequential(data, len(data), out) == 0
        assert out.raw == hashlib.blake2s(data, digest_size=32).digest()


def test_tensor_root_from_library_nodes(hc):
    """Rebuild the oracle's per-tensor tree with the library's node function."""
    from oracle import cmerge_oracle as om
    rng = np.random.default_rng(3)
    buf = rng.integers(0, 256, size=262144 + 5 * 4096 + 1024, dtype=np.uint8).tobytes()
    leaves = om.tensor_leaves(buf)
    m = len(leaves)
    level = [_node(hc, leaf, k, 0, k == m - 1) for k, leaf in enumerate(leaves)]
    depth = 0
    while len(level) > 1:
        depth += 1
        mm = (len(level) + 1) // 2
        level = [_node(hc, level[2 * j] + level[2 * j + 1], j, depth, j == mm - 1)
                 if 2 * j + 1 < len(level) else level[2 * j] for j in range(mm)]
    assert level[0] == oracle.tensor_root(np.frombuffer(buf, np.uint8))


def test_single_step_bf16_conversion(hc):
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.standard_normal(100000) * np.exp2(rng.integers(-130, 128, 100000)),
                        [1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -8, 3.3961e38, 2.0 ** -134,
                         -0.0, np.inf, -np.inf]])
    y = np.zeros(x.size, np.uint16)
    hc.hc_f64_to_bf16(x.ctypes.data, y.ctypes.data, x.size)
    assert np.array_equal(y, oracle.f64_to_bf16_bits(x))
