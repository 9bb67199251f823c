"""The library's BLAKE3 code (csrc/blake3.h), compiled for the host by the
test harness tests/native/hostcheck.hip, against the published BLAKE3 test
vectors and the oracle, with the chunk counters, flags and parent nodes the GPU
path uses; and the compiler's single-step fp64 -> bf16 conversion used by the
render kernel, against the oracle."""

import ctypes
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
    L.hc_blake3_chunk.argtypes = [ctypes.c_char_p, ctypes.c_uint64, ctypes.c_uint64,
                                  ctypes.c_int, ctypes.c_char_p]
    L.hc_blake3_parent.argtypes = [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int,
                                   ctypes.c_char_p]
    L.hc_f64_to_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    return L


def _chunk(hc, data, index, root):
    out = ctypes.create_string_buffer(32)
    assert hc.hc_blake3_chunk(data, len(data), index, int(root), out) == 0
    return out.raw


def _parent(hc, left, right, root):
    out = ctypes.create_string_buffer(32)
    assert hc.hc_blake3_parent(left, right, int(root), out) == 0
    return out.raw


def _library_blake3(hc, data):
    """BLAKE3 of a message (a positive multiple of 64 bytes) built from the
    library's chunk and parent functions the way the GPU builds it: chunks
    paired level by level, an unpaired last node carried up, ROOT on the top."""
    chunks = [data[k:k + 1024] for k in range(0, len(data), 1024)]
    if len(chunks) == 1:
        return _chunk(hc, chunks[0], 0, True)
    level = [_chunk(hc, c, k, False) for k, c in enumerate(chunks)]
    while len(level) > 1:
        top = len(level) == 2
        level = [_parent(hc, level[2 * j], level[2 * j + 1], top) if 2 * j + 1 < len(level)
                 else level[2 * j] for j in range((len(level) + 1) // 2)]
    return level[0]


def test_library_blake3_matches_published_vectors(hc, golden):
    g = golden("blake3_vectors.json")
    checked = 0
    for case in g["cases"]:
        n = case["input_len"]
        if n == 0 or n % 64:
            continue                           # the library hashes whole 64-byte blocks
        data = (np.arange(n, dtype=np.int64) % 251).astype(np.uint8).tobytes()
        assert _library_blake3(hc, data).hex() == case["hash_hex"], n
        checked += 1
    assert checked >= 8


@pytest.mark.parametrize("nblocks", [1, 15, 16, 17, 48, 80, 16 * 37 + 5])
def test_library_blake3_matches_oracle(hc, nblocks):
    rng = np.random.default_rng(nblocks)
    data = rng.integers(0, 256, size=64 * nblocks, dtype=np.uint8).tobytes()
    assert _library_blake3(hc, data) == oracle.blake3(data)


def test_tensor_root_from_library_nodes(hc):
    """The oracle's tensor root rebuilt from the library's chunk and parent code
    over the tensor's bytes in memory order (two 64 KiB stripes and a rest with
    a short last chunk)."""
    rng = np.random.default_rng(3)
    buf = rng.integers(0, 256, size=2 * 65536 + 5 * 1024 + 192, dtype=np.uint8)
    assert _library_blake3(hc, buf.tobytes()) == oracle.tensor_root(buf)


def test_single_step_bf16_conversion(hc):
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.standard_normal(100000) * np.exp2(rng.integers(-130, 128, 100000)),
                        [1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -8, 3.3961e38, 2.0 ** -134,
                         -0.0, np.inf, -np.inf]])
    y = np.zeros(x.size, np.uint16)
    hc.hc_f64_to_bf16(x.ctypes.data, y.ctypes.data, x.size)
    assert np.array_equal(y, oracle.f64_to_bf16_bits(x))
