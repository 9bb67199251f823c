"""Pins for the oracle's content address Id (Alg. 2; hash tiebreak of §4.3).

The paper fixes what the hash covers (shapes, dtypes and raw bytes of every
layer's K and V, unshifted, in layer order) and that it is collision-resistant;
it does not name the function. The oracle's reading: each tensor's root is the
BLAKE3-256 of its raw bytes in memory order, and the Id is the BLAKE3-256 of a
64-byte shape/dtype header followed by the roots of K^0, V^0, ..., K^{L-1},
V^{L-1}.

Pins: the BLAKE3 implementation against the published BLAKE3 test vectors
(empty input, one block, multi-block chunks, trees of 2 to 100 chunks); tensor
roots of tensors whose memory holds exactly a published vector's input (so the
root is that vector's digest, with no arithmetic of the oracle's own in the
expected value); and the coverage properties the paper states (every byte,
every shape and dtype field, K/V and layer order)."""

import struct

import numpy as np
import pytest

import oracle
from oracle import cmerge_oracle as om
from helpers import copy_fragment, rand_fragment


def _vector_input(n):
    """Input of the published BLAKE3 vectors: byte i is i mod 251."""
    return (np.arange(n, dtype=np.int64) % 251).astype(np.uint8)


def test_blake3_matches_published_vectors(golden):
    g = golden("blake3_vectors.json")
    assert len(g["cases"]) >= 16
    for case in g["cases"]:
        n = case["input_len"]
        assert oracle.blake3(_vector_input(n).tobytes()).hex() == case["hash_hex"], n
    for case in g["ascii_cases"]:
        assert oracle.blake3(case["message_ascii"].encode()).hex() == case["hash_hex"]


def test_blake3_accepts_any_buffer_layout():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 256, size=3000, dtype=np.uint8)
    want = oracle.blake3(a.tobytes())
    assert oracle.blake3(a) == want
    assert oracle.blake3(bytearray(a.tobytes())) == want
    assert oracle.blake3(a.view(np.uint16)) == want


# (published input length, H, d, storage dtype): tensors [1, H, T, d] whose bytes
# are exactly that input, for every row size the library supports (64 B .. 1 KiB)
# and one to 100 chunks.
VECTOR_TENSORS = [
    (1024, 2, 32, np.uint16),      # rows of 64 B, one chunk
    (2048, 1, 64, np.uint16),      # 128 B rows, two chunks
    (3072, 3, 64, np.float32),     # 256 B rows, three chunks (unpaired node)
    (4096, 2, 128, np.uint16),     # 256 B rows
    (5120, 5, 128, np.float32),    # 512 B rows
    (8192, 4, 256, np.float32),    # 1 KiB rows
    (16384, 8, 128, np.uint16),
    (31744, 31, 256, np.float32),  # 31 chunks
    (102400, 8, 128, np.uint16),   # 100 chunks: a tree with carried-up nodes
]


@pytest.mark.parametrize("n,H,d,dt", VECTOR_TENSORS)
def test_tensor_root_is_blake3_of_memory_bytes(golden, n, H, d, dt):
    """A [1, H, T, d] tensor whose memory holds the published input: its root is
    the published digest, whatever the row size and element type."""
    want = {c["input_len"]: c["hash_hex"] for c in golden("blake3_vectors.json")["cases"]}[n]
    esize = np.dtype(dt).itemsize
    T = n // (H * d * esize)
    assert T * H * d * esize == n
    t = _vector_input(n).view(dt).reshape(1, H, T, d)
    assert om.tensor_root(t).hex() == want
    # a transposed view of other bytes in memory order is not what is hashed:
    # the root follows the tensor's logical row-major order
    tt = np.ascontiguousarray(np.swapaxes(t, 1, 2))
    assert om.tensor_root(tt).hex() != want or H == 1 or T == 1


def test_fragment_id_from_published_roots(golden):
    """Id of a fragment whose every tensor holds the published 4096-byte input:
    each root is the published digest, and the Id is BLAKE3 of the header bytes
    (written out here field by field) followed by those roots."""
    want = {c["input_len"]: c["hash_hex"] for c in golden("blake3_vectors.json")["cases"]}[4096]
    t = _vector_input(4096).view(np.uint16).reshape(1, 2, 8, 128)
    L = 3
    f = oracle.Fragment("bfloat16", [(t.copy(), t.copy()) for _ in range(L)])
    header = (b"CMFRAG01" + (1).to_bytes(4, "little") + (2).to_bytes(4, "little")
              + L.to_bytes(4, "little") + (1).to_bytes(4, "little") + (2).to_bytes(4, "little")
              + (8).to_bytes(8, "little") + (128).to_bytes(4, "little") + bytes(24))
    assert oracle.fragment_id(f) == oracle.blake3(header + bytes.fromhex(want) * (2 * L))


def test_root_changes_on_every_single_byte_flip():
    rng = np.random.default_rng(0)
    buf = rng.integers(0, 256, size=3 * 4096 + 1024, dtype=np.uint8)
    base = om.tensor_root(buf)
    positions = [0, 1, 63, 64, 1023, 1024, 4095, 4096, 8191, 8192, 12287, 12288, buf.size - 1]
    positions += [int(p) for p in rng.integers(0, buf.size, size=40)]
    seen = {base}
    for p in positions:
        b = buf.copy()
        b[p] ^= 0x01
        r = om.tensor_root(b)
        assert r != base
        seen.add(r)
    assert len(seen) == len(set(positions)) + 1


def test_root_is_order_and_length_sensitive():
    rng = np.random.default_rng(1)
    buf = rng.integers(0, 256, size=4 * 4096, dtype=np.uint8)
    base = om.tensor_root(buf)
    swapped = np.concatenate([buf[1024:2048], buf[:1024], buf[2048:]])     # two chunks swapped
    assert om.tensor_root(swapped) != base
    blocks = np.concatenate([buf[64:128], buf[:64], buf[128:]])            # two blocks swapped
    assert om.tensor_root(blocks) != base
    assert om.tensor_root(np.concatenate([buf, np.zeros(64, np.uint8)])) != base
    assert om.tensor_root(buf[:-64]) != base


def test_header_layout():
    h = oracle.fragment_header("bfloat16", 36, 8, 4096, 128)
    assert len(h) == 64
    assert h[:8] == b"CMFRAG01"
    code, esize, L, B, H = struct.unpack_from("<5I", h, 8)
    (T,) = struct.unpack_from("<Q", h, 28)
    (d,) = struct.unpack_from("<I", h, 36)
    assert (code, esize, L, B, H, T, d) == (1, 2, 36, 1, 8, 4096, 128)
    assert h[40:] == bytes(24)
    assert oracle.fragment_header("float32", 2, 2, 16, 64)[8:16] == struct.pack("<II", 0, 4)


def test_id_covers_every_tensor_byte_and_is_content_only():
    rng = np.random.default_rng(2)
    f = rand_fragment(rng, L=2, H=2, T=40, d=32)
    fid = oracle.fragment_id(f)
    assert oracle.fragment_id(copy_fragment(f)) == fid          # allocation does not matter
    for l in range(f.L):
        for kv in range(2):
            g = copy_fragment(f)
            flat = g.layers[l][kv].reshape(-1).view(np.uint8)
            flat[rng.integers(0, flat.size)] ^= 0x80
            assert oracle.fragment_id(g) != fid


def test_id_covers_kv_and_layer_order():
    rng = np.random.default_rng(3)
    f = rand_fragment(rng, L=2, H=1, T=8, d=16)
    fid = oracle.fragment_id(f)
    kv_swapped = oracle.Fragment(f.dtype, [(V, K) for K, V in f.layers])
    layers_swapped = oracle.Fragment(f.dtype, list(reversed(f.layers)))
    assert oracle.fragment_id(kv_swapped) != fid
    assert oracle.fragment_id(layers_swapped) != fid


def test_id_covers_shapes_and_dtype():
    """The same bytes under another shape or dtype are another fragment."""
    rng = np.random.default_rng(4)
    raw = rng.standard_normal((1, 2, 6, 16)).astype(np.float32)
    a = oracle.Fragment("float32", [(raw, raw.copy())])
    b = oracle.Fragment("float32", [(raw.reshape(1, 3, 4, 16), raw.reshape(1, 3, 4, 16).copy())])
    c = oracle.Fragment("float32", [(raw.reshape(1, 2, 12, 8), raw.reshape(1, 2, 12, 8).copy())])
    as_bf16 = raw.view(np.uint16).reshape(1, 2, 6, 32)
    e = oracle.Fragment("bfloat16", [(as_bf16, as_bf16.copy())])
    ids = {oracle.fragment_id(x) for x in (a, b, c, e)}
    assert len(ids) == 4
    two = oracle.Fragment("float32", [(raw, raw.copy()), (raw, raw.copy())])
    assert oracle.fragment_id(two) not in ids                  # the layer count is covered too
