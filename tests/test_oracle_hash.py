"""Pins for the oracle's content address Id (Alg. 2; hash tiebreak of §4.3).

The paper fixes what the hash covers (shapes, dtypes and raw bytes of every
layer's K and V, unshifted, in layer order) and that it is collision-resistant;
it does not name the function. The oracle's reading is BLAKE3-256 over each
tensor's bytes in a fixed interleaved order, then over a header and the tensor
roots. The pins below: the BLAKE3 implementation against the published BLAKE3
test vectors (single blocks, multi-block chunks, trees of 2 to 100 chunks), the
message order against its closed form, and the coverage properties the paper
states (every byte, every shape/dtype field, K/V and layer order)."""

import struct

import numpy as np
import pytest

import oracle
from oracle import cmerge_oracle as om
from helpers import copy_fragment, rand_fragment


def test_blake3_matches_published_vectors(golden):
    g = golden("blake3_vectors.json")
    assert len(g["cases"]) >= 16
    for case in g["cases"]:
        n = case["input_len"]
        data = (np.arange(n, dtype=np.int64) % 251).astype(np.uint8).tobytes()
        assert oracle.blake3(data).hex() == case["hash_hex"], n
    for case in g["ascii_cases"]:
        assert oracle.blake3(case["message_ascii"].encode()).hex() == case["hash_hex"]


def test_blake3_accepts_any_buffer_layout():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 256, size=3000, dtype=np.uint8)
    want = oracle.blake3(a.tobytes())
    assert oracle.blake3(a) == want
    assert oracle.blake3(bytearray(a.tobytes())) == want
    assert oracle.blake3(a.view(np.uint16)) == want


@pytest.mark.parametrize("nblocks", [1, 5, 16, 17, 64, 1023, 1024, 1025, 1024 + 70, 2048, 3 * 1024 + 17])
def test_message_order_closed_form(nblocks):
    """Closed form of the message order: inside a full 64 KiB stripe s, chunk
    64 s + k holds, for each 4 KiB step in turn, the 16-byte pieces k, k+64,
    k+128, k+192 of the step; after the last full stripe the pieces keep their
    order. The message is a permutation of the pieces."""
    npieces = nblocks * 4
    ids = np.arange(npieces * 4, dtype=np.uint32)           # 4 words per 16-byte piece
    buf = ids.view(np.uint8)
    msg = om.tensor_message(buf)
    assert msg.size == buf.size
    got = (msg.view(np.uint32).reshape(-1, 4)[:, 0] // 4).tolist()
    want = []
    full = npieces // 4096                                   # pieces per stripe: 4096
    for s in range(full):
        for k in range(64):
            for step in range(16):
                base = s * 4096 + step * 256
                want += [base + k + 64 * q for q in range(4)]
    want += list(range(full * 4096, npieces))
    assert got == want
    assert sorted(got) == list(range(npieces))


def test_short_tensor_root_is_plain_blake3():
    """A tensor shorter than one stripe is hashed in its own byte order."""
    rng = np.random.default_rng(6)
    for n in (64, 1024, 5000 - 5000 % 64, 65536 - 64):
        buf = rng.integers(0, 256, size=n, dtype=np.uint8)
        assert om.tensor_root(buf) == oracle.blake3(buf.tobytes())


def test_root_changes_on_every_single_byte_flip():
    rng = np.random.default_rng(0)
    buf = rng.integers(0, 256, size=65536 + 3 * 4096 + 1024, dtype=np.uint8)
    base = om.tensor_root(buf)
    positions = [0, 1, 15, 16, 63, 64, 1023, 1024, 4095, 4096, 65535, 65536, 69631, 69632,
                 buf.size - 1]
    positions += list(rng.integers(0, buf.size, size=40))
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
    swapped = np.concatenate([buf[4096:8192], buf[:4096], buf[8192:]])
    assert om.tensor_root(swapped) != base
    assert om.tensor_root(np.concatenate([buf, np.zeros(4096, np.uint8)])) != base
    assert om.tensor_root(buf[:-64]) != base
    big = rng.integers(0, 256, size=2 * 65536 + 3072, dtype=np.uint8)  # two full stripes + rest
    for a, b in ((0, 16), (0, 1024), (65536, 65536 + 16), (131072, 131072 + 64)):
        sw = big.copy()
        sw[a:a + 16], sw[b:b + 16] = big[b:b + 16], big[a:a + 16]    # swap two pieces
        assert om.tensor_root(sw) != om.tensor_root(big)


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
            arr = g.layers[l][kv]
            flat = arr.reshape(-1).view(np.uint8)
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
    rng = np.random.default_rng(4)
    raw = rng.standard_normal((1, 2, 6, 16)).astype(np.float32)
    a = oracle.Fragment("float32", [(raw, raw.copy())])
    b = oracle.Fragment("float32", [(raw.reshape(1, 3, 4, 16), raw.reshape(1, 3, 4, 16).copy())])
    c = oracle.Fragment("float32", [(raw.reshape(1, 2, 12, 8), raw.reshape(1, 2, 12, 8).copy())])
    as_bf16 = raw.view(np.uint16).reshape(1, 2, 6, 32)
    e = oracle.Fragment("bfloat16", [(as_bf16, as_bf16.copy())])
    ids = {oracle.fragment_id(x) for x in (a, b, c, e)}
    assert len(ids) == 4                                       # same bytes, four identities
    two = oracle.Fragment("float32", [(raw, raw.copy()), (raw, raw.copy())])
    assert oracle.fragment_id(two) not in ids                  # layer count is covered too
