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


ROW_BYTES = (64, 128, 256, 512, 1024)


@pytest.mark.parametrize("row_bytes", ROW_BYTES)
@pytest.mark.parametrize("nblocks", [1, 5, 16, 17, 64, 1023, 1024, 1025, 1024 + 70, 2048, 3 * 1024 + 17])
def test_message_order_closed_form(nblocks, row_bytes):
    """Closed form of the message order: inside a full 64 KiB stripe s, chunk
    64 s + k holds, for each 4 KiB step in turn, the 16-byte pieces f, f + P,
    f + 128, f + 128 + P of the step, with P = row_bytes / 32 and
    f = (k // P) * 2P + k % P; after the last full stripe the pieces keep their
    order. The message is a permutation of the pieces."""
    P = row_bytes // 32
    npieces = nblocks * 4
    ids = np.arange(npieces * 4, dtype=np.uint32)           # 4 words per 16-byte piece
    buf = ids.view(np.uint8)
    msg = om.tensor_message(buf, row_bytes)
    assert msg.size == buf.size
    got = (msg.view(np.uint32).reshape(-1, 4)[:, 0] // 4).tolist()
    want = []
    full = npieces // 4096                                   # pieces per stripe: 4096
    for s in range(full):
        for k in range(64):
            f = (k // P) * 2 * P + k % P
            for step in range(16):
                base = s * 4096 + step * 256
                want += [base + f, base + f + P, base + f + 128, base + f + 128 + P]
    want += list(range(full * 4096, npieces))
    assert got == want
    assert sorted(got) == list(range(npieces))


@pytest.mark.parametrize("row_bytes", ROW_BYTES)
def test_lane_pieces_hold_both_halves_of_their_pairs(row_bytes):
    """What the order is for: a lane's four pieces are two (first half, second
    half) pairs of one row column each, and the 64 lanes cover the step once."""
    lanes = oracle.stripe_lane_pieces(row_bytes)
    ppr = row_bytes // 16
    assert sorted(lanes.reshape(-1).tolist()) == list(range(256))
    for a, b in ((0, 1), (2, 3)):
        ra, ca = np.divmod(lanes[:, a], ppr)
        rb, cb = np.divmod(lanes[:, b], ppr)
        assert np.array_equal(ra, rb)
        assert np.all(ca < ppr // 2) and np.array_equal(cb, ca + ppr // 2)


