"""Pins for the oracle's content address Id (Alg. 2; hash tiebreak of §4.3).

The paper fixes what the hash covers (shapes, dtypes and raw bytes of every
layer's K and V, unshifted, in layer order) and that it is collision-resistant;
it does not name the function. The oracle's reading is a BLAKE2s-256 tree.
The pins below: the primitive against RFC 7693's published vector, the tree's
node schedule against its closed form, and the coverage properties the paper
states (every byte, every shape/dtype field, K/V and layer order)."""

import hashlib
import struct

import numpy as np
import pytest

import oracle
from oracle import cmerge_oracle as om
from helpers import copy_fragment, rand_fragment


def test_blake2s_primitive_matches_rfc7693(golden):
    g = golden("rfc7693_blake2s.json")
    assert hashlib.blake2s(g["message_ascii"].encode()).hexdigest() == g["blake2s_256_hex"]


def test_tree_parameters_take_effect():
    data = b"\x01" * 100
    plain = hashlib.blake2s(data).digest()
    node = om._blake2s_node(data, 0, 0, True)
    assert node != plain
    assert om._blake2s_node(data, 1, 0, True) != node      # node offset
    assert om._blake2s_node(data, 0, 1, True) != node      # node depth
    assert om._blake2s_node(data, 0, 0, False) != node     # last-node flag


def _expected_leaves(nbytes):
    blocks = nbytes // 64
    full, rest = divmod(blocks, 4096)
    return 64 * full + min(64, rest)


@pytest.mark.parametrize("nblocks", [1, 5, 64, 65, 130, 4096, 4096 + 1, 4096 * 2 + 70, 4096 * 3])
def test_striped_leaves_closed_form(nblocks):
    """Closed form of the leaf layout: in a full 4 KiB step leaf k takes the
    16-byte pieces k, k+64, k+128, k+192; in a shorter final step it takes
    block k whole. The leaves are a permutation of the 16-byte pieces."""
    npieces = nblocks * 4
    ids = np.arange(npieces * 4, dtype=np.uint32)           # 4 words per 16-byte piece
    buf = ids.view(np.uint8)
    leaves = om.tensor_leaves(buf)
    assert len(leaves) == _expected_leaves(buf.nbytes)
    seen = []
    for idx, leaf in enumerate(leaves):
        assert 0 < len(leaf) <= 4096 and len(leaf) % 64 == 0
        pieces = (np.frombuffer(leaf, np.uint32).reshape(-1, 4)[:, 0] // 4).tolist()
        s, k = divmod(idx, 64)
        want = []
        stripe_pieces = min(16384, npieces - s * 16384)
        for t0 in range(0, stripe_pieces, 256):
            base = s * 16384 + t0
            step = min(256, stripe_pieces - t0)
            if step == 256:
                want += [base + k + 64 * q for q in range(4)]
            elif 4 * k < step:
                want += [base + 4 * k + q for q in range(4)]
        assert pieces == want
        seen += pieces
    assert sorted(seen) == list(range(npieces))


@pytest.mark.parametrize("nblocks", [1, 2, 64, 65, 130, 4096 + 3, 3 * 4096])
def test_tree_schedule_closed_form(monkeypatch, nblocks):
    """A binary tree with m leaves and carried-up odd nodes hashes exactly m
    leaves (offsets 0..m-1, depth 0, last flag on leaf m-1) and m-1 parents,
    with depth = ceil(log2 m) at the root."""
    calls = []
    real = om._blake2s_node

    def spy(data, off, depth, last):
        calls.append((len(bytes(data)), off, depth, last))
        return real(data, off, depth, last)

    monkeypatch.setattr(om, "_blake2s_node", spy)
    buf = np.arange(nblocks * 64, dtype=np.uint8)
    m = _expected_leaves(buf.nbytes)
    om.tensor_root(buf)
    leaves = [c for c in calls if c[2] == 0]
    parents = [c for c in calls if c[2] > 0]
    assert [c[1] for c in leaves] == list(range(m))
    assert [c[3] for c in leaves] == [k == m - 1 for k in range(m)]
    assert sum(c[0] for c in leaves) == buf.nbytes
    assert len(parents) == m - 1
    assert all(c[0] == 64 for c in parents)
    if m > 1:
        assert max(c[2] for c in parents) == int(np.ceil(np.log2(m)))
        root_call = parents[-1]
        assert root_call[1] == 0 and root_call[3] is True


def test_root_changes_on_every_single_byte_flip():
    rng = np.random.default_rng(0)
    buf = rng.integers(0, 256, size=3 * 4096 + 1024, dtype=np.uint8)
    base = om.tensor_root(buf)
    positions = [0, 1, 63, 64, 4095, 4096, 8191, 8192, 12287, 12288, buf.size - 1]
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
    big = rng.integers(0, 256, size=2 * 262144, dtype=np.uint8)       # two full stripes
    sw = big.copy()
    sw[:64], sw[64:128] = big[64:128], big[:64]                      # swap blocks of two leaves
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
