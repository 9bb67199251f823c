"""CPU oracle: CanonicalMerge render of a LatentFragmentSet, written from the paper.

TEST INFRASTRUCTURE ONLY (see the package docstring). Plain Python + numpy,
plus a plain C BLAKE3 (blake3_ref.c, loaded through ctypes); fp64 for every
floating-point step, no blocking or fusion.

What each function follows:
  * fragment_id / tensor_root / fragment_header: the content address Id of
    Alg. 2 (§4.5) and the hash tiebreak of §4.3 ("shapes, dtypes and raw bytes
    of every layer's K and V", order K1,V1,...,KL,VL, unshifted). The paper names
    no hash function; the reading used here is BLAKE3-256 of each tensor's raw
    bytes in memory order (its root), then BLAKE3-256 of a 64-byte shape/dtype
    header followed by the roots of K1, V1, ..., KL, VL.
  * FragmentSet: Ingest and Merge of Alg. 2 — set union keyed by Id, Eq. (5).
  * fragment_key / mean_knorm: Eq. (3) (§4.3) and Alg. 1 — mean L2 norm of the
    routing layer's K rows over the last T* = min_j T_j positions, averaged over
    heads (batch is 1). The sum order is fixed as adjacent-pair trees so that a
    second implementation can reproduce the key bit for bit; ordering uses the
    sum S = rho * H * T*.
  * canonical_order: Alg. 1 — argsort(-rho, -h): descending score, ties broken
    by descending hash (digest read as a big-endian unsigned integer).
  * offsets_of: §4.2 — s_pi(1) = 0, s_pi(i) = s_pi(i-1) + T_pi(i-1).
  * rope_*, rotate_pairs: §4.1 RoPE R(t) and Eq. (1): K of the fragment in slot
    i is multiplied by R(s_i) R(0)^-1 = R(s_i); half-split pairs (j, j + d/2),
    theta_j = base^(-2j/d), rotation by +s * theta_j.
  * render_in_order / canonical_merge: Eq. (1)-(2) — per layer, concatenate the
    rotated K and the unchanged V along the sequence axis.
  * render_multiset_naive: §5.9 — the naive policy that renders every delivery
    (no absorption); a foil for the re-delivery test only.
"""

from __future__ import annotations

import ctypes
import os
import struct
from dataclasses import dataclass
from typing import Dict, Iterable, List, Sequence, Tuple

import numpy as np

CHUNK_BYTES = 1024         # BLAKE3 chunk
_DIGEST = 32               # BLAKE3-256
# dtype -> (header code, element bytes)
_DTYPE_INFO = {"float32": (0, 4), "bfloat16": (1, 2)}
_MAGIC = b"CMFRAG01"


# --------------------------------------------------------------------------- fragments

@dataclass
class Fragment:
    """One thinker's unshifted legacy KV cache (§4.4): per layer (K, V), each an
    array of shape [1, H, T, d]; float32 values, or bfloat16 as uint16 bits."""
    dtype: str
    layers: List[Tuple[np.ndarray, np.ndarray]]

    def __post_init__(self):
        if self.dtype not in _DTYPE_INFO:
            raise ValueError(f"unsupported dtype {self.dtype}")
        want = np.float32 if self.dtype == "float32" else np.uint16
        shape = self.layers[0][0].shape
        for K, V in self.layers:
            if K.shape != shape or V.shape != shape or K.dtype != want or V.dtype != want:
                raise ValueError("every layer's K and V must share shape and storage dtype")
        if len(shape) != 4 or shape[0] != 1:
            raise ValueError("tensors must be [1, H, T, d]")

    @property
    def L(self) -> int:
        return len(self.layers)

    @property
    def H(self) -> int:
        return self.layers[0][0].shape[1]

    @property
    def T(self) -> int:
        return self.layers[0][0].shape[2]

    @property
    def d(self) -> int:
        return self.layers[0][0].shape[3]


# --------------------------------------------------------------------------- Id (Alg. 2)

_B3_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libblake3_ref.so")
_b3 = None


def _b3_lib():
    global _b3
    if _b3 is None:
        if not os.path.exists(_B3_LIB):
            raise RuntimeError(f"{_B3_LIB} is missing: build it with oracle/build_native.py "
                               "(__graft_entry__.build() does)")
        lib = ctypes.CDLL(_B3_LIB)
        lib.oracle_blake3.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_char_p]
        lib.oracle_blake3.restype = None
        _b3 = lib
    return _b3


def blake3(data) -> bytes:
    """BLAKE3-256 (unkeyed hash mode) of a byte string, computed by the plain C
    implementation in blake3_ref.c, written from the BLAKE3 specification."""
    raw = np.ascontiguousarray(np.frombuffer(memoryview(data).cast("B"), dtype=np.uint8))
    out = ctypes.create_string_buffer(_DIGEST)
    _b3_lib().oracle_blake3(raw.ctypes.data if raw.size else None, raw.size, out)
    return out.raw


def tensor_root(buf) -> bytes:
    """Root of one tensor: BLAKE3-256 of its raw bytes in memory order (a
    [1, H, T, d] row-major tensor: head by head, row by row, element by element,
    each element's bytes little-endian as stored)."""
    return blake3(np.ascontiguousarray(np.frombuffer(memoryview(buf).cast("B"), dtype=np.uint8)))


def fragment_header(dtype: str, L: int, H: int, T: int, d: int) -> bytes:
    """64-byte little-endian header carrying the fragment's shapes and dtype:
    magic, dtype code, element bytes, L, batch (=1), H, T (u64), d, zero pad."""
    code, esize = _DTYPE_INFO[dtype]
    hdr = struct.pack("<8sIIIIIQI", _MAGIC, code, esize, L, 1, H, T, d)
    return hdr + bytes(64 - len(hdr))


def fragment_id_from_roots(header: bytes, roots: Sequence[bytes]) -> bytes:
    return blake3(header + b"".join(roots))


def fragment_id(frag: Fragment) -> bytes:
    """Id(C) of Alg. 2: BLAKE3-256(header || root(K1) || root(V1) || ... ||
    root(KL) || root(VL)), each root the BLAKE3-256 of the tensor's bytes."""
    roots = []
    for K, V in frag.layers:
        roots.append(tensor_root(np.ascontiguousarray(K)))
        roots.append(tensor_root(np.ascontiguousarray(V)))
    return fragment_id_from_roots(fragment_header(frag.dtype, frag.L, frag.H, frag.T, frag.d), roots)


# --------------------------------------------------------------------------- state (Alg. 2)

class FragmentSet:
    """LatentFragmentSet state: a set of (Id, fragment) pairs; Merge is set
    union (Eq. (5)), Ingest adds one delivery, a byte-identical copy is absorbed."""

    def __init__(self, items: Dict[bytes, Fragment] | None = None):
        self.items: Dict[bytes, Fragment] = dict(items or {})

    def ingest(self, frag: Fragment) -> bytes:
        fid = fragment_id(frag)
        if fid not in self.items:
            self.items[fid] = frag
        return fid

    def merge(self, other: "FragmentSet") -> "FragmentSet":
        out = dict(self.items)
        for k, v in other.items.items():
            out.setdefault(k, v)
        return FragmentSet(out)

    def ids(self) -> frozenset:
        return frozenset(self.items)

    def __len__(self) -> int:
        return len(self.items)

    def render(self, routing_layer: int, rope_base: float, style: str = "half"):
        """Render of Alg. 2: CanonicalMerge over the set's fragments."""
        frags = list(self.items.values())
        ids = list(self.items.keys())
        return canonical_merge(frags, routing_layer, rope_base, style=style, ids=ids)


# --------------------------------------------------------------------------- score (Eq. (3))

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (bf16 is the top half of fp32)."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f64(x) if dtype == "bfloat16" else x.astype(np.float64)


def pairwise_sum(x: np.ndarray) -> np.ndarray:
    """Sum along the last axis by a level-wise adjacent-pair tree, after
    zero-padding that axis to a power of two."""
    n = x.shape[-1]
    p = 1 << max(0, (n - 1).bit_length())
    if p != n:
        pad = np.zeros(x.shape[:-1] + (p - n,), dtype=x.dtype)
        x = np.concatenate([x, pad], axis=-1)
    while x.shape[-1] > 1:
        x = x[..., 0::2] + x[..., 1::2]
    return x[..., 0]


def fragment_key(frag: Fragment, routing_layer: int, tail_len: int) -> float:
    """S_i = sum over heads h and the last tail_len rows r of ||K[0, h, r, :]||_2.

    Eq. (3) divides this by H * T*; the division is common to every fragment of
    a set, so the canonical order is taken on S_i itself."""
    K = frag.layers[routing_layer][0]
    T = frag.T
    if not 1 <= tail_len <= T:
        raise ValueError("tail_len must be in [1, T]")
    x = to_f64(K[0, :, T - tail_len:, :], frag.dtype)   # [H, T*, d]
    row_sq = pairwise_sum(x * x)                         # squares are exact in fp64
    norms = np.sqrt(row_sq)                              # IEEE, correctly rounded
    return float(pairwise_sum(norms.reshape(-1)))        # rows flattened (h, r) row-major


def mean_knorm(frag: Fragment, routing_layer: int, tail_len: int) -> float:
    """rho_i of Eq. (3)."""
    return fragment_key(frag, routing_layer, tail_len) / (frag.H * tail_len)


# --------------------------------------------------------------------------- order (Alg. 1)

def canonical_order(keys: Sequence[float], ids: Sequence[bytes]) -> List[int]:
    """pi* = argsort(-rho, -h): descending key; equal keys by descending digest."""
    return sorted(range(len(keys)), key=lambda i: (-keys[i], -int.from_bytes(ids[i], "big")))


def offsets_of(lengths: Sequence[int]) -> List[int]:
    """Exclusive prefix sum of the lengths in slot order (§4.2)."""
    out, s = [], 0
    for t in lengths:
        out.append(s)
        s += int(t)
    return out


# --------------------------------------------------------------------------- RoPE (§4.1, Eq. (1))

def rope_inv_freq(d: int, base: float) -> np.ndarray:
    """theta_j = base^(-2j/d), j < d/2."""
    return np.array([float(base) ** (-(2 * j) / d) for j in range(d // 2)], dtype=np.float64)


def rope_angles(s: int, d: int, base: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos and sin of s * theta_j in fp64."""
    phi = np.float64(s) * rope_inv_freq(d, base)
    return np.cos(phi), np.sin(phi)


def rotate_pairs(x: np.ndarray, c: np.ndarray, sn: np.ndarray, style: str = "half") -> np.ndarray:
    """Apply R(s) to fp64 rows x[..., d]: each pair (x1, x2) becomes
    (x1 c - x2 sn, x2 c + x1 sn), two products then one add/subtract."""
    d = x.shape[-1]
    if style == "half":
        x1, x2 = x[..., : d // 2], x[..., d // 2:]
    elif style == "interleaved":
        x1, x2 = x[..., 0::2], x[..., 1::2]
    else:
        raise ValueError(style)
    y1 = x1 * c - x2 * sn
    y2 = x2 * c + x1 * sn
    if style == "half":
        return np.concatenate([y1, y2], axis=-1)
    y = np.empty_like(x)
    y[..., 0::2] = y1
    y[..., 1::2] = y2
    return y


def f64_to_bf16_bits(y: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16, ties to even, in one step
    (no intermediate fp32 rounding). NaN becomes the quiet NaN 0x7FC0."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    with np.errstate(over="ignore", invalid="ignore"):
        _, e = np.frexp(a)                               # a = m * 2^e, m in [0.5, 1)
        qe = np.maximum(e - 1, -126) - 7                 # exponent of one bf16 ulp at a
        r = np.rint(np.ldexp(a, -qe))                    # exact scaling, then RNE to integer
        v = np.ldexp(r, qe)                              # a bf16 value (or >= 2^128)
        bits = (v.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)  # exact; overflow -> inf
    bits = bits | (np.signbit(y).astype(np.uint16) << 15)
    bits = np.where(np.isnan(y), np.uint16(0x7FC0), bits)
    return bits.astype(np.uint16)


def round_to_dtype(y: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bfloat16":
        return f64_to_bf16_bits(y)
    with np.errstate(over="ignore"):
        return y.astype(np.float32)                      # IEEE RNE


# --------------------------------------------------------------------------- render (Eq. (1)-(2))

def render_in_order(frags: Sequence[Fragment], rope_base: float, style: str = "half"):
    """BagMerge with the given order: per layer, K of slot i rotated by R(s_i)
    (slot with s_i = 0 copied byte for byte) and V copied; both concatenated
    along T. Returns a list of (K, V) arrays of shape [1, H, sum T, d]."""
    dtype = frags[0].dtype
    offs = offsets_of([f.T for f in frags])
    d = frags[0].d
    tables = [None if s == 0 else rope_angles(s, d, rope_base) for s in offs]
    out = []
    for l in range(frags[0].L):
        ks, vs = [], []
        for f, tab in zip(frags, tables):
            K, V = f.layers[l]
            if tab is None:
                ks.append(K.copy())
            else:
                ks.append(round_to_dtype(rotate_pairs(to_f64(K, dtype), tab[0], tab[1], style), dtype))
            vs.append(V.copy())
        out.append((np.concatenate(ks, axis=2), np.concatenate(vs, axis=2)))
    return out


def _check_compatible(frags: Sequence[Fragment]):
    f0 = frags[0]
    for f in frags:
        if (f.dtype, f.L, f.H, f.d) != (f0.dtype, f0.L, f0.H, f0.d):
            raise ValueError("fragments of one set must share dtype, L, H and d")


def canonical_merge(frags: Sequence[Fragment], routing_layer: int, rope_base: float,
                    style: str = "half", ids: Sequence[bytes] | None = None):
    """Alg. 1 over distinct fragments. Returns dict(cache, order, keys, ids, offsets)."""
    _check_compatible(frags)
    t_star = min(f.T for f in frags)
    keys = [fragment_key(f, routing_layer, t_star) for f in frags]
    if ids is None:
        ids = [fragment_id(f) for f in frags]
    order = canonical_order(keys, ids)
    ordered = [frags[i] for i in order]
    return {
        "cache": render_in_order(ordered, rope_base, style),
        "order": order,
        "keys": keys,
        "ids": list(ids),
        "offsets": offsets_of([f.T for f in ordered]),
        "tail_len": t_star,
    }


def render_deliveries(deliveries: Sequence[Fragment], routing_layer: int, rope_base: float,
                      style: str = "half"):
    """Ingest every delivery into an empty set, then Render (Alg. 2).

    Returns the merged cache plus, per delivery, its Id and the slot its content
    occupies; 'order' lists the delivery index kept for each slot (the first
    arrival of each distinct Id)."""
    ids = [fragment_id(f) for f in deliveries]
    first: Dict[bytes, int] = {}
    for i, fid in enumerate(ids):
        first.setdefault(fid, i)
    kept = sorted(first.values())
    res = canonical_merge([deliveries[i] for i in kept], routing_layer, rope_base, style,
                          ids=[ids[i] for i in kept])
    order = [kept[j] for j in res["order"]]
    slot_of_id = {ids[i]: s for s, i in enumerate(order)}
    return {
        "cache": res["cache"],
        "ids": ids,
        "order": order,
        "n_unique": len(kept),
        "slot_of_delivery": [slot_of_id[fid] for fid in ids],
        "offsets": res["offsets"],
        "lengths": [deliveries[i].T for i in order],
        "T_out": int(sum(deliveries[i].T for i in order)),
        "tail_len": res["tail_len"],
        "keys": {kept[j]: res["keys"][j] for j in range(len(kept))},
    }


def render_multiset_naive(deliveries: Sequence[Fragment], routing_layer: int, rope_base: float,
                          style: str = "half"):
    """Naive re-render of §5.9: every delivery is a separate operand (no
    absorption), laid out in canonical order; identical copies tie on key and
    hash and sit next to each other."""
    _check_compatible(deliveries)
    t_star = min(f.T for f in deliveries)
    keys = [fragment_key(f, routing_layer, t_star) for f in deliveries]
    ids = [fragment_id(f) for f in deliveries]
    order = canonical_order(keys, ids)
    return render_in_order([deliveries[i] for i in order], rope_base, style)


def iter_layer_bytes(cache) -> Iterable[Tuple[bytes, bytes]]:
    for K, V in cache:
        yield np.ascontiguousarray(K).tobytes(), np.ascontiguousarray(V).tobytes()
