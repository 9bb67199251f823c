"""Small builders shared by the CPU tests (numpy only, no method arithmetic)."""

import numpy as np

from oracle import Fragment


def rand_fragment(rng, L=2, H=2, T=6, d=16, dtype="float32", k_scale=1.0):
    layers = []
    for _ in range(L):
        K = (rng.standard_normal((1, H, T, d)) * k_scale).astype(np.float32)
        V = rng.standard_normal((1, H, T, d)).astype(np.float32)
        if dtype == "bfloat16":
            K = (K.view(np.uint32) >> 16).astype(np.uint16)
            V = (V.view(np.uint32) >> 16).astype(np.uint16)
        layers.append((K, V))
    return Fragment(dtype, layers)


def copy_fragment(f):
    return Fragment(f.dtype, [(K.copy(), V.copy()) for K, V in f.layers])


def cache_bytes(cache):
    return [(np.ascontiguousarray(K).tobytes(), np.ascontiguousarray(V).tobytes()) for K, V in cache]
