"""Draw the tensors of a Workload as legacy KV caches (torch tensors).

A legacy cache is a tuple over layers of (K, V), each a contiguous tensor of
shape [1, H, T, d]. Values: K ~ N(0, k_scale_i^2), V ~ N(0, 1), drawn in fp32
and stored in the workload dtype. Every (fragment, layer, K|V) tensor has a
seed of its own derived from the workload seed, so any tensor can be drawn
alone (draw_tensor) and equals the one inside make_fragments.
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np
import torch

from .configs import Workload

TORCH_DTYPES = {"float32": torch.float32, "bfloat16": torch.bfloat16}


def _stream_seed(seed: int, frag: int, layer: int, kind: int) -> int:
    state = np.random.SeedSequence([seed, frag, layer, kind]).generate_state(1, np.uint64)[0]
    return int(state & np.uint64(0x7FFF_FFFF_FFFF_FFFF))


def draw_tensor(w: Workload, i: int, layer: int, kind: str, device="cpu") -> torch.Tensor:
    """K (kind='k') or V (kind='v') of distinct fragment i at one layer."""
    if kind == "k":
        for src, dst in w.shared_k:
            if dst == i:
                if w.lengths[src] != w.lengths[dst]:
                    raise ValueError("a shared-K pair must have equal lengths")
                i = src
        scale, k = w.k_scale[i], 0
    elif kind == "v":
        scale, k = 1.0, 1
    else:
        raise ValueError(kind)
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(_stream_seed(w.seed, i, layer, k))
    x = torch.randn((1, w.H, w.lengths[i], w.d), generator=g, dtype=torch.float32, device=dev)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(TORCH_DTYPES[w.dtype]).contiguous()


def make_fragments(w: Workload, device="cpu") -> List[Tuple[Tuple[torch.Tensor, torch.Tensor], ...]]:
    """One legacy cache per distinct fragment of the workload."""
    return [tuple((draw_tensor(w, i, l, "k", device), draw_tensor(w, i, l, "v", device))
                  for l in range(w.L))
            for i in range(w.n_distinct)]


def make_deliveries(w: Workload, frags: Sequence) -> list:
    """Arrival list: the first delivery of a fragment is the fragment itself,
    every re-delivery is a byte copy in a buffer of its own."""
    seen = set()
    out = []
    for i in w.deliveries:
        if i in seen:
            out.append(tuple((K.clone(), V.clone()) for K, V in frags[i]))
        else:
            seen.add(i)
            out.append(frags[i])
    return out


def tensor_to_numpy(x: torch.Tensor) -> np.ndarray:
    """Host copy: float32 stays float32, bfloat16 becomes its uint16 bit patterns."""
    x = x.detach().to("cpu").contiguous()
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16).copy()
    if x.dtype == torch.float32:
        return x.numpy().copy()
    raise TypeError(f"unsupported dtype {x.dtype}")


def to_numpy_cache(cache) -> Tuple[str, list]:
    """Host copy of a legacy cache: (dtype name, [(K, V) numpy arrays])."""
    dtype = {torch.bfloat16: "bfloat16", torch.float32: "float32"}[cache[0][0].dtype]
    return dtype, [(tensor_to_numpy(K), tensor_to_numpy(V)) for K, V in cache]


def make_paged(caches: Sequence, block: int, spare_pages: int, seed: int = 0, device=None):
    """The same fragments stored in a page pool [L, 2, P, H, B, d] (pages of B
    tokens of every head), each fragment on ceil(T / B) pages drawn at random from
    the pool, plus `spare_pages` pages left free. Returns (pool, lengths,
    page_lists, free_pages). Unused rows of a fragment's last page are zero."""
    K0 = caches[0][0][0]
    L, (_, H, _, d) = len(caches[0]), K0.shape
    device = device if device is not None else K0.device
    lengths = [int(c[0][0].shape[2]) for c in caches]
    need = [(T + block - 1) // block for T in lengths]
    P = sum(need) + spare_pages
    perm = np.random.default_rng(seed).permutation(P)
    pool = torch.zeros((L, 2, P, H, block, d), dtype=K0.dtype, device=device)
    page_lists, k = [], 0
    for c, T, nb in zip(caches, lengths, need):
        pages = perm[k:k + nb].tolist()
        k += nb
        page_lists.append(pages)
        idx = torch.tensor(pages, dtype=torch.long, device=device)
        for l, (K, V) in enumerate(c):
            for kv, x in enumerate((K, V)):
                padded = torch.zeros((H, nb * block, d), dtype=x.dtype, device=device)
                padded[:, :T] = x[0]
                pool[l, kv, idx] = padded.reshape(H, nb, block, d).permute(1, 0, 2, 3)
    free = perm[k:].tolist()
    return pool, lengths, page_lists, free


def gather_paged(pool: torch.Tensor, table, T: int) -> torch.Tensor:
    """Dense [L, 2, 1, H, T, d] view-copy of a sequence stored on pages `table`
    (one page id per B rows)."""
    L, _, _, H, B, d = pool.shape
    idx = torch.as_tensor(np.asarray(table, dtype=np.int64), device=pool.device)
    pages = pool[:, :, idx]                                  # [L, 2, nb, H, B, d]
    dense = pages.permute(0, 1, 3, 2, 4, 5).reshape(L, 2, H, -1, d)[:, :, :, :T]
    return dense.unsqueeze(2).contiguous()
