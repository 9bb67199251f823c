"""Seeded synthetic KV-cache fragments with the shapes of the paper's workloads.

This package is shared by the CPU oracle's tests, the HIP path's tests and the
benchmark. It draws random numbers and lays them out as per-layer K/V tensors;
it holds none of the merge method's arithmetic (no hashing, no norms, no
ordering, no rotation).
"""

from .configs import (  # noqa: F401
    Workload,
    WORKLOADS,
    custom,
    qwen3_17b_n2,
    qwen3_17b_n5,
    qwen3_4b_large,
    qwen3_4b_n4,
    tiny,
    workload,
)
from .generate import (  # noqa: F401
    TORCH_DTYPES,
    draw_tensor,
    gather_paged,
    make_deliveries,
    make_fragments,
    make_paged,
    tensor_to_numpy,
    to_numpy_cache,
)
