"""CPU oracle for the CanonicalMerge render of a LatentFragmentSet.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this package. It shares no code with
the HIP path (no kernels, headers, helpers, tables or constants) and imports
nothing from it; the product path never calls it.
"""

from .cmerge_oracle import (  # noqa: F401
    CHUNK_BYTES,
    Fragment,
    FragmentSet,
    bf16_bits_to_f64,
    blake3,
    canonical_merge,
    canonical_order,
    f64_to_bf16_bits,
    fragment_header,
    fragment_id,
    fragment_key,
    mean_knorm,
    offsets_of,
    pairwise_sum,
    render_deliveries,
    render_in_order,
    render_multiset_naive,
    rope_angles,
    rope_inv_freq,
    rotate_pairs,
    round_to_dtype,
    tensor_root,
)
