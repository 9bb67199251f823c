"""MI355X-native CanonicalMerge render of a LatentFragmentSet (arXiv 2607.01308,
§4.3-§4.5, Alg. 1-2): HIP kernels for gfx950 behind the C ABI of
include/cmerge.h, with a thin torch binding."""

from ._cabi import CmError, LIB_PATH  # noqa: F401
from .binding import (  # noqa: F401
    KERNELS,
    FragmentBatch,
    PagedSet,
    bag_plan,
    canonical_order,
    equal_key_mask,
    fragment_hash,
    fragment_hash_select,
    fragment_knorm,
    multiset_order,
    paged_render,
    paged_tables,
    paged_workspace_size,
    plan_elems,
    render_merge,
    render_merge_devplan,
    render_merge_range,
    render_merge_hash,
    render_deliveries_async,
    timing_enable,
    timing_query,
    timing_reset,
    workspace_size,
)
from .fragset import (  # noqa: F401
    LatentFragmentSet,
    MergedCache,
    PagedRender,
    PIPELINES,
    RenderResult,
    bag_merge,
    fragment_ids,
    release_workspace,
    render_deliveries,
    render_multiset,
    render_paged,
)
