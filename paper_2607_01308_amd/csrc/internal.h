// Internal interface between the C-ABI layer (api.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cmerge.h"

namespace cm {

// Device pointers read from the fragment table arrive as integers; casting them
// into the global address space lets the compiler emit global (not flat) loads.
#define CM_GLOBAL __attribute__((address_space(1)))
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <class T>
__device__ __forceinline__ const CM_GLOBAL T* global_ptr(const void* p) {
  return (const CM_GLOBAL T*)p;
}

// Validated description of a fragment set (see cm_fragset in cmerge.h).
struct SetDesc {
  int32_t n, L, H, d, dtype;
  int32_t esize;              // bytes per element
  int64_t stride;             // int64 entries per table row = 1 + 2L
  int64_t row_bytes;          // bytes of one [d] row = d * esize
  const int64_t* table_dev;   // device table (kernels)
  const int64_t* table_host;  // host table (sizing)
  int64_t T(int i) const { return table_host[(int64_t)i * stride]; }
};

// Bytes of one token of one tensor: H rows of d elements.
inline int64_t token_bytes_of(const SetDesc& s) { return (int64_t)s.H * s.row_bytes; }

constexpr size_t kWsAlign = 256;

// Hash geometry (see cm_fragment_hash): 64-byte blocks, BLAKE3 chunks of 16
// blocks (1 KiB of consecutive tensor bytes), and the work unit of the hash
// kernels: a stripe of 1024 blocks (64 KiB), i.e. 64 consecutive chunks, one per
// lane of a wave; a tensor's last stripe may be shorter.
constexpr int64_t kStripeBlocks = 1024;
constexpr int kStripeChunks = 64;

// BLAKE3 chunks of a tensor of `bytes` (a positive multiple of 64): ceil(bytes / 1 KiB).
__host__ __device__ __forceinline__ int64_t chunks_of(int64_t bytes) {
  return (bytes + 1023) >> 10;
}

// (tensor, stripe) work items per tensor: full stripes plus one for the rest.
__host__ __device__ __forceinline__ int64_t stripes_of(int64_t bytes) {
  return ((bytes >> 6) + kStripeBlocks - 1) / kStripeBlocks;
}

// Nodes per tensor at tree level v: ceil(m0 / 2^v).
__host__ __device__ __forceinline__ int64_t nodes_at(int64_t m0, int v) {
  return (m0 + (((int64_t)1 << v) - 1)) >> v;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Threads of a one-workgroup table kernel: at least n (one per delivery), and
// about one per 16 table entries of `work`, a power of two in [64, 1024].
inline int table_threads(int32_t n, int64_t work) {
  int t = 64;
  while (t < 1024 && (t < n || (int64_t)t * 16 < work)) t <<= 1;
  return t;
}

// Compute units of the current device (cached per device).
int device_cu_count();

// Tree-hash geometry of a set: a tensor of B bytes has m0 = ceil(B / 1 KiB)
// BLAKE3 chunks; level v of its tree has ceil(m0 / 2^v) nodes (adjacent pairs,
// an unpaired last node carried up, which is BLAKE3's left-balanced tree).
struct HashLayout {
  int32_t levels;         // parent levels above the chunks (0 if every tensor is one chunk)
  int64_t tasks;          // (tensor, stripe) work items of the chunk kernel
  int64_t total0;         // nodes at level 0 over all tensors
  int64_t total1;         // nodes at level 1 over all tensors (0 if levels == 0)
  size_t off_tables;      // int64 [levels+2][n+1]: per-level node bases, then task bases
  size_t off_arrived;     // int32 [n]: roots written per fragment (the tail kernel's Id step)
  size_t off_buf0;        // level-0 (and even levels) node digests
  size_t off_buf1;        // odd levels
  size_t bytes;           // total workspace bytes
};
HashLayout hash_layout(const SetDesc& s);

struct KnormLayout {
  int64_t rows;           // H * tail_len
  int64_t padded;         // next power of two >= rows
  int32_t rows_per_block; // min(256, padded)
  int64_t count0;         // partial sums per fragment after the row pass
  size_t off_a, off_b;    // ping-pong partial buffers (doubles)
  size_t bytes;
};
KnormLayout knorm_layout(const SetDesc& s, int64_t tail_len);
size_t knorm_max_bytes(const SetDesc& s);  // over every legal tail_len
// Partial sums of the score tree that a one-workgroup kernel finishes
// (knorm_fold.h): at most this many over the whole set.
constexpr int64_t kKnormFoldMax = 4096;
// A set small enough to score inside the one-workgroup kernel that needs the
// keys (no score launch): layer >= 0 names the routing layer.
struct KnormDirect {
  int32_t layer;          // -1: the scores come from the knorm launches
  int32_t esize;
  int64_t tail;           // T*
  int64_t padded;         // leaves per fragment: next power of two >= H * T*
};

struct KnormPartials {
  const double* parts;    // count per fragment, fragment-major (keys itself if count == 1)
  int64_t count;
  KnormDirect direct{-1, 0, 0, 0};
};
// Largest score tree computed inside the consumer instead of launched: leaves
// (n * padded) and 16-byte row pieces (at most four passes of 1024 threads).
constexpr int64_t kKnormDirectPieces = 4096;

struct RenderLayout {
  size_t off_tiles;       // int64 [n+1] work-unit bases per slot (fused hash+render tasks)
  size_t off_angles;      // double [n][d/2][2] cos, sin per slot (rotate.h: piece-ordered for
                          // the unit and paged renders, pair order for the fused kernel)
  size_t off_hsel;        // uint8 [n]: 0 = slot delivery hashed by the fused kernel
  size_t off_src_base;    // int64 [n][2LH]: per slot and row block, the source base of row 0
  size_t off_unit_slot;   // int32 [render units]: slot of each unit of a row block
  size_t off_flag;        // int32: 1 if the plan passed its device check
  size_t bytes;
};
RenderLayout render_layout(const SetDesc& s);
// Units of one merged row block (the render grid's x extent).
int64_t render_units(const SetDesc& s, int64_t T_out);

// Launchers (enqueue on `stream`, return the first HIP error).
// select == nullptr hashes every fragment; otherwise only fragments i with
// select[i] == want (the other digests are left untouched).
// tables_ready: the node-base tables are already in ws (launch_mask_hash_prep).
hipError_t launch_hash(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                       uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream,
                       bool tables_ready = false);
// launch_equal_key_mask and launch_hash_prep in one launch, after folding the
// score partials into keys (kp.count > 1).
hipError_t launch_mask_hash_prep(const SetDesc& s, const HashLayout& lay, const KnormPartials& kp,
                                 double* keys, uint8_t* mask, uint8_t* ws, hipStream_t stream);
// The stages of launch_hash: node-base tables, then (after the leaves) the
// parent levels and the final Id.
hipError_t launch_hash_prep(const SetDesc& s, const HashLayout& lay, uint8_t* ws,
                            hipStream_t stream);
hipError_t launch_hash_tree(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                            uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream);
hipError_t launch_equal_key_mask(const SetDesc& s, const double* keys, uint8_t* mask,
                                 hipStream_t stream);
hipError_t launch_knorm(const SetDesc& s, const KnormLayout& lay, int32_t layer, int64_t tail_len,
                        double* keys, uint8_t* ws, hipStream_t stream);
// The score kernels up to the last fold_max (or fewer) partial sums of the set,
// which a later one-workgroup kernel folds (knorm_fold); with count == 1 the
// keys are already written.
hipError_t launch_knorm_partial(const SetDesc& s, const KnormLayout& lay, int32_t layer,
                                int64_t tail_len, double* keys, uint8_t* ws, hipStream_t stream,
                                int64_t fold_max, KnormPartials* out);
// dedupe = false: every delivery gets a slot (naive multiset order).
hipError_t launch_order(const SetDesc& s, const double* keys, const uint8_t* digests,
                        bool dedupe, int64_t* plan, hipStream_t stream);
// Order (with dedupe) and, in the same launch, the per-slot render tables of
// launch_render_prep (rws: the render's part of the workspace).
hipError_t launch_order_render_prep(const SetDesc& s, const double* keys, const uint8_t* digests,
                                    int64_t* plan, const RenderLayout& rlay, double base,
                                    int32_t style, int32_t stripe_blocks, const uint8_t* select,
                                    uint8_t* rws, hipStream_t stream);
// Render of a set of distinct fragments, steps 2-5 after the score partials:
// one workgroup folds the scores (kp.count > 1), orders, and builds the unit
// render's tables for T_out rows; a plan whose T_out differs (the set held
// byte-identical members) gets CM_ESHAPE in its status, and neither it nor a
// plan with a non-finite score is rendered. Then the unit render.
hipError_t launch_render_set(const SetDesc& s, const RenderLayout& lay, const KnormPartials& kp,
                             double* keys, const uint8_t* digests, int64_t* plan, int64_t T_out,
                             double base, int32_t style, void* out, uint8_t* rws,
                             hipStream_t stream);
// Per-slot angle tables; with stripe_blocks > 0 also the per-slot task bases of
// 2L * stripes of that many 64-byte blocks (and hsel when select is given).
hipError_t launch_render_prep(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                              int32_t n_unique, double base, int32_t style, int32_t stripe_blocks,
                              const uint8_t* select, uint8_t* ws, hipStream_t stream);
// Render plus, for every slot delivery i with select[i] == 0, its Id (chunk
// level fused into the render, then the tree). ws = hash workspace, then
// render's. The slot count, T_out and the task count are read from the plan on
// the device; out must hold the merged cache of the plan's T_out rows.
// tables_ready: the hash workspace already holds this set's node-base tables
// (written by launch_hash_prep earlier on the same stream); prep_ready: the
// render's per-slot tables too (launch_order_render_prep).
hipError_t launch_render_hash(const SetDesc& s, const HashLayout& hlay, const RenderLayout& rlay,
                              const int64_t* plan_dev, double base, int32_t style,
                              const uint8_t* select, uint8_t* digests, void* out, uint8_t* ws,
                              hipStream_t stream, bool tables_ready = false,
                              bool prep_ready = false);
// Rows [row0, T_out) of every row block are rendered into `out`, whose row
// blocks are T_cap rows long (row0 = 0, T_cap = T_out: the whole merged cache).
struct RenderRange {
  int64_t row0, T_out, T_cap;
};
// check_on_device: the plan was not validated on the host; the prep kernel checks
// it against the set and T_out and, if it fails, skips the render and writes
// CM_ESHAPE into the plan's status.
hipError_t launch_render(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                         const RenderRange& rr, double base, int32_t style, bool check_on_device,
                         void* out, uint8_t* ws, hipStream_t stream);
// The unit render alone, its tables (angles, unit slots, source bases) already in ws.
hipError_t launch_render_units(const SetDesc& s, const RenderLayout& lay,
                               const int64_t* plan_dev, const RenderRange& rr, int32_t style,
                               void* out, uint8_t* ws, hipStream_t stream);

// Validated paged set (see cm_pagedset): s describes the fragments with a table
// of 2 int64 per fragment {T, first page index}.
struct PagedDesc {
  SetDesc s;
  int32_t block, b_shift;
  int64_t pages;
  void* pool;
  const int32_t* blocks_dev;
};
// Steps 1-2 on paged fragments: scores (full tree) and the Id of every fragment
// (the same content address as the dense form's: each tensor hashed in the
// byte order of its dense layout).
hipError_t launch_knorm_paged(const PagedDesc& p, const KnormLayout& lay, int32_t layer,
                              int64_t tail_len, double* keys, uint8_t* ws, hipStream_t stream);
// select as launch_hash; blocks_per_cu > 0 caps the chunk kernel's persistent
// grid (fewer workgroups leave room for a kernel running beside it).
hipError_t launch_hash_paged(const PagedDesc& p, const HashLayout& lay, const uint8_t* select,
                             uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream,
                             int blocks_per_cu = 0);
// Steps 1 and 4-5 in one pass over paged storage: the render of the fragment
// rows into the pages of the merged K and V block tables (rows whose merged
// page is the page they are read from are left in place) and, for the slot
// deliveries with select[i] == 0, their Ids (hsel as launch_render_hash).
// Workspace: the hash layout, then the render layout (launch_render_hash's).
hipError_t launch_paged_render_hash(const PagedDesc& p, const HashLayout& hlay,
                                    const RenderLayout& rlay, const int64_t* plan_dev, double base,
                                    int32_t style, const uint8_t* select, const int32_t* k_table,
                                    const int32_t* v_table, uint8_t* digests, uint8_t* ws,
                                    hipStream_t stream);
// Merged K and V block tables of the plan on the device (cm_paged_tables' rule;
// paged.hip). nbo_cap: the tables' capacity in blocks.
hipError_t launch_paged_tables(const PagedDesc& p, int64_t* plan_dev, const int32_t* free_dev,
                               int64_t n_free, int64_t nbo_cap, int32_t* k_table,
                               int32_t* v_table, int64_t* n_fresh, hipStream_t stream);
hipError_t launch_paged_render(const PagedDesc& p, const int64_t* plan_dev, int32_t n_unique,
                               double base, int32_t style, const int32_t* k_table,
                               const int32_t* v_table, const int32_t* fresh, int64_t n_fresh,
                               uint8_t* ws, hipStream_t stream);

// Per-kernel event timing (no-op unless cm_timing_enable(1)).
class ScopedTiming {
 public:
  ScopedTiming(int kernel_id, hipStream_t stream);
  ~ScopedTiming();
  ScopedTiming(const ScopedTiming&) = delete;
  ScopedTiming& operator=(const ScopedTiming&) = delete;

 private:
  int id_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
};

enum KernelId {
  K_HASH_PREP = 0,
  K_HASH_LEAF,
  K_HASH_PARENT,
  K_HASH_FINAL,
  K_KNORM_ROWS,
  K_KNORM_TREE,
  K_ORDER,
  K_KEY_MASK,
  K_RENDER_PREP,
  K_RENDER,
  K_RENDER_HASH,
  K_PAGED,
  K_PAGED_HASH_RENDER,
  K_COUNT
};

}  // namespace cm
