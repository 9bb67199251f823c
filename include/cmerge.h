/*
 * cmerge.h — C ABI of libcmerge: the CanonicalMerge render of a LatentFragmentSet
 * on AMD Instinct MI355X (gfx950).
 *
 * Paper: "Cache Merging as a Convergent Replicated State for Multi-Agent Latent
 * Reasoning" (arXiv 2607.01308). The calls below are the steps of Alg. 1
 * (CanonicalMerge) run inside Render of Alg. 2 (LatentFragmentSet):
 *   cm_fragment_hash        Id of Alg. 2 / the hash tiebreak h_i of §4.3
 *   cm_fragment_knorm       the mean K-norm score rho_i of Eq. (3)
 *   cm_canonical_order      Ingest dedupe (Eq. (5)) + argsort(-rho, -h) of Alg. 1
 *                           + the offsets s of §4.2
 *   cm_render_merge         Eq. (1)-(2): K of slot i rotated by R(s_i), V copied,
 *                           both concatenated along the sequence axis
 *   cm_render_merge_devplan the same with the plan left on the device
 *   cm_render_merge_range   the slots from a given rank on (incremental render)
 *   cm_render_set           steps 2-5 for a set with known Ids, in one call
 *   cm_paged_order / cm_paged_hash_select / cm_paged_tables / cm_paged_render /
 *   cm_paged_render_hash    steps 1-5 over paged storage
 *   cm_paged_deliveries     steps 1-5 over paged storage in one call, with no host
 *                           round trip
 * the paper's baselines over the same render:
 *   cm_multiset_order       the naive re-render order of §5.9 (no dedupe)
 *   cm_bag_plan             BagMerge with a caller-supplied order (§4.2)
 * and, to run step 1 without a second read of the fragments:
 *   cm_equal_key_mask       the deliveries whose digest the order needs
 *   cm_fragment_hash_select the Id of a subset of the deliveries
 *   cm_render_merge_hash    the render plus the remaining Ids from its loads
 *   cm_render_deliveries    steps 1-5 over a batch of deliveries in one call, with
 *                           no host round trip
 *   cm_render_deliveries_noalloc
 *                           the same with no workspace argument, for callers that
 *                           cannot allocate
 *   cm_render_deliveries_graph / cm_graph_launch / cm_graph_destroy
 *                           the same call captured into a HIP graph and replayed
 *
 * Conventions
 *   - Every function returns int32_t: CM_OK (0) or a negative cm_status. No
 *     exception crosses the ABI. cm_last_error() returns a thread-local message
 *     for the last failing call on the calling thread.
 *   - Device work is enqueued on `stream` (a hipStream_t passed as void*; NULL is
 *     the null stream) and the call returns without waiting for it. Argument
 *     checks happen on the host before anything is enqueued; a call that returns
 *     an error has enqueued nothing.
 *   - All buffers are owned by the caller. The library allocates no device
 *     memory: calls that need scratch take a workspace of at least
 *     cm_workspace_size() bytes (device memory, 256-byte aligned). Buffers must
 *     stay valid until the enqueued work has finished. Calls that share a
 *     workspace must be ordered (same stream, or synchronised).
 *   - Tensors: a fragment is a HuggingFace legacy KV cache: per layer l a K and a
 *     V tensor of shape [1, H, T, d], contiguous, row-major, dtype bf16 or fp32.
 *     K is stored post-RoPE at local positions 0..T-1 (§4.1). Every tensor
 *     address must be 16-byte aligned.
 *   - Supported shapes: d a power of two with d * element_bytes in [64, 1024];
 *     1 <= n <= CM_MAX_FRAGMENTS; L, H >= 1; T >= 1.
 */
#ifndef CMERGE_H
#define CMERGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CM_ABI_VERSION 1
#define CM_MAX_FRAGMENTS 1024

typedef enum {
  CM_OK = 0,
  CM_EINVAL = -1,      /* NULL pointer, count or index out of range, misaligned buffer */
  CM_ESHAPE = -2,      /* unsupported or inconsistent shape; T_out != sum of slot lengths */
  CM_EDTYPE = -3,      /* unsupported dtype */
  CM_ENONFINITE = -4,  /* a score is NaN or infinite (reported through the plan) */
  CM_EHIP = -5,        /* a HIP runtime call failed; the message carries hipGetErrorString */
  CM_EWORKSPACE = -6,  /* workspace NULL, misaligned or smaller than cm_workspace_size() */
} cm_status;

typedef enum { CM_F32 = 0, CM_BF16 = 1 } cm_dtype;

/* RoPE pairing (§4.1 leaves it open): CM_ROPE_HALF pairs (j, j + d/2), the
 * HuggingFace Qwen3 layout and the default. CM_ROPE_INTERLEAVED pairs (2j, 2j+1). */
typedef enum { CM_ROPE_HALF = 0, CM_ROPE_INTERLEAVED = 1 } cm_rope_style;

/* A set of n fragments (deliveries; byte-identical duplicates allowed) sharing
 * L, H, d and dtype.
 * table_host: host memory, n rows of (1 + 2L) int64:
 *     row i = { T_i, addr(K_i^0), addr(V_i^0), ..., addr(K_i^{L-1}), addr(V_i^{L-1}) }
 *     with device addresses of the [1, H, T_i, d] tensors.
 * table_dev: device memory holding the same n * (1 + 2L) values (the kernels read
 *     it; the host validates table_host). The caller keeps the two identical. */
typedef struct {
  int32_t n;
  int32_t L;
  int32_t H;
  int32_t d;
  int32_t dtype;     /* cm_dtype */
  int32_t reserved;  /* must be 0 */
  const int64_t* table_host;
  const int64_t* table_dev;
} cm_fragset;

/* RoPE of the model: theta_j = base^(-2j/d) (§4.1). */
typedef struct {
  double base;
  int32_t style;     /* cm_rope_style */
  int32_t reserved;  /* must be 0 */
} cm_rope;

/* ---------------------------------------------------------------- plan layout
 * A plan is an int64 array of cm_plan_elems(n) entries, written on the device by
 * cm_canonical_order (or cm_multiset_order; on the host by cm_bag_plan) and read
 * by cm_render_merge:
 *   [0]                 status: CM_OK, or CM_ENONFINITE if a score is not finite
 *   [1]                 n (deliveries)
 *   [2]                 n_unique: distinct fragments = slots of the merged cache
 *   [3]                 T_out: merged length, the sum of the slot lengths
 *   [4 + s]             delivery index rendered in slot s (s < n_unique)
 *   [4 + n + s]         offset s_pi(s) of slot s (§4.2)
 *   [4 + 2n + s]        length of slot s
 *   [4 + 3n + i]        slot holding the content of delivery i (duplicates point
 *                       at the slot of their first arrival)
 * Entries for s >= n_unique are -1. */
#define CM_PLAN_STATUS 0
#define CM_PLAN_N 1
#define CM_PLAN_NUNIQUE 2
#define CM_PLAN_TOUT 3
#define CM_PLAN_HEADER 4

/* ---------------------------------------------------------------- utilities */

int32_t cm_version(void);                    /* CM_ABI_VERSION */
const char* cm_last_error(void);             /* "" when the last call succeeded */
const char* cm_status_string(int32_t status);
size_t cm_plan_elems(int32_t n);             /* 4 + 4n */

/* Workspace bytes that every call below needs for this set (the maximum over
 * the calls). The set is validated (host table only). */
int32_t cm_workspace_size(const cm_fragset* set, size_t* bytes_out);

/* ---------------------------------------------------------------- step 1
 * Id of Alg. 2 (content address; also the hash tiebreak of §4.3): for every
 * fragment, a 32-byte digest of its shapes, dtype and the raw bytes of
 * K^0, V^0, ..., K^{L-1}, V^{L-1} in that order. Function: BLAKE3-256 (unkeyed
 * hash mode of the BLAKE3 specification). Per tensor, the root is the BLAKE3-256
 * of its raw bytes in memory order (the [1, H, T, d] row-major bytes: what any
 * BLAKE3 implementation gives for the buffer).
 * Then the Id is the BLAKE3-256 of a 64-byte header (magic "CMFRAG01", u32 dtype
 * code 0=fp32 1=bf16, u32 element bytes, u32 L, u32 batch=1, u32 H, u64 T, u32 d,
 * zero pad; little-endian) followed by the 2L tensor roots.
 * digests_dev: device, n * 32 bytes, written in delivery order. */
int32_t cm_fragment_hash(const cm_fragset* set, uint8_t* digests_dev,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Same Id, computed only for the fragments i with select_dev[i] == select_value
 * (select_dev: device, n bytes; select_value in [0, 255]); the other digests are
 * left untouched. Two calls with complementary selections may run concurrently
 * on different streams if each has a workspace of its own. */
int32_t cm_fragment_hash_select(const cm_fragset* set, const uint8_t* select_dev,
                                int32_t select_value, uint8_t* digests_dev, void* workspace,
                                size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------- step 2
 * Score of Eq. (3) / Alg. 1: for every fragment i,
 *   keys_dev[i] = S_i = sum over heads h and rows r in [T_i - tail_len, T_i) of
 *                 || K_i^{(routing_layer)}[0, h, r, :] ||_2
 * and rho_i = S_i / (H * tail_len). tail_len is T* = min_j T_j of the set.
 * Arithmetic (identical on every device and in the CPU oracle): fp64; squares
 * exact; each row sum by a level-wise adjacent-pair tree over d; correctly
 * rounded sqrt; the H * tail_len row norms, flattened (h, r) row-major and
 * zero-padded to a power of two, summed by the same kind of tree.
 * routing_layer: 0-based, in [0, L). tail_len in [1, min_i T_i].
 * keys_dev: device, n doubles. Non-finite inputs give non-finite keys (reported
 * by cm_canonical_order). */
int32_t cm_fragment_knorm(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                          double* keys_dev, void* workspace, size_t workspace_bytes,
                          void* stream);

/* ---------------------------------------------------------------- step 3
 * Which digests the order needs (for running the rest of step 1 concurrently
 * with steps 4-5): mask_dev[i] = 1 if another fragment has a bitwise-equal key,
 * else 0. Byte-identical copies always share their key, and ties need equal
 * keys, so cm_canonical_order and cm_multiset_order read exactly these digests.
 * keys_dev: output of cm_fragment_knorm (device); mask_dev: device, n bytes. */
int32_t cm_equal_key_mask(const cm_fragset* set, const double* keys_dev, uint8_t* mask_dev,
                          void* stream);

/* Ingest dedupe (Alg. 2; Eq. (5)) and canonical order (Alg. 1): deliveries with
 * equal digests are one fragment (the first arrival is kept); the distinct
 * fragments are sorted by descending key, equal keys by descending digest read
 * as a 256-bit big-endian unsigned integer; offsets are the exclusive prefix sum
 * of the lengths in that order (§4.2). Runs on the device in one workgroup.
 * keys_dev, digests_dev: outputs of steps 1-2 (device); only the digests of
 * fragments marked by cm_equal_key_mask are read, the others may still be in
 * flight. plan_dev: device, cm_plan_elems(n) int64 (layout above). A non-finite
 * key sets plan status CM_ENONFINITE; the call itself still returns CM_OK. */
int32_t cm_canonical_order(const cm_fragset* set, const double* keys_dev,
                           const uint8_t* digests_dev, int64_t* plan_dev, void* stream);

/* The naive re-render of §5.9 (Table 10's foil): the order of
 * cm_canonical_order over every delivery, without Ingest's dedupe. Each
 * delivery gets a slot; byte-identical copies tie on key and digest and keep
 * their delivery order. Same arguments and plan layout as cm_canonical_order
 * (n_unique = n, slot_of_delivery[i] = the slot of delivery i). */
int32_t cm_multiset_order(const cm_fragset* set, const double* keys_dev,
                          const uint8_t* digests_dev, int64_t* plan_dev, void* stream);
/* BagMerge of Eq. (1)-(2) with a caller-supplied order pi (the paper's fixed
 * orders, e.g. default and swap, §4.2): slot k renders delivery order_host[k]
 * at the offset of the lengths before it; no dedupe, no scores. Host only: writes
 * the cm_plan_elems(n) int64 plan to plan_host (the caller copies it to the
 * device for cm_render_merge). order_host: host, count indices in [0, n), each
 * one delivery (a delivery may appear more than once); 1 <= count <= n.
 * slot_of_delivery[i] is the first slot rendering delivery i, or -1. */
int32_t cm_bag_plan(const cm_fragset* set, const int32_t* order_host, int32_t count,
                    int64_t* plan_host);
/* ---------------------------------------------------------------- steps 4-5
 * Eq. (1)-(2) with pi = the plan's slot order: for every layer l and head h,
 *   out K rows [s, s + T) = R(s) K_slot  (rotation in fp64, rounded to nearest
 *                                          even in the storage dtype; s = 0 is a
 *                                          byte copy)
 *   out V rows [s, s + T) = V_slot       (byte copy)
 * R(s) rotates pair (x1, x2) by s * theta_j: (x1 c - x2 sn, x2 c + x1 sn).
 * plan_dev: the plan on the device; plan_host: the same plan copied to the host
 * (the host validates it and sizes the launch from it).
 * out_dev: device, 16-byte aligned, 2 * L * H * T_out * d elements laid out as
 * [L][2][1][H][T_out][d]: layer l's K is the contiguous [1, H, T_out, d] block at
 * element offset (2l) * H * T_out * d and its V the block after it.
 * T_out must equal the plan's T_out. The plan status must be CM_OK. */
int32_t cm_render_merge(const cm_fragset* set, const int64_t* plan_dev,
                        const int64_t* plan_host, const cm_rope* rope, void* out_dev,
                        int64_t T_out, void* workspace, size_t workspace_bytes,
                        void* stream);

/* Incremental render (the lazy Render of Alg. 2 without re-rendering the whole
 * set): renders only slots [first_slot, n_unique) of the plan, i.e. rows
 * [offset of first_slot, T_out) of every row block, into a merged cache whose row
 * blocks are T_cap >= T_out rows long: out_dev laid out [L][2][1][H][T_cap][d]
 * (layer l's K is the block at element offset (2l) * H * T_cap * d, rows
 * [0, T_out) of each head in use). Rows before the first slot's offset are not
 * touched. After a fragment is inserted into a set at rank r, the slots before r
 * keep their fragments and offsets, so rendering the new plan from slot r into
 * the cache rendered for the old plan (same T_cap) gives exactly the full render.
 * plan_dev / plan_host as in cm_render_merge (T_out is the plan's);
 * 0 <= first_slot < n_unique. */
int32_t cm_render_merge_range(const cm_fragset* set, const int64_t* plan_dev,
                              const int64_t* plan_host, const cm_rope* rope, int32_t first_slot,
                              void* out_dev, int64_t T_cap, void* workspace,
                              size_t workspace_bytes, void* stream);
/* As cm_render_merge for a plan that is only on the device (e.g. just written by
 * cm_canonical_order on the same stream): nothing waits for the plan. The caller
 * gives T_out (for a set of distinct fragments, the sum of their lengths;
 * 1 <= T_out <= the sum of all lengths). Before any byte moves, the device checks
 * the plan against the set and T_out (status CM_OK, n, n_unique, each slot's
 * delivery and length, offsets as prefix sums, T_out); a plan that fails is not
 * rendered (out_dev is left untouched) and CM_ESHAPE is written into its status
 * entry plan_dev[0], which the caller reads after the stream has finished. The
 * call itself returns CM_OK for such a plan. */
int32_t cm_render_merge_devplan(const cm_fragset* set, int64_t* plan_dev, const cm_rope* rope,
                                void* out_dev, int64_t T_out, void* workspace,
                                size_t workspace_bytes, void* stream);
/* Render of Alg. 2 for a set whose members are distinct and whose Ids are
 * known (computed at Ingest): steps 2-5 in one call with nothing waiting for the
 * host. cm_fragment_knorm (keys_dev), cm_canonical_order (plan_dev) and the
 * render of cm_render_merge_devplan, with the order and the render's tables
 * built in one launch. digests_dev: n * 32 bytes, device, 16-byte aligned, the
 * members' Ids; routing_layer, tail_len as cm_fragment_knorm. T_out must be the
 * sum of all member lengths (CM_ESHAPE otherwise): out_dev holds
 * [L][2][1][H][T_out][d]. After the stream has finished the caller reads
 * plan_dev's status: CM_ENONFINITE (a score is not finite) or CM_ESHAPE (two
 * members have the same Id, so the plan's T_out is shorter) mean nothing was
 * rendered. Workspace: cm_workspace_size() bytes. */
int32_t cm_render_set(const cm_fragset* set, const uint8_t* digests_dev, int32_t routing_layer,
                      int64_t tail_len, const cm_rope* rope, double* keys_dev, int64_t* plan_dev,
                      void* out_dev, int64_t T_out, void* workspace, size_t workspace_bytes,
                      void* stream);
/* Steps 1 and 4-5 in one pass: the render of cm_render_merge and, for every
 * slot delivery i with select_dev[i] == 0, its Id (as cm_fragment_hash) written
 * to digests_dev[i]; the Id's chunk level is computed from the same loads that
 * feed the render, so each fragment byte is read once. The digests of all
 * other deliveries are left untouched (give them select 1 and compute them
 * before, e.g. with cm_fragment_hash_select: with select = the output of
 * cm_equal_key_mask, every delivery not rendered in a slot is among them).
 * select_dev: device, n bytes. Workspace: cm_workspace_size() bytes. */
int32_t cm_render_merge_hash(const cm_fragset* set, const int64_t* plan_dev,
                             const int64_t* plan_host, const cm_rope* rope,
                             const uint8_t* select_dev, uint8_t* digests_dev, void* out_dev,
                             int64_t T_out, void* workspace, size_t workspace_bytes,
                             void* stream);

/* Steps 1-5 over a batch of deliveries (Render of Alg. 2 after Ingest of each
 * delivery), enqueued on `stream` in one call with nothing waiting for the host:
 * cm_fragment_knorm (keys_dev), cm_equal_key_mask (mask_dev), the Ids of the
 * deliveries whose keys collide (cm_fragment_hash_select with mask 1), the
 * dedupe and canonical order (plan_dev, as cm_canonical_order), then the render
 * fused with every other Id (cm_render_merge_hash), reading the plan on the
 * device. The merged cache of the plan's length T_out is written to the start of
 * out_dev as [L][2][1][H][T_out][d] (each layer's K then V), so out_dev must hold
 * that for T_out = T_cap rows: T_cap >= the sum of all delivery lengths (which
 * bounds T_out) is required. After the stream has finished, the caller reads
 * plan_dev: its status (CM_ENONFINITE if a score is not finite; then nothing is
 * rendered and the digests of the non-colliding deliveries are not written), T_out,
 * the order, offsets and the slot of each delivery.
 * routing_layer, tail_len: as cm_fragment_knorm (tail_len = the smallest length
 * for Eq. (3)'s T*). keys_dev: n doubles; mask_dev: n bytes; digests_dev: n * 32
 * bytes, 16-byte aligned; plan_dev: cm_plan_elems(n) int64; all device, written by
 * the call. Workspace: cm_workspace_size() bytes, used by each stage in turn. */
int32_t cm_render_deliveries(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                             const cm_rope* rope, double* keys_dev, uint8_t* mask_dev,
                             uint8_t* digests_dev, int64_t* plan_dev, void* out_dev,
                             int64_t T_cap, void* workspace, size_t workspace_bytes,
                             void* stream);

/* cm_render_deliveries for callers that cannot allocate device memory or
 * cannot hand over a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc. Same arguments, outputs and errors as
 * cm_render_deliveries, without the workspace: the scratch is a fixed array of
 * CM_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, created when the
 * library's code object is loaded on that GPU and held until the process ends.
 * The call allocates nothing (no hipMalloc, no library allocation); its first
 * call on a device looks up that device's copy of the array. A set whose
 * workspace (cm_workspace_size) exceeds CM_NOALLOC_SCRATCH_BYTES is rejected
 * with CM_EWORKSPACE before anything is enqueued. Every call on one GPU shares
 * its array, and no stage reads scratch it has not written in the same call:
 * calls on one GPU must be ordered (one stream, or synchronised); two calls that
 * overlap on one GPU race and give undefined results. */
#define CM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int32_t cm_render_deliveries_noalloc(const cm_fragset* set, int32_t routing_layer,
                                     int64_t tail_len, const cm_rope* rope, double* keys_dev,
                                     uint8_t* mask_dev, uint8_t* digests_dev, int64_t* plan_dev,
                                     void* out_dev, int64_t T_cap, void* stream);

/* cm_render_deliveries captured into a HIP graph, for callers that repeat the
 * same merge shape (Render of Alg. 2 after Ingest; steps 1-5) and are bound by
 * kernel launches (small sets): cm_graph_launch then enqueues every kernel of
 * the call with one launch. The graph holds the call's arguments: the set's
 * device table and fragment tensors, keys_dev, mask_dev, digests_dev, plan_dev,
 * out_dev and the workspace must stay allocated, at the same addresses, until
 * cm_graph_destroy, and each launch reads the fragment tensors as they are then
 * (write new contents of the same shapes into them between launches). The
 * arguments are checked as in cm_render_deliveries (the host tables are read
 * once, here); nothing is enqueued by this call. Launches that overlap (or that
 * overlap other calls using the same buffers) race. *graph_out: an opaque
 * handle, NULL on error. */
typedef struct cm_graph cm_graph;
int32_t cm_render_deliveries_graph(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                                   const cm_rope* rope, double* keys_dev, uint8_t* mask_dev,
                                   uint8_t* digests_dev, int64_t* plan_dev, void* out_dev,
                                   int64_t T_cap, void* workspace, size_t workspace_bytes,
                                   cm_graph** graph_out);
/* Enqueue the captured kernels on `stream`. CM_EINVAL for a NULL graph. */
int32_t cm_graph_launch(cm_graph* graph, void* stream);
/* Free a graph (NULL is allowed). Launches already enqueued still run. */
int32_t cm_graph_destroy(cm_graph* graph);

/* ---------------------------------------------------------------- paged render
 * Paged KV storage (the merge as a permutation of already-allocated blocks plus
 * the RoPE rotation, §4.5): one page pool holds, for every layer and K/V, P pages
 * of B tokens of all H heads: pool laid out [L][2][P][H][B][d] (page p of layer
 * l's K is the [H][B][d] block at element offset (2l * P + p) * H * B * d; its V
 * at ((2l + 1) * P + p) * H * B * d). Fragment i is its length T_i and
 * ceil(T_i / B) page ids, the same for every layer and K/V: its row t lives in
 * row t % B of page blocks[first_i + t / B].
 * table_host / table_dev: n rows of 2 int64 {T_i, first_i}; blocks_host /
 * blocks_dev: n_blocks int32 page ids in [0, P). B is a power of two with
 * B * d * element_bytes in [1 KiB, 16 KiB]. The pool address is 16-byte aligned.
 */
typedef struct {
  int32_t n;
  int32_t L;
  int32_t H;
  int32_t d;
  int32_t dtype;     /* cm_dtype */
  int32_t block;     /* B, tokens per page */
  int64_t pages;     /* P */
  void* pool_dev;
  const int64_t* table_host;
  const int64_t* table_dev;
  const int32_t* blocks_host;
  const int32_t* blocks_dev;
  int64_t n_blocks;
} cm_pagedset;

/* Steps 1-3 on fragments that live only in the pool, enqueued with nothing
 * waiting for the host: cm_fragment_knorm's keys (keys_dev, n doubles), the mask
 * of cm_equal_key_mask (mask_dev, n bytes: 1 for a delivery whose key equals
 * another's), the Ids of the deliveries with mask 1 (digests_dev, n * 32 bytes,
 * 16-byte aligned; the same content address as the dense form's: each tensor is
 * hashed in the byte order of its [1, H, T, d] layout, Alg. 2 Id), then
 * cm_canonical_order's dedupe, order and offsets (plan_dev, cm_plan_elems(n)
 * int64), which read only those digests. The Ids of the deliveries with mask 0
 * are not written: compute them with cm_paged_hash_select(mask_dev, 0), e.g.
 * on another stream beside cm_paged_render. routing_layer, tail_len as
 * cm_fragment_knorm. Workspace: cm_paged_workspace_size() bytes. */
int32_t cm_paged_order(const cm_pagedset* set, int32_t routing_layer, int64_t tail_len,
                       double* keys_dev, uint8_t* mask_dev, uint8_t* digests_dev,
                       int64_t* plan_dev, void* workspace, size_t workspace_bytes, void* stream);

/* The Id of every paged fragment i with select_dev[i] == select_value (as
 * cm_fragment_hash_select; the other digests are left untouched).
 * workgroups_per_cu: the chunk kernel's persistent grid per compute unit, 0 for
 * the default (4); fewer leave room for a kernel running beside it on another
 * stream, such as the paged render. It reads the pool and writes only
 * digests_dev and its workspace, so it may run concurrently with
 * cm_paged_render over the same set (which writes only fresh pages) if the two
 * have separate workspaces. Workspace: cm_paged_workspace_size() bytes. */
int32_t cm_paged_hash_select(const cm_pagedset* set, const uint8_t* select_dev,
                             int32_t select_value, uint8_t* digests_dev, int32_t workgroups_per_cu,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Block tables of the merged cache for a plan over the paged fragments (any plan
 * of this file's layout whose slots index the paged set's fragments, e.g. from
 * cm_canonical_order over the same fragments or cm_bag_plan). Merged block j
 * holds rows [jB, min(jB + B, T_out)). It reuses a fragment page, with no copy,
 * when all its rows come from one slot s, start at a page boundary of that
 * fragment (jB - offset_s a multiple of B) and, for K, offset_s = 0 (R(0) = I);
 * otherwise it gets the next page of free_host, to be written by
 * cm_paged_render. Outputs (host, ceil(T_out / B) entries each): k_table_host,
 * v_table_host (page ids); fresh_host: the fresh pages to write as codes
 * 2j + kv (at most 2 ceil(T_out / B) entries; K pages first, each kind in
 * ascending page id), their count in *n_fresh.
 * Host only. CM_EINVAL if free_host has fewer than the pages needed (*n_fresh
 * then holds the number needed). */
int32_t cm_paged_tables(const cm_pagedset* set, const int64_t* plan_host, const int32_t* free_host,
                        int64_t n_free, int32_t* k_table_host, int32_t* v_table_host,
                        int32_t* fresh_host, int64_t* n_fresh);
/* Writes the fresh pages of cm_paged_tables: for each code 2j + kv of fresh_dev
 * (device, n_fresh int32), every layer and head, rows [jB, min(jB + B, T_out)) of
 * the merged cache into page (kv ? v_table : k_table)[j] — K of a slot at offset
 * s rotated by R(s) as in cm_render_merge, V copied; rows past T_out in the last
 * page are left untouched. Pages not listed are neither read as destinations
 * nor written. k_table_dev, v_table_dev: device copies of the tables.
 * plan_dev / plan_host as in cm_render_merge. Workspace: cm_paged_workspace_size()
 * bytes. */
int32_t cm_paged_render(const cm_pagedset* set, const int64_t* plan_dev, const int64_t* plan_host,
                        const cm_rope* rope, const int32_t* k_table_dev,
                        const int32_t* v_table_dev, const int32_t* fresh_dev, int64_t n_fresh,
                        void* workspace, size_t workspace_bytes, void* stream);
/* Steps 1 and 4-5 in one pass over paged storage (§4.5; Alg. 2 Id; Eq. (1)-(2)),
 * the paged counterpart of cm_render_merge_hash: every row of the plan's merged
 * cache whose page in the block tables is not the page it is read from is
 * written there (K of a slot at offset s rotated by R(s), V copied), rows in a
 * reused fragment page stay in place, rows past T_out in the last page are left
 * untouched; from the same loads, the Id of every slot delivery i with
 * select_dev[i] == 0 is written to digests_dev (the others are left untouched;
 * with the mask of cm_paged_order, the deliveries whose Id it did not compute).
 * The result equals cm_paged_render with the same tables plus
 * cm_paged_hash_select(select_dev, 0), with each byte read once.
 * k_table_host / v_table_host: the block tables (ceil(T_out / B) page ids each,
 * e.g. from cm_paged_tables), checked on the host: every entry a page of the
 * pool, a fragment page only where cm_paged_tables would reuse it, no other
 * page twice (CM_EINVAL otherwise); k_table_dev / v_table_dev: their device
 * copies, read by the kernel. select_dev: device, n bytes; digests_dev: n * 32
 * bytes, 16-byte aligned. plan_dev / plan_host as in cm_render_merge.
 * P * H * B must not exceed 2^32 - 1 (CM_ESHAPE; the kernel names a pool row
 * with 32 bits). Workspace: cm_paged_workspace_size() bytes. */
int32_t cm_paged_render_hash(const cm_pagedset* set, const int64_t* plan_dev,
                             const int64_t* plan_host, const cm_rope* rope,
                             const int32_t* k_table_host, const int32_t* v_table_host,
                             const int32_t* k_table_dev, const int32_t* v_table_dev,
                             const uint8_t* select_dev, uint8_t* digests_dev, void* workspace,
                             size_t workspace_bytes, void* stream);
/* Steps 1-5 over paged storage in one call with nothing waiting for the host
 * (Render of Alg. 2 over deliveries that live only in the pool, §4.5): the steps
 * of cm_paged_order (keys_dev, mask_dev, the colliding deliveries' digests,
 * plan_dev), the merged K and V block tables built on the device by
 * cm_paged_tables' rule from the free pages in list order (k_table_dev,
 * v_table_dev; *n_fresh_dev = the free pages taken), then cm_paged_render_hash
 * with them and mask_dev (every other Id). After the stream has finished the
 * caller reads plan_dev (status, T_out, order, offsets, slots) and the first
 * ceil(T_out / B) entries of each table. A plan status of CM_ENONFINITE (a score
 * is not finite) or CM_EINVAL (the free list is shorter than the render needs;
 * *n_fresh_dev then holds the number needed) means nothing was rendered and the
 * non-colliding Ids were not written.
 * free_host / free_dev: n_free page ids (host, checked: pages of the pool,
 * distinct, no fragment page; and its device copy). k_table_dev, v_table_dev:
 * device, ceil(sum of the lengths / B) int32 each; n_fresh_dev: device, one
 * int64. Other arguments as cm_paged_order and cm_paged_render_hash (the same
 * P * H * B limit). Workspace: cm_paged_workspace_size() bytes. */
int32_t cm_paged_deliveries(const cm_pagedset* set, int32_t routing_layer, int64_t tail_len,
                            const cm_rope* rope, const int32_t* free_host,
                            const int32_t* free_dev, int64_t n_free, double* keys_dev,
                            uint8_t* mask_dev, uint8_t* digests_dev, int64_t* plan_dev,
                            int32_t* k_table_dev, int32_t* v_table_dev, int64_t* n_fresh_dev,
                            void* workspace, size_t workspace_bytes, void* stream);
int32_t cm_paged_workspace_size(const cm_pagedset* set, size_t* bytes_out);

/* ---------------------------------------------------------------- timing
 * Optional per-kernel timing with HIP events recorded on the launch stream
 * around every kernel this library enqueues (off by default; a process-wide
 * switch). cm_timing_query waits for the recorded events, adds their durations
 * to the per-kernel totals and returns the total milliseconds and launch count
 * for one kernel name ("hash_prep", "hash_leaf", "hash_parent", "hash_final",
 * "knorm_rows", "knorm_tree", "order", "key_mask", "render_prep", "render",
 * "render_hash", "paged", "paged_hash_render"). */
int32_t cm_timing_enable(int32_t on);
int32_t cm_timing_reset(void);
int32_t cm_timing_query(const char* kernel, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* CMERGE_H */
