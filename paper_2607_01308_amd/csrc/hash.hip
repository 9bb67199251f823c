// Step 1 — content address Id of Alg. 2 (also the hash tiebreak of §4.3).
//
// Per tensor, BLAKE3-256 of its raw bytes in memory order; per fragment,
// BLAKE3-256 of a 64-byte shape/dtype header followed by the 2L tensor roots
// (K^0, V^0, ..., K^{L-1}, V^{L-1}). One wave takes one stripe of 64
// consecutive BLAKE3 chunks (64 KiB) and lane k hashes chunk k of it: 16
// dependent compressions, each 64-byte block loaded as four 16-byte pieces (the
// lanes' loads are 1 KiB apart, so each lane reads whole 64-byte halves of
// cache lines and the other half one block later), two blocks ahead of the
// compression. The work is VALU-bound (12 VALU ops per G step, 672 per block);
// the tree above the chunks takes one launch per three levels over all tensors
// at full lane occupancy (the parents add 1/16 of the chunk work) until at most
// nine levels remain, then one launch folds the top of every tensor's tree (and,
// for a small set, computes each fragment's Id in its last workgroup; otherwise
// one more launch does). Fragments stored in a page pool are hashed by a chunk
// kernel that walks each chunk's blocks through the page list in the order of
// the dense layout, so the Id does not depend on the storage.
#include "blake3_quad.h"
#include "chunk_ops.h"
#include "key_mask.h"
#include "knorm_fold.h"

namespace cm {

namespace {

constexpr int kBlock = 256;
// Grid of CUs x CM_HASH_BLOCKS_PER_CU workgroups of 4 waves (3 fit on a SIMD at
// this kernel's register count); measured on 2.7 GB of hashing: 2 per CU
// 1.10 ms, 3 per CU 1.06 ms, 4 per CU 1.03 ms.
#ifndef CM_HASH_BLOCKS_PER_CU
#define CM_HASH_BLOCKS_PER_CU 4
#endif
constexpr int kLeafBlocksPerCu = CM_HASH_BLOCKS_PER_CU;

// Largest i in [0, n) with base[i] <= g (bases strictly increase).
__device__ __forceinline__ int find_fragment(const int64_t* __restrict__ base, int n, int64_t g) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (base[mid] <= g) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// base[v][i] = number of level-v nodes of fragments 0..i-1 (all 2L tensors each);
// base[v][n] = total nodes at level v; row levels+1 holds the same prefix sums
// of the (tensor, stripe) tasks of the chunk kernel. One workgroup. For n <= 64
// each row gets a thread that walks the fragments in order, all rows at once;
// more fragments take a block-wide inclusive scan per row.
__device__ __forceinline__ void hash_tables(const int64_t* __restrict__ table, int32_t n,
                                            int64_t stride, int64_t token_bytes, int32_t L,
                                            int32_t levels, int64_t* __restrict__ base,
                                            int32_t* __restrict__ arrived) {
  __shared__ int64_t sc[1024];
  const int tid = threadIdx.x;
  if (tid < n) arrived[tid] = 0;
  if (n <= 64) {
    if (tid < n) sc[tid] = table[(int64_t)tid * stride] * token_bytes;
    __syncthreads();
    for (int v = tid; v <= levels + 1; v += (int)blockDim.x) {
      int64_t* row = base + (int64_t)v * (n + 1);
      int64_t acc = 0;
      for (int i = 0; i < n; ++i) {
        const int64_t bytes = sc[i];
        row[i] = acc;
        acc += 2 * (int64_t)L * (v <= levels ? nodes_at(chunks_of(bytes), v) : stripes_of(bytes));
      }
      row[n] = acc;
    }
    __syncthreads();
    return;
  }
  const int64_t bytes = tid < n ? table[(int64_t)tid * stride] * token_bytes : 0;
  const int64_t m0 = tid < n ? chunks_of(bytes) : 0;
  for (int v = 0; v <= levels + 1; ++v) {
    const int64_t per = v <= levels ? nodes_at(m0, v) : stripes_of(bytes);
    const int64_t x = tid < n ? 2 * (int64_t)L * per : 0;
    sc[tid] = x;
    __syncthreads();
    for (int off = 1; off < (int)blockDim.x; off <<= 1) {
      const int64_t t = tid >= off ? sc[tid - off] : 0;
      __syncthreads();
      sc[tid] += t;
      __syncthreads();
    }
    int64_t* row = base + (int64_t)v * (n + 1);
    if (tid < n) row[tid] = sc[tid] - x;
    if (tid == (int)blockDim.x - 1) row[n] = sc[tid];
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void hash_prep_kernel(const int64_t* __restrict__ table,
                                                         int32_t n, int64_t stride,
                                                         int64_t token_bytes, int32_t L,
                                                         int32_t levels,
                                                         int64_t* __restrict__ base,
                                                         int32_t* __restrict__ arrived) {
  hash_tables(table, n, stride, token_bytes, L, levels, base, arrived);
}

// The last levels of the scores (count > 1), the key mask and the node-base
// tables in one launch (the tables depend only on the lengths). The score
// partials may share workspace with the tables: the fold reads all of them
// into LDS before a table entry is written.
__global__ __launch_bounds__(1024) void mask_hash_prep_kernel(
    const int64_t* __restrict__ table, int32_t n, int64_t stride, int64_t token_bytes, int32_t L,
    int32_t levels, const double* parts, int64_t count, KnormDirect kd, int32_t H, int32_t d,
    double* keys, uint8_t* __restrict__ mask, int64_t* base, int32_t* __restrict__ arrived) {
  knorm_finish(table, stride, n, H, d, kd, parts, count, keys);
  equal_key_mask_body(n, keys, mask);
  hash_tables(table, n, stride, token_bytes, L, levels, base, arrived);
}

// One wave = one (tensor, stripe) task at a time: lane k hashes chunk k of the
// stripe, 1 KiB of consecutive bytes (the tensor's last chunk may be shorter,
// lanes past it idle). The grid is bounded (a few workgroups per CU) and strides
// over all tasks.
__global__ __launch_bounds__(kBlock) void hash_chunk_kernel(const int64_t* __restrict__ table,
                                                            int32_t n, int64_t stride,
                                                            int64_t token_bytes,
                                                            const int64_t* __restrict__ base0,
                                                            const int64_t* __restrict__ task_base,
                                                            int64_t total_tasks,
                                                            const uint8_t* __restrict__ select,
                                                            uint32_t want,
                                                            uint8_t* __restrict__ nodes) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
  const int64_t waves = (int64_t)gridDim.x * (kBlock / 64);
  for (int64_t task = (int64_t)blockIdx.x * (kBlock / 64) + wave; task < total_tasks;
       task += waves) {
    const int i = find_fragment(task_base, n, task);
    if (select && select[i] != want) continue;
    const int64_t bytes = table[(int64_t)i * stride] * token_bytes;
    const int64_t stripes = stripes_of(bytes);
    const int64_t m = chunks_of(bytes);
    const int64_t local = task - task_base[i];
    const int64_t t = local / stripes;
    const int64_t sidx = local - t * stripes;
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const uint64_t chunk0 = (uint64_t)sidx * kStripeChunks;
    const uint8_t* p = reinterpret_cast<const uint8_t*>(table[(int64_t)i * stride + 1 + t]) +
                       ((sidx * kStripeBlocks) << 6);
    B3Cv s;
    if (!hash_lane_chunk(s, p, in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks, lane,
                         chunk0, m == 1))
      continue;
    store_cv(nodes + (base0[i] + t * m + (int64_t)chunk0 + lane) * 32, s);
  }
}

// The chunk kernel for fragments in a paged pool ([L][2][P][H][B][d]; the
// fragment's row t in row t % B of page blocks[first + t / B]). The Id is the
// same content address as for the dense form, so each tensor's bytes are hashed
// in the order of its dense [1, H, T, d] layout: lane k of a stripe walks chunk
// k's blocks row by row through the pages (a 64-byte block never straddles a
// row, rows being 64-byte multiples).
__global__ __launch_bounds__(kBlock) void paged_hash_chunk_kernel(
    const uint8_t* __restrict__ pool, int64_t P, int32_t H, int32_t b_shift, int32_t rb_shift,
    const int64_t* __restrict__ table, const int32_t* __restrict__ blocks, int32_t n,
    int64_t token_bytes, const int64_t* __restrict__ base0, const int64_t* __restrict__ task_base,
    int64_t total_tasks, const uint8_t* __restrict__ select, uint32_t want,
    uint8_t* __restrict__ nodes) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
  const int64_t waves = (int64_t)gridDim.x * (kBlock / 64);
  const int64_t rb = (int64_t)1 << rb_shift;
  const int64_t bmask = ((int64_t)1 << b_shift) - 1;
  for (int64_t task = (int64_t)blockIdx.x * (kBlock / 64) + wave; task < total_tasks;
       task += waves) {
    const int i = find_fragment(task_base, n, task);
    if (select && select[i] != want) continue;
    const int64_t T = table[2 * (int64_t)i];
    const int64_t first = table[2 * (int64_t)i + 1];
    const int64_t bytes = T * token_bytes;
    const int64_t stripes = stripes_of(bytes);
    const int64_t m = chunks_of(bytes);
    const int64_t local = task - task_base[i];
    const int64_t t = local / stripes;                 // tensor 2l + kv
    const int64_t sidx = local - t * stripes;
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const int64_t stripe_blocks = in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks;
    const int64_t b0 = (int64_t)lane * kB3ChunkBlocks;
    if (b0 >= stripe_blocks) continue;                 // lane past the tensor's last chunk
    const int64_t nb = stripe_blocks - b0 < kB3ChunkBlocks ? stripe_blocks - b0 : kB3ChunkBlocks;
    const int64_t c = sidx * kStripeChunks + lane;     // chunk index in the tensor
    // dense byte 1024 c = head h, row tr, column col
    const int64_t o = c << 10;
    int64_t h = o / (T << rb_shift);
    const int64_t r = o - h * (T << rb_shift);
    int64_t tr = r >> rb_shift;
    int64_t col = r & (rb - 1);
    // b3_chunk asks for the chunk's blocks in order, one call each
    auto load = [&](int64_t, uint32_t (&w)[16]) {
      const int64_t page = blocks[first + (tr >> b_shift)];
      const int64_t row = ((((t * P + page) * H + h) << b_shift) + (tr & bmask));
      load_block64(pool + (row << rb_shift) + col, w);
      col += 64;
      if (col == rb) {
        col = 0;
        if (++tr == T) {
          tr = 0;
          ++h;
        }
      }
    };
    B3Cv st;
    b3_chunk(st, nb, (uint64_t)c, m == 1, load);
    store_cv(nodes + (base0[i] + t * m + c) * 32, st);
  }
}

constexpr int kSubLevels = 3;
constexpr int kSubLanes = 64;

// Fold one lane's cur (1 .. 2^K) consecutive level-v0 nodes at c (32 bytes each)
// into their level-(v0 + K) node, level by level in the lane's own LDS slots
// (word w of the lane's node p at [p * 8 + w][lane]: consecutive lanes hit
// consecutive banks). The first level is folded straight from the children in
// memory, so the slots hold at most half of them. m0: the tensor's chunk count,
// which places ROOT on the compression that leaves the tensor one node.
__device__ __forceinline__ void fold_children(const uint8_t* c, int cur, int64_t m0, int v0, int K,
                                              uint32_t (*lds)[kSubLanes], int lane,
                                              uint32_t (&w)[8]) {
  for (int lev = 1; lev <= K; ++lev) {
    const uint32_t flags = kB3Parent | (nodes_at(m0, v0 + lev) == 1 ? kB3Root : 0u);
    const int nn = (cur + 1) >> 1;
    for (int p = 0; p < nn; ++p) {
      uint32_t m[16];
      const bool pair = 2 * p + 1 < cur;
      if (lev == 1) {
        // children 2p and 2p + 1 (an unpaired last child alone)
        const uint4* q = reinterpret_cast<const uint4*>(c + (int64_t)(2 * p) * 32);
        const int words = pair ? 4 : 2;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (k < words) {
            const uint4 v = q[k];
            m[4 * k + 0] = v.x;
            m[4 * k + 1] = v.y;
            m[4 * k + 2] = v.z;
            m[4 * k + 3] = v.w;
          }
        }
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) m[k] = lds[2 * p * 8 + k][lane];
        if (pair) {
#pragma unroll
          for (int k = 0; k < 8; ++k) m[8 + k] = lds[(2 * p + 1) * 8 + k][lane];
        }
      }
      if (pair) {
        B3Cv cv;
        b3_init(cv);
        b3_compress(cv, m, 0, 64, flags);
#pragma unroll
        for (int k = 0; k < 8; ++k) m[k] = cv.h[k];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) lds[p * 8 + k][lane] = m[k];
    }
    cur = nn;
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) w[k] = lds[k][lane];
}

// Tree levels v0+1 .. v0+K (K <= kSubLevels) of every tensor in one launch:
// lane g computes node g of level v0+K (numbered over all tensors) from its up to
// 2^K children at level v0, level by level in the lane's own LDS slots. Node j
// of a level is the BLAKE3 parent of children 2j and 2j+1 of the level below (ROOT
// on the compression that leaves the tensor one node); an unpaired last child
// is carried up unchanged. Pairing level by level this way builds BLAKE3's
// left-balanced tree: every complete subtree of 2^v chunks starts at a multiple
// of 2^v and the unpaired tail joins at the level where it has a sibling. A lane
// does up to 2^K - 1 dependent compressions, so a launch covers K levels at full
// lane occupancy and the level below is read once.
__global__ __launch_bounds__(kSubLanes) void hash_subtree_kernel(
    const int64_t* __restrict__ table, int32_t n, int64_t stride, int64_t token_bytes, int32_t v0,
    int32_t K, const int64_t* __restrict__ base_lo, const int64_t* __restrict__ base_hi,
    int64_t total_hi, const uint8_t* __restrict__ select, uint32_t want,
    const uint8_t* __restrict__ in, uint8_t* __restrict__ out) {
  __shared__ uint32_t lds[(1 << (kSubLevels - 1)) * 8][kSubLanes];
  const int lane = threadIdx.x;
  const int64_t g = (int64_t)blockIdx.x * kSubLanes + lane;
  if (g >= total_hi) return;
  const int i = find_fragment(base_hi, n, g);
  if (select && select[i] != want) return;
  const int64_t m0 = chunks_of(table[(int64_t)i * stride] * token_bytes);
  const int64_t m_lo = nodes_at(m0, v0);
  const int64_t m_hi = nodes_at(m0, v0 + K);
  const int64_t local = g - base_hi[i];
  const int64_t t = local / m_hi;
  const int64_t j = local - t * m_hi;
  const int64_t first = j << K;
  const int cur = (int)(m_lo - first < ((int64_t)1 << K) ? m_lo - first : ((int64_t)1 << K));
  uint32_t w[8];
  fold_children(in + (base_lo[i] + t * m_lo + first) * 32, cur, m0, v0, K, lds, lane, w);
  uint4* o = reinterpret_cast<uint4*>(out + g * 32);
  o[0] = make_uint4(w[0], w[1], w[2], w[3]);
  o[1] = make_uint4(w[4], w[5], w[6], w[7]);
}

// Fold cnt (>= 1) chaining values held in LDS (word w of value p at
// [p * 8 + w][lane slot], lds_w words apart per value) into one, level by level:
// value j of a level is the BLAKE3 parent of values 2j and 2j+1 of the level
// below, an unpaired last value is carried up. ROOT marks the final compression
// when root is set. All 64 lanes of the (one-wave) workgroup take part. A level
// of at most 16 values is made by quads (b3_compress_quad: value j by lanes
// 4j .. 4j + 3), which shortens the chain of dependent compressions about 2x;
// a wider level takes one lane per value.
__device__ __forceinline__ void fold_cvs(uint32_t* lds, int cnt, bool root, int lane) {
  const int Q = lane >> 2;
  const int q = lane & 3;
  while (cnt > 1) {
    const int nn = (cnt + 1) >> 1;
    const uint32_t flags = kB3Parent | (root && nn == 1 ? kB3Root : 0u);
    if (nn <= 16) {
      uint32_t m[16];
      uint32_t lo = 0, hi = 0;
      const bool pair = Q < nn && 2 * Q + 1 < cnt;   // uniform over the quad
      if (pair) {
#pragma unroll
        for (int k = 0; k < 16; ++k) m[k] = lds[(2 * Q) * 8 + k];
      } else if (Q < nn) {
        lo = lds[(2 * Q) * 8 + q];
        hi = lds[(2 * Q) * 8 + 4 + q];
      }
      __syncthreads();
      if (pair) {
        b3_init_quad(lo, hi, (q & 1) != 0, (q & 2) != 0);
        b3_compress_quad(lo, hi, m, 0, 64, flags, (q & 1) != 0, (q & 2) != 0);
      }
      if (Q < nn) {
        lds[Q * 8 + q] = lo;
        lds[Q * 8 + 4 + q] = hi;
      }
      __syncthreads();
      cnt = nn;
      continue;
    }
    uint32_t m[16];
    const bool pair = lane < nn && 2 * lane + 1 < cnt;
    const bool copy = lane < nn && 2 * lane + 1 >= cnt;
    if (lane < nn) {
#pragma unroll
      for (int k = 0; k < 8; ++k) m[k] = lds[(2 * lane) * 8 + k];
      if (pair) {
#pragma unroll
        for (int k = 0; k < 8; ++k) m[8 + k] = lds[(2 * lane + 1) * 8 + k];
      }
    }
    __syncthreads();
    if (pair) {
      B3Cv cv;
      b3_init(cv);
      b3_compress(cv, m, 0, 64, flags);
#pragma unroll
      for (int k = 0; k < 8; ++k) lds[lane * 8 + k] = cv.h[k];
    } else if (copy) {
#pragma unroll
      for (int k = 0; k < 8; ++k) lds[lane * 8 + k] = m[k];
    }
    __syncthreads();
    cnt = nn;
  }
}

// Id = BLAKE3-256(header || root(K^0) || root(V^0) || ...) of fragment i by
// one 64-lane workgroup. The message is L + 1 blocks (the header, then per
// layer the pair of roots K, V) in C = ceil((L + 1) / 16) chunks. Lane k hashes
// chunk 64 g + k of each group g of 64 chunks; a full group is an aligned
// complete subtree of BLAKE3's left-balanced tree and is folded into one value,
// the last group into the value of its own subtree (carries included); then the
// group values are folded. ROOT marks the single chunk (C = 1) or the last
// compression.
constexpr int kFinalGroups = 32;   // 32 x 64 chunks: L + 1 <= 32768 blocks

struct IdShape {
  int32_t L, H, d;
  uint32_t dtype_code, esize;
};

__device__ __forceinline__ void fragment_id(uint64_t T, const IdShape& sh,
                                            const uint8_t* __restrict__ r,
                                            uint8_t* __restrict__ digest, int lane) {
  __shared__ uint32_t chunk_cv[64 * 8];
  __shared__ uint32_t group_cv[kFinalGroups * 8];
  const int64_t blocks = (int64_t)sh.L + 1;
  const int64_t chunks = (blocks + kB3ChunkBlocks - 1) / kB3ChunkBlocks;
  const int groups = (int)((chunks + 63) / 64);
  auto load = [&](int64_t g, uint32_t (&w)[16]) {
    if (g == 0) {
      const uint32_t h[16] = {0x52464D43u, 0x31304741u,  // "CMFRAG01"
                              sh.dtype_code, sh.esize, (uint32_t)sh.L, 1u, (uint32_t)sh.H,
                              (uint32_t)T, (uint32_t)(T >> 32), (uint32_t)sh.d,
                              0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
      for (int k = 0; k < 16; ++k) w[k] = h[k];
    } else {
      load_block64(r + (g - 1) * 64, w);
    }
  };
  if (chunks <= 16) {
    // up to 255 layers: quad j hashes chunk j (b3_chunk_quad), a chain of at
    // most 16 compressions of about half the latency of one lane's
    const int Q = lane >> 2;
    const int q = lane & 3;
    if (Q < chunks) {
      const int64_t g0 = (int64_t)Q * kB3ChunkBlocks;
      const int64_t nb = blocks - g0 < kB3ChunkBlocks ? blocks - g0 : kB3ChunkBlocks;
      uint32_t lo, hi;
      b3_chunk_quad(lo, hi, nb, (uint64_t)Q, chunks == 1, (q & 1) != 0, (q & 2) != 0,
                    [&](int64_t b, uint32_t (&w)[16]) { load(g0 + b, w); });
      chunk_cv[Q * 8 + q] = lo;
      chunk_cv[Q * 8 + 4 + q] = hi;
    }
    __syncthreads();
    fold_cvs(chunk_cv, (int)chunks, true, lane);
    if (lane < 8) reinterpret_cast<uint32_t*>(digest)[lane] = chunk_cv[lane];
    return;
  }
  for (int g = 0; g < groups; ++g) {
    const int64_t c = (int64_t)g * 64 + lane;
    const int cnt = (int)(chunks - (int64_t)g * 64 < 64 ? chunks - (int64_t)g * 64 : 64);
    if (c < chunks) {
      const int64_t g0 = c * kB3ChunkBlocks;
      const int64_t nb = blocks - g0 < kB3ChunkBlocks ? blocks - g0 : kB3ChunkBlocks;
      B3Cv cv;
      b3_chunk(cv, nb, (uint64_t)c, chunks == 1,
               [&](int64_t b, uint32_t (&w)[16]) { load(g0 + b, w); });
#pragma unroll
      for (int k = 0; k < 8; ++k) chunk_cv[lane * 8 + k] = cv.h[k];
    }
    __syncthreads();
    fold_cvs(chunk_cv, cnt, groups == 1, lane);
    if (lane < 8) group_cv[g * 8 + lane] = chunk_cv[lane];
    __syncthreads();
  }
  fold_cvs(group_cv, groups, true, lane);
  if (lane < 8) reinterpret_cast<uint32_t*>(digest)[lane] = group_cv[lane];
}

// The top of every tensor's tree in one launch, one 64-lane workgroup per
// (tensor t, fragment i): its m <= 64 x 8 nodes of level v0 are folded in runs
// of r consecutive ones per lane (r the smallest power of two with m <= 64 r:
// an aligned complete subtree, or the tail of the level with its carries), then
// the lane values level by level across the workgroup, so the chain of
// dependent compressions is about log2(m) long; the root goes to node
// base_top[i] + t of the top level.
constexpr int kTailLevels = kSubLevels + 6;   // 2^3 nodes per lane x 64 lanes
// Largest tail grid (2L x n workgroups) whose last workgroups compute the Ids
// (Tiny 8, Qwen3-1.7B N=2 112; measured at 2304 on the Qwen3-4B large set, the
// fences cost about 0.1 ms more than the Id launch).
constexpr int64_t kFuseIdMaxGroups = 256;

//
// With `arrived` (small sets): the workgroup that writes the last of fragment
// i's 2L roots then computes its Id (fragment_id), which saves the Id launch.
// Each workgroup makes its root visible device-wide and counts itself in
// arrived[i] (zeroed by the node-table kernel of the same call); the one that
// sees 2L - 1 arrivals before its own reads every root (after an acquire fence)
// and resets the counter for a later pass. The release fence writes back the
// XCD's L2, which across thousands of workgroups costs more than the launch it
// saves, so large sets take the separate Id kernel.
__global__ __launch_bounds__(kSubLanes) void hash_tail_kernel(
    const int64_t* __restrict__ table, int64_t stride, int64_t token_bytes, int32_t v0,
    const int64_t* __restrict__ base_lo, const int64_t* __restrict__ base_top,
    const uint8_t* __restrict__ select, uint32_t want, const uint8_t* __restrict__ in,
    uint8_t* out, IdShape sh, int32_t* __restrict__ arrived, uint8_t* __restrict__ digests) {
  __shared__ uint32_t lds[(1 << (kSubLevels - 1)) * 8][kSubLanes];
  __shared__ uint32_t vals[kSubLanes * 8];
  __shared__ int32_t seen;
  const int t = blockIdx.x;
  const int i = blockIdx.y;
  const int lane = threadIdx.x;
  if (select && select[i] != want) return;   // uniform over the workgroup
  const int64_t m0 = chunks_of(table[(int64_t)i * stride] * token_bytes);
  const int64_t m = nodes_at(m0, v0);                  // <= 2^kTailLevels (checked by the host)
  int K = 0;                                           // r = 2^K nodes per lane
  while (K < kSubLevels && m > ((int64_t)kSubLanes << K)) ++K;
  const int cnt = (int)nodes_at(m, K);                 // lane values, <= 64
  if (lane < cnt) {
    const int64_t first = (int64_t)lane << K;
    const uint8_t* c = in + (base_lo[i] + t * m + first) * 32;
    uint32_t w[8];
    if (K == 0) {
      const uint4* q = reinterpret_cast<const uint4*>(c);
      const uint4 a = q[0], b = q[1];
      w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
      w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
    } else {
      const int cur = (int)(m - first < ((int64_t)1 << K) ? m - first : ((int64_t)1 << K));
      fold_children(c, cur, m0, v0, K, lds, lane, w);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) vals[lane * 8 + k] = w[k];
  }
  __syncthreads();
  fold_cvs(vals, cnt, true, lane);
  if (lane < 8) reinterpret_cast<uint32_t*>(out + (base_top[i] + t) * 32)[lane] = vals[lane];
  if (!arrived) return;                  // the Ids come from hash_final_kernel
  __threadfence();                       // release this root to the other workgroups
  __syncthreads();
  if (lane == 0) seen = atomicAdd(&arrived[i], 1);
  __syncthreads();
  if (seen != 2 * sh.L - 1) return;      // uniform over the workgroup
  __threadfence();                       // acquire the other workgroups' roots
  fragment_id((uint64_t)table[(int64_t)i * stride], sh, out + base_top[i] * 32,
              digests + (int64_t)i * 32, lane);
  if (lane == 0) arrived[i] = 0;
}

// The Id alone (every tensor of the set is a single chunk, so there is no tail
// launch to compute it), one workgroup per fragment.
__global__ __launch_bounds__(64) void hash_final_kernel(
    const int64_t* __restrict__ table, int64_t stride, IdShape sh,
    const int64_t* __restrict__ base_last, const uint8_t* __restrict__ select, uint32_t want,
    const uint8_t* __restrict__ roots, uint8_t* __restrict__ digests) {
  const int i = blockIdx.x;
  if (select && select[i] != want) return;   // uniform over the workgroup
  fragment_id((uint64_t)table[(int64_t)i * stride], sh, roots + base_last[i] * 32,
              digests + (int64_t)i * 32, threadIdx.x);
}

}  // namespace

HashLayout hash_layout(const SetDesc& s) {
  HashLayout lay{};
  int64_t max_m0 = 1;
  for (int i = 0; i < s.n; ++i) {
    lay.tasks += 2 * (int64_t)s.L * stripes_of(s.T(i) * token_bytes_of(s));
    const int64_t m0 = chunks_of(s.T(i) * token_bytes_of(s));
    if (m0 > max_m0) max_m0 = m0;
    lay.total0 += 2 * (int64_t)s.L * m0;
    lay.total1 += 2 * (int64_t)s.L * nodes_at(m0, 1);
  }
  while (((int64_t)1 << lay.levels) < max_m0) ++lay.levels;
  if (lay.levels == 0) lay.total1 = 0;
  size_t off = 0;
  lay.off_tables = off;
  off = align_up(off + sizeof(int64_t) * (size_t)(lay.levels + 2) * (size_t)(s.n + 1), kWsAlign);
  lay.off_arrived = off;
  off = align_up(off + sizeof(int32_t) * (size_t)s.n, kWsAlign);
  lay.off_buf0 = off;
  off = align_up(off + 32 * (size_t)lay.total0, kWsAlign);
  lay.off_buf1 = off;
  off = align_up(off + 32 * (size_t)lay.total1, kWsAlign);
  lay.bytes = off;
  return lay;
}

hipError_t launch_hash_prep(const SetDesc& s, const HashLayout& lay, uint8_t* ws,
                            hipStream_t stream) {
  ScopedTiming tm(K_HASH_PREP, stream);
  int threads = 64;
  while (threads < s.n) threads <<= 1;
  hipLaunchKernelGGL(hash_prep_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev, s.n,
                     s.stride, token_bytes_of(s), s.L, lay.levels,
                     reinterpret_cast<int64_t*>(ws + lay.off_tables),
                     reinterpret_cast<int32_t*>(ws + lay.off_arrived));
  return hipGetLastError();
}

hipError_t launch_hash_tree(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                            uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream) {
  int64_t* base = reinterpret_cast<int64_t*>(ws + lay.off_tables);
  // level 0 is in buf0; each launch reads one buffer and writes the other
  // (buf1 holds every level it receives: they are no larger than level 1)
  uint8_t* buf[2] = {ws + lay.off_buf0, ws + lay.off_buf1};
  const int64_t nb1 = s.n + 1;
  hipError_t e = hipSuccess;
  int launch = 0;
  int v0 = 0;
  // three levels per launch over all tensors while more than kTailLevels remain
  // (every tensor then has at most 2^kTailLevels nodes), then the rest at once
  for (; lay.levels - v0 > kTailLevels; v0 += kSubLevels, ++launch) {
    const int K = kSubLevels;
    int64_t total = 0;
    for (int i = 0; i < s.n; ++i)
      total += 2 * (int64_t)s.L * nodes_at(chunks_of(s.T(i) * token_bytes_of(s)), v0 + K);
    ScopedTiming tm(K_HASH_PARENT, stream);
    const int64_t grid = (total + kSubLanes - 1) / kSubLanes;
    hipLaunchKernelGGL(hash_subtree_kernel, dim3((uint32_t)grid), dim3(kSubLanes), 0, stream,
                       s.table_dev, s.n, s.stride, token_bytes_of(s), v0, K, base + v0 * nb1,
                       base + (v0 + K) * nb1, total, select, want, buf[launch & 1],
                       buf[(launch + 1) & 1]);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // the cm_dtype value doubles as the header's dtype code
  const IdShape sh{s.L, s.H, s.d, (uint32_t)s.dtype, (uint32_t)s.esize};
  int32_t* arrived = reinterpret_cast<int32_t*>(ws + lay.off_arrived);
  if (v0 < lay.levels) {
    // the top levels of every tensor; for a small set also each fragment's Id, in
    // the workgroup that finishes its last root
    const bool fuse_id = (int64_t)2 * s.L * s.n <= kFuseIdMaxGroups;
    {
      ScopedTiming tm(K_HASH_PARENT, stream);
      hipLaunchKernelGGL(hash_tail_kernel, dim3((uint32_t)(2 * s.L), (uint32_t)s.n),
                         dim3(kSubLanes), 0, stream, s.table_dev, s.stride, token_bytes_of(s), v0,
                         base + v0 * nb1, base + lay.levels * nb1, select, want, buf[launch & 1],
                         buf[(launch + 1) & 1], sh, fuse_id ? arrived : nullptr, digests);
    }
    if ((e = hipGetLastError()) != hipSuccess || fuse_id) return e;
    ++launch;
  }
  ScopedTiming tm(K_HASH_FINAL, stream);
  hipLaunchKernelGGL(hash_final_kernel, dim3((uint32_t)s.n), dim3(64), 0, stream, s.table_dev,
                     s.stride, sh, base + lay.levels * nb1, select, want, buf[launch & 1],
                     digests);
  return hipGetLastError();
}

hipError_t launch_mask_hash_prep(const SetDesc& s, const HashLayout& lay, const KnormPartials& kp,
                                 double* keys, uint8_t* mask, uint8_t* ws, hipStream_t stream) {
  ScopedTiming tm(K_KEY_MASK, stream);
  // at least n threads (the scans over fragments); the node tables' scans cost a
  // barrier per step, so no more threads than that (the fold's few thousand
  // additions do not need them)
  int threads = 64;
  while (threads < s.n) threads <<= 1;
  if (kp.direct.layer >= 0) threads = 1024;   // the score rows too
  hipLaunchKernelGGL(mask_hash_prep_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev, s.n,
                     s.stride, token_bytes_of(s), s.L, lay.levels, kp.parts, kp.count, kp.direct,
                     s.H, s.d, keys, mask,
                     reinterpret_cast<int64_t*>(ws + lay.off_tables),
                     reinterpret_cast<int32_t*>(ws + lay.off_arrived));
  return hipGetLastError();
}

hipError_t launch_hash(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                       uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream,
                       bool tables_ready) {
  hipError_t e = hipSuccess;
  if (!tables_ready && (e = launch_hash_prep(s, lay, ws, stream)) != hipSuccess) return e;
  {
    int64_t* base = reinterpret_cast<int64_t*>(ws + lay.off_tables);
    const int64_t nb1 = s.n + 1;
    ScopedTiming tm(K_HASH_LEAF, stream);
    const int64_t full = (lay.tasks + (kBlock / 64) - 1) / (kBlock / 64);
    const int64_t cap = (int64_t)device_cu_count() * kLeafBlocksPerCu;
    const int64_t grid = full < cap ? full : cap;
    hipLaunchKernelGGL(hash_chunk_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, stream,
                       s.table_dev, s.n, s.stride, token_bytes_of(s), base,
                       base + (int64_t)(lay.levels + 1) * nb1, lay.tasks, select, want,
                       ws + lay.off_buf0);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, lay, select, want, digests, ws, stream);
}

hipError_t launch_hash_paged(const PagedDesc& p, const HashLayout& lay, const uint8_t* select,
                             uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream,
                             int blocks_per_cu) {
  const SetDesc& s = p.s;
  hipError_t e = launch_hash_prep(s, lay, ws, stream);
  if (e != hipSuccess) return e;
  {
    int64_t* base = reinterpret_cast<int64_t*>(ws + lay.off_tables);
    const int64_t nb1 = s.n + 1;
    ScopedTiming tm(K_HASH_LEAF, stream);
    const int64_t full = (lay.tasks + (kBlock / 64) - 1) / (kBlock / 64);
    const int64_t cap =
        (int64_t)device_cu_count() * (blocks_per_cu > 0 ? blocks_per_cu : kLeafBlocksPerCu);
    const int64_t grid = full < cap ? full : cap;
    hipLaunchKernelGGL(paged_hash_chunk_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, stream,
                       static_cast<const uint8_t*>(p.pool), p.pages, s.H, p.b_shift,
                       (int32_t)__builtin_ctzll((unsigned long long)s.row_bytes), s.table_dev,
                       p.blocks_dev, s.n, token_bytes_of(s), base,
                       base + (int64_t)(lay.levels + 1) * nb1, lay.tasks, select, want,
                       ws + lay.off_buf0);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, lay, select, want, digests, ws, stream);
}

}  // namespace cm
