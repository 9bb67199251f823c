// Step 1 — content address Id of Alg. 2 (also the hash tiebreak of §4.3).
//
// Per tensor, a BLAKE2s-256 binary tree over striped leaves; per fragment, a
// sequential BLAKE2s-256 of a 64-byte shape/dtype header followed by the 2L
// tensor roots (K^0, V^0, ..., K^{L-1}, V^{L-1}). A tensor is cut into stripes
// of 256 KiB and steps of 4 KiB; in every step each of the stripe's 64 leaves
// takes one 64-byte block: leaf k the 16-byte pieces k, k+64, k+128, k+192 (a
// shorter final step keeps block k whole). That layout is chosen for 64-wide
// wavefronts: one wave takes one stripe, lane k hashes leaf k (64 dependent
// compressions with the next blocks in flight), and each of the four 16-byte
// loads of a step reads 1 KiB of contiguous memory across the wave. The work is
// VALU-bound (12 VALU ops per G step, 960 per block); each upper tree level is
// one launch over all tensors at full lane occupancy (the parents add 1/64 of
// the leaf work).
#include "blake2s.h"
#include "internal.h"

namespace cm {

namespace {

constexpr int kBlock = 256;
#ifndef CM_HASH_BLOCKS_PER_CU
#define CM_HASH_BLOCKS_PER_CU 2
#endif
constexpr int kLeafBlocksPerCu = CM_HASH_BLOCKS_PER_CU;

__device__ __forceinline__ void load64(const uint8_t* p, uint32_t (&m)[16]) {
  const CM_GLOBAL u32x4* q = global_ptr<u32x4>(p);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u32x4 v = q[k];
    m[4 * k + 0] = v[0];
    m[4 * k + 1] = v[1];
    m[4 * k + 2] = v[2];
    m[4 * k + 3] = v[3];
  }
}

// Block of leaf `lane` in step j of a stripe starting at p: the 16-byte pieces
// lane, lane+64, lane+128, lane+192 of a full step; block `lane` of the final
// short step (j == full_steps).
__device__ __forceinline__ void load_leaf_block(const uint8_t* p, int lane, int64_t j,
                                               int64_t full_steps, uint32_t (&m)[16]) {
  if (j < full_steps) {
    const CM_GLOBAL u32x4* q = global_ptr<u32x4>(p + (j << 12) + lane * 16);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const u32x4 v = q[k * 64];
      m[4 * k + 0] = v[0];
      m[4 * k + 1] = v[1];
      m[4 * k + 2] = v[2];
      m[4 * k + 3] = v[3];
    }
  } else {
    load64(p + (j << 12) + lane * 64, m);
  }
}

__device__ __forceinline__ void store_digest(uint8_t* out, const B2sState& s) {
  uint4* q = reinterpret_cast<uint4*>(out);
  q[0] = make_uint4(s.h[0], s.h[1], s.h[2], s.h[3]);
  q[1] = make_uint4(s.h[4], s.h[5], s.h[6], s.h[7]);
}

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
// of the (tensor, stripe) tasks of the leaf kernel. One workgroup, block-wide
// inclusive scans.
__global__ __launch_bounds__(1024) void hash_prep_kernel(const int64_t* __restrict__ table,
                                                         int32_t n, int64_t stride,
                                                         int64_t token_bytes, int32_t L,
                                                         int32_t levels,
                                                         int64_t* __restrict__ base) {
  __shared__ int64_t sc[1024];
  const int tid = threadIdx.x;
  const int64_t bytes = tid < n ? table[(int64_t)tid * stride] * token_bytes : 0;
  const int64_t m0 = tid < n ? leaves_of(bytes) : 0;
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

// One wave = one (tensor, stripe) task at a time; lane k hashes leaf k of the
// stripe, whose blocks lie 4 KiB apart. The grid is bounded (a few workgroups
// per CU) and strides over all tasks: a VALU-bound kernel saturates the SIMDs
// with a couple of waves each, and the wave slots left free let an HBM-bound
// kernel on another stream run on the same CUs.
__global__ __launch_bounds__(kBlock) void hash_leaf_kernel(const int64_t* __restrict__ table,
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
    const int64_t m = leaves_of(bytes);
    const int64_t local = task - task_base[i];
    const int64_t t = local / stripes;
    const int64_t sidx = local - t * stripes;
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const int64_t blocks_here = in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks;
    if (lane >= blocks_here) continue;
    const int64_t nb = (blocks_here - lane + kStripeLeaves - 1) / kStripeLeaves;
    const int64_t full_steps = blocks_here / kStripeLeaves;
    const int64_t leaf = sidx * kStripeLeaves + lane;
    const uint8_t* p = reinterpret_cast<const uint8_t*>(table[(int64_t)i * stride + 1 + t]) +
                       ((sidx * kStripeBlocks) << 6);
    B2sState s;
    b2s_init_tree(s, (uint64_t)leaf, 0);
    b2s_node(s, (uint64_t)nb, leaf == m - 1, [&](uint64_t b, uint32_t (&w)[16]) {
      load_leaf_block(p, lane, (int64_t)b, full_steps, w);
    });
    store_digest(nodes + (base0[i] + t * m + leaf) * 32, s);
  }
}

// Level v >= 1: node j of a tensor hashes children 2j, 2j+1 of level v-1;
// an unpaired last child is carried up unchanged.
__global__ __launch_bounds__(kBlock) void hash_parent_kernel(
    const int64_t* __restrict__ table, int32_t n, int64_t stride, int64_t token_bytes, int32_t v,
    const int64_t* __restrict__ base_prev, const int64_t* __restrict__ base_cur,
    int64_t total_cur, const uint8_t* __restrict__ select, uint32_t want,
    const uint8_t* __restrict__ in, uint8_t* __restrict__ out) {
  const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (g >= total_cur) return;
  const int i = find_fragment(base_cur, n, g);
  if (select && select[i] != want) return;
  const int64_t m0 = leaves_of(table[(int64_t)i * stride] * token_bytes);
  const int64_t m_prev = nodes_at(m0, v - 1);
  const int64_t m_cur = nodes_at(m0, v);
  const int64_t local = g - base_cur[i];
  const int64_t t = local / m_cur;
  const int64_t j = local - t * m_cur;
  const uint8_t* c = in + (base_prev[i] + t * m_prev + 2 * j) * 32;
  if (2 * j + 1 < m_prev) {
    uint32_t m[16];
    load64(c, m);
    B2sState s;
    b2s_init_tree(s, (uint64_t)j, (uint32_t)v);
    b2s_compress(s, m, 64, true, j == m_cur - 1);
    store_digest(out + g * 32, s);
  } else {
    const uint4* q = reinterpret_cast<const uint4*>(c);
    uint4* o = reinterpret_cast<uint4*>(out + g * 32);
    o[0] = q[0];
    o[1] = q[1];
  }
}

// Id = BLAKE2s-256(header || root(K^0) || root(V^0) || ...), one lane per fragment.
__global__ __launch_bounds__(64) void hash_final_kernel(
    const int64_t* __restrict__ table, int32_t n, int64_t stride, int32_t L, int32_t H,
    int32_t d, uint32_t dtype_code, uint32_t esize, const int64_t* __restrict__ base_last,
    const uint8_t* __restrict__ select, uint32_t want, const uint8_t* __restrict__ roots,
    uint8_t* __restrict__ digests) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (select && select[i] != want) return;
  const uint64_t T = (uint64_t)table[(int64_t)i * stride];
  uint32_t m[16] = {0x52464D43u, 0x31304741u,  // "CMFRAG01"
                    dtype_code, esize, (uint32_t)L, 1u, (uint32_t)H,
                    (uint32_t)T, (uint32_t)(T >> 32), (uint32_t)d,
                    0u, 0u, 0u, 0u, 0u, 0u};
  B2sState s;
  b2s_init_sequential(s);
  b2s_compress(s, m, 64, false, false);
  const uint8_t* r = roots + base_last[i] * 32;
  for (int l = 0; l < L; ++l) {
    load64(r + (int64_t)l * 64, m);
    b2s_compress(s, m, (uint64_t)(l + 2) * 64, l == L - 1, false);
  }
  store_digest(digests + (int64_t)i * 32, s);
}

}  // namespace

HashLayout hash_layout(const SetDesc& s) {
  HashLayout lay{};
  int64_t max_m0 = 1;
  for (int i = 0; i < s.n; ++i) {
    lay.tasks += 2 * (int64_t)s.L * stripes_of(s.T(i) * token_bytes_of(s));
    const int64_t m0 = leaves_of(s.T(i) * token_bytes_of(s));
    if (m0 > max_m0) max_m0 = m0;
    lay.total0 += 2 * (int64_t)s.L * m0;
    lay.total1 += 2 * (int64_t)s.L * nodes_at(m0, 1);
  }
  while (((int64_t)1 << lay.levels) < max_m0) ++lay.levels;
  if (lay.levels == 0) lay.total1 = 0;
  size_t off = 0;
  lay.off_tables = off;
  off = align_up(off + sizeof(int64_t) * (size_t)(lay.levels + 2) * (size_t)(s.n + 1), kWsAlign);
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
                     reinterpret_cast<int64_t*>(ws + lay.off_tables));
  return hipGetLastError();
}

hipError_t launch_hash_tree(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                            uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream) {
  int64_t* base = reinterpret_cast<int64_t*>(ws + lay.off_tables);
  uint8_t* buf[2] = {ws + lay.off_buf0, ws + lay.off_buf1};
  const int64_t nb1 = s.n + 1;
  hipError_t e = hipSuccess;
  for (int v = 1; v <= lay.levels; ++v) {
    int64_t total = 0;
    for (int i = 0; i < s.n; ++i)
      total += 2 * (int64_t)s.L * nodes_at(leaves_of(s.T(i) * token_bytes_of(s)), v);
    ScopedTiming tm(K_HASH_PARENT, stream);
    const int64_t grid = (total + kBlock - 1) / kBlock;
    hipLaunchKernelGGL(hash_parent_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, stream,
                       s.table_dev, s.n, s.stride, token_bytes_of(s), v, base + (v - 1) * nb1,
                       base + v * nb1, total, select, want, buf[(v - 1) & 1], buf[v & 1]);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    ScopedTiming tm(K_HASH_FINAL, stream);
    const uint32_t code = s.dtype;  // cm_dtype value doubles as the header dtype code
    hipLaunchKernelGGL(hash_final_kernel, dim3((uint32_t)((s.n + 63) / 64)), dim3(64), 0,
                       stream, s.table_dev, s.n, s.stride, s.L, s.H, s.d, code,
                       (uint32_t)s.esize, base + lay.levels * nb1, select, want,
                       buf[lay.levels & 1], digests);
  }
  return hipGetLastError();
}

hipError_t launch_hash(const SetDesc& s, const HashLayout& lay, const uint8_t* select,
                       uint32_t want, uint8_t* digests, uint8_t* ws, hipStream_t stream) {
  hipError_t e = launch_hash_prep(s, lay, ws, stream);
  if (e != hipSuccess) return e;
  {
    int64_t* base = reinterpret_cast<int64_t*>(ws + lay.off_tables);
    const int64_t nb1 = s.n + 1;
    ScopedTiming tm(K_HASH_LEAF, stream);
    const int64_t full = (lay.tasks + (kBlock / 64) - 1) / (kBlock / 64);
    const int64_t cap = (int64_t)device_cu_count() * kLeafBlocksPerCu;
    const int64_t grid = full < cap ? full : cap;
    hipLaunchKernelGGL(hash_leaf_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, stream,
                       s.table_dev, s.n, s.stride, token_bytes_of(s), base,
                       base + (int64_t)(lay.levels + 1) * nb1, lay.tasks, select, want,
                       ws + lay.off_buf0);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, lay, select, want, digests, ws, stream);
}

}  // namespace cm
