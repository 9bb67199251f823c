// Step 3 — Ingest dedupe (Alg. 2, Eq. (5)) and canonical order (Alg. 1):
// pi* = argsort(-S, -h) over the distinct fragments, offsets by exclusive prefix
// sum of the lengths in that order (§4.2). Without dedupe the same order over
// every delivery is the naive re-render of §5.9: byte-identical copies tie on
// key and digest and keep their delivery order.
//
// n <= 1024 deliveries fit one workgroup (one lane per delivery), so the order
// is built by exact counting, with no sort network and no host round trip: a
// delivery is absorbed if an earlier one has the same digest; the slot of a
// kept delivery is the number of kept deliveries that precede it (larger key,
// or equal key and larger big-endian digest, or equal both and earlier).
// Keys are compared as IEEE doubles and only bitwise-equal keys tie.
// Everything is integer or comparison work, so the plan is exact and
// independent of thread timing.
//
// Byte-identical deliveries have bitwise-equal keys (the key is a
// deterministic function of the bytes), and ties need equal keys, so the
// digest of a delivery is read only when another delivery has the same key.
// That lets the digests of every other delivery be computed concurrently with
// the render (equal_key_mask marks the ones needed first).
#include "key_mask.h"
#include "knorm_fold.h"
#include "render_tables.h"

namespace cm {

namespace {

__device__ __forceinline__ uint32_t bswap32(uint32_t x) {
  return __builtin_bswap32(x);
}

// Digest words in big-endian significance order (byte 0 most significant).
__device__ __forceinline__ void load_digest_be(const uint8_t* __restrict__ digests, int i,
                                               uint32_t (&w)[8]) {
  const uint32_t* p = reinterpret_cast<const uint32_t*>(digests + (int64_t)i * 32);
#pragma unroll
  for (int k = 0; k < 8; ++k) w[k] = bswap32(p[k]);
}

// -1, 0, +1 for a <, ==, > b as 256-bit big-endian unsigned integers.
__device__ __forceinline__ int cmp_digest(const uint32_t (&a)[8], const uint32_t (&b)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k)
    if (a[k] != b[k]) return a[k] > b[k] ? 1 : -1;
  return 0;
}

// The plan, by one workgroup of at least n threads (see the top of this file).
__device__ __forceinline__ void order_body(const int64_t* __restrict__ table, int64_t stride,
                                           int32_t n, const double* __restrict__ keys,
                                           const uint8_t* __restrict__ digests, int32_t dedupe,
                                           int64_t* __restrict__ plan) {
  __shared__ double s_key[1024];
  __shared__ int64_t s_len[1024];     // by delivery, then by slot
  __shared__ int32_t s_first[1024];   // first delivery with the same digest
  __shared__ int32_t s_rank[1024];    // slot of each distinct delivery
  __shared__ int32_t s_src[1024];     // delivery of each slot
  __shared__ int64_t s_slot_len[1024];
  const int tid = threadIdx.x;
  const bool live = tid < n;
  uint32_t mine[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  double key = 0.0;
  int64_t len = 0;
  s_src[tid] = -1;
  s_slot_len[tid] = 0;
  s_rank[tid] = 0;
  if (live) {
    key = keys[tid];
    len = table[(int64_t)tid * stride];
    s_key[tid] = key;
    s_len[tid] = len;
  }
  const int bad = __syncthreads_or(live && !isfinite(key));
  if (bad) {
    // a non-finite score leaves the order undefined: the plan says so and
    // holds no slots (nothing is rendered from it)
    if (tid < n) {
      const int64_t nn = n;
      plan[CM_PLAN_HEADER + tid] = -1;
      plan[CM_PLAN_HEADER + nn + tid] = -1;
      plan[CM_PLAN_HEADER + 2 * nn + tid] = -1;
      plan[CM_PLAN_HEADER + 3 * nn + tid] = -1;
    }
    if (tid == 0) {
      plan[CM_PLAN_STATUS] = CM_ENONFINITE;
      plan[CM_PLAN_N] = n;
      plan[CM_PLAN_NUNIQUE] = 0;
      plan[CM_PLAN_TOUT] = 0;
    }
    return;
  }
  if (live) {
    bool shared = false;
    for (int j = 0; j < n; ++j) shared |= (j != tid && s_key[j] == key);
    if (shared) load_digest_be(digests, tid, mine);
  }

  // Absorption: the first arrival of each content is kept (copies share key,
  // length and digest).
  int first = tid;
  if (live) {
    for (int j = 0; dedupe && j < tid; ++j) {
      if (s_key[j] != key || s_len[j] != len) continue;
      uint32_t other[8];
      load_digest_be(digests, j, other);
      if (cmp_digest(other, mine) == 0) { first = j; break; }
    }
    s_first[tid] = first;
  }
  __syncthreads();
  const bool distinct = live && first == tid;
  const int n_unique = __syncthreads_count(distinct);

  // Slot = number of kept deliveries ordered before this one.
  if (distinct) {
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      if (j == tid || s_first[j] != j) continue;
      const double kj = s_key[j];
      bool before = kj > key;
      if (!before && kj == key) {
        uint32_t other[8];
        load_digest_be(digests, j, other);
        const int c = cmp_digest(other, mine);
        before = c > 0 || (c == 0 && j < tid);   // equal content (no dedupe): delivery order
      }
      rank += before ? 1 : 0;
    }
    s_rank[tid] = rank;
    if (rank < 1024) {
      s_src[rank] = tid;
      s_slot_len[rank] = len;
    }
  }
  __syncthreads();

  // Offsets: exclusive prefix sum of slot lengths (exact integers).
  int64_t off = 0;
  if (tid < n_unique) {
    for (int s2 = 0; s2 < tid; ++s2) off += s_slot_len[s2];
  }
  if (tid < n) {
    const int64_t nn = n;
    if (tid < n_unique) {
      plan[CM_PLAN_HEADER + tid] = s_src[tid];
      plan[CM_PLAN_HEADER + nn + tid] = off;
      plan[CM_PLAN_HEADER + 2 * nn + tid] = s_slot_len[tid];
    } else {
      plan[CM_PLAN_HEADER + tid] = -1;
      plan[CM_PLAN_HEADER + nn + tid] = -1;
      plan[CM_PLAN_HEADER + 2 * nn + tid] = -1;
    }
    plan[CM_PLAN_HEADER + 3 * nn + tid] = s_rank[s_first[tid]];
  }
  if (tid == n_unique - 1) {
    plan[CM_PLAN_STATUS] = CM_OK;
    plan[CM_PLAN_N] = n;
    plan[CM_PLAN_NUNIQUE] = n_unique;
    plan[CM_PLAN_TOUT] = off + s_slot_len[tid];
  }
}

__global__ __launch_bounds__(1024) void order_kernel(const int64_t* __restrict__ table,
                                                     int64_t stride, int32_t n,
                                                     const double* __restrict__ keys,
                                                     const uint8_t* __restrict__ digests,
                                                     int32_t dedupe, int64_t* __restrict__ plan) {
  order_body(table, stride, n, keys, digests, dedupe, plan);
}

// The plan, then (same workgroup, after a barrier that makes the plan visible to
// every thread) the render's per-slot tables: one launch where the path would
// otherwise take two.
__global__ __launch_bounds__(1024) void order_render_prep_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const double* __restrict__ keys,
    const uint8_t* __restrict__ digests, int64_t* __restrict__ plan, int32_t d, int32_t ep,
    int32_t style, double base, int32_t stripe_blocks, int64_t tensor_pairs, int64_t token_bytes,
    const uint8_t* __restrict__ select, uint8_t* __restrict__ hsel,
    int64_t* __restrict__ unit_base, double* __restrict__ angles) {
  order_body(table, stride, n, keys, digests, 1, plan);
  __syncthreads();
  render_tables(plan, n, d, ep, style, base, stripe_blocks, tensor_pairs, token_bytes, select,
                hsel, unit_base, angles, table, stride, 0, nullptr, nullptr);
}

// Steps 2-5 of a set render before the render itself: the last levels of the
// scores (count > 1), the plan, then the unit render's tables for T_out rows.
// The members of a set are distinct, so the plan's T_out is the sum of all
// lengths; a plan whose T_out differs (byte-identical members were absorbed)
// gets CM_ESHAPE, and it, like a plan with a non-finite score, is not rendered.
__global__ __launch_bounds__(1024) void order_set_prep_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n,
    const double* __restrict__ parts, int64_t count, KnormDirect kd, double* __restrict__ keys,
    const uint8_t* __restrict__ digests, int64_t* __restrict__ plan, int64_t T_out, int32_t d,
    int32_t ep, int32_t style, double base, double* __restrict__ angles,
    int64_t* __restrict__ unit_base, int32_t H, int32_t n_lkh, int32_t rb_shift, int64_t units,
    int32_t* __restrict__ unit_slot, int64_t* __restrict__ src_base) {
  knorm_finish(table, stride, n, H, d, kd, parts, count, keys);
  order_body(table, stride, n, keys, digests, 1, plan);
  __syncthreads();
  bool ok = plan[CM_PLAN_STATUS] == CM_OK;
  if (ok && plan[CM_PLAN_TOUT] != T_out) {
    ok = false;
    if (threadIdx.x == 0) plan[CM_PLAN_STATUS] = CM_ESHAPE;
  }
  if (ok)
    render_tables(plan, n, d, ep, style, base, 0, 0, 0, nullptr, nullptr, unit_base, angles,
                  table, stride, T_out, nullptr, nullptr);
  unit_tables(table, stride, plan, n, H, n_lkh, rb_shift, 0, T_out, units, ok, unit_slot,
              src_base);
}

__global__ __launch_bounds__(1024) void equal_key_mask_kernel(const int64_t* __restrict__ table,
                                                              int64_t stride, int32_t n,
                                                              const double* __restrict__ keys,
                                                              uint8_t* __restrict__ mask) {
  equal_key_mask_body(n, keys, mask);
}

}  // namespace

hipError_t launch_equal_key_mask(const SetDesc& s, const double* keys, uint8_t* mask,
                                 hipStream_t stream) {
  int threads = 64;
  while (threads < s.n) threads <<= 1;
  ScopedTiming tm(K_KEY_MASK, stream);
  hipLaunchKernelGGL(equal_key_mask_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev,
                     s.stride, s.n, keys, mask);
  return hipGetLastError();
}

hipError_t launch_order(const SetDesc& s, const double* keys, const uint8_t* digests,
                        bool dedupe, int64_t* plan, hipStream_t stream) {
  int threads = 64;
  while (threads < s.n) threads <<= 1;
  ScopedTiming tm(K_ORDER, stream);
  hipLaunchKernelGGL(order_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev, s.stride,
                     s.n, keys, digests, dedupe ? 1 : 0, plan);
  return hipGetLastError();
}

hipError_t launch_order_render_prep(const SetDesc& s, const double* keys, const uint8_t* digests,
                                    int64_t* plan, const RenderLayout& rlay, double base,
                                    int32_t style, int32_t stripe_blocks, const uint8_t* select,
                                    uint8_t* rws, hipStream_t stream) {
  ScopedTiming tm(K_ORDER, stream);
  // at least n threads (one per delivery), and enough for about two angle
  // pairs each (fp64 pow, cos and sin per pair: 31 pairs per thread of 64 took
  // 43 us on a 32-delivery set)
  int threads = 64;
  while (threads < 1024 && (threads < s.n || (int64_t)threads * 2 < (int64_t)s.n * (s.d / 2)))
    threads <<= 1;
  hipLaunchKernelGGL(order_render_prep_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev,
                     s.stride, s.n, keys, digests, plan, s.d, 16 / s.esize, style, base,
                     stripe_blocks, (int64_t)s.L, token_bytes_of(s), select,
                     select ? rws + rlay.off_hsel : nullptr,
                     reinterpret_cast<int64_t*>(rws + rlay.off_tiles),
                     reinterpret_cast<double*>(rws + rlay.off_angles));
  return hipGetLastError();
}

hipError_t launch_render_set(const SetDesc& s, const RenderLayout& lay, const KnormPartials& kp,
                             double* keys, const uint8_t* digests, int64_t* plan, int64_t T_out,
                             double base, int32_t style, void* out, uint8_t* rws,
                             hipStream_t stream) {
  const int64_t units = render_units(s, T_out);
  // the score rows too when the set is scored here
  const int threads = kp.direct.layer >= 0 ? 1024
                                           : table_threads(s.n, units + (int64_t)s.n * 2 * s.L * s.H);
  {
    ScopedTiming tm(K_ORDER, stream);
    hipLaunchKernelGGL(order_set_prep_kernel, dim3(1), dim3(threads), 0, stream, s.table_dev,
                       s.stride, s.n, kp.parts, kp.count, kp.direct, keys, digests, plan, T_out, s.d,
                       16 / s.esize, style, base, reinterpret_cast<double*>(rws + lay.off_angles),
                       reinterpret_cast<int64_t*>(rws + lay.off_tiles), s.H, 2 * s.L * s.H,
                       (int32_t)__builtin_ctzll((unsigned long long)s.row_bytes), units,
                       reinterpret_cast<int32_t*>(rws + lay.off_unit_slot),
                       reinterpret_cast<int64_t*>(rws + lay.off_src_base));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_render_units(s, lay, plan, RenderRange{0, T_out, T_out}, style, out, rws, stream);
}

}  // namespace cm
