// Steps 1 and 4-5 in one pass: the render of Eq. (1)-(2) and, for the
// fragments whose Id is still missing, the leaf level of their hash tree (Id
// of Alg. 2), from the same loads.
//
// Hashing is VALU-bound (960 VALU ops per 64-byte block) and the render is
// HBM-bound; done separately they read every byte twice. Here one wave takes
// one (slot, tensor, stripe) task: at step j every lane loads one 64-byte block
// (block 64j + lane of the 256 KiB stripe, so the wave reads 4 KiB of
// contiguous memory), compresses it into its leaf (leaf = lane of the stripe,
// exactly the striped leaf layout of the tree) and writes it to its place in
// the merged cache: V and offset-0 K unchanged, other K rotated by R(off).
// A row is row_bytes / 64 consecutive lanes, so the other half of a lane's
// pairs sits in lane ^ (blocks per row / 2) and one xor shuffle brings it in.
// The slot's cos/sin table lives in LDS, one copy per wave. HBM traffic is the
// algorithmic minimum (each byte read once, written once); the kernel is bound
// by the VALU work of the hash plus the fp64 rotation.
#include "blake2s.h"
#include "internal.h"
#include "stream_ops.h"

namespace cm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxD = 512;  // largest head dimension (d * element bytes <= 1024)
#ifndef CM_FUSED_BLOCKS_PER_CU
#define CM_FUSED_BLOCKS_PER_CU 2
#endif

__device__ __forceinline__ void load64(const uint8_t* p, uint32_t (&m)[16]) {
  const CM_GLOBAL u32x4* q = global_ptr<u32x4>(p);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u32x4 v = __builtin_nontemporal_load(q + k);
    m[4 * k + 0] = v[0];
    m[4 * k + 1] = v[1];
    m[4 * k + 2] = v[2];
    m[4 * k + 3] = v[3];
  }
}

__device__ __forceinline__ void store64(uint8_t* p, const uint32_t (&y)[16]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    u32x4 v;
    v[0] = y[4 * k + 0];
    v[1] = y[4 * k + 1];
    v[2] = y[4 * k + 2];
    v[3] = y[4 * k + 3];
    st_stream(p + 16 * k, v);
  }
}

template <int ESIZE>
__device__ __forceinline__ void put_bits(uint32_t (&y)[16], int e, uint32_t bits) {
  if constexpr (ESIZE == 2) {
    if (e & 1) y[e >> 1] |= bits << 16;
    else y[e >> 1] = bits;
  } else {
    y[e] = bits;
  }
}

// Rotate the block x (lane's chunk c of a row; bpr blocks per row) into y.
// ang holds (cos, sin) of pair j at [2j], [2j+1]. Must be reached by every lane
// of the wave (the half-row partner comes from a cross-lane shuffle).
template <int ESIZE, int STYLE>
__device__ __forceinline__ void rotate_block(const uint32_t (&x)[16], int c, int bpr,
                                             const double* ang, uint32_t (&y)[16]) {
#pragma clang fp contract(off)
  constexpr int E = 64 / ESIZE;  // elements per block
  if constexpr (STYLE == CM_ROPE_INTERLEAVED) {
    const int j0 = c * (E / 2);
#pragma unroll
    for (int p = 0; p < E / 2; ++p) {
      const double x1 = elem_f64<ESIZE>(x, 2 * p), x2 = elem_f64<ESIZE>(x, 2 * p + 1);
      const double cs = ang[2 * (j0 + p)], sn = ang[2 * (j0 + p) + 1];
      put_bits<ESIZE>(y, 2 * p, round_bits<ESIZE>(x1 * cs - x2 * sn));
      put_bits<ESIZE>(y, 2 * p + 1, round_bits<ESIZE>(x2 * cs + x1 * sn));
    }
  } else if (bpr == 1) {
    // the whole row is this block: pairs (e, e + E/2)
#pragma unroll
    for (int e = 0; e < E / 2; ++e) {
      const double x1 = elem_f64<ESIZE>(x, e), x2 = elem_f64<ESIZE>(x, e + E / 2);
      const double cs = ang[2 * e], sn = ang[2 * e + 1];
      put_bits<ESIZE>(y, e, round_bits<ESIZE>(x1 * cs - x2 * sn));
      put_bits<ESIZE>(y, e + E / 2, round_bits<ESIZE>(x2 * cs + x1 * sn));
    }
  } else {
    const int hb = bpr >> 1;
    uint32_t p[16];
#pragma unroll
    for (int w = 0; w < 16; ++w) p[w] = __shfl_xor(x[w], hb, 64);
    const bool second = c >= hb;
    const int j0 = (second ? c - hb : c) * E;
    // first half: y = x c - p s; second half: y = x c + p s = x c - (-p) s
    const double sg = second ? -1.0 : 1.0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const double xv = elem_f64<ESIZE>(x, e);
      const double pv = sg * elem_f64<ESIZE>(p, e);
      const double cs = ang[2 * (j0 + e)], sn = ang[2 * (j0 + e) + 1];
      put_bits<ESIZE>(y, e, round_bits<ESIZE>(xv * cs - pv * sn));
    }
  }
}

template <int ESIZE, int STYLE>
__global__ __launch_bounds__(kThreads) void render_hash_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, int32_t n_u, int64_t total_tasks,
    const double* __restrict__ angles, int32_t H, int32_t d, int64_t T_out,
    const uint8_t* __restrict__ select, const int64_t* __restrict__ base0,
    uint8_t* __restrict__ nodes, uint8_t* __restrict__ out) {
  __shared__ double sh_ang[kWaves][kMaxD];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t row_bytes = (int64_t)d * ESIZE;
  const int bpr = (int)(row_bytes >> 6);  // 64-byte blocks per row: 1, 2, 4, 8 or 16
  const int c = lane & (bpr - 1);         // this lane's block within its row
  const int rows_step = 64 / bpr;         // rows covered by one wave step
  const int64_t waves = (int64_t)gridDim.x * kWaves;
  double* ang = sh_ang[wave];
  for (int64_t task = (int64_t)blockIdx.x * kWaves + wave; task < total_tasks; task += waves) {
    int lo = 0, hi = n_u - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (task_base[mid] <= task) lo = mid; else hi = mid - 1;
    }
    const int s = lo;
    const int64_t i = plan[CM_PLAN_HEADER + s];
    const int64_t off = plan[CM_PLAN_HEADER + n + s];
    const int64_t T = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
    const bool hashing = select[i] == 0;
    const int64_t bytes = (int64_t)H * T * row_bytes;
    const int64_t stripes = stripes_of(bytes);
    const int64_t local = task - task_base[s];
    const int64_t t = local / stripes;            // tensor: 2l + kv
    const int64_t sidx = local - t * stripes;
    const bool rotate = (t & 1) == 0 && off != 0;
    if (rotate) {
      for (int q = lane; q < d; q += 64) ang[q] = angles[(int64_t)s * d + q];
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const int bh = (int)(in_stripe < kStripeBlocks ? in_stripe : kStripeBlocks);
    const int steps = (bh + kStripeLeaves - 1) / kStripeLeaves;
    const int nb = lane < bh ? (bh - lane + kStripeLeaves - 1) / kStripeLeaves : 0;
    const int64_t first_block = sidx * kStripeBlocks + lane;
    const uint8_t* src = reinterpret_cast<const uint8_t*>(table[i * stride + 1 + t]) +
                         (first_block << 6);
    uint8_t* out_t = out + t * (int64_t)H * T_out * row_bytes;
    const int64_t leaf = sidx * kStripeLeaves + lane;
    const int64_t m = leaves_of(bytes);
    int64_t row = first_block / bpr;
    int64_t hh = row / T;
    int64_t tt = row - hh * T;
    B2sState st;
    b2s_init_tree(st, (uint64_t)leaf, 0);
    uint32_t cur[16], nxt[16];
    if (nb > 0) load64(src, cur);
    for (int j = 0; j < steps; ++j) {
      const bool active = j < nb;
      if (j + 1 < nb) load64(src + (int64_t)(j + 1) * (kStripeLeaves * 64), nxt);
      if (hashing && active)
        b2s_compress(st, cur, (uint64_t)(j + 1) << 6, j + 1 == nb, j + 1 == nb && leaf == m - 1);
      uint32_t y[16];
      if (rotate) {
        rotate_block<ESIZE, STYLE>(cur, c, bpr, ang, y);
      } else {
#pragma unroll
        for (int w = 0; w < 16; ++w) y[w] = cur[w];
      }
      if (active) store64(out_t + ((hh * T_out + off + tt) * row_bytes + c * 64), y);
      tt += rows_step;
      while (tt >= T) {
        tt -= T;
        ++hh;
      }
#pragma unroll
      for (int w = 0; w < 16; ++w) cur[w] = nxt[w];
    }
    if (hashing && nb > 0) {
      uint4* q = reinterpret_cast<uint4*>(nodes + (base0[i] + t * m + leaf) * 32);
      q[0] = make_uint4(st.h[0], st.h[1], st.h[2], st.h[3]);
      q[1] = make_uint4(st.h[4], st.h[5], st.h[6], st.h[7]);
    }
  }
}

}  // namespace

int64_t render_hash_tasks(const SetDesc& s, const int64_t* plan_host) {
  const int64_t nu = plan_host[CM_PLAN_NUNIQUE];
  int64_t tasks = 0;
  for (int64_t k = 0; k < nu; ++k) {
    const int64_t len = plan_host[CM_PLAN_HEADER + 2 * (int64_t)s.n + k];
    tasks += 2 * (int64_t)s.L * stripes_of(len * token_bytes_of(s));
  }
  return tasks;
}

hipError_t launch_render_hash(const SetDesc& s, const HashLayout& hlay, const RenderLayout& rlay,
                              const int64_t* plan_dev, int32_t n_unique, int64_t total_tasks,
                              int64_t T_out, double base, int32_t style, const uint8_t* select,
                              uint8_t* digests, void* out, uint8_t* ws, hipStream_t stream) {
  uint8_t* hws = ws;
  uint8_t* rws = ws + align_up(hlay.bytes, kWsAlign);
  hipError_t e = launch_hash_prep(s, hlay, hws, stream);
  if (e != hipSuccess) return e;
  if ((e = launch_render_prep(s, rlay, plan_dev, n_unique, base, /*stripe_tasks=*/true, select,
                              rws, stream)) != hipSuccess)
    return e;
  const uint8_t* hsel = rws + rlay.off_hsel;  // 0: slot delivery whose Id is computed here
  {
    const int64_t* base_tab = reinterpret_cast<const int64_t*>(hws + hlay.off_tables);
    const int64_t* tasks = reinterpret_cast<const int64_t*>(rws + rlay.off_tiles);
    const double* angles = reinterpret_cast<const double*>(rws + rlay.off_angles);
    const int64_t full = (total_tasks + kWaves - 1) / kWaves;
    const int64_t cap = (int64_t)device_cu_count() * CM_FUSED_BLOCKS_PER_CU;
    const dim3 grid((uint32_t)(full < cap ? full : cap));
    ScopedTiming tm(K_RENDER_HASH, stream);
    uint8_t* nodes = hws + hlay.off_buf0;
    uint8_t* o = reinterpret_cast<uint8_t*>(out);
    if (s.esize == 2) {
      if (style == CM_ROPE_HALF)
        hipLaunchKernelGGL((render_hash_kernel<2, CM_ROPE_HALF>), grid, dim3(kThreads), 0, stream,
                           s.table_dev, s.stride, s.n, plan_dev, tasks, n_unique, total_tasks,
                           angles, s.H, s.d, T_out, hsel, base_tab, nodes, o);
      else
        hipLaunchKernelGGL((render_hash_kernel<2, CM_ROPE_INTERLEAVED>), grid, dim3(kThreads), 0,
                           stream, s.table_dev, s.stride, s.n, plan_dev, tasks, n_unique,
                           total_tasks, angles, s.H, s.d, T_out, hsel, base_tab, nodes, o);
    } else {
      if (style == CM_ROPE_HALF)
        hipLaunchKernelGGL((render_hash_kernel<4, CM_ROPE_HALF>), grid, dim3(kThreads), 0, stream,
                           s.table_dev, s.stride, s.n, plan_dev, tasks, n_unique, total_tasks,
                           angles, s.H, s.d, T_out, hsel, base_tab, nodes, o);
      else
        hipLaunchKernelGGL((render_hash_kernel<4, CM_ROPE_INTERLEAVED>), grid, dim3(kThreads), 0,
                           stream, s.table_dev, s.stride, s.n, plan_dev, tasks, n_unique,
                           total_tasks, angles, s.H, s.d, T_out, hsel, base_tab, nodes, o);
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, hlay, hsel, 0, digests, hws, stream);
}

}  // namespace cm
