// Steps 4-5 — Eq. (1)-(2): for every layer l, K/V and head h, the merged
// [T_out, d] block is the concatenation over slots s of the fragment rows, K
// multiplied by R(off_s) (byte copy when off_s = 0), V copied.
//
// HBM-bound streaming (about 0.4 flop per byte moved), so the design is about
// bytes in flight: each (l, kv, h, slot) segment is contiguous in both source
// and destination and is cut into 32 KiB tiles; one 256-lane workgroup moves
// one tile with all of its 16-byte nontemporal loads issued before the first
// store. A K lane owns the same 16-byte column chunk of both halves of a row
// (pairs j and j + d/2, or the adjacent pairs of an interleaved chunk), so its
// cos/sin values are loaded once per tile from the per-slot angle table and
// kept in registers. The rotation runs in fp64 with the products and the
// add/subtract rounded separately, then rounds once to the storage dtype
// (round-to-nearest-even; bf16 via the compiler's single-step conversion).
#include "internal.h"
#include "stream_ops.h"

namespace cm {

namespace {

#ifndef CM_RENDER_TILE_BYTES
#define CM_RENDER_TILE_BYTES 32768
#endif
constexpr int kThreads = 256;
constexpr int kTileBytes = CM_RENDER_TILE_BYTES;

// 16 bytes <-> fp64 lanes
template <int ESIZE>
struct Chunk;

template <>
struct Chunk<2> {
  static constexpr int E = 8;
  __device__ __forceinline__ static void unpack(const u32x4 v, double (&x)[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] = (double)__uint_as_float(v[k] << 16);
      x[2 * k + 1] = (double)__uint_as_float(v[k] & 0xFFFF0000u);
    }
  }
  __device__ __forceinline__ static u32x4 pack(const double (&y)[8]) {
    u32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = bf16_bits_rne(y[2 * k]) | (bf16_bits_rne(y[2 * k + 1]) << 16);
    return v;
  }
};

template <>
struct Chunk<4> {
  static constexpr int E = 4;
  __device__ __forceinline__ static void unpack(const u32x4 v, double (&x)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = (double)__uint_as_float(v[k]);
  }
  __device__ __forceinline__ static u32x4 pack(const double (&y)[4]) {
    u32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __float_as_uint((float)y[k]);
    return v;
  }
};

__device__ __forceinline__ void copy_tile(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                          int64_t bytes) {
  constexpr int U = kTileBytes / 16 / kThreads;
  const int tid = threadIdx.x;
  const int64_t chunks = bytes >> 4;
  if (chunks == (int64_t)U * kThreads) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = ld_stream(src + (int64_t)(tid + u * kThreads) * 16);
#pragma unroll
    for (int u = 0; u < U; ++u) st_stream(dst + (int64_t)(tid + u * kThreads) * 16, v[u]);
  } else {
    for (int64_t c = tid; c < chunks; c += kThreads) st_stream(dst + c * 16, ld_stream(src + c * 16));
  }
}

// Rotate rows of one slot. HALF: lane pairs column chunk q of the first half with
// chunk q of the second half (P = chunks per half row). INTERLEAVED: lane owns
// chunk c of the row, whose EPC elements are EPC/2 adjacent pairs.
template <int ESIZE, int STYLE>
__device__ __forceinline__ void rotate_tile(const uint8_t* __restrict__ src,
                                            uint8_t* __restrict__ dst, int64_t rows, int d,
                                            const double* __restrict__ cs) {
#pragma clang fp contract(off)
  using C = Chunk<ESIZE>;
  constexpr int E = C::E;
  const int row_bytes = d * ESIZE;
  const int tid = threadIdx.x;
  if constexpr (STYLE == CM_ROPE_HALF) {
    const int P = row_bytes >> 5;          // 16-byte chunks per half row
    const int rpi = kThreads / P;          // rows per iteration
    const int q = tid % P;
    const int rsub = tid / P;
    const int half = row_bytes >> 1;
    double c[E], sn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      c[e] = cs[2 * (q * E + e)];
      sn[e] = cs[2 * (q * E + e) + 1];
    }
    constexpr int U = kTileBytes / 32 / kThreads;  // iterations of a full tile
    auto body = [&](const u32x4 a, const u32x4 b, u32x4& ya, u32x4& yb) {
      double x1[E], x2[E], y1[E], y2[E];
      C::unpack(a, x1);
      C::unpack(b, x2);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        y1[e] = x1[e] * c[e] - x2[e] * sn[e];
        y2[e] = x2[e] * c[e] + x1[e] * sn[e];
      }
      ya = C::pack(y1);
      yb = C::pack(y2);
    };
    if (rows == (int64_t)U * rpi) {
      u32x4 a[U], b[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t off = (int64_t)(rsub + u * rpi) * row_bytes + q * 16;
        a[u] = ld_stream(src + off);
        b[u] = ld_stream(src + off + half);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t off = (int64_t)(rsub + u * rpi) * row_bytes + q * 16;
        u32x4 ya, yb;
        body(a[u], b[u], ya, yb);
        st_stream(dst + off, ya);
        st_stream(dst + off + half, yb);
      }
    } else {
      for (int64_t r = rsub; r < rows; r += rpi) {
        const int64_t off = r * row_bytes + q * 16;
        u32x4 ya, yb;
        body(ld_stream(src + off), ld_stream(src + off + half), ya, yb);
        st_stream(dst + off, ya);
        st_stream(dst + off + half, yb);
      }
    }
  } else {
    const int CPR = row_bytes >> 4;        // chunks per row
    const int rpi = kThreads / CPR;
    const int cq = tid % CPR;
    const int rsub = tid / CPR;
    constexpr int PP = E / 2;              // pairs per chunk
    double c[PP], sn[PP];
#pragma unroll
    for (int p = 0; p < PP; ++p) {
      c[p] = cs[2 * (cq * PP + p)];
      sn[p] = cs[2 * (cq * PP + p) + 1];
    }
    for (int64_t r = rsub; r < rows; r += rpi) {
      const int64_t off = r * row_bytes + cq * 16;
      double x[E], y[E];
      C::unpack(ld_stream(src + off), x);
#pragma unroll
      for (int p = 0; p < PP; ++p) {
        y[2 * p] = x[2 * p] * c[p] - x[2 * p + 1] * sn[p];
        y[2 * p + 1] = x[2 * p + 1] * c[p] + x[2 * p] * sn[p];
      }
      st_stream(dst + off, C::pack(y));
    }
  }
}

// grid (tiles per (l, kv, h), 2*L*H); block (x, y) moves tile x of row block
// y = (l*2 + kv)*H + h of the output.
template <int ESIZE, int STYLE>
__global__ __launch_bounds__(kThreads) void render_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ tile_base, int32_t n_unique, const double* __restrict__ angles,
    int32_t H, int32_t d, int64_t T_out, int32_t tile_rows, uint8_t* __restrict__ out) {
  const int64_t k = blockIdx.x;
  const int32_t lkh = blockIdx.y;
  int lo = 0, hi = n_unique - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tile_base[mid] <= k) lo = mid; else hi = mid - 1;
  }
  const int s = lo;
  const int64_t src_i = plan[CM_PLAN_HEADER + s];
  const int64_t off = plan[CM_PLAN_HEADER + n + s];
  const int64_t len = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
  const int64_t r0 = (k - tile_base[s]) * tile_rows;
  const int64_t rows = len - r0 < tile_rows ? len - r0 : tile_rows;
  if (rows <= 0) return;
  const int h = lkh % H;
  const int lk = lkh / H;
  const int kv = lk & 1;
  const int l = lk >> 1;
  const int64_t row_bytes = (int64_t)d * ESIZE;
  const uint8_t* src = reinterpret_cast<const uint8_t*>(table[src_i * stride + 1 + 2 * l + kv]) +
                       ((int64_t)h * len + r0) * row_bytes;
  uint8_t* dst = out + ((int64_t)lkh * T_out + off + r0) * row_bytes;
  if (kv == 1 || off == 0)
    copy_tile(src, dst, rows * row_bytes);
  else
    rotate_tile<ESIZE, STYLE>(src, dst, rows, d, angles + (int64_t)s * d);
}

// One workgroup: per-slot work-unit bases (exclusive scan of the units of each
// slot: ceil(len / tile_rows) tiles, or 2L * stripes for the fused hash+render)
// and cos/sin(off_s * theta_j), theta_j = base^(-2j/d), in fp64. With a select
// mask it also writes hsel[i] = 0 for the slot deliveries whose Id the fused
// kernel computes (select[i] == 0), 1 for every other delivery.
__global__ __launch_bounds__(1024) void render_prep_kernel(
    const int64_t* __restrict__ plan, int32_t n, int32_t d, double base, int32_t tile_rows,
    int32_t stripe_mode, int64_t tensor_pairs, int64_t token_bytes,
    const uint8_t* __restrict__ select, uint8_t* __restrict__ hsel,
    int64_t* __restrict__ unit_base, double* __restrict__ angles) {
  __shared__ int64_t sc[1024];
  const int tid = threadIdx.x;
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t len = tid < n_u ? plan[CM_PLAN_HEADER + 2 * (int64_t)n + tid] : 0;
  int64_t x = 0;
  if (tid < n_u)
    x = stripe_mode ? 2 * tensor_pairs * stripes_of(len * token_bytes)
                    : (len + tile_rows - 1) / tile_rows;
  sc[tid] = x;
  if (hsel && tid < n) hsel[tid] = 1;
  __syncthreads();
  for (int o = 1; o < (int)blockDim.x; o <<= 1) {
    const int64_t t = tid >= o ? sc[tid - o] : 0;
    __syncthreads();
    sc[tid] += t;
    __syncthreads();
  }
  if (tid < n_u) unit_base[tid] = sc[tid] - x;
  if (tid == (int)blockDim.x - 1) unit_base[n_u] = sc[tid];
  if (hsel && tid < n_u) {
    const int64_t i = plan[CM_PLAN_HEADER + tid];
    if (select[i] == 0) hsel[i] = 0;
  }
  const int halfd = d >> 1;
  for (int idx = tid; idx < n_u * halfd; idx += blockDim.x) {
    const int s = idx / halfd;
    const int j = idx - s * halfd;
    const double theta = pow(base, -(double)(2 * j) / (double)d);
    const double phi = (double)plan[CM_PLAN_HEADER + n + s] * theta;
    angles[2 * idx] = cos(phi);
    angles[2 * idx + 1] = sin(phi);
  }
}

template <int ESIZE>
hipError_t launch_render_t(const SetDesc& s, const RenderLayout& lay, const int64_t* plan,
                           int32_t n_unique, int64_t total_tiles, int64_t T_out, int32_t style,
                           void* out, uint8_t* ws, hipStream_t stream) {
  const int64_t* tiles = reinterpret_cast<const int64_t*>(ws + lay.off_tiles);
  const double* angles = reinterpret_cast<const double*>(ws + lay.off_angles);
  const dim3 grid((uint32_t)total_tiles, (uint32_t)(2 * s.L * s.H));
  ScopedTiming tm(K_RENDER, stream);
  if (style == CM_ROPE_HALF)
    hipLaunchKernelGGL((render_kernel<ESIZE, CM_ROPE_HALF>), grid, dim3(kThreads), 0, stream,
                       s.table_dev, s.stride, s.n, plan, tiles, n_unique, angles, s.H, s.d, T_out,
                       lay.tile_rows, reinterpret_cast<uint8_t*>(out));
  else
    hipLaunchKernelGGL((render_kernel<ESIZE, CM_ROPE_INTERLEAVED>), grid, dim3(kThreads), 0,
                       stream, s.table_dev, s.stride, s.n, plan, tiles, n_unique, angles, s.H, s.d,
                       T_out, lay.tile_rows, reinterpret_cast<uint8_t*>(out));
  return hipGetLastError();
}

}  // namespace

RenderLayout render_layout(const SetDesc& s) {
  RenderLayout lay{};
  lay.tile_rows = (int32_t)(kTileBytes / s.row_bytes);
  lay.off_tiles = 0;
  lay.off_angles = align_up(sizeof(int64_t) * (size_t)(s.n + 1), kWsAlign);
  lay.off_hsel = align_up(lay.off_angles + sizeof(double) * (size_t)s.n * (size_t)s.d, kWsAlign);
  lay.bytes = align_up(lay.off_hsel + (size_t)s.n, kWsAlign);
  return lay;
}

hipError_t launch_render_prep(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                              int32_t n_unique, double base, bool stripe_tasks,
                              const uint8_t* select, uint8_t* ws, hipStream_t stream) {
  ScopedTiming tm(K_RENDER_PREP, stream);
  int threads = 64;
  const int need = n_unique > s.n ? n_unique : s.n;
  while (threads < need) threads <<= 1;
  hipLaunchKernelGGL(render_prep_kernel, dim3(1), dim3(threads), 0, stream, plan_dev, s.n, s.d,
                     base, lay.tile_rows, stripe_tasks ? 1 : 0, (int64_t)s.L, token_bytes_of(s),
                     select, select ? ws + lay.off_hsel : nullptr,
                     reinterpret_cast<int64_t*>(ws + lay.off_tiles),
                     reinterpret_cast<double*>(ws + lay.off_angles));
  return hipGetLastError();
}

hipError_t launch_render(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                         int32_t n_unique, int64_t total_tiles, int64_t T_out, double base,
                         int32_t style, void* out, uint8_t* ws, hipStream_t stream) {
  hipError_t e = launch_render_prep(s, lay, plan_dev, n_unique, base, false, nullptr, ws, stream);
  if (e != hipSuccess) return e;
  if (s.esize == 2)
    return launch_render_t<2>(s, lay, plan_dev, n_unique, total_tiles, T_out, style, out, ws, stream);
  return launch_render_t<4>(s, lay, plan_dev, n_unique, total_tiles, T_out, style, out, ws, stream);
}

}  // namespace cm
