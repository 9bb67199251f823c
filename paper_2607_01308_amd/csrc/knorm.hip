// Step 2 — score of Eq. (3) / Alg. 1: S_i = sum over heads and the last T* rows
// of the routing layer's K of the row L2 norms (rho_i = S_i / (H T*)).
//
// The summation order is fixed so that the key is bit-identical on any device
// and in the CPU oracle: squares in fp64 (exact for bf16 and fp32 inputs), each
// row summed by a level-wise adjacent-pair tree over d, correctly rounded sqrt,
// and the H*T* row norms (flattened (h, r), zero-padded to a power of two)
// summed by the same kind of tree. A row is spread over d*e/16 consecutive
// lanes (one 16-byte load each): the lane's own elements form the bottom levels
// of the row tree in registers and an xor-butterfly over those lanes forms the
// upper levels (fp addition is commutative, so both partners hold the same
// node). An aligned block of up to 256 row norms is one subtree, reduced in LDS;
// further levels run as small tree launches, the last few of them, where a
// one-workgroup kernel follows, inside that kernel (knorm_fold.h). Reads only
// the H*T*d*e tail bytes of one layer per fragment.
#include "internal.h"
#include "knorm_fold.h"

namespace cm {

namespace {

// In-place level-wise adjacent-pair tree over sh[0..count), count a power of two.
__device__ __forceinline__ double lds_tree(double* sh, int count) {
  const int tid = threadIdx.x;
  for (int w = count >> 1; w >= 1; w >>= 1) {
    double t = 0.0;
    if (tid < w) t = sh[2 * tid] + sh[2 * tid + 1];
    __syncthreads();
    if (tid < w) sh[tid] = t;
    __syncthreads();
  }
  return sh[0];
}

constexpr int kInFlight = 16;   // row loads in flight per thread

// Where row t of head h of fragment i's routing-layer K lives: a dense
// [1, H, T, d] tensor named by the fragment table, or a page of a paged pool
// ([L][2][P][H][B][d], the fragment's row t in row t % B of its page t / B).
struct DenseRows {
  const int64_t* table;
  int64_t stride;
  int32_t layer;
  __device__ __forceinline__ int64_t length(int i) const { return table[(int64_t)i * stride]; }
  __device__ __forceinline__ const uint8_t* row(int i, int64_t T, int64_t h, int64_t t,
                                                int rb_shift) const {
    return reinterpret_cast<const uint8_t*>(table[(int64_t)i * stride + 1 + 2 * layer]) +
           ((h * T + t) << rb_shift);
  }
};

struct PagedRows {
  const uint8_t* pool;
  const int64_t* table;    // {T_i, first page index}
  const int32_t* blocks;
  int64_t P;
  int32_t H, b_shift, layer;
  __device__ __forceinline__ int64_t length(int i) const { return table[2 * (int64_t)i]; }
  __device__ __forceinline__ const uint8_t* row(int i, int64_t, int64_t h, int64_t t,
                                                int rb_shift) const {
    const int64_t page = blocks[table[2 * (int64_t)i + 1] + (t >> b_shift)];
    const int64_t r = ((((int64_t)2 * layer * P + page) * H + h) << b_shift) +
                      (t & (((int64_t)1 << b_shift) - 1));
    return pool + (r << rb_shift);
  }
};

// grid (count0, n), 256 threads: block b of fragment i sums rows
// [b*rpb, (b+1)*rpb) of the padded (h, r) row space.
template <int ESIZE, class Rows>
__global__ __launch_bounds__(256) void knorm_rows_kernel(Rows src, int64_t tail, int32_t d,
                                                         int64_t rows, int32_t rpb,
                                                         int64_t count0,
                                                         double* __restrict__ out) {
#pragma clang fp contract(off)
  __shared__ double sh[256];
  const int i = blockIdx.y;
  const int64_t blk = blockIdx.x;
  const int64_t T = src.length(i);
  const int row_bytes = d * ESIZE;
  const int rb_shift = __builtin_ctz((unsigned)row_bytes);
  const int lpr = row_bytes >> 4;  // lanes per row: a power of two in [4, 64]
  const int rpp = 256 / lpr;       // rows per pass
  const int tid = threadIdx.x;
  const int q = tid & (lpr - 1);
  // kInFlight passes at a time: their loads are all issued before the first is
  // used, so the block waits for memory once per group instead of once per pass
  // row f = h * tail + r of the (h, r) space: one division for the thread's
  // first row, then steps of rpp rows
  const int64_t f0 = blk * rpb + tid / lpr;
  int64_t h = f0 / tail;
  int64_t r = f0 - h * tail;
  for (int p0 = 0; p0 < rpb; p0 += rpp * kInFlight) {
    u32x4 v[kInFlight];
    bool valid[kInFlight];
#pragma unroll
    for (int g = 0; g < kInFlight; ++g) {
      const int fl = p0 + g * rpp + tid / lpr;
      const int64_t f = blk * rpb + fl;
      valid[g] = fl < rpb && f < rows;
      v[g] = u32x4{0u, 0u, 0u, 0u};
      if (valid[g]) v[g] = *global_ptr<u32x4>(src.row(i, T, h, T - tail + r, rb_shift) + q * 16);
      r += rpp;
      if (r >= tail) {               // a division only for tails shorter than a pass
        const int64_t k = r < 2 * tail ? 1 : r / tail;
        h += k;
        r -= k * tail;
      }
    }
    // each level of the butterfly over all kInFlight rows before the next, so
    // their cross-lane moves overlap instead of forming one long chain
    double acc[kInFlight];
#pragma unroll
    for (int g = 0; g < kInFlight; ++g) acc[g] = valid[g] ? row_chunk_sumsq<ESIZE>(v[g]) : 0.0;
    for (int o = 1; o < lpr; o <<= 1) {
#pragma unroll
      for (int g = 0; g < kInFlight; ++g) acc[g] = acc[g] + __shfl_xor(acc[g], o, 64);
    }
#pragma unroll
    for (int g = 0; g < kInFlight; ++g) {
      const int fl = p0 + g * rpp + tid / lpr;
      if (fl < rpb && q == 0) sh[fl] = valid[g] ? sqrt(acc[g]) : 0.0;
    }
  }
  __syncthreads();
  const double s = lds_tree(sh, rpb);
  if (tid == 0) out[(int64_t)i * count0 + blk] = s;
}

// grid (cout, n), g threads: out[i][b] = tree of in[i][b*g .. b*g+g).
__global__ __launch_bounds__(256) void knorm_tree_kernel(const double* __restrict__ in,
                                                         int64_t cin, double* __restrict__ out,
                                                         int64_t cout) {
#pragma clang fp contract(off)
  __shared__ double sh[256];
  const int i = blockIdx.y;
  const int g = blockDim.x;
  sh[threadIdx.x] = in[(int64_t)i * cin + (int64_t)blockIdx.x * g + threadIdx.x];
  __syncthreads();
  const double s = lds_tree(sh, g);
  if (threadIdx.x == 0) out[(int64_t)i * cout + blockIdx.x] = s;
}

int64_t next_pow2(int64_t x) {
  int64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

}  // namespace

KnormLayout knorm_layout(const SetDesc& s, int64_t tail_len) {
  KnormLayout lay{};
  lay.rows = (int64_t)s.H * tail_len;
  lay.padded = next_pow2(lay.rows);
  // one subtree of 256 rows per workgroup, or of fewer (down to 64) when that
  // leaves too few workgroups to keep the loads of a short tail in flight (2048:
  // eight per CU)
  int64_t rpb = lay.padded < 256 ? lay.padded : 256;
  while (rpb > 64 && (int64_t)s.n * (lay.padded / rpb) < 2048) rpb >>= 1;
  lay.rows_per_block = (int32_t)rpb;
  lay.count0 = lay.padded / lay.rows_per_block;
  const size_t a = sizeof(double) * (size_t)s.n * (size_t)lay.count0;
  const size_t b = sizeof(double) * (size_t)s.n * (size_t)((lay.count0 + 255) / 256);
  lay.off_a = 0;
  lay.off_b = align_up(a, kWsAlign);
  lay.bytes = align_up(lay.off_b + b, kWsAlign);
  return lay;
}

size_t knorm_max_bytes(const SetDesc& s) {
  int64_t tmin = s.T(0);
  for (int i = 1; i < s.n; ++i)
    if (s.T(i) < tmin) tmin = s.T(i);
  return knorm_layout(s, tmin).bytes;  // grows with tail_len, which is at most min T
}

namespace {

// knorm_rows over `src`, then tree launches down to fold_max partial sums.
template <class Rows>
hipError_t knorm_launches(const SetDesc& s, const KnormLayout& lay, Rows src, int64_t tail_len,
                          double* keys, uint8_t* ws, hipStream_t stream, int64_t fold_max,
                          KnormPartials* out) {
  double* bufs[2] = {reinterpret_cast<double*>(ws + lay.off_a),
                     reinterpret_cast<double*>(ws + lay.off_b)};
  {
    ScopedTiming tm(K_KNORM_ROWS, stream);
    double* o = lay.count0 == 1 ? keys : bufs[0];
    const dim3 grid((uint32_t)lay.count0, (uint32_t)s.n);
    if (s.esize == 2)
      hipLaunchKernelGGL((knorm_rows_kernel<2, Rows>), grid, dim3(256), 0, stream, src, tail_len,
                         s.d, lay.rows, lay.rows_per_block, lay.count0, o);
    else
      hipLaunchKernelGGL((knorm_rows_kernel<4, Rows>), grid, dim3(256), 0, stream, src, tail_len,
                         s.d, lay.rows, lay.rows_per_block, lay.count0, o);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t c = lay.count0;
  int cur = 0;
  while (c > 1 && (int64_t)s.n * c > fold_max) {
    // one launch takes up to 8 levels; the last one folds no further than needed
    int64_t g = c < 256 ? c : 256;
    while (g > 2 && (int64_t)s.n * (c / (g >> 1)) <= fold_max) g >>= 1;
    const int64_t cout = c / g;
    double* o = cout == 1 ? keys : bufs[cur ^ 1];
    ScopedTiming tm(K_KNORM_TREE, stream);
    hipLaunchKernelGGL(knorm_tree_kernel, dim3((uint32_t)cout, (uint32_t)s.n), dim3((uint32_t)g),
                       0, stream, bufs[cur], c, o, cout);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    cur ^= 1;
    c = cout;
  }
  out->parts = c == 1 ? keys : bufs[cur];
  out->count = c;
  return hipSuccess;
}

}  // namespace

hipError_t launch_knorm_partial(const SetDesc& s, const KnormLayout& lay, int32_t layer,
                                int64_t tail_len, double* keys, uint8_t* ws, hipStream_t stream,
                                int64_t fold_max, KnormPartials* out) {
  // a small set (Tiny: 64 rows) is scored inside the consumer: no launch
  const int64_t leaves = (int64_t)s.n * lay.padded;
  if (fold_max >= kKnormFoldMax && leaves <= kKnormFoldMax &&
      leaves * (s.row_bytes / 16) <= kKnormDirectPieces) {
    out->parts = nullptr;
    out->count = lay.padded;
    out->direct = KnormDirect{layer, s.esize, tail_len, lay.padded};
    return hipSuccess;
  }
  return knorm_launches(s, lay, DenseRows{s.table_dev, s.stride, layer}, tail_len, keys, ws,
                        stream, fold_max, out);
}

hipError_t launch_knorm_paged(const PagedDesc& p, const KnormLayout& lay, int32_t layer,
                              int64_t tail_len, double* keys, uint8_t* ws, hipStream_t stream) {
  KnormPartials kp;
  const PagedRows src{static_cast<const uint8_t*>(p.pool), p.s.table_dev, p.blocks_dev, p.pages,
                      p.s.H, p.b_shift, layer};
  return knorm_launches(p.s, lay, src, tail_len, keys, ws, stream, 1, &kp);
}

hipError_t launch_knorm(const SetDesc& s, const KnormLayout& lay, int32_t layer, int64_t tail_len,
                        double* keys, uint8_t* ws, hipStream_t stream) {
  KnormPartials kp;
  return launch_knorm_partial(s, lay, layer, tail_len, keys, ws, stream, 1, &kp);
}

}  // namespace cm
