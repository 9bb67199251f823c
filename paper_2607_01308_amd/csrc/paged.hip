// Steps 4-5 over paged storage (§4.5: the merge as a permutation of blocks that
// are already allocated, plus the RoPE rotation). The block tables of the merged
// cache reuse fragment pages wherever a merged block is one whole fragment page
// (every V page of a page-aligned slot, K only at offset 0); this kernel writes
// the other pages, one 64-lane workgroup per (fresh page, layer, head): the
// page's B rows of that head, B * row_bytes bytes, 16 bytes per lane and piece,
// pieces 1 KiB apart (one column per lane, so the lane's angles are loaded once
// when the page comes from one slot). A prep pass resolves each fresh page to
// its slot and the one or two fragment pages its rows come from.
#include "rotate.h"

namespace cm {

namespace {

// Per fresh page (one lane each): what the render of that page needs, so that a
// wave's data loads wait on one scalar load. desc[2f] = {out page, kv | one_slot
// << 1, slot s of the block's first row, fragment page A holding that row},
// desc[2f + 1] = {the fragment's page after A (or -1), row of the first row in
// A, rows of the block in use, block index j}. one_slot: every row of the block
// comes from slot s. out page -1: not a block of this merged cache.
__global__ __launch_bounds__(256) void paged_prep_kernel(
    const int64_t* __restrict__ table, const int32_t* __restrict__ blocks,
    const int64_t* __restrict__ plan, int32_t n, int32_t b_shift,
    const int32_t* __restrict__ k_table, const int32_t* __restrict__ v_table,
    const int32_t* __restrict__ fresh, int64_t n_fresh, int4* __restrict__ desc) {
  const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (f >= n_fresh) return;
  const int32_t code = fresh[f];
  const int64_t B = (int64_t)1 << b_shift;
  const int64_t T_out = plan[CM_PLAN_TOUT];
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t j = code >> 1;
  const int kv = code & 1;
  int4 lo = make_int4(-1, 0, 0, 0), hi = make_int4(-1, 0, 0, 0);
  if (code >= 0 && j * B < T_out) {
    const int64_t* offs = plan + CM_PLAN_HEADER + n;
    const int64_t r0 = j * B;
    const int64_t rows = (r0 + B < T_out ? r0 + B : T_out) - r0;
    int s = 0, top = n_u - 1;
    while (s < top) {
      const int mid = (s + top + 1) >> 1;
      if (offs[mid] <= r0) s = mid; else top = mid - 1;
    }
    const bool one_slot = s + 1 >= n_u || offs[s + 1] > r0 + rows - 1;
    const int64_t i = plan[CM_PLAN_HEADER + s];
    const int64_t T = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
    const int64_t t0 = r0 - offs[s];
    const int64_t first = table[2 * i + 1];
    const int64_t k0 = t0 >> b_shift;
    const bool has_next = (k0 + 1) * B < T;
    lo = make_int4((kv ? v_table : k_table)[j], kv | (one_slot ? 2 : 0), s, blocks[first + k0]);
    hi = make_int4(has_next ? blocks[first + k0 + 1] : -1, (int)(t0 & (B - 1)), (int)rows, (int)j);
  }
  desc[2 * f] = lo;
  desc[2 * f + 1] = hi;
}

// Grid (fresh pages x H, L): consecutive workgroups write the heads of one
// page, i.e. one contiguous page of the pool after another.
template <int ESIZE, int STYLE, int HB>
__global__ __launch_bounds__(64) void paged_render_kernel(
    uint8_t* __restrict__ pool, int64_t P, int32_t b_shift, const int64_t* __restrict__ table,
    const int32_t* __restrict__ blocks, const int64_t* __restrict__ plan, int32_t n,
    const double* __restrict__ angles, const int4* __restrict__ desc, int32_t H, int32_t d,
    int32_t pieces) {
  constexpr int EP = 16 / ESIZE;
  constexpr int NA = STYLE == CM_ROPE_HALF ? EP : EP / 2;
  const int lane = threadIdx.x;
  const int rb_shift = __builtin_ctz((unsigned)(d * ESIZE));
  const int64_t row_mask = ((int64_t)1 << rb_shift) - 1;
  const int ppr = (d * ESIZE) >> 4;
  const int64_t f = blockIdx.x / H;
  const int h = (int)(blockIdx.x - f * H);
  const int l = blockIdx.y;
  const int4 d0 = desc[2 * f], d1 = desc[2 * f + 1];
  const int64_t out_page = d0.x;
  if (out_page < 0 || out_page >= P) return;
  const int kv = d0.y & 1;
  const bool one_slot = (d0.y & 2) != 0;
  const int s0 = d0.z;
  const int64_t B = (int64_t)1 << b_shift;
  const int64_t* offs = plan + CM_PLAN_HEADER + n;
  const int64_t page_bytes = (int64_t)H << (b_shift + rb_shift);
  const int64_t head_off = (int64_t)h << (b_shift + rb_shift);
  const int64_t lk = 2 * (int64_t)l + kv;
  uint8_t* dst = pool + (lk * P + out_page) * page_bytes + head_off;
  const uint8_t* src_pool = pool + lk * P * page_bytes + head_off;
  const int cp = (int)(((lane * 16) & row_mask) >> 4);
  if (one_slot) {
    const bool rotate = kv == 0 && offs[s0] != 0;
    double cs[NA], sn[NA];
    if (rotate) piece_angles<ESIZE, STYLE>(angles + (int64_t)s0 * d, cp, ppr, cs, sn);
    // kBatch pieces at a time: all their loads are issued before the first store
    constexpr int kBatch = 4;
    for (int k0 = 0; k0 < pieces; k0 += kBatch) {
      u32x4 x[kBatch];
      bool valid[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int64_t b = lane * 16 + 1024 * (int64_t)(k0 + u);   // byte of the page's [B][row] block
        const int64_t row_in = b >> rb_shift;
        const int64_t q = d1.y + row_in;                 // row counted from page A's start
        const int64_t page = q < B ? d0.w : d1.x;
        valid[u] = k0 + u < pieces && row_in < d1.z;
        x[u] = u32x4{0u, 0u, 0u, 0u};
        if (valid[u])
          x[u] = ld16(src_pool + page * page_bytes + ((q & (B - 1)) << rb_shift) + (b & row_mask));
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (k0 + u >= pieces) break;                    // uniform over the wave
        u32x4 y = x[u];
        if constexpr (STYLE == CM_ROPE_HALF) {
          const u32x4 p = lane_xor4<HB>(x[u]);           // every lane takes part
          if (rotate) y = rotate_piece_half<ESIZE>(x[u], p, cs, sn);
        } else {
          if (rotate) y = rotate_piece_il<ESIZE>(x[u], cs, sn);
        }
        if (valid[u]) st_stream(dst + lane * 16 + 1024 * (int64_t)(k0 + u), y);
      }
    }
    return;
  }
  // the block crosses a slot boundary: slot, fragment page and angles per lane
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t r0 = (int64_t)d1.w << b_shift;
  for (int k = 0; k < pieces; ++k) {
    const int64_t b = lane * 16 + 1024 * (int64_t)k;
    const int64_t row_in = b >> rb_shift;
    const int64_t r = r0 + row_in;
    const bool valid = row_in < d1.z;
    int s = s0;
    while (s + 1 < n_u && offs[s + 1] <= r) ++s;
    const int64_t i = plan[CM_PLAN_HEADER + s];
    const int64_t off = offs[s];
    u32x4 x = {0u, 0u, 0u, 0u};
    if (valid) {
      const int64_t t = r - off;                       // row of fragment i
      const int64_t page = blocks[table[2 * i + 1] + (t >> b_shift)];
      x = ld16(src_pool + page * page_bytes + ((t & (B - 1)) << rb_shift) + (b & row_mask));
    }
    const bool rotate = kv == 0 && off != 0;
    u32x4 y = x;
    double cs[NA], sn[NA];
    if constexpr (STYLE == CM_ROPE_HALF) {
      const u32x4 p = lane_xor4<HB>(x);              // every lane takes part
      if (rotate) {
        piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cs, sn);
        y = rotate_piece_half<ESIZE>(x, p, cs, sn);
      }
    } else {
      if (rotate) {
        piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cs, sn);
        y = rotate_piece_il<ESIZE>(x, cs, sn);
      }
    }
    if (valid) st_stream(dst + b, y);
  }
}

// Block tables of a plan's merged cache, built on the device by one workgroup
// with the rule of cm_paged_tables: merged block j (rows [jB, min(jB + B,
// T_out))) keeps the page of its slot's fragment when all its rows come from
// that slot and start at one of the fragment's page boundaries (V), and the
// slot is at offset 0 (K: R(0) = I); every other block takes the next page of
// `free` in block order, K before V. Each thread takes a run of consecutive
// blocks: a count, a scan of the counts, then the assignment. A free list too
// short for the plan leaves the tables unwritten and the plan's status
// CM_EINVAL (n_fresh: the pages needed), so nothing is rendered; a plan whose
// status is already an error is left as it is (n_fresh: 0).
__global__ __launch_bounds__(1024) void paged_tables_kernel(
    int64_t* __restrict__ plan, int32_t n, const int64_t* __restrict__ table,
    const int32_t* __restrict__ blocks, int32_t b_shift, const int32_t* __restrict__ free_pages,
    int64_t n_free, int64_t nbo_cap, int32_t* __restrict__ k_table,
    int32_t* __restrict__ v_table, int64_t* __restrict__ n_fresh) {
  __shared__ int64_t s_off[CM_MAX_FRAGMENTS];
  __shared__ int64_t s_len[CM_MAX_FRAGMENTS];
  __shared__ int64_t s_first[CM_MAX_FRAGMENTS];
  __shared__ int64_t scan[1024];
  const int tid = threadIdx.x, nt = blockDim.x;
  if (plan[CM_PLAN_STATUS] != CM_OK) {
    if (tid == 0) *n_fresh = 0;
    return;
  }
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t T_out = plan[CM_PLAN_TOUT];
  const int64_t B = (int64_t)1 << b_shift;
  const int64_t nbo = (T_out + B - 1) >> b_shift;
  if (n_u < 1 || n_u > n || nbo > nbo_cap) {     // not a plan of this set (checked on the
    if (tid == 0) {                              // host for every other entry point)
      *n_fresh = 0;
      plan[CM_PLAN_STATUS] = CM_ESHAPE;
    }
    return;
  }
  for (int s = tid; s < n_u; s += nt) {
    s_off[s] = plan[CM_PLAN_HEADER + n + s];
    s_len[s] = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
    s_first[s] = table[2 * plan[CM_PLAN_HEADER + s] + 1];
  }
  __syncthreads();
  const int64_t per = (nbo + nt - 1) / nt;
  const int64_t j0 = (int64_t)tid * per < nbo ? (int64_t)tid * per : nbo;
  const int64_t j1 = j0 + per < nbo ? j0 + per : nbo;
  // slot holding row j0 * B (offsets increase over the slots)
  int s0 = 0;
  {
    int hi = n_u - 1;
    while (s0 < hi) {
      const int mid = (s0 + hi + 1) >> 1;
      if (s_off[mid] <= j0 * B) s0 = mid; else hi = mid - 1;
    }
  }
  // block j: the fragment page it may keep (-1: none) and whether K may keep it
  auto reuse = [&](int64_t j, int& s, int32_t& page, bool& k_too) {
    const int64_t r0 = j * B;
    while (s + 1 < n_u && s_off[s + 1] <= r0) ++s;
    const int64_t e = r0 + B < T_out ? r0 + B : T_out;
    const int64_t t0 = r0 - s_off[s];
    const bool whole = e <= s_off[s] + s_len[s] && (t0 & (B - 1)) == 0;
    page = whole ? blocks[s_first[s] + (t0 >> b_shift)] : -1;
    k_too = s_off[s] == 0;
  };
  int64_t cnt = 0;
  {
    int s = s0;
    for (int64_t j = j0; j < j1; ++j) {
      int32_t page;
      bool k_too;
      reuse(j, s, page, k_too);
      cnt += (page >= 0 ? 0 : 1) + ((page >= 0 && k_too) ? 0 : 1);
    }
  }
  scan[tid] = cnt;
  __syncthreads();
  for (int o = 1; o < nt; o <<= 1) {
    const int64_t t = tid >= o ? scan[tid - o] : 0;
    __syncthreads();
    scan[tid] += t;
    __syncthreads();
  }
  const int64_t total = scan[nt - 1];
  if (total > n_free) {
    if (tid == 0) {
      *n_fresh = total;
      plan[CM_PLAN_STATUS] = CM_EINVAL;
    }
    return;
  }
  int64_t next = scan[tid] - cnt;
  int s = s0;
  for (int64_t j = j0; j < j1; ++j) {
    int32_t page;
    bool k_too;
    reuse(j, s, page, k_too);
    k_table[j] = (page >= 0 && k_too) ? page : free_pages[next++];
    v_table[j] = page >= 0 ? page : free_pages[next++];
  }
  if (tid == 0) *n_fresh = total;
}

}  // namespace

hipError_t launch_paged_tables(const PagedDesc& p, int64_t* plan_dev, const int32_t* free_dev,
                               int64_t n_free, int64_t nbo_cap, int32_t* k_table,
                               int32_t* v_table, int64_t* n_fresh, hipStream_t stream) {
  ScopedTiming tm(K_RENDER_PREP, stream);
  hipLaunchKernelGGL(paged_tables_kernel, dim3(1), dim3(1024), 0, stream, plan_dev, p.s.n,
                     p.s.table_dev, p.blocks_dev, p.b_shift, free_dev, n_free, nbo_cap, k_table,
                     v_table, n_fresh);
  return hipGetLastError();
}

hipError_t launch_paged_render(const PagedDesc& p, const int64_t* plan_dev, int32_t n_unique,
                               double base, int32_t style, const int32_t* k_table,
                               const int32_t* v_table, const int32_t* fresh, int64_t n_fresh,
                               uint8_t* ws, hipStream_t stream) {
  RenderLayout lay{};                 // angles at the start of the workspace
  hipError_t e = launch_render_prep(p.s, lay, plan_dev, n_unique, base, style, 0, nullptr, ws,
                                    stream);
  if (e != hipSuccess || n_fresh == 0) return e;
  const double* angles = reinterpret_cast<const double*>(ws);
  int4* desc = reinterpret_cast<int4*>(ws + align_up(sizeof(double) * (size_t)p.s.n * p.s.d,
                                                     kWsAlign));
  {
    ScopedTiming tm(K_RENDER_PREP, stream);
    hipLaunchKernelGGL(paged_prep_kernel, dim3((uint32_t)((n_fresh + 255) / 256)), dim3(256), 0,
                       stream, p.s.table_dev, p.blocks_dev, plan_dev, p.s.n, p.b_shift, k_table,
                       v_table, fresh, n_fresh, desc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int32_t pieces = (int32_t)(((int64_t)p.block * p.s.row_bytes) >> 10);
  const dim3 grid((uint32_t)(n_fresh * p.s.H), (uint32_t)p.s.L);
  uint8_t* pool = static_cast<uint8_t*>(p.pool);
  ScopedTiming tm(K_PAGED, stream);
  auto go = [&](auto tag) {
    constexpr int STYLE = decltype(tag)::style, HB = decltype(tag)::hb;
    if (p.s.esize == 2)
      hipLaunchKernelGGL((paged_render_kernel<2, STYLE, HB>), grid, dim3(64), 0, stream, pool,
                         p.pages, p.b_shift, p.s.table_dev, p.blocks_dev, plan_dev, p.s.n, angles,
                         desc, p.s.H, p.s.d, pieces);
    else
      hipLaunchKernelGGL((paged_render_kernel<4, STYLE, HB>), grid, dim3(64), 0, stream, pool,
                         p.pages, p.b_shift, p.s.table_dev, p.blocks_dev, plan_dev, p.s.n, angles,
                         desc, p.s.H, p.s.d, pieces);
  };
  dispatch_style(style, p.s.row_bytes, go);
  return hipGetLastError();
}

}  // namespace cm
