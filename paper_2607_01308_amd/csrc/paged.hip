// Steps 4-5 over paged storage (§4.5: the merge as a permutation of blocks that
// are already allocated, plus the RoPE rotation). The block tables of the merged
// cache reuse fragment pages wherever a merged block is one whole fragment page
// (every V page of a page-aligned slot, K only at offset 0); this kernel writes
// the other pages, one 64-lane workgroup per (fresh page, layer, head): the
// page's B rows of that head, B * row_bytes bytes, 16 bytes per lane and piece,
// pieces 1 KiB apart (one column per lane, so the lane's angles are loaded once
// when the page comes from one slot). Rows are looked up through the plan's
// slot offsets and the fragment's page list.
#include "rotate.h"

namespace cm {

namespace {

template <int ESIZE, int STYLE, int HB>
__global__ __launch_bounds__(64) void paged_render_kernel(
    uint8_t* __restrict__ pool, int64_t P, int32_t b_shift, const int64_t* __restrict__ table,
    const int32_t* __restrict__ blocks, const int64_t* __restrict__ plan, int32_t n,
    const double* __restrict__ angles, const int32_t* __restrict__ k_table,
    const int32_t* __restrict__ v_table, const int32_t* __restrict__ fresh, int32_t H, int32_t d,
    int32_t pieces) {
  constexpr int EP = 16 / ESIZE;
  constexpr int NA = STYLE == CM_ROPE_HALF ? EP : EP / 2;
  const int lane = threadIdx.x;
  const int rb_shift = __builtin_ctz((unsigned)(d * ESIZE));
  const int64_t row_mask = ((int64_t)1 << rb_shift) - 1;
  const int ppr = (d * ESIZE) >> 4;
  const int l = blockIdx.y / H;
  const int h = blockIdx.y - l * H;
  const int32_t code = fresh[blockIdx.x];
  const int64_t j = code >> 1;
  const int kv = code & 1;
  const int64_t T_out = plan[CM_PLAN_TOUT];
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t B = (int64_t)1 << b_shift;
  if (code < 0 || j * B >= T_out) return;              // not a block of this merged cache
  const int64_t out_page = (kv ? v_table : k_table)[j];
  if (out_page < 0 || out_page >= P) return;
  const int64_t page_bytes = (int64_t)H << (b_shift + rb_shift);
  const int64_t lk = 2 * (int64_t)l + kv;
  uint8_t* dst = pool + (lk * P + out_page) * page_bytes + ((int64_t)h << (b_shift + rb_shift));
  const uint8_t* src_pool = pool + lk * P * page_bytes + ((int64_t)h << (b_shift + rb_shift));
  const int64_t* offs = plan + CM_PLAN_HEADER + n;
  const int64_t r0 = j * B;
  const int64_t r_last = (r0 + B < T_out ? r0 + B : T_out) - 1;
  int s0 = 0, hi = n_u - 1;                            // last slot with offset <= r0
  while (s0 < hi) {
    const int mid = (s0 + hi + 1) >> 1;
    if (offs[mid] <= r0) s0 = mid; else hi = mid - 1;
  }
  const bool one_slot = s0 + 1 >= n_u || offs[s0 + 1] > r_last;
  const int cp = (int)(((lane * 16) & row_mask) >> 4);
  double cs[NA], sn[NA];
  if (one_slot && kv == 0 && offs[s0] != 0)
    piece_angles<ESIZE, STYLE>(angles + (int64_t)s0 * d, cp, ppr, cs, sn);
  for (int k = 0; k < pieces; ++k) {
    const int64_t b = lane * 16 + 1024 * (int64_t)k;   // byte of the page's [B][row] block
    const int64_t r = r0 + (b >> rb_shift);
    const bool valid = r < T_out;
    int s = s0;
    if (!one_slot)
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
    if constexpr (STYLE == CM_ROPE_HALF) {
      const u32x4 p = lane_xor4<HB>(x);              // every lane takes part
      if (rotate) {
        double cl[NA], sl[NA];
        if (!one_slot) piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cl, sl);
        y = rotate_piece_half<ESIZE>(x, p, one_slot ? cs : cl, one_slot ? sn : sl);
      }
    } else {
      if (rotate) {
        double cl[NA], sl[NA];
        if (!one_slot) piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cl, sl);
        y = rotate_piece_il<ESIZE>(x, one_slot ? cs : cl, one_slot ? sn : sl);
      }
    }
    if (valid) st_stream(dst + b, y);
  }
}

}  // namespace

hipError_t launch_paged_render(const PagedDesc& p, const int64_t* plan_dev, int32_t n_unique,
                               double base, int32_t style, const int32_t* k_table,
                               const int32_t* v_table, const int32_t* fresh, int64_t n_fresh,
                               uint8_t* ws, hipStream_t stream) {
  RenderLayout lay{};                 // angles at the start of the workspace
  hipError_t e = launch_render_prep(p.s, lay, plan_dev, n_unique, base, style, 0, nullptr, ws,
                                    stream);
  if (e != hipSuccess || n_fresh == 0) return e;
  const double* angles = reinterpret_cast<const double*>(ws);
  const int32_t pieces = (int32_t)(((int64_t)p.block * p.s.row_bytes) >> 10);
  const dim3 grid((uint32_t)n_fresh, (uint32_t)(p.s.L * p.s.H));
  uint8_t* pool = static_cast<uint8_t*>(p.pool);
  ScopedTiming tm(K_PAGED, stream);
  auto go = [&](auto tag) {
    constexpr int STYLE = decltype(tag)::style, HB = decltype(tag)::hb;
    if (p.s.esize == 2)
      hipLaunchKernelGGL((paged_render_kernel<2, STYLE, HB>), grid, dim3(64), 0, stream, pool,
                         p.pages, p.b_shift, p.s.table_dev, p.blocks_dev, plan_dev, p.s.n, angles,
                         k_table, v_table, fresh, p.s.H, p.s.d, pieces);
    else
      hipLaunchKernelGGL((paged_render_kernel<4, STYLE, HB>), grid, dim3(64), 0, stream, pool,
                         p.pages, p.b_shift, p.s.table_dev, p.blocks_dev, plan_dev, p.s.n, angles,
                         k_table, v_table, fresh, p.s.H, p.s.d, pieces);
  };
  dispatch_style(style, p.s.row_bytes, go);
  return hipGetLastError();
}

}  // namespace cm
