// Steps 4-5 — Eq. (1)-(2): for every layer l, K/V and head h, the merged
// [T_out, d] block is the concatenation over slots s of the fragment rows, K
// multiplied by R(off_s) (byte copy when off_s = 0), V copied.
//
// HBM-bound streaming (about 0.4 flop per byte moved). On this chip a copy
// reaches its highest bandwidth when the grid walks memory in address order in
// small units, so the render is a one-shot grid of one-wave workgroups, each
// writing one 4 KiB unit of the merged cache in output order: block (x, y)
// writes bytes [4096 x, 4096 x + 4096) of row block y = (l*2 + kv)*H + h, lane
// pieces lane + 64 k (each load and store 1 KiB contiguous across the wave, all
// pieces of a lane in one column). The lookups are precomputed by a prep pass so
// that a wave's data load waits on two scalar loads only: the slot of its unit
// (every row block has the same row -> slot map) and the source base of that
// slot in its row block (render_tables.h). A unit crossing a slot boundary
// resolves the slot per lane. K at a non-zero offset is rotated with the
// partner piece fetched from the lane P pieces away.
#include "render_geometry.h"
#include "render_tables.h"

namespace cm {

namespace {

constexpr int kUnitPieces = kRenderUnitPieces;       // 16-byte pieces per lane
constexpr int kUnitBytes = kRenderUnitBytes;

template <int ESIZE, int STYLE, int HB>
__global__ __launch_bounds__(64) void render_unit_kernel(
    const int32_t* __restrict__ unit_slot, const int64_t* __restrict__ src_base,
    const int64_t* __restrict__ plan, int32_t n, const double* __restrict__ angles,
    int32_t H, int32_t d, int64_t row0, int64_t T_out, int64_t T_cap, uint8_t* __restrict__ out) {
  constexpr int EP = 16 / ESIZE;
  constexpr int NA = STYLE == CM_ROPE_HALF ? EP : EP / 2;
  const int lane = threadIdx.x;
  const int rb_shift = __builtin_ctz((unsigned)(d * ESIZE));
  const int64_t row_mask = ((int64_t)1 << rb_shift) - 1;
  const int ppr = (d * ESIZE) >> 4;                    // 16-byte pieces per row
  const int lkh = blockIdx.y;                          // (l * 2 + kv) * H + h
  const bool is_k = ((lkh / H) & 1) == 0;
  const int64_t end = T_out << rb_shift;               // rendered bytes of a row block end here
  const int64_t R = T_cap << rb_shift;                 // bytes of one row block of `out`
  // units tile rows [row0, T_out) of every row block; piece k of the lane is
  // byte lb + 1024 k of the row block
  const int64_t lb = (row0 << rb_shift) + (int64_t)blockIdx.x * kUnitBytes + lane * 16;
  const int cp = (int)((lb & row_mask) >> 4);          // column piece of this lane
  const int64_t* offs = plan + CM_PLAN_HEADER + n;
  const int64_t n_lkh = gridDim.y;
  // piece k from slot s: load, rotate (K at a non-zero offset), store
  auto piece = [&](int k, int s, const double* cs, const double* sn) {
    const int64_t b = lb + 1024 * k;
    const bool valid = b < end;
    const uint8_t* src = reinterpret_cast<const uint8_t*>(src_base[s * n_lkh + lkh]);
    u32x4 x = {0u, 0u, 0u, 0u};
    if (valid) x = ld16(src + b);                      // row b >> rb_shift, same column
    const bool rotate = is_k && offs[s] != 0;
    u32x4 y = x;
    double cl[NA], sl[NA];
    if constexpr (STYLE == CM_ROPE_HALF) {
      const u32x4 p = lane_xor4<HB>(x);              // every lane takes part
      if (rotate) {
        if (!cs) piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cl, sl);
        y = rotate_piece_half<ESIZE>(x, p, cs ? cs : cl, cs ? sn : sl);
      }
    } else {
      if (rotate) {
        if (!cs) piece_angles<ESIZE, STYLE>(angles + (int64_t)s * d, cp, ppr, cl, sl);
        y = rotate_piece_il<ESIZE>(x, cs ? cs : cl, cs ? sn : sl);
      }
    }
    if (valid) st_stream(out + lkh * R + b, y);
  };
  const int32_t us = unit_slot[blockIdx.x];
  if (us < 0) return;                                  // the plan failed its device check
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int s0 = us & (kUnitCrosses - 1);
  if (!(us & kUnitCrosses)) {
    // one slot for the whole unit: angles once, every piece
    double cs[NA], sn[NA];
    if (is_k && offs[s0] != 0) piece_angles<ESIZE, STYLE>(angles + (int64_t)s0 * d, cp, ppr, cs, sn);
#pragma unroll
    for (int k = 0; k < kUnitPieces; ++k) piece(k, s0, cs, sn);
  } else {
    // the unit crosses a slot boundary: slot per lane and piece
#pragma unroll
    for (int k = 0; k < kUnitPieces; ++k)
      piece(k, unit_piece_slot(offs, n_u, us, (lb + 1024 * k) >> rb_shift), nullptr, nullptr);
  }
}

// The plan check (check_on_device), the angle tables and the unit render's
// lookups in one workgroup.
__global__ __launch_bounds__(1024) void render_prep_units_kernel(
    const int64_t* __restrict__ plan, int32_t n, int32_t d, int32_t ep, int32_t style,
    double base, int64_t* __restrict__ unit_base, double* __restrict__ angles,
    const int64_t* __restrict__ table, int64_t stride, int64_t T_out, int32_t* plan_ok,
    int64_t* plan_status, int32_t H, int32_t n_lkh, int32_t rb_shift, int64_t row0,
    int64_t units, int32_t* __restrict__ unit_slot, int64_t* __restrict__ src_base) {
  const bool ok = render_tables(plan, n, d, ep, style, base, 0, 0, 0, nullptr, nullptr, unit_base,
                                angles, table, stride, T_out, plan_ok, plan_status);
  unit_tables(table, stride, plan, n, H, n_lkh, rb_shift, row0, ok ? plan[CM_PLAN_TOUT] : 0, units,
              ok, unit_slot, src_base);
}

__global__ __launch_bounds__(1024) void render_prep_kernel(
    const int64_t* __restrict__ plan, int32_t n, int32_t d, int32_t ep, int32_t style,
    double base, int32_t stripe_blocks, int64_t tensor_pairs, int64_t token_bytes,
    const uint8_t* __restrict__ select, uint8_t* __restrict__ hsel,
    int64_t* __restrict__ unit_base, double* __restrict__ angles,
    const int64_t* __restrict__ table, int64_t stride, int64_t T_out, int32_t* plan_ok,
    int64_t* plan_status) {
  render_tables(plan, n, d, ep, style, base, stripe_blocks, tensor_pairs, token_bytes, select, hsel,
                unit_base, angles, table, stride, T_out, plan_ok, plan_status);
}

}  // namespace

int64_t render_units(const SetDesc& s, int64_t T_out) {
  return (T_out * s.row_bytes + kUnitBytes - 1) / kUnitBytes;
}

RenderLayout render_layout(const SetDesc& s) {
  int64_t T_all = 0;                      // T_out never exceeds the sum over all deliveries
  for (int i = 0; i < s.n; ++i) T_all += s.T(i);
  RenderLayout lay{};
  lay.off_tiles = 0;
  lay.off_angles = align_up(sizeof(int64_t) * (size_t)(s.n + 1), kWsAlign);
  lay.off_hsel = align_up(lay.off_angles + sizeof(double) * (size_t)s.n * (size_t)s.d, kWsAlign);
  lay.off_src_base = align_up(lay.off_hsel + (size_t)s.n, kWsAlign);
  lay.off_unit_slot = align_up(lay.off_src_base + sizeof(int64_t) * (size_t)s.n * 2 * s.L * s.H,
                               kWsAlign);
  lay.off_flag = align_up(lay.off_unit_slot + sizeof(int32_t) * (size_t)render_units(s, T_all),
                          kWsAlign);
  lay.bytes = align_up(lay.off_flag + sizeof(int32_t), kWsAlign);
  return lay;
}

hipError_t launch_render_prep(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                              int32_t n_unique, double base, int32_t style, int32_t stripe_blocks,
                              const uint8_t* select, uint8_t* ws, hipStream_t stream) {
  ScopedTiming tm(K_RENDER_PREP, stream);
  int threads = 64;
  const int need = n_unique > s.n ? n_unique : s.n;
  while (threads < need) threads <<= 1;
  hipLaunchKernelGGL(render_prep_kernel, dim3(1), dim3(threads), 0, stream, plan_dev, s.n, s.d,
                     16 / s.esize, style, base, stripe_blocks, (int64_t)s.L, token_bytes_of(s),
                     select, select ? ws + lay.off_hsel : nullptr,
                     reinterpret_cast<int64_t*>(ws + lay.off_tiles),
                     reinterpret_cast<double*>(ws + lay.off_angles), s.table_dev, s.stride,
                     (int64_t)0, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_render_units(const SetDesc& s, const RenderLayout& lay,
                               const int64_t* plan_dev, const RenderRange& rr, int32_t style,
                               void* out, uint8_t* ws, hipStream_t stream) {
  const int64_t units = render_units(s, rr.T_out - rr.row0);
  if (units <= 0) return hipSuccess;
  const int32_t n_lkh = 2 * s.L * s.H;
  const int32_t* unit_slot = reinterpret_cast<const int32_t*>(ws + lay.off_unit_slot);
  const int64_t* src_base = reinterpret_cast<const int64_t*>(ws + lay.off_src_base);
  const double* angles = reinterpret_cast<const double*>(ws + lay.off_angles);
  const dim3 grid((uint32_t)units, (uint32_t)n_lkh);
  uint8_t* o = reinterpret_cast<uint8_t*>(out);
  ScopedTiming tm(K_RENDER, stream);
  auto go = [&](auto tag) {
    constexpr int STYLE = decltype(tag)::style, HB = decltype(tag)::hb;
    if (s.esize == 2)
      hipLaunchKernelGGL((render_unit_kernel<2, STYLE, HB>), grid, dim3(64), 0, stream, unit_slot,
                         src_base, plan_dev, s.n, angles, s.H, s.d, rr.row0, rr.T_out, rr.T_cap, o);
    else
      hipLaunchKernelGGL((render_unit_kernel<4, STYLE, HB>), grid, dim3(64), 0, stream, unit_slot,
                         src_base, plan_dev, s.n, angles, s.H, s.d, rr.row0, rr.T_out, rr.T_cap, o);
  };
  dispatch_style(style, s.row_bytes, go);
  return hipGetLastError();
}

hipError_t launch_render(const SetDesc& s, const RenderLayout& lay, const int64_t* plan_dev,
                         const RenderRange& rr, double base, int32_t style, bool check_on_device,
                         void* out, uint8_t* ws, hipStream_t stream) {
  int32_t* plan_ok = check_on_device ? reinterpret_cast<int32_t*>(ws + lay.off_flag) : nullptr;
  const int64_t units = render_units(s, rr.T_out - rr.row0);
  {
    ScopedTiming tm(K_RENDER_PREP, stream);
    const int threads = table_threads(s.n, units + (int64_t)s.n * 2 * s.L * s.H);
    hipLaunchKernelGGL(render_prep_units_kernel, dim3(1), dim3(threads), 0, stream, plan_dev, s.n,
                       s.d, 16 / s.esize, style, base,
                       reinterpret_cast<int64_t*>(ws + lay.off_tiles),
                       reinterpret_cast<double*>(ws + lay.off_angles), s.table_dev, s.stride,
                       rr.T_out, plan_ok, const_cast<int64_t*>(plan_dev), s.H, 2 * s.L * s.H,
                       (int32_t)__builtin_ctzll((unsigned long long)s.row_bytes), rr.row0,
                       units, reinterpret_cast<int32_t*>(ws + lay.off_unit_slot),
                       reinterpret_cast<int64_t*>(ws + lay.off_src_base));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_render_units(s, lay, plan_dev, rr, style, out, ws, stream);
}

}  // namespace cm
