// Per-slot tables of the render, built by one workgroup once the plan exists
// (shared by the render's own prep kernel and the order kernels of the one-call
// paths, which build them right after the plan, in the same workgroup).
#pragma once

#include "render_geometry.h"
#include "rotate.h"

namespace cm {

// One workgroup: per-slot cos/sin(off_s * theta_j), theta_j = base^(-2j/d), in
// fp64: in the piece-ordered layout of rotate.h for the unit render
// (stripe_blocks == 0), in pair order (entry j holds pair j) for the fused
// hash+render, whose lanes read them wave-uniformly. With stripe_blocks > 0 also the
// per-slot work-unit bases of the fused hash+render (2L * stripes of that many
// 64-byte blocks per slot, exclusive scan; the total at index n as well, none if
// the plan's status is an error) and, with a select mask, hsel[i] = 0
// for the slot deliveries whose Id the fused kernel computes (select[i] == 0),
// 1 for every other delivery. Returns false (the same in every thread) for a
// plan that fails the device check; nothing else is written then.
__device__ __forceinline__ bool render_tables(
    const int64_t* __restrict__ plan, int32_t n, int32_t d, int32_t ep, int32_t style,
    double base, int32_t stripe_blocks, int64_t tensor_pairs, int64_t token_bytes,
    const uint8_t* __restrict__ select, uint8_t* __restrict__ hsel,
    int64_t* __restrict__ unit_base, double* __restrict__ angles,
    const int64_t* __restrict__ table, int64_t stride, int64_t T_out, int32_t* plan_ok,
    int64_t* plan_status) {
  __shared__ int64_t sc[1024];
  const int tid = threadIdx.x;
  int n_u = (int)plan[CM_PLAN_NUNIQUE];
  if (plan_ok) {
    // A plan the host has not seen: status, n, n_unique, T_out, every slot's
    // delivery and length, and the offsets as exclusive prefix sums. The block
    // holds at least n threads, one per slot.
    const bool head = plan[CM_PLAN_STATUS] == CM_OK && plan[CM_PLAN_N] == n && n_u >= 1 &&
                      n_u <= n && plan[CM_PLAN_TOUT] == T_out;
    bool ok = true;
    int64_t len = 0;
    if (head && tid < n_u) {
      const int64_t src = plan[CM_PLAN_HEADER + tid];
      len = plan[CM_PLAN_HEADER + 2 * (int64_t)n + tid];
      ok = src >= 0 && src < n && len >= 1 && len == table[src * stride];
    }
    sc[tid] = ok ? len : 0;
    __syncthreads();
    for (int o = 1; o < (int)blockDim.x; o <<= 1) {
      const int64_t t = tid >= o ? sc[tid - o] : 0;
      __syncthreads();
      sc[tid] += t;
      __syncthreads();
    }
    if (head && tid < n_u) ok = ok && plan[CM_PLAN_HEADER + n + tid] == sc[tid] - len;
    const bool all = __syncthreads_and(ok) && head && sc[blockDim.x - 1] == T_out;
    if (tid == 0) {
      *plan_ok = all ? 1 : 0;
      // a plan that already reports an error (a non-finite score) keeps it
      if (!all && plan[CM_PLAN_STATUS] == CM_OK) *plan_status = CM_ESHAPE;
    }
    if (!all) return false;
    __syncthreads();
  }
  if (stripe_blocks > 0) {
    // a plan whose status is an error (a non-finite score) gets no tasks
    if (plan[CM_PLAN_STATUS] != CM_OK || n_u < 0 || n_u > n) n_u = 0;
    const int64_t len = tid < n_u ? plan[CM_PLAN_HEADER + 2 * (int64_t)n + tid] : 0;
    int64_t x = 0;
    if (tid < n_u)
      x = 2 * tensor_pairs * ((((len * token_bytes) >> 6) + stripe_blocks - 1) / stripe_blocks);
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
    if (tid == (int)blockDim.x - 1) {
      unit_base[n_u] = sc[tid];
      unit_base[n] = sc[tid];          // the task total, where the fused kernel reads it
    }
    if (hsel && tid < n_u) {
      const int64_t i = plan[CM_PLAN_HEADER + tid];
      if (select[i] == 0) hsel[i] = 0;
    }
  }
  const int halfd = d >> 1;
  const int ppr = d / ep;                    // pieces per row
  // theta_j is computed once per column a thread visits (with a block of at
  // least d / 2 threads, a thread keeps one column for every slot)
  int tj = -1;
  double theta = 0.0;
  for (int idx = tid; idx < n_u * halfd; idx += blockDim.x) {
    const int s = idx / halfd;
    const int j = idx - s * halfd;
    if (j != tj) {
      theta = pow(base, -(double)(2 * j) / (double)d);
      tj = j;
    }
    const double phi = (double)plan[CM_PLAN_HEADER + n + s] * theta;
    const int k = stripe_blocks > 0 ? j
                  : style == CM_ROPE_HALF ? angle_slot_half(j / ep, j % ep, ppr >> 1)
                                          : angle_slot_il(j / (ep >> 1), j % (ep >> 1), ppr);
    angles[2 * ((int64_t)s * halfd + k)] = cos(phi);
    angles[2 * ((int64_t)s * halfd + k) + 1] = sin(phi);
  }
  return true;
}

// The lookups of the unit render (render.hip) for rows [row0, T_out) of a plan,
// by one workgroup: unit_slot[x] = slot of the first row of unit x (|
// kUnitCrosses if a later row of the unit lies in another slot), src_base[s][lkh]
// = the address that row r of slot s in row block lkh = (l * 2 + kv) * H + h is
// read from when offset by r * row_bytes. ok == false (a plan that is not
// rendered): every unit gets -1, which the render skips. The slots' delivery,
// length and offset are staged in LDS first.
__device__ __forceinline__ void unit_tables(const int64_t* __restrict__ table, int64_t stride,
                                            const int64_t* __restrict__ plan, int32_t n,
                                            int32_t H, int32_t n_lkh, int32_t rb_shift,
                                            int64_t row0, int64_t T_out, int64_t units, bool ok,
                                            int32_t* __restrict__ unit_slot,
                                            int64_t* __restrict__ src_base) {
  __shared__ int64_t u_off[1024];
  __shared__ int64_t u_len[1024];
  __shared__ int64_t u_src[1024];
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  if (!ok) {
    for (int64_t x = tid; x < units; x += nt) unit_slot[x] = -1;
    return;
  }
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  for (int s = tid; s < n_u; s += nt) {
    u_src[s] = plan[CM_PLAN_HEADER + s];
    u_off[s] = plan[CM_PLAN_HEADER + n + s];
    u_len[s] = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
  }
  __syncthreads();
  for (int64_t x = tid; x < units; x += nt)
    unit_slot[x] = unit_slot_code(u_off, n_u, T_out, rb_shift, row0, x);
  for (int64_t e = tid; e < (int64_t)n_u * n_lkh; e += nt) {
    const int s = (int)(e / n_lkh);
    const int lkh = (int)(e - (int64_t)s * n_lkh);
    const int64_t base = table[u_src[s] * stride + 1 + lkh / H];
    src_base[e] = base + unit_src_offset(lkh % H, u_len[s], u_off[s], rb_shift, 0);
  }
}

}  // namespace cm
