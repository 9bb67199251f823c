// C ABI of libcmerge (include/cmerge.h): argument validation on the host, workspace
// sizing, error reporting and the optional per-kernel event timing. Every check
// runs before anything is enqueued, so a failing call leaves the stream untouched.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "cmerge.h"
#include "internal.h"

namespace {

thread_local std::string g_err;

int32_t fail(int32_t code, const std::string& msg) {
  g_err = msg;
  return code;
}

int32_t fail_hip(hipError_t e, const char* where) {
  return fail(CM_EHIP, std::string(where) + ": " + hipGetErrorName(e) + ": " + hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int32_t check_set(const cm_fragset* set, cm::SetDesc* out) {
  if (!set) return fail(CM_EINVAL, "set is NULL");
  if (set->n < 1 || set->n > CM_MAX_FRAGMENTS)
    return fail(CM_EINVAL, "n must be in [1, " + std::to_string(CM_MAX_FRAGMENTS) + "], got " +
                               std::to_string(set->n));
  if (set->L < 1 || set->H < 1) return fail(CM_EINVAL, "L and H must be >= 1");
  if ((int64_t)2 * set->L * set->H > 65535)
    return fail(CM_ESHAPE, "2 * L * H must be <= 65535");
  int esize = 0;
  if (set->dtype == CM_F32) esize = 4;
  else if (set->dtype == CM_BF16) esize = 2;
  else return fail(CM_EDTYPE, "dtype must be CM_F32 or CM_BF16, got " + std::to_string(set->dtype));
  const int64_t row_bytes = (int64_t)set->d * esize;
  if (!is_pow2(set->d) || row_bytes < 64 || row_bytes > 1024)
    return fail(CM_ESHAPE, "d must be a power of two with d * element_bytes in [64, 1024], got d=" +
                               std::to_string(set->d));
  if (set->reserved != 0) return fail(CM_EINVAL, "reserved field must be 0");
  if (!set->table_host || !set->table_dev) return fail(CM_EINVAL, "fragment tables are NULL");
  if (!aligned(set->table_dev, 8)) return fail(CM_EINVAL, "table_dev must be 8-byte aligned");
  const int64_t stride = 1 + 2 * (int64_t)set->L;
  for (int i = 0; i < set->n; ++i) {
    const int64_t* row = set->table_host + (int64_t)i * stride;
    const int64_t T = row[0];
    if (T < 1) return fail(CM_EINVAL, "fragment " + std::to_string(i) + " has T < 1");
    if (T > ((int64_t)1 << 40) / ((int64_t)set->H * row_bytes))
      return fail(CM_ESHAPE, "fragment " + std::to_string(i) + " tensor exceeds 1 TiB");
    for (int64_t t = 1; t < stride; ++t) {
      const uintptr_t a = (uintptr_t)row[t];
      if (a == 0 || (a & 15) != 0)
        return fail(CM_EINVAL, "fragment " + std::to_string(i) + " tensor " + std::to_string(t - 1) +
                                   " address is NULL or not 16-byte aligned");
    }
  }
  out->n = set->n;
  out->L = set->L;
  out->H = set->H;
  out->d = set->d;
  out->dtype = set->dtype;
  out->esize = esize;
  out->stride = stride;
  out->row_bytes = row_bytes;
  out->table_dev = set->table_dev;
  out->table_host = set->table_host;
  return CM_OK;
}

int32_t check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return CM_OK;
  if (!ws) return fail(CM_EWORKSPACE, "workspace is NULL");
  if (!aligned(ws, cm::kWsAlign)) return fail(CM_EWORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return fail(CM_EWORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, got " +
                                   std::to_string(ws_bytes));
  return CM_OK;
}

// Scratch of cm_render_deliveries_noalloc: one copy per GPU, created with the
// library's code object on that device and held until the process ends. On the
// host `scratch` names a stand-in, not device memory, so host code never passes
// it to a kernel: device_scratch() looks up the current device's own address
// once (hipGetSymbolAddress) and every launch takes that.
constexpr size_t kScratchBytes = (size_t)CM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int32_t device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "cm_render_deliveries_noalloc: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CM_EINVAL, "cm_render_deliveries_noalloc: device index " + std::to_string(dev) +
                               " is beyond the library's table of " + std::to_string(kMaxDevices));
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail_hip(e, "cm_render_deliveries_noalloc: hipGetSymbolAddress");
    if (!p || !aligned(p, cm::kWsAlign))
      return fail(CM_EHIP, "cm_render_deliveries_noalloc: scratch address is NULL or misaligned");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return CM_OK;
}

// Every call fits in this many bytes: the render's tables follow the hash
// workspace (fused render+hash) or the score partials (set render, which keeps
// them until the order kernel has folded them).
size_t render_ws_offset(const cm::SetDesc& s) {
  const size_t hb = cm::hash_layout(s).bytes;
  const size_t kn = cm::knorm_max_bytes(s);
  return cm::align_up(hb > kn ? hb : kn, cm::kWsAlign);
}

size_t workspace_need(const cm::SetDesc& s) {
  return render_ws_offset(s) + cm::render_layout(s).bytes;
}

int64_t min_T(const cm::SetDesc& s) {
  int64_t m = s.T(0);
  for (int i = 1; i < s.n; ++i) m = s.T(i) < m ? s.T(i) : m;
  return m;
}

// ------------------------------------------------------------------ timing registry
const char* const kKernelNames[cm::K_COUNT] = {
    "hash_prep", "hash_leaf", "hash_parent", "hash_final", "knorm_rows", "knorm_tree",
    "order",     "key_mask",  "render_prep", "render",     "render_hash", "paged",
    "paged_hash_render"};
std::atomic<bool> g_timing{false};
// set while this thread captures a call into a graph: no timing events then
thread_local bool t_capturing = false;
std::mutex g_tmu;
struct Pending {
  int id;
  hipEvent_t a, b;
};
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
double g_total_ms[cm::K_COUNT];
int64_t g_count[cm::K_COUNT];

hipEvent_t take_event() {
  {
    std::lock_guard<std::mutex> lk(g_tmu);
    if (!g_pool.empty()) {
      hipEvent_t e = g_pool.back();
      g_pool.pop_back();
      return e;
    }
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

hipError_t drain_pending() {
  std::lock_guard<std::mutex> lk(g_tmu);
  hipError_t first = hipSuccess;
  for (const Pending& p : g_pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e == hipSuccess) {
      g_total_ms[p.id] += ms;
      g_count[p.id] += 1;
    } else if (first == hipSuccess) {
      first = e;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
  return first;
}

}  // namespace

namespace cm {

int device_cu_count() {
  static std::mutex mu;
  static int counts[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lk(mu);
  if (counts[dev] == 0) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0)
      cu = 256;
    counts[dev] = cu;
  }
  return counts[dev];
}

ScopedTiming::ScopedTiming(int kernel_id, hipStream_t stream) : id_(kernel_id), stream_(stream) {
  if (t_capturing || !g_timing.load(std::memory_order_relaxed)) return;
  start_ = take_event();
  if (start_ && hipEventRecord(start_, stream_) != hipSuccess) start_ = nullptr;
}

ScopedTiming::~ScopedTiming() {
  if (!start_) return;
  hipEvent_t end = take_event();
  if (!end || hipEventRecord(end, stream_) != hipSuccess) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  g_pending.push_back({id_, start_, end});
}

}  // namespace cm

extern "C" {

int32_t cm_version(void) { return CM_ABI_VERSION; }

const char* cm_last_error(void) { return g_err.c_str(); }

const char* cm_status_string(int32_t status) {
  switch (status) {
    case CM_OK: return "CM_OK";
    case CM_EINVAL: return "CM_EINVAL";
    case CM_ESHAPE: return "CM_ESHAPE";
    case CM_EDTYPE: return "CM_EDTYPE";
    case CM_ENONFINITE: return "CM_ENONFINITE";
    case CM_EHIP: return "CM_EHIP";
    case CM_EWORKSPACE: return "CM_EWORKSPACE";
    default: return "CM_UNKNOWN";
  }
}

size_t cm_plan_elems(int32_t n) { return n < 0 ? 0 : (size_t)CM_PLAN_HEADER + 4 * (size_t)n; }

int32_t cm_workspace_size(const cm_fragset* set, size_t* bytes_out) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!bytes_out) return fail(CM_EINVAL, "bytes_out is NULL");
  *bytes_out = workspace_need(s);
  return CM_OK;
}

static int32_t hash_common(const cm_fragset* set, const uint8_t* select, uint32_t want,
                           uint8_t* digests_dev, void* workspace, size_t workspace_bytes,
                           void* stream, const char* where) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if (want > 255) return fail(CM_EINVAL, "select_value must be in [0, 255]");
  const cm::HashLayout lay = cm::hash_layout(s);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  hipError_t e = cm::launch_hash(s, lay, select, want, digests_dev,
                                 static_cast<uint8_t*>(workspace), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, where);
}

int32_t cm_fragment_hash(const cm_fragset* set, uint8_t* digests_dev, void* workspace,
                         size_t workspace_bytes, void* stream) {
  return hash_common(set, nullptr, 0, digests_dev, workspace, workspace_bytes, stream,
                     "cm_fragment_hash");
}

int32_t cm_fragment_hash_select(const cm_fragset* set, const uint8_t* select_dev,
                                int32_t select_value, uint8_t* digests_dev, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (!select_dev) {
    g_err.clear();
    return fail(CM_EINVAL, "select_dev is NULL");
  }
  if (select_value < 0) {
    g_err.clear();
    return fail(CM_EINVAL, "select_value must be in [0, 255]");
  }
  return hash_common(set, select_dev, (uint32_t)select_value, digests_dev, workspace,
                     workspace_bytes, stream, "cm_fragment_hash_select");
}

int32_t cm_equal_key_mask(const cm_fragset* set, const double* keys_dev, uint8_t* mask_dev,
                          void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!mask_dev) return fail(CM_EINVAL, "mask_dev is NULL");
  hipError_t e = cm::launch_equal_key_mask(s, keys_dev, mask_dev, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_equal_key_mask");
}

int32_t cm_fragment_knorm(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                          double* keys_dev, void* workspace, size_t workspace_bytes,
                          void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (routing_layer < 0 || routing_layer >= s.L)
    return fail(CM_EINVAL, "routing_layer must be in [0, L), got " + std::to_string(routing_layer));
  const int64_t tmin = min_T(s);
  if (tail_len < 1 || tail_len > tmin)
    return fail(CM_EINVAL, "tail_len must be in [1, min T] = [1, " + std::to_string(tmin) + "], got " +
                               std::to_string(tail_len));
  if (!keys_dev || !aligned(keys_dev, 8))
    return fail(CM_EINVAL, "keys_dev is NULL or not 8-byte aligned");
  const cm::KnormLayout lay = cm::knorm_layout(s, tail_len);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  hipError_t e = cm::launch_knorm(s, lay, routing_layer, tail_len, keys_dev,
                                  static_cast<uint8_t*>(workspace), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_fragment_knorm");
}

int32_t cm_canonical_order(const cm_fragset* set, const double* keys_dev,
                           const uint8_t* digests_dev, int64_t* plan_dev, void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!digests_dev || !aligned(digests_dev, 4))
    return fail(CM_EINVAL, "digests_dev is NULL or misaligned");
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  hipError_t e =
      cm::launch_order(s, keys_dev, digests_dev, true, plan_dev, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_canonical_order");
}

int32_t cm_multiset_order(const cm_fragset* set, const double* keys_dev,
                          const uint8_t* digests_dev, int64_t* plan_dev, void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!digests_dev || !aligned(digests_dev, 4))
    return fail(CM_EINVAL, "digests_dev is NULL or misaligned");
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  hipError_t e =
      cm::launch_order(s, keys_dev, digests_dev, false, plan_dev, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_multiset_order");
}

int32_t cm_bag_plan(const cm_fragset* set, const int32_t* order_host, int32_t count,
                    int64_t* plan_host) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!order_host || !plan_host) return fail(CM_EINVAL, "order_host / plan_host is NULL");
  if (count < 1 || count > s.n)
    return fail(CM_EINVAL, "count must be in [1, n] = [1, " + std::to_string(s.n) + "], got " +
                               std::to_string(count));
  const int64_t n = s.n;
  for (int64_t k = 0; k < 4 + 4 * n; ++k) plan_host[k] = -1;
  int64_t off = 0;
  for (int32_t k = 0; k < count; ++k) {
    const int32_t i = order_host[k];
    if (i < 0 || i >= s.n)
      return fail(CM_EINVAL, "order entry " + std::to_string(k) + " = " + std::to_string(i) +
                                 " is not a delivery index");
    plan_host[CM_PLAN_HEADER + k] = i;
    plan_host[CM_PLAN_HEADER + n + k] = off;
    plan_host[CM_PLAN_HEADER + 2 * n + k] = s.T(i);
    if (plan_host[CM_PLAN_HEADER + 3 * n + i] < 0) plan_host[CM_PLAN_HEADER + 3 * n + i] = k;
    off += s.T(i);
  }
  plan_host[CM_PLAN_STATUS] = CM_OK;
  plan_host[CM_PLAN_N] = n;
  plan_host[CM_PLAN_NUNIQUE] = count;
  plan_host[CM_PLAN_TOUT] = off;
  return CM_OK;
}

}  // extern "C"

namespace {

// Checks shared by the render entry points; returns the slot count.
int32_t check_rope(const cm_rope* rope) {
  if (!rope) return fail(CM_EINVAL, "rope is NULL");
  if (!std::isfinite(rope->base) || rope->base <= 0.0)
    return fail(CM_EINVAL, "rope base must be finite and > 0");
  if (rope->style != CM_ROPE_HALF && rope->style != CM_ROPE_INTERLEAVED)
    return fail(CM_EINVAL, "rope style must be CM_ROPE_HALF or CM_ROPE_INTERLEAVED");
  if (rope->reserved != 0) return fail(CM_EINVAL, "rope reserved field must be 0");
  return CM_OK;
}

int32_t check_render_args(const cm::SetDesc& s, const int64_t* plan_dev, const int64_t* plan_host,
                          const cm_rope* rope, void* out_dev, int64_t T_out, int64_t* nu_out) {
  int32_t st = check_rope(rope);
  if (st != CM_OK) return st;
  if (!plan_dev || !aligned(plan_dev, 8) || !plan_host)
    return fail(CM_EINVAL, "plan_dev / plan_host is NULL or misaligned");
  if (!out_dev || !aligned(out_dev, 16)) return fail(CM_EINVAL, "out_dev is NULL or not 16-byte aligned");
  if (plan_host[CM_PLAN_STATUS] == CM_ENONFINITE)
    return fail(CM_ENONFINITE, "the plan reports a non-finite score");
  if (plan_host[CM_PLAN_STATUS] != CM_OK) return fail(CM_EINVAL, "plan status is not CM_OK");
  if (plan_host[CM_PLAN_N] != s.n) return fail(CM_EINVAL, "plan was built for another n");
  const int64_t nu = plan_host[CM_PLAN_NUNIQUE];
  if (nu < 1 || nu > s.n) return fail(CM_EINVAL, "plan n_unique out of range");
  if (T_out < 1 || plan_host[CM_PLAN_TOUT] != T_out)
    return fail(CM_ESHAPE, "T_out does not match the plan");
  int64_t off = 0;
  for (int64_t k = 0; k < nu; ++k) {
    const int64_t src = plan_host[CM_PLAN_HEADER + k];
    const int64_t o = plan_host[CM_PLAN_HEADER + s.n + k];
    const int64_t len = plan_host[CM_PLAN_HEADER + 2 * (int64_t)s.n + k];
    if (src < 0 || src >= s.n) return fail(CM_EINVAL, "plan slot refers to no delivery");
    if (len != s.T((int)src)) return fail(CM_ESHAPE, "plan slot length differs from the fragment's T");
    if (o != off) return fail(CM_ESHAPE, "plan offsets are not the prefix sum of slot lengths");
    off += len;
  }
  if (off != T_out) return fail(CM_ESHAPE, "T_out differs from the sum of slot lengths");
  if (cm::render_units(s, T_out) >= ((int64_t)1 << 31))
    return fail(CM_ESHAPE, "merged cache too long for one launch");
  *nu_out = nu;
  return CM_OK;
}

}  // namespace

extern "C" {

int32_t cm_render_merge(const cm_fragset* set, const int64_t* plan_dev, const int64_t* plan_host,
                        const cm_rope* rope, void* out_dev, int64_t T_out, void* workspace,
                        size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  int64_t nu = 0;
  if ((st = check_render_args(s, plan_dev, plan_host, rope, out_dev, T_out, &nu)) != CM_OK)
    return st;
  const cm::RenderLayout lay = cm::render_layout(s);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  hipError_t e = cm::launch_render(s, lay, plan_dev, {0, T_out, T_out}, rope->base, rope->style,
                                   false, out_dev, static_cast<uint8_t*>(workspace),
                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_render_merge");
}

int32_t cm_render_merge_range(const cm_fragset* set, const int64_t* plan_dev,
                              const int64_t* plan_host, const cm_rope* rope, int32_t first_slot,
                              void* out_dev, int64_t T_cap, void* workspace,
                              size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if (!plan_host) return fail(CM_EINVAL, "plan_host is NULL");
  const int64_t T_out = plan_host[CM_PLAN_TOUT];
  int64_t nu = 0;
  if ((st = check_render_args(s, plan_dev, plan_host, rope, out_dev, T_out, &nu)) != CM_OK)
    return st;
  if (first_slot < 0 || first_slot >= nu)
    return fail(CM_EINVAL, "first_slot must be in [0, n_unique)");
  if (T_cap < T_out) return fail(CM_ESHAPE, "T_cap must be >= the plan's T_out");
  const cm::RenderLayout lay = cm::render_layout(s);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  const int64_t row0 = plan_host[CM_PLAN_HEADER + s.n + first_slot];
  hipError_t e = cm::launch_render(s, lay, plan_dev, {row0, T_out, T_cap}, rope->base,
                                   rope->style, false, out_dev, static_cast<uint8_t*>(workspace),
                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_render_merge_range");
}

int32_t cm_render_merge_devplan(const cm_fragset* set, int64_t* plan_dev, const cm_rope* rope,
                                void* out_dev, int64_t T_out, void* workspace,
                                size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if ((st = check_rope(rope)) != CM_OK) return st;
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  if (!out_dev || !aligned(out_dev, 16)) return fail(CM_EINVAL, "out_dev is NULL or not 16-byte aligned");
  int64_t T_all = 0;
  for (int i = 0; i < s.n; ++i) T_all += s.T(i);
  if (T_out < 1 || T_out > T_all)
    return fail(CM_ESHAPE, "T_out must be in [1, sum of the fragment lengths]");
  if (cm::render_units(s, T_out) >= ((int64_t)1 << 31))
    return fail(CM_ESHAPE, "merged cache too long for one launch");
  const cm::RenderLayout lay = cm::render_layout(s);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  hipError_t e = cm::launch_render(s, lay, plan_dev, {0, T_out, T_out}, rope->base, rope->style,
                                   true, out_dev, static_cast<uint8_t*>(workspace),
                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_render_merge_devplan");
}

int32_t cm_render_set(const cm_fragset* set, const uint8_t* digests_dev, int32_t routing_layer,
                      int64_t tail_len, const cm_rope* rope, double* keys_dev, int64_t* plan_dev,
                      void* out_dev, int64_t T_out, void* workspace, size_t workspace_bytes,
                      void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if ((st = check_rope(rope)) != CM_OK) return st;
  if (routing_layer < 0 || routing_layer >= s.L)
    return fail(CM_EINVAL, "routing_layer must be in [0, L), got " + std::to_string(routing_layer));
  const int64_t tmin = min_T(s);
  if (tail_len < 1 || tail_len > tmin)
    return fail(CM_EINVAL, "tail_len must be in [1, min T] = [1, " + std::to_string(tmin) + "], got " +
                               std::to_string(tail_len));
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  if (!out_dev || !aligned(out_dev, 16))
    return fail(CM_EINVAL, "out_dev is NULL or not 16-byte aligned");
  int64_t T_all = 0;
  for (int i = 0; i < s.n; ++i) T_all += s.T(i);
  if (T_out != T_all)
    return fail(CM_ESHAPE, "T_out must be the sum of the member lengths (" + std::to_string(T_all) +
                               "), got " + std::to_string(T_out));
  if (cm::render_units(s, T_out) >= ((int64_t)1 << 31))
    return fail(CM_ESHAPE, "merged cache too long for one launch");
  if ((st = check_ws(workspace, workspace_bytes, workspace_need(s))) != CM_OK) return st;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  hipStream_t sm = static_cast<hipStream_t>(stream);
  // score partials at the start of the workspace, the render's tables after them
  cm::KnormPartials kp{};
  hipError_t e = cm::launch_knorm_partial(s, cm::knorm_layout(s, tail_len), routing_layer,
                                          tail_len, keys_dev, ws, sm, cm::kKnormFoldMax, &kp);
  if (e == hipSuccess)
    e = cm::launch_render_set(s, cm::render_layout(s), kp, keys_dev, digests_dev, plan_dev, T_out,
                              rope->base, rope->style, out_dev, ws + render_ws_offset(s), sm);
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_render_set");
}

int32_t cm_render_merge_hash(const cm_fragset* set, const int64_t* plan_dev,
                             const int64_t* plan_host, const cm_rope* rope,
                             const uint8_t* select_dev, uint8_t* digests_dev, void* out_dev,
                             int64_t T_out, void* workspace, size_t workspace_bytes,
                             void* stream) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  int64_t nu = 0;
  if ((st = check_render_args(s, plan_dev, plan_host, rope, out_dev, T_out, &nu)) != CM_OK)
    return st;
  if (!select_dev) return fail(CM_EINVAL, "select_dev is NULL");
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  const cm::HashLayout hlay = cm::hash_layout(s);
  const cm::RenderLayout rlay = cm::render_layout(s);
  const size_t need = cm::align_up(hlay.bytes, cm::kWsAlign) + rlay.bytes;
  if ((st = check_ws(workspace, workspace_bytes, need)) != CM_OK) return st;
  hipError_t e = cm::launch_render_hash(s, hlay, rlay, plan_dev, rope->base, rope->style,
                                        select_dev, digests_dev, out_dev,
                                        static_cast<uint8_t*>(workspace),
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_render_merge_hash");
}

}  // extern "C"

namespace {

// Steps 1-5 of cm_render_deliveries after its argument checks. The workspace is
// the caller's (workspace_bytes its size) or, with fixed_scratch, this device's
// copy of `scratch`, once the set's need is known to fit it.
int32_t render_deliveries_common(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                                 const cm_rope* rope, double* keys_dev, uint8_t* mask_dev,
                                 uint8_t* digests_dev, int64_t* plan_dev, void* out_dev,
                                 int64_t T_cap, void* workspace, size_t workspace_bytes,
                                 bool fixed_scratch, void* stream, const char* where,
                                 bool check_only = false) {
  g_err.clear();
  cm::SetDesc s;
  int32_t st = check_set(set, &s);
  if (st != CM_OK) return st;
  if ((st = check_rope(rope)) != CM_OK) return st;
  if (routing_layer < 0 || routing_layer >= s.L)
    return fail(CM_EINVAL, "routing_layer must be in [0, L), got " + std::to_string(routing_layer));
  const int64_t tmin = min_T(s);
  if (tail_len < 1 || tail_len > tmin)
    return fail(CM_EINVAL, "tail_len must be in [1, min T] = [1, " + std::to_string(tmin) + "], got " +
                               std::to_string(tail_len));
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!mask_dev) return fail(CM_EINVAL, "mask_dev is NULL");
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  if (!out_dev || !aligned(out_dev, 16))
    return fail(CM_EINVAL, "out_dev is NULL or not 16-byte aligned");
  int64_t T_all = 0;
  for (int i = 0; i < s.n; ++i) T_all += s.T(i);
  if (T_cap < T_all)
    return fail(CM_ESHAPE, "T_cap must be at least the sum of the delivery lengths (" +
                               std::to_string(T_all) + "), got " + std::to_string(T_cap));
  const size_t need = workspace_need(s);
  if (fixed_scratch) {
    if (need > kScratchBytes)
      return fail(CM_EWORKSPACE, std::string(where) + ": this set needs " + std::to_string(need) +
                                     " bytes of scratch, more than the fixed " +
                                     std::to_string(kScratchBytes) +
                                     " (CM_NOALLOC_SCRATCH_BYTES); call cm_render_deliveries "
                                     "with a workspace instead");
    if ((st = device_scratch(&workspace)) != CM_OK) return st;
  } else if ((st = check_ws(workspace, workspace_bytes, need)) != CM_OK) {
    return st;
  }
  if (check_only) return CM_OK;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  hipStream_t sm = static_cast<hipStream_t>(stream);
  // the workspace is reused by each stage in turn: they run in order on one stream
  cm::KnormPartials kp{};
  hipError_t e = cm::launch_knorm_partial(s, cm::knorm_layout(s, tail_len), routing_layer,
                                          tail_len, keys_dev, ws, sm, cm::kKnormFoldMax, &kp);
  const cm::HashLayout hlay = cm::hash_layout(s);
  // the last score levels, the key mask and the hash trees' node tables in one
  // launch (the tables depend only on the lengths); it reads the score partials
  // before it writes over them
  if (e == hipSuccess) e = cm::launch_mask_hash_prep(s, hlay, kp, keys_dev, mask_dev, ws, sm);
  if (e == hipSuccess) e = cm::launch_hash(s, hlay, mask_dev, 1, digests_dev, ws, sm, true);
  // the order kernel also builds the render's per-slot tables; the node-base
  // tables written for the first Ids are still in the workspace (the render's
  // tables live after them), so the fused pass reuses both
  const cm::RenderLayout rlay = cm::render_layout(s);
  if (e == hipSuccess)
    e = cm::launch_order_render_prep(s, keys_dev, digests_dev, plan_dev, rlay, rope->base,
                                     rope->style, (int32_t)cm::kStripeBlocks, mask_dev,
                                     ws + cm::align_up(hlay.bytes, cm::kWsAlign), sm);
  if (e == hipSuccess)
    e = cm::launch_render_hash(s, hlay, rlay, plan_dev, rope->base, rope->style, mask_dev,
                               digests_dev, out_dev, ws, sm, true, true);
  return e == hipSuccess ? CM_OK : fail_hip(e, where);
}

}  // namespace

extern "C" {

int32_t cm_render_deliveries(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                             const cm_rope* rope, double* keys_dev, uint8_t* mask_dev,
                             uint8_t* digests_dev, int64_t* plan_dev, void* out_dev,
                             int64_t T_cap, void* workspace, size_t workspace_bytes,
                             void* stream) {
  return render_deliveries_common(set, routing_layer, tail_len, rope, keys_dev, mask_dev,
                                  digests_dev, plan_dev, out_dev, T_cap, workspace,
                                  workspace_bytes, false, stream, "cm_render_deliveries");
}

int32_t cm_render_deliveries_noalloc(const cm_fragset* set, int32_t routing_layer,
                                     int64_t tail_len, const cm_rope* rope, double* keys_dev,
                                     uint8_t* mask_dev, uint8_t* digests_dev, int64_t* plan_dev,
                                     void* out_dev, int64_t T_cap, void* stream) {
  return render_deliveries_common(set, routing_layer, tail_len, rope, keys_dev, mask_dev,
                                  digests_dev, plan_dev, out_dev, T_cap, nullptr, 0, true, stream,
                                  "cm_render_deliveries_noalloc");
}

}  // extern "C"

struct cm_graph {
  hipGraph_t graph;
  hipGraphExec_t exec;
};

extern "C" {

int32_t cm_render_deliveries_graph(const cm_fragset* set, int32_t routing_layer, int64_t tail_len,
                                   const cm_rope* rope, double* keys_dev, uint8_t* mask_dev,
                                   uint8_t* digests_dev, int64_t* plan_dev, void* out_dev,
                                   int64_t T_cap, void* workspace, size_t workspace_bytes,
                                   cm_graph** graph_out) {
  g_err.clear();
  if (!graph_out) return fail(CM_EINVAL, "graph_out is NULL");
  *graph_out = nullptr;
  // the arguments first, on the host
  int32_t st = render_deliveries_common(set, routing_layer, tail_len, rope, keys_dev, mask_dev,
                                        digests_dev, plan_dev, out_dev, T_cap, workspace,
                                        workspace_bytes, false, nullptr,
                                        "cm_render_deliveries_graph", true);
  if (st != CM_OK) return st;
  // capture on a stream of this call's own (the caller's may be the null
  // stream, which cannot be captured); nothing runs until the graph is launched
  hipStream_t cs = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  if (e != hipSuccess) return fail_hip(e, "cm_render_deliveries_graph");
  e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    (void)hipStreamDestroy(cs);
    return fail_hip(e, "cm_render_deliveries_graph");
  }
  t_capturing = true;
  st = render_deliveries_common(set, routing_layer, tail_len, rope, keys_dev, mask_dev,
                                digests_dev, plan_dev, out_dev, T_cap, workspace, workspace_bytes,
                                false, cs, "cm_render_deliveries_graph");
  t_capturing = false;
  const std::string err = g_err;       // a failed launch's message, if any
  hipGraph_t g = nullptr;
  e = hipStreamEndCapture(cs, &g);
  (void)hipStreamDestroy(cs);
  if (st != CM_OK) {
    if (g) (void)hipGraphDestroy(g);
    g_err = err;
    return st;
  }
  if (e != hipSuccess) return fail_hip(e, "cm_render_deliveries_graph");
  if (!g) return fail(CM_EHIP, "cm_render_deliveries_graph: the capture gave no graph");
  hipGraphExec_t x = nullptr;
  e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    (void)hipGraphDestroy(g);
    return fail_hip(e, "cm_render_deliveries_graph");
  }
  *graph_out = new cm_graph{g, x};
  return CM_OK;
}

int32_t cm_graph_launch(cm_graph* graph, void* stream) {
  g_err.clear();
  if (!graph) return fail(CM_EINVAL, "graph is NULL");
  const hipError_t e = hipGraphLaunch(graph->exec, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_graph_launch");
}

int32_t cm_graph_destroy(cm_graph* graph) {
  g_err.clear();
  if (!graph) return CM_OK;
  hipError_t e = hipGraphExecDestroy(graph->exec);
  const hipError_t e2 = hipGraphDestroy(graph->graph);
  delete graph;
  if (e == hipSuccess) e = e2;
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_graph_destroy");
}

}  // extern "C"

namespace {

int32_t check_pagedset(const cm_pagedset* set, cm::PagedDesc* out) {
  if (!set) return fail(CM_EINVAL, "set is NULL");
  if (set->n < 1 || set->n > CM_MAX_FRAGMENTS)
    return fail(CM_EINVAL, "n must be in [1, " + std::to_string(CM_MAX_FRAGMENTS) + "]");
  if (set->L < 1 || set->H < 1) return fail(CM_EINVAL, "L and H must be >= 1");
  if ((int64_t)2 * set->L * set->H > 65535) return fail(CM_ESHAPE, "2 * L * H must be <= 65535");
  int esize = 0;
  if (set->dtype == CM_F32) esize = 4;
  else if (set->dtype == CM_BF16) esize = 2;
  else return fail(CM_EDTYPE, "dtype must be CM_F32 or CM_BF16");
  const int64_t row_bytes = (int64_t)set->d * esize;
  if (!is_pow2(set->d) || row_bytes < 64 || row_bytes > 1024)
    return fail(CM_ESHAPE, "d must be a power of two with d * element_bytes in [64, 1024]");
  if (set->block < 1 || !is_pow2(set->block) || set->block * row_bytes < 1024 ||
      set->block * row_bytes > 16384)
    return fail(CM_ESHAPE, "block must be a power of two with block * d * element_bytes in "
                           "[1024, 16384]");
  if (set->pages < 1 || set->pages > ((int64_t)1 << 31) - 1)
    return fail(CM_EINVAL, "pages must be in [1, 2^31)");
  if (!set->pool_dev || !aligned(set->pool_dev, 16))
    return fail(CM_EINVAL, "pool_dev is NULL or not 16-byte aligned");
  if (!set->table_host || !set->table_dev || !set->blocks_host || !set->blocks_dev)
    return fail(CM_EINVAL, "paged tables are NULL");
  if (!aligned(set->table_dev, 8) || !aligned(set->blocks_dev, 4))
    return fail(CM_EINVAL, "table_dev / blocks_dev misaligned");
  if (set->n_blocks < 1) return fail(CM_EINVAL, "n_blocks must be >= 1");
  for (int64_t k = 0; k < set->n_blocks; ++k)
    if (set->blocks_host[k] < 0 || set->blocks_host[k] >= set->pages)
      return fail(CM_EINVAL, "page id " + std::to_string(k) + " outside the pool");
  for (int i = 0; i < set->n; ++i) {
    const int64_t T = set->table_host[2 * (int64_t)i], first = set->table_host[2 * (int64_t)i + 1];
    if (T < 1) return fail(CM_EINVAL, "fragment " + std::to_string(i) + " has T < 1");
    const int64_t nb = (T + set->block - 1) / set->block;
    if (first < 0 || first > set->n_blocks - nb)
      return fail(CM_EINVAL, "fragment " + std::to_string(i) + " page list outside blocks");
  }
  cm::SetDesc& s = out->s;
  s.n = set->n;
  s.L = set->L;
  s.H = set->H;
  s.d = set->d;
  s.dtype = set->dtype;
  s.esize = esize;
  s.stride = 2;
  s.row_bytes = row_bytes;
  s.table_dev = set->table_dev;
  s.table_host = set->table_host;
  out->block = set->block;
  out->b_shift = __builtin_ctz((unsigned)set->block);
  out->pages = set->pages;
  out->pool = set->pool_dev;
  out->blocks_dev = set->blocks_dev;
  return CM_OK;
}

// Workspace of the paged render: angles, then 32 bytes per fresh page (at most
// two per merged block of B rows, T_out at most the sum of the lengths).
size_t paged_render_ws(const cm::PagedDesc& p) {
  int64_t T_all = 0;
  for (int i = 0; i < p.s.n; ++i) T_all += p.s.T(i);
  const int64_t blocks = (T_all + p.block - 1) / p.block;
  return cm::align_up(sizeof(double) * (size_t)p.s.n * p.s.d, cm::kWsAlign) +
         cm::align_up(32 * 2 * (size_t)blocks, cm::kWsAlign);
}

// Workspace of the paged hash + render: the hash layout, then the render's.
size_t paged_fused_ws(const cm::PagedDesc& p) {
  return cm::align_up(cm::hash_layout(p.s).bytes, cm::kWsAlign) + cm::render_layout(p.s).bytes;
}

// Every paged call fits: the render's, the fused hash + render's, or the
// scores' and Ids' of cm_paged_order (which run one after the other over the
// same bytes).
size_t paged_ws(const cm::PagedDesc& p) {
  size_t need = paged_render_ws(p);
  const size_t kn = cm::knorm_max_bytes(p.s);
  const size_t hb = cm::hash_layout(p.s).bytes;
  const size_t fu = paged_fused_ws(p);
  if (kn > need) need = kn;
  if (hb > need) need = hb;
  if (fu > need) need = fu;
  return need;
}

// Plan checks against the fragments' lengths (slots, lengths, prefix offsets).
int32_t check_plan_host(const cm::SetDesc& s, const int64_t* plan_host, int64_t* nu_out) {
  if (!plan_host) return fail(CM_EINVAL, "plan_host is NULL");
  if (plan_host[CM_PLAN_STATUS] != CM_OK) return fail(CM_EINVAL, "plan status is not CM_OK");
  if (plan_host[CM_PLAN_N] != s.n) return fail(CM_EINVAL, "plan was built for another n");
  const int64_t nu = plan_host[CM_PLAN_NUNIQUE];
  if (nu < 1 || nu > s.n) return fail(CM_EINVAL, "plan n_unique out of range");
  int64_t off = 0;
  for (int64_t k = 0; k < nu; ++k) {
    const int64_t src = plan_host[CM_PLAN_HEADER + k];
    if (src < 0 || src >= s.n) return fail(CM_EINVAL, "plan slot refers to no fragment");
    if (plan_host[CM_PLAN_HEADER + 2 * (int64_t)s.n + k] != s.T((int)src))
      return fail(CM_ESHAPE, "plan slot length differs from the fragment's T");
    if (plan_host[CM_PLAN_HEADER + s.n + k] != off)
      return fail(CM_ESHAPE, "plan offsets are not the prefix sum of slot lengths");
    off += s.T((int)src);
  }
  if (plan_host[CM_PLAN_TOUT] != off) return fail(CM_ESHAPE, "plan T_out is not the sum of lengths");
  *nu_out = nu;
  return CM_OK;
}

// Merged block j of a plan's cache (rows [jB, min(jB + B, T_out))) can keep a
// fragment page, with no copy, when all its rows come from one slot and start at
// a page boundary of that slot's fragment: that page (-1 if none), and whether
// the slot is at offset 0 (K pages only then: R(0) = I). s: the slot holding
// row jB, advanced from the previous block's.
struct Reuse {
  int32_t page;
  bool k_too;
};
Reuse reusable_page(const cm_pagedset* set, const int64_t* plan_host, int64_t nu, int64_t j,
                    int64_t* s) {
  const int64_t n = set->n, B = set->block;
  const int64_t T_out = plan_host[CM_PLAN_TOUT];
  const int64_t r0 = j * B, e = std::min(r0 + B, T_out);
  while (*s + 1 < nu && plan_host[CM_PLAN_HEADER + n + *s + 1] <= r0) ++*s;
  const int64_t i = plan_host[CM_PLAN_HEADER + *s];
  const int64_t off = plan_host[CM_PLAN_HEADER + n + *s];
  const int64_t T = plan_host[CM_PLAN_HEADER + 2 * n + *s];
  const bool whole_page = e <= off + T && (r0 - off) % B == 0;
  Reuse r;
  r.page = whole_page ? set->blocks_host[set->table_host[2 * i + 1] + (r0 - off) / B] : -1;
  r.k_too = off == 0;
  return r;
}

// Block tables given by the caller for a render that writes every row whose
// merged page is not the page it is read from: every entry a page of the pool;
// a fragment page only where reusable_page allows it (then it is that page);
// every other page used once.
int32_t check_block_tables(const cm_pagedset* set, const int64_t* plan_host, int64_t nu,
                           const int32_t* k_table_host, const int32_t* v_table_host) {
  if (!k_table_host || !v_table_host) return fail(CM_EINVAL, "k_table_host / v_table_host NULL");
  std::vector<uint8_t> used((size_t)set->pages, 0);
  for (int64_t k = 0; k < set->n_blocks; ++k) used[(size_t)set->blocks_host[k]] = 1;
  const int64_t nbo = (plan_host[CM_PLAN_TOUT] + set->block - 1) / set->block;
  int64_t s = 0;
  for (int64_t j = 0; j < nbo; ++j) {
    const Reuse r = reusable_page(set, plan_host, nu, j, &s);
    for (int kv = 0; kv < 2; ++kv) {
      const int32_t q = (kv ? v_table_host : k_table_host)[j];
      const std::string where = std::string(kv ? "v" : "k") + "_table[" + std::to_string(j) + "]";
      if (q < 0 || q >= set->pages) return fail(CM_EINVAL, where + " is outside the pool");
      if (used[(size_t)q] == 1) {
        if (q != r.page || (kv == 0 && !r.k_too))
          return fail(CM_EINVAL, where + " is a fragment page that this block cannot reuse");
      } else {
        if (used[(size_t)q] == 2) return fail(CM_EINVAL, where + " repeats a page");
        used[(size_t)q] = 2;
      }
    }
  }
  return CM_OK;
}

}  // namespace

extern "C" {

int32_t cm_paged_workspace_size(const cm_pagedset* set, size_t* bytes_out) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if (!bytes_out) return fail(CM_EINVAL, "bytes_out is NULL");
  *bytes_out = paged_ws(p);
  return CM_OK;
}

}  // extern "C"

namespace {

// Argument checks of steps 1-3 on a paged set (cm_paged_order and
// cm_paged_deliveries).
int32_t check_paged_order_args(const cm::PagedDesc& p, int32_t routing_layer, int64_t tail_len,
                               const double* keys_dev, const uint8_t* mask_dev,
                               const uint8_t* digests_dev, const int64_t* plan_dev) {
  const cm::SetDesc& s = p.s;
  if (routing_layer < 0 || routing_layer >= s.L)
    return fail(CM_EINVAL, "routing_layer must be in [0, L), got " + std::to_string(routing_layer));
  const int64_t tmin = min_T(s);
  if (tail_len < 1 || tail_len > tmin)
    return fail(CM_EINVAL, "tail_len must be in [1, min T] = [1, " + std::to_string(tmin) + "], got " +
                               std::to_string(tail_len));
  if (!keys_dev || !aligned(keys_dev, 8)) return fail(CM_EINVAL, "keys_dev is NULL or misaligned");
  if (!mask_dev) return fail(CM_EINVAL, "mask_dev is NULL");
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  return CM_OK;
}

// Steps 1-3 on a paged set: scores, the deliveries whose digest the order reads
// (a key equal to another's), their Ids, the order. The other Ids are left to
// the caller (cm_paged_hash_select beside the render, or the fused render).
hipError_t enqueue_paged_order(const cm::PagedDesc& p, int32_t routing_layer, int64_t tail_len,
                               double* keys_dev, uint8_t* mask_dev, uint8_t* digests_dev,
                               int64_t* plan_dev, uint8_t* ws, hipStream_t sm) {
  const cm::SetDesc& s = p.s;
  hipError_t e = cm::launch_knorm_paged(p, cm::knorm_layout(s, tail_len), routing_layer, tail_len,
                                        keys_dev, ws, sm);
  if (e == hipSuccess) e = cm::launch_equal_key_mask(s, keys_dev, mask_dev, sm);
  if (e == hipSuccess)
    e = cm::launch_hash_paged(p, cm::hash_layout(s), mask_dev, 1, digests_dev, ws, sm);
  if (e == hipSuccess) e = cm::launch_order(s, keys_dev, digests_dev, true, plan_dev, sm);
  return e;
}

// A free-page list: pages of the pool, distinct, holding no fragment row.
int32_t check_free_pages(const cm_pagedset* set, const int32_t* free_host, int64_t n_free) {
  if (n_free < 0 || (n_free > 0 && !free_host)) return fail(CM_EINVAL, "free_host is NULL");
  std::vector<uint8_t> used((size_t)set->pages, 0);
  for (int64_t k = 0; k < set->n_blocks; ++k) used[(size_t)set->blocks_host[k]] = 1;
  for (int64_t k = 0; k < n_free; ++k) {
    const int32_t q = free_host[k];
    if (q < 0 || q >= set->pages || used[(size_t)q])
      return fail(CM_EINVAL, "free page " + std::to_string(k) +
                                 " is outside the pool, repeated or holds a fragment page");
    used[(size_t)q] = 2;
  }
  return CM_OK;
}

}  // namespace

extern "C" {

int32_t cm_paged_order(const cm_pagedset* set, int32_t routing_layer, int64_t tail_len,
                       double* keys_dev, uint8_t* mask_dev, uint8_t* digests_dev,
                       int64_t* plan_dev, void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if ((st = check_paged_order_args(p, routing_layer, tail_len, keys_dev, mask_dev, digests_dev,
                                   plan_dev)) != CM_OK)
    return st;
  if ((st = check_ws(workspace, workspace_bytes, paged_ws(p))) != CM_OK) return st;
  hipError_t e = enqueue_paged_order(p, routing_layer, tail_len, keys_dev, mask_dev, digests_dev,
                                     plan_dev, static_cast<uint8_t*>(workspace),
                                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_paged_order");
}

int32_t cm_paged_deliveries(const cm_pagedset* set, int32_t routing_layer, int64_t tail_len,
                            const cm_rope* rope, const int32_t* free_host,
                            const int32_t* free_dev, int64_t n_free, double* keys_dev,
                            uint8_t* mask_dev, uint8_t* digests_dev, int64_t* plan_dev,
                            int32_t* k_table_dev, int32_t* v_table_dev, int64_t* n_fresh_dev,
                            void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if ((uint64_t)set->pages * (uint64_t)set->H * (uint64_t)set->block > 0xFFFFFFFFull)
    return fail(CM_ESHAPE, "pages * H * block must be below 2^32 for the fused paged render");
  if ((st = check_rope(rope)) != CM_OK) return st;
  if ((st = check_paged_order_args(p, routing_layer, tail_len, keys_dev, mask_dev, digests_dev,
                                   plan_dev)) != CM_OK)
    return st;
  if ((st = check_free_pages(set, free_host, n_free)) != CM_OK) return st;
  if (n_free > 0 && (!free_dev || !aligned(free_dev, 4)))
    return fail(CM_EINVAL, "free_dev is NULL or misaligned");
  if (!k_table_dev || !v_table_dev || !aligned(k_table_dev, 4) || !aligned(v_table_dev, 4))
    return fail(CM_EINVAL, "k_table_dev / v_table_dev NULL or misaligned");
  if (!n_fresh_dev || !aligned(n_fresh_dev, 8))
    return fail(CM_EINVAL, "n_fresh_dev is NULL or misaligned");
  if ((st = check_ws(workspace, workspace_bytes, paged_ws(p))) != CM_OK) return st;
  int64_t T_all = 0;
  for (int i = 0; i < p.s.n; ++i) T_all += p.s.T(i);
  const int64_t nbo_cap = (T_all + p.block - 1) / p.block;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  hipStream_t sm = static_cast<hipStream_t>(stream);
  // steps 1-3 (the colliding deliveries' Ids), the block tables, then the
  // render with every other Id from its loads, in workspace that each step
  // takes over from the one before
  hipError_t e = enqueue_paged_order(p, routing_layer, tail_len, keys_dev, mask_dev, digests_dev,
                                     plan_dev, ws, sm);
  if (e == hipSuccess)
    e = cm::launch_paged_tables(p, plan_dev, free_dev, n_free, nbo_cap, k_table_dev, v_table_dev,
                                n_fresh_dev, sm);
  if (e == hipSuccess)
    e = cm::launch_paged_render_hash(p, cm::hash_layout(p.s), cm::render_layout(p.s), plan_dev,
                                     rope->base, rope->style, mask_dev, k_table_dev, v_table_dev,
                                     digests_dev, ws, sm);
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_paged_deliveries");
}

int32_t cm_paged_hash_select(const cm_pagedset* set, const uint8_t* select_dev,
                             int32_t select_value, uint8_t* digests_dev, int32_t workgroups_per_cu,
                             void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if (select_value < 0 || select_value > 255)
    return fail(CM_EINVAL, "select_value must be in [0, 255]");
  if (workgroups_per_cu < 0 || workgroups_per_cu > 64)
    return fail(CM_EINVAL, "workgroups_per_cu must be in [0, 64]");
  const cm::HashLayout lay = cm::hash_layout(p.s);
  if ((st = check_ws(workspace, workspace_bytes, lay.bytes)) != CM_OK) return st;
  hipError_t e = cm::launch_hash_paged(p, lay, select_dev, (uint32_t)select_value, digests_dev,
                                       static_cast<uint8_t*>(workspace),
                                       static_cast<hipStream_t>(stream), workgroups_per_cu);
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_paged_hash_select");
}

int32_t cm_paged_tables(const cm_pagedset* set, const int64_t* plan_host, const int32_t* free_host,
                        int64_t n_free, int32_t* k_table_host, int32_t* v_table_host,
                        int32_t* fresh_host, int64_t* n_fresh) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  int64_t nu = 0;
  if ((st = check_plan_host(p.s, plan_host, &nu)) != CM_OK) return st;
  if (!k_table_host || !v_table_host || !fresh_host || !n_fresh)
    return fail(CM_EINVAL, "output pointer is NULL");
  if ((st = check_free_pages(set, free_host, n_free)) != CM_OK) return st;
  const int64_t B = p.block;
  const int64_t T_out = plan_host[CM_PLAN_TOUT];
  const int64_t nbo = (T_out + B - 1) / B;
  int64_t taken = 0, count = 0;
  int64_t s = 0;                                   // slot holding row j * B
  for (int64_t j = 0; j < nbo; ++j) {
    const Reuse r = reusable_page(set, plan_host, nu, j, &s);
    for (int kv = 0; kv < 2; ++kv) {
      int32_t* tab = kv ? v_table_host : k_table_host;
      if (r.page >= 0 && (kv == 1 || r.k_too)) {
        tab[j] = r.page;
      } else {
        tab[j] = taken < n_free ? free_host[taken] : -1;
        ++taken;
        fresh_host[count++] = (int32_t)(2 * j + kv);
      }
    }
  }
  *n_fresh = count;
  if (taken <= n_free) {
    std::sort(fresh_host, fresh_host + count, [&](int32_t a, int32_t b) {
      const int32_t pa = (a & 1 ? v_table_host : k_table_host)[a >> 1];
      const int32_t pb = (b & 1 ? v_table_host : k_table_host)[b >> 1];
      return (a & 1) != (b & 1) ? (a & 1) < (b & 1) : pa < pb;
    });
  }
  if (taken > n_free)
    return fail(CM_EINVAL, "need " + std::to_string(taken) + " free pages, got " +
                               std::to_string(n_free));
  return CM_OK;
}

int32_t cm_paged_render(const cm_pagedset* set, const int64_t* plan_dev, const int64_t* plan_host,
                        const cm_rope* rope, const int32_t* k_table_dev,
                        const int32_t* v_table_dev, const int32_t* fresh_dev, int64_t n_fresh,
                        void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if ((st = check_rope(rope)) != CM_OK) return st;
  int64_t nu = 0;
  if ((st = check_plan_host(p.s, plan_host, &nu)) != CM_OK) return st;
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  const int64_t nbo = (plan_host[CM_PLAN_TOUT] + p.block - 1) / p.block;
  if (n_fresh < 0 || n_fresh > 2 * nbo) return fail(CM_EINVAL, "n_fresh out of range");
  if (n_fresh > 0 && (!fresh_dev || !k_table_dev || !v_table_dev))
    return fail(CM_EINVAL, "fresh_dev / tables are NULL");
  if ((st = check_ws(workspace, workspace_bytes, paged_render_ws(p))) != CM_OK) return st;
  hipError_t e = cm::launch_paged_render(p, plan_dev, (int32_t)nu, rope->base, rope->style,
                                         k_table_dev, v_table_dev, fresh_dev, n_fresh,
                                         static_cast<uint8_t*>(workspace),
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_paged_render");
}

int32_t cm_paged_render_hash(const cm_pagedset* set, const int64_t* plan_dev,
                             const int64_t* plan_host, const cm_rope* rope,
                             const int32_t* k_table_host, const int32_t* v_table_host,
                             const int32_t* k_table_dev, const int32_t* v_table_dev,
                             const uint8_t* select_dev, uint8_t* digests_dev, void* workspace,
                             size_t workspace_bytes, void* stream) {
  g_err.clear();
  cm::PagedDesc p;
  int32_t st = check_pagedset(set, &p);
  if (st != CM_OK) return st;
  if ((uint64_t)set->pages * (uint64_t)set->H * (uint64_t)set->block > 0xFFFFFFFFull)
    return fail(CM_ESHAPE, "pages * H * block must be below 2^32 for the fused paged render");
  if ((st = check_rope(rope)) != CM_OK) return st;
  int64_t nu = 0;
  if ((st = check_plan_host(p.s, plan_host, &nu)) != CM_OK) return st;
  if (!plan_dev || !aligned(plan_dev, 8)) return fail(CM_EINVAL, "plan_dev is NULL or misaligned");
  if ((st = check_block_tables(set, plan_host, nu, k_table_host, v_table_host)) != CM_OK) return st;
  if (!k_table_dev || !v_table_dev || !aligned(k_table_dev, 4) || !aligned(v_table_dev, 4))
    return fail(CM_EINVAL, "k_table_dev / v_table_dev NULL or misaligned");
  if (!select_dev) return fail(CM_EINVAL, "select_dev is NULL");
  if (!digests_dev || !aligned(digests_dev, 16))
    return fail(CM_EINVAL, "digests_dev is NULL or not 16-byte aligned");
  if ((st = check_ws(workspace, workspace_bytes, paged_fused_ws(p))) != CM_OK) return st;
  const cm::HashLayout hlay = cm::hash_layout(p.s);
  const cm::RenderLayout rlay = cm::render_layout(p.s);
  hipError_t e = cm::launch_paged_render_hash(p, hlay, rlay, plan_dev, rope->base, rope->style,
                                              select_dev, k_table_dev, v_table_dev, digests_dev,
                                              static_cast<uint8_t*>(workspace),
                                              static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_paged_render_hash");
}

int32_t cm_timing_enable(int32_t on) {
  g_err.clear();
  g_timing.store(on != 0);
  return CM_OK;
}

int32_t cm_timing_reset(void) {
  g_err.clear();
  hipError_t e = drain_pending();
  std::lock_guard<std::mutex> lk(g_tmu);
  for (int k = 0; k < cm::K_COUNT; ++k) {
    g_total_ms[k] = 0.0;
    g_count[k] = 0;
  }
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_timing_reset");
}

int32_t cm_timing_query(const char* kernel, double* total_ms, int64_t* launches) {
  g_err.clear();
  if (!kernel || !total_ms || !launches) return fail(CM_EINVAL, "NULL argument");
  int id = -1;
  for (int k = 0; k < cm::K_COUNT; ++k)
    if (std::strcmp(kernel, kKernelNames[k]) == 0) id = k;
  if (id < 0) return fail(CM_EINVAL, std::string("unknown kernel name ") + kernel);
  hipError_t e = drain_pending();
  std::lock_guard<std::mutex> lk(g_tmu);
  *total_ms = g_total_ms[id];
  *launches = g_count[id];
  return e == hipSuccess ? CM_OK : fail_hip(e, "cm_timing_query");
}

}  // extern "C"
