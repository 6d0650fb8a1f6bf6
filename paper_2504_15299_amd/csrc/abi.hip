// C ABI of libd2moe: argument validation on the host, then asynchronous
// launches on the caller's stream.  No allocation.  The only global state is
// the per-device address of the fixed scratch array that the allocation-free
// forward uses (d2moe_moe_forward_noalloc).
#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.h"

using namespace d2moe;

// Fixed forward workspace for callers that cannot allocate (HIP graph
// capture, serving loops that forbid hipMalloc).  Each GPU the library runs
// on holds its own copy until the process ends.  Host code never uses the
// array's name as an address: its device address is looked up once per
// device with hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) uint8_t scratch[D2MOE_NOALLOC_SCRATCH_BYTES];

namespace {

bool ladder_ok(int b_min, int b_max) { return b_min >= 1 && b_min <= b_max && b_max <= 8; }

bool shape_ok(int rows, int cols, int group) {
  if (group != 64 && group != 128) return false;
  if (rows <= 0 || cols <= 0 || cols % group != 0) return false;
  return rows % (2048 / group) == 0;
}

bool mwq_ok(const d2moe_mwq* m) {
  return m && m->n_experts >= 1 && shape_ok(m->rows, m->cols, m->group) &&
         ladder_ok(m->b_min, m->b_max) && m->planes && m->scales && m->zeros;
}

d2moe_status from_hip(hipError_t e) { return e == hipSuccess ? D2MOE_OK : D2MOE_EHIP; }

// Device address of `scratch` on the current device, looked up at the first
// call on that device (with that device current) and kept for the process.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

d2moe_status noalloc_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return D2MOE_EHIP;
  if (dev >= kMaxDevices) return D2MOE_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return D2MOE_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return D2MOE_OK;
}

}  // namespace

extern "C" {

const char* d2moe_status_string(d2moe_status s) {
  switch (s) {
    case D2MOE_OK: return "ok";
    case D2MOE_EINVAL: return "invalid argument";
    case D2MOE_EUNSUPPORTED: return "unsupported";
    case D2MOE_EHIP: return "HIP error";
    case D2MOE_EWORKSPACE: return "workspace too small";
    case D2MOE_ESCRATCH: return "sizes need more than the fixed no-allocation scratch";
    default: return "unknown status";
  }
}

d2moe_status d2moe_mwq_size(int32_t n_experts, int32_t rows, int32_t cols, int32_t group,
                            int32_t b_min, int32_t b_max, size_t* planes_bytes,
                            size_t* scales_bytes, size_t* zeros_bytes) {
  if (n_experts < 1 || !shape_ok(rows, cols, group) || !ladder_ok(b_min, b_max))
    return D2MOE_EINVAL;
  const size_t E = (size_t)n_experts, N = (size_t)rows, K = (size_t)cols;
  if (planes_bytes) *planes_bytes = E * N * K / 32 * (size_t)b_max * 4;
  if (scales_bytes) *scales_bytes = E * N * (K / group) * (size_t)(b_max - b_min + 1) * 2;
  if (zeros_bytes) *zeros_bytes = E * N * (K / group);
  return D2MOE_OK;
}

d2moe_status d2moe_pack_mwq(const void* W, d2moe_dtype w_dtype, const d2moe_mwq* out,
                            void* stream) {
  if (!W || !mwq_ok(out)) return D2MOE_EINVAL;
  if (w_dtype != D2MOE_F32) return D2MOE_EUNSUPPORTED;
  return from_hip(launch_pack((const float*)W, out, (hipStream_t)stream));
}

d2moe_status d2moe_mwq_calib_factor_workspace(int32_t h, size_t* bytes) {
  if (h < 64 || h % 64 != 0 || !bytes) return D2MOE_EINVAL;
  *bytes = calib_factor_workspace(h);
  return D2MOE_OK;
}

d2moe_status d2moe_mwq_calib_factor(const float* X, int32_t tokens, int32_t h, double lambda,
                                    float* U, int32_t* info, void* workspace, size_t ws_bytes,
                                    void* stream) {
  if (h < 64 || h % 64 != 0 || tokens < 0 || !(lambda >= 0.0) || !U || !info ||
      (tokens > 0 && !X))
    return D2MOE_EINVAL;
  if ((long long)tokens * h > (1ll << 40)) return D2MOE_EINVAL;
  if (!workspace || ws_bytes < calib_factor_workspace(h) || ((uintptr_t)workspace & 255u) != 0)
    return D2MOE_EWORKSPACE;
  return from_hip(launch_calib_factor(X, tokens, h, lambda, U, workspace, info,
                                      (hipStream_t)stream));
}

d2moe_status d2moe_pack_mwq_calibrated_workspace(int32_t rows, int32_t cols, int32_t gamma,
                                                 size_t* bytes) {
  if (rows < 1 || cols < 1 || (gamma != 64 && gamma != 128) || cols % gamma != 0 || !bytes)
    return D2MOE_EINVAL;
  *bytes = calib_pack_workspace(rows, cols, gamma);
  return D2MOE_OK;
}

d2moe_status d2moe_pack_mwq_calibrated(const void* W, d2moe_dtype w_dtype, const float* U,
                                       int32_t gamma, const d2moe_mwq* out, void* workspace,
                                       size_t ws_bytes, void* stream) {
  if (!W || !U || !mwq_ok(out)) return D2MOE_EINVAL;
  if (w_dtype != D2MOE_F32) return D2MOE_EUNSUPPORTED;
  if ((gamma != 64 && gamma != 128) || gamma % out->group != 0 || out->cols % gamma != 0)
    return D2MOE_EINVAL;
  if (!workspace || ws_bytes < calib_pack_workspace(out->rows, out->cols, gamma) ||
      ((uintptr_t)workspace & 255u) != 0)
    return D2MOE_EWORKSPACE;
  return from_hip(launch_pack_calibrated((const float*)W, U, gamma, out, workspace,
                                         (hipStream_t)stream));
}

d2moe_status d2moe_debug_unpack(const d2moe_mwq* w, int32_t expert, int32_t bits, uint8_t* q1,
                                int8_t* signs, void* stream) {
  if (!mwq_ok(w) || expert < 0 || expert >= w->n_experts || bits < w->b_min ||
      bits > w->b_max || !q1 || (bits > w->b_min && !signs))
    return D2MOE_EINVAL;
  return from_hip(launch_debug_unpack(w, expert, bits, q1, signs, (hipStream_t)stream));
}

d2moe_status d2moe_route(const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d,
                         const float* Wg, const float* bias, int32_t E, int32_t k,
                         const int32_t* token_req, const uint8_t* bit_table, int32_t R,
                         int32_t b_min, int32_t b_max, const d2moe_routing* out, void* stream) {
  if (T < 0 || d < 1 || E < 1 || E > 64 || k < 1 || k > E || R < 1 || !ladder_ok(b_min, b_max))
    return D2MOE_EINVAL;
  if (x_dtype != D2MOE_F32 && x_dtype != D2MOE_BF16) return D2MOE_EUNSUPPORTED;
  if (!out || !out->hist || !out->offsets || !out->expert_maxbit || !out->flags)
    return D2MOE_EINVAL;
  if (T > 0 && (!out->topk_idx || !out->topk_w || !out->topk_bits || !out->perm ||
                !out->slot_of || !out->logits))
    return D2MOE_EINVAL;
  if (T > 0 && (!x || !Wg || !bit_table)) return D2MOE_EINVAL;
  if ((long long)T * k > (1ll << 30)) return D2MOE_EINVAL;
  return from_hip(launch_route(x, x_dtype, T, d, Wg, bias, E, k, token_req, bit_table, R, b_min,
                               b_max, out, (hipStream_t)stream));
}

d2moe_status d2moe_route_learned(const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d,
                                 const float* Wg, const float* bias, int32_t E, int32_t k,
                                 const float* Wr, const float* br, int32_t b_min, int32_t b_max,
                                 float* bit_logits, const d2moe_routing* out, void* stream) {
  if (T < 0 || d < 1 || E < 1 || E > 64 || k < 1 || k > E || !ladder_ok(b_min, b_max))
    return D2MOE_EINVAL;
  if (x_dtype != D2MOE_F32 && x_dtype != D2MOE_BF16) return D2MOE_EUNSUPPORTED;
  if (!out || !out->hist || !out->offsets || !out->expert_maxbit || !out->flags)
    return D2MOE_EINVAL;
  if (T > 0 && (!out->topk_idx || !out->topk_w || !out->topk_bits || !out->perm ||
                !out->slot_of || !out->logits))
    return D2MOE_EINVAL;
  if (T > 0 && (!x || !Wg || !Wr || !bit_logits)) return D2MOE_EINVAL;
  if ((long long)T * k > (1ll << 30) || (long long)T * E * (b_max - b_min + 1) > (1ll << 31))
    return D2MOE_EINVAL;
  return from_hip(launch_route_learned(x, x_dtype, T, d, Wg, bias, E, k, Wr, br, b_min, b_max,
                                       bit_logits, out, (hipStream_t)stream));
}

d2moe_status d2moe_moe_forward_workspace(int32_t T, int32_t d, int32_t d_ff, int32_t E,
                                         int32_t k, int32_t shared_d_ff, size_t* bytes) {
  if (T < 0 || d < 1 || d_ff < 1 || E < 1 || E > 64 || k < 1 || k > E || shared_d_ff < 0 ||
      !bytes)
    return D2MOE_EINVAL;
  *bytes = fwd_workspace_layout(T, d, d_ff, E, k, shared_d_ff).total;
  return D2MOE_OK;
}

static d2moe_status forward_impl(const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d,
                                 int32_t d_ff, int32_t E, int32_t k, const d2moe_mwq* w13,
                                 const d2moe_mwq* w2, const d2moe_routing* r,
                                 const d2moe_mwq* shared_w13, const d2moe_mwq* shared_w2,
                                 int32_t shared_bits, int32_t shared_d_ff, void* out,
                                 void* workspace, size_t ws_bytes, void* stream,
                                 void* const* events, bool concurrent) {
  if (T < 0 || d < 1 || d_ff < 1 || E < 1 || E > 64 || k < 1 || k > E) return D2MOE_EINVAL;
  if (x_dtype != D2MOE_F32 && x_dtype != D2MOE_BF16) return D2MOE_EUNSUPPORTED;
  if (!mwq_ok(w13) || !mwq_ok(w2) || !r) return D2MOE_EINVAL;
  if (w13->n_experts != E || w13->rows != 2 * d_ff || w13->cols != d) return D2MOE_EINVAL;
  if (w2->n_experts != E || w2->rows != d || w2->cols != d_ff) return D2MOE_EINVAL;
  if (w13->b_min != w2->b_min || w13->b_max != w2->b_max) return D2MOE_EINVAL;
  // output tiling: 32-row slices of W1/W3, 64-row slices of W2
  if (d_ff % 32 != 0 || d % 64 != 0) return D2MOE_EUNSUPPORTED;
  if (!r->hist || !r->offsets || !r->expert_maxbit) return D2MOE_EINVAL;
  if (T > 0 && (!r->topk_w || !r->topk_bits || !r->perm || !r->slot_of)) return D2MOE_EINVAL;
  const bool has_shared = shared_w13 || shared_w2;
  if (has_shared) {
    if (!mwq_ok(shared_w13) || !mwq_ok(shared_w2) || shared_d_ff < 1) return D2MOE_EINVAL;
    if (shared_w13->n_experts != 1 || shared_w13->rows != 2 * shared_d_ff ||
        shared_w13->cols != d || shared_w2->n_experts != 1 || shared_w2->rows != d ||
        shared_w2->cols != shared_d_ff)
      return D2MOE_EINVAL;
    if (shared_w13->b_min != shared_w2->b_min || shared_w13->b_max != shared_w2->b_max ||
        shared_bits < shared_w13->b_min || shared_bits > shared_w13->b_max)
      return D2MOE_EINVAL;
    if (shared_d_ff % 32 != 0) return D2MOE_EUNSUPPORTED;
  }
  if (T > 0 && (!x || !out)) return D2MOE_EINVAL;
  const size_t need = fwd_workspace_layout(T, d, d_ff, E, k, has_shared ? shared_d_ff : 0).total;
  if (T > 0 && (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255u) != 0))
    return D2MOE_EWORKSPACE;
  return from_hip(launch_forward(x, x_dtype, T, d, d_ff, E, k, w13, w2, r,
                                 has_shared ? shared_w13 : nullptr,
                                 has_shared ? shared_w2 : nullptr, shared_bits,
                                 has_shared ? shared_d_ff : 0, out, workspace,
                                 (hipStream_t)stream, (hipEvent_t const*)events, concurrent));
}

d2moe_status d2moe_moe_forward(const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d,
                               int32_t d_ff, int32_t E, int32_t k, const d2moe_mwq* w13,
                               const d2moe_mwq* w2, const d2moe_routing* r,
                               const d2moe_mwq* shared_w13, const d2moe_mwq* shared_w2,
                               int32_t shared_bits, int32_t shared_d_ff, void* out,
                               void* workspace, size_t ws_bytes, void* stream) {
  return forward_impl(x, x_dtype, T, d, d_ff, E, k, w13, w2, r, shared_w13, shared_w2,
                      shared_bits, shared_d_ff, out, workspace, ws_bytes, stream, nullptr, true);
}

d2moe_status d2moe_moe_forward_noalloc(const void* x, d2moe_dtype x_dtype, int32_t T,
                                       int32_t d, int32_t d_ff, int32_t E, int32_t k,
                                       const d2moe_mwq* w13, const d2moe_mwq* w2,
                                       const d2moe_routing* r, const d2moe_mwq* shared_w13,
                                       const d2moe_mwq* shared_w2, int32_t shared_bits,
                                       int32_t shared_d_ff, void* out, void* stream) {
  // the workspace size check comes first so that an oversized call is
  // reported as such, with nothing launched
  if (T < 0 || d < 1 || d_ff < 1 || E < 1 || E > 64 || k < 1 || k > E || shared_d_ff < 0)
    return D2MOE_EINVAL;
  const bool has_shared = shared_w13 || shared_w2;
  const size_t need = fwd_workspace_layout(T, d, d_ff, E, k, has_shared ? shared_d_ff : 0).total;
  if (need > (size_t)D2MOE_NOALLOC_SCRATCH_BYTES) return D2MOE_ESCRATCH;
  void* ws = nullptr;
  const d2moe_status st = noalloc_scratch(&ws);
  if (st != D2MOE_OK) return st;
  return forward_impl(x, x_dtype, T, d, d_ff, E, k, w13, w2, r, shared_w13, shared_w2,
                      shared_bits, shared_d_ff, out, ws, (size_t)D2MOE_NOALLOC_SCRATCH_BYTES,
                      stream, nullptr, false);
}

d2moe_status d2moe_moe_forward_profiled(const void* x, d2moe_dtype x_dtype, int32_t T,
                                        int32_t d, int32_t d_ff, int32_t E, int32_t k,
                                        const d2moe_mwq* w13, const d2moe_mwq* w2,
                                        const d2moe_routing* r, const d2moe_mwq* shared_w13,
                                        const d2moe_mwq* shared_w2, int32_t shared_bits,
                                        int32_t shared_d_ff, void* out, void* workspace,
                                        size_t ws_bytes, void* stream, void* const* events) {
  if (!events || !events[0] || !events[1] || !events[2] || !events[3]) return D2MOE_EINVAL;
  return forward_impl(x, x_dtype, T, d, d_ff, E, k, w13, w2, r, shared_w13, shared_w2,
                      shared_bits, shared_d_ff, out, workspace, ws_bytes, stream, events, false);
}

d2moe_status d2moe_residual_rmsnorm(float* x, const void* y, d2moe_dtype y_dtype, int32_t T,
                                    int32_t d, float eps, void* h, d2moe_dtype h_dtype,
                                    void* stream) {
  if (T < 0 || d < 1 || d > norm_max_cols() || !(eps >= 0.0f)) return D2MOE_EINVAL;
  if ((y_dtype != D2MOE_F32 && y_dtype != D2MOE_BF16) ||
      (h_dtype != D2MOE_F32 && h_dtype != D2MOE_BF16))
    return D2MOE_EINVAL;
  if (T > 0 && (!x || !h)) return D2MOE_EINVAL;
  return from_hip(launch_residual_rmsnorm(x, y, y_dtype, T, d, eps, h, h_dtype,
                                          (hipStream_t)stream));
}

d2moe_status d2moe_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t blocks,
                               void* stream) {
  if (!buf || !sink || blocks < 1 || bytes % 16 != 0 || ((uintptr_t)buf & 15u) != 0)
    return D2MOE_EINVAL;
  return from_hip(launch_stream_read(buf, bytes, sink, blocks, (hipStream_t)stream));
}

d2moe_status d2moe_moe_forward_streamed(
    const void* x, d2moe_dtype x_dtype, int32_t T, int32_t d, int32_t d_ff, int32_t E, int32_t k,
    const d2moe_mwq* host_w13, const d2moe_mwq* host_w2, const d2moe_mwq* w13,
    const d2moe_mwq* w2, uint8_t* resident, const d2moe_routing* r, const int32_t* hist_host,
    const d2moe_unit* units, int32_t n_units, void* out, void* workspace, size_t ws_bytes,
    void* stream, void* io_stream, void* const* events) {
  if (T < 0 || d < 1 || d_ff < 1 || E < 1 || E > 64 || k < 1 || k > E) return D2MOE_EINVAL;
  if (x_dtype != D2MOE_F32 && x_dtype != D2MOE_BF16) return D2MOE_EUNSUPPORTED;
  if (!mwq_ok(w13) || !mwq_ok(w2) || !mwq_ok(host_w13) || !mwq_ok(host_w2) || !r || !resident ||
      !hist_host || n_units < 0 || (n_units > 0 && (!units || !events)))
    return D2MOE_EINVAL;
  if (w13->n_experts != E || w13->rows != 2 * d_ff || w13->cols != d) return D2MOE_EINVAL;
  if (w2->n_experts != E || w2->rows != d || w2->cols != d_ff) return D2MOE_EINVAL;
  if (w13->b_min != w2->b_min || w13->b_max != w2->b_max) return D2MOE_EINVAL;
  for (const d2moe_mwq* hm : {host_w13, host_w2}) {
    const d2moe_mwq* dm = hm == host_w13 ? w13 : w2;
    if (hm->n_experts != dm->n_experts || hm->rows != dm->rows || hm->cols != dm->cols ||
        hm->group != dm->group || hm->b_min != dm->b_min || hm->b_max != dm->b_max)
      return D2MOE_EINVAL;
  }
  if (d_ff % 32 != 0 || d % 64 != 0) return D2MOE_EUNSUPPORTED;
  if (T > 0 && (!x || !out || !r->topk_w || !r->perm || !r->slot_of)) return D2MOE_EINVAL;
  const int b_min = w13->b_min, b_max = w13->b_max, L = b_max - b_min + 1;
  // the units must load each expert's planes in the order they are needed and
  // compute every nonempty bucket exactly once
  uint8_t have[64];
  int seen[64 * 8] = {0};
  long total = 0;
  for (int e = 0; e < E; ++e) {
    if (resident[e] != 0 && (resident[e] < b_min || resident[e] > b_max)) return D2MOE_EINVAL;
    have[e] = resident[e];
  }
  for (int i = 0; i < n_units; ++i) {
    const d2moe_unit& u = units[i];
    if (u.expert < 0 || u.expert >= E || u.bits < b_min || u.bits > b_max) return D2MOE_EINVAL;
    const int want_to = have[u.expert] > u.bits ? have[u.expert] : u.bits;
    if (u.load_from != have[u.expert] || u.load_to != want_to) return D2MOE_EINVAL;
    const int bk = u.expert * L + (u.bits - b_min);
    if (u.count < 1 || u.count != hist_host[bk] || seen[bk]) return D2MOE_EINVAL;
    seen[bk] = 1;
    have[u.expert] = (uint8_t)want_to;
    total += u.count;
  }
  for (int i = 0; i < E * L; ++i)
    if (hist_host[i] < 0 || (hist_host[i] > 0 && !seen[i])) return D2MOE_EINVAL;
  if (total != (long)T * k) return D2MOE_EINVAL;
  const size_t need = fwd_workspace_layout(T, d, d_ff, E, k, 0).total;
  if (T > 0 && (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255u) != 0))
    return D2MOE_EWORKSPACE;
  for (int i = 0; i < n_units; ++i)
    if (!events[i]) return D2MOE_EINVAL;
  return from_hip(launch_forward_streamed(x, x_dtype, T, d, d_ff, E, k, host_w13, host_w2, w13,
                                          w2, resident, r, hist_host, units, n_units, out,
                                          workspace, (hipStream_t)stream, (hipStream_t)io_stream,
                                          (hipEvent_t const*)events));
}

d2moe_status d2moe_hebf_order(const int32_t* hist, int32_t E, int32_t b_min, int32_t b_max,
                              const uint8_t* resident, d2moe_unit* units, int32_t* n_units) {
  if (!hist || E < 1 || E > 64 || !ladder_ok(b_min, b_max) || !units || !n_units)
    return D2MOE_EINVAL;
  if (resident)
    for (int j = 0; j < E; ++j)
      if (resident[j] != 0 && (resident[j] < b_min || resident[j] > b_max)) return D2MOE_EINVAL;
  *n_units = hebf_order(hist, E, b_min, b_max, resident, units);
  return D2MOE_OK;
}

d2moe_status d2moe_budget_plan(const uint8_t* want, int32_t n_layers, int32_t E,
                               const int64_t* level_bytes, int32_t K, int64_t budget,
                               uint8_t* resident, d2moe_budget_action* actions,
                               int32_t max_actions, int32_t* n_actions) {
  if (!want || n_layers < 1 || E < 1 || !level_bytes || K < 1 || K > 8 || !resident ||
      !n_actions || max_actions < 0 || (max_actions > 0 && !actions))
    return D2MOE_EINVAL;
  for (long i = 0; i < (long)n_layers * E; ++i)
    if (want[i] > K || resident[i] > K) return D2MOE_EINVAL;
  for (int l = 0; l < K; ++l)
    if (level_bytes[l] < 0) return D2MOE_EINVAL;
  // plan on a copy, so that a too-small action array leaves the caller's
  // residency untouched
  std::vector<uint8_t> res(resident, resident + (size_t)n_layers * E);
  const int n = budget_plan(want, n_layers, E, level_bytes, K, budget, res.data(), actions,
                            max_actions);
  if (n < 0) {
    *n_actions = -n - 1;
    return D2MOE_EINVAL;
  }
  std::copy(res.begin(), res.end(), resident);
  *n_actions = n;
  return D2MOE_OK;
}

}  // extern "C"
