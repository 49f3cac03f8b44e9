// Host side of the C ABI declared in include/xshare.h: argument validation (before any
// HIP call), workspace carving and kernel launches.  No allocation, no synchronisation.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "internal.h"
#include "xshare.h"

namespace {

using xs::kMaxAssignments;
using xs::kMaxExperts;
using xs::kMaxTokens;
using xs::kMaxTopK;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Parameter checks shared by every entry point.  `hier` enables the m_r check; `ep` (GPU
// groups) requires the per-group budget mode, which is valid only there.
xshare_status check_params(int32_t T, const xshare_route_params* p, bool hier, bool ep = false) {
  if (!p) return XSHARE_EINVAL;
  if (T < 0 || p->n_experts < 1 || p->top_k < 1 || p->top_k > p->n_experts) return XSHARE_EINVAL;
  if (p->warmup_k0 < 0 || p->warmup_k0 > p->top_k || p->budget < 0) return XSHARE_EINVAL;
  if (ep ? p->budget_mode != XSHARE_BUDGET_PER_GROUP
         : (p->budget_mode != XSHARE_BUDGET_TOTAL && p->budget_mode != XSHARE_BUDGET_EXTRA &&
            p->budget_mode != XSHARE_BUDGET_THRESHOLD))
    return XSHARE_EINVAL;
  if (p->budget_mode == XSHARE_BUDGET_THRESHOLD &&
      !(std::isfinite(p->threshold) && p->threshold >= 0.0f))
    return XSHARE_EINVAL;
  if (p->score_mode != XSHARE_SCORE_TOPK && p->score_mode != XSHARE_SCORE_DENSE)
    return XSHARE_EINVAL;
  if (p->budget_mode == XSHARE_BUDGET_TOTAL && p->budget < p->top_k) return XSHARE_EINVAL;
  if (hier && p->per_request_budget < 0) return XSHARE_EINVAL;
  if (p->n_experts > kMaxExperts || p->top_k > kMaxTopK || T > kMaxTokens ||
      (int64_t)T * p->top_k > kMaxAssignments)
    return XSHARE_EUNSUPPORTED;
  return XSHARE_OK;
}

xshare_status check_offsets(int32_t T, const int32_t* req_offsets, const int32_t* host_offsets,
                            int32_t R) {
  if (R < 0 || R > T || (R == 0) != (T == 0)) return XSHARE_EINVAL;
  if (R > 0 && !req_offsets) return XSHARE_EINVAL;
  if (host_offsets) {
    if (host_offsets[0] != 0 || host_offsets[R] != T) return XSHARE_EINVAL;
    for (int r = 0; r < R; ++r)
      if (host_offsets[r + 1] <= host_offsets[r]) return XSHARE_EINVAL;
  }
  return XSHARE_OK;
}

// GPU-group layout: 1 <= G <= N; equal contiguous blocks need G | N; a host copy of the
// map is validated; `forward` also checks the local group.
xshare_status check_ep(int32_t N, const xshare_ep_layout* ep, bool forward) {
  if (!ep) return XSHARE_OK;
  const int G = ep->n_groups;
  if (G < 1 || G > N) return XSHARE_EINVAL;
  if (!ep->expert_group && N % G != 0) return XSHARE_EINVAL;
  if (ep->host_expert_group)
    for (int j = 0; j < N; ++j)
      if (ep->host_expert_group[j] < 0 || ep->host_expert_group[j] >= G) return XSHARE_EINVAL;
  if (forward && (ep->local_group < -1 || ep->local_group >= G)) return XSHARE_EINVAL;
  return XSHARE_OK;
}

// Bound on the experts the expert GEMMs are launched for (grid size; blocks beyond the
// device-side count exit at once).  Active experts never exceed the selected set (<= budget
// under a total budget) nor the (token, slot) pairs.  One group's share also stays within
// the group and within its load, which is at most max(m_g, |S_0 on the group|) after the
// rounds, or at most k after a top-up to k experts; |S_0| <= T * k0.
int layer_bound(int32_t T, const xshare_route_params* p, const xshare_ep_layout* ep) {
  const int N = p->n_experts, k = p->top_k;
  int b = xs::active_bound(T, N, k, p->budget_mode, p->budget);
  if (ep && ep->local_group >= 0) {
    int size = N;
    if (!ep->expert_group) {
      size = N / ep->n_groups;
    } else if (ep->host_expert_group) {
      size = 0;
      for (int j = 0; j < N; ++j) size += ep->host_expert_group[j] == ep->local_group;
    }
    const int64_t load = std::max<int64_t>(std::max<int64_t>(p->budget, k),
                                           (int64_t)T * p->warmup_k0);
    b = (int)std::min<int64_t>(std::min(b, size), load);
  }
  return b;
}

// Experts expected to be active, for the choice of split counts (speed only): a group's
// share is expected to hold about m_g experts, other calls up to the bound.
int layer_estimate(int32_t T, const xshare_route_params* p, const xshare_ep_layout* ep) {
  const int b = layer_bound(T, p, ep);
  if (ep && ep->local_group >= 0) return std::min(b, std::max(p->budget, 1));
  return b;
}

template <typename P>
P* at(void* ws, size_t off) {
  return reinterpret_cast<P*>(static_cast<char*>(ws) + off);
}

// Fills the routing arguments; outputs may be redirected to workspace scratch.
xs::RouteArgs route_args(const float* logits, int32_t T, const xshare_route_params* p,
                         const int32_t* req_offsets, int32_t R, const xshare_ep_layout* ep,
                         int32_t* group_load, uint8_t* sel_mask, int32_t* ids, float* w,
                         xshare_stats* stats, void* ws, const xs::RouteLayout& L) {
  xs::RouteArgs a{};
  a.logits = logits;
  a.T = T;
  a.N = p->n_experts;
  a.k = p->top_k;
  a.k0 = p->warmup_k0;
  a.budget = std::min(p->budget, p->n_experts);  // a larger budget selects the same set
  a.budget_mode = p->budget_mode;
  a.score_mode = p->score_mode;
  a.m_r = std::min(p->per_request_budget, p->n_experts);
  a.tau = p->threshold;
  a.req_offsets = req_offsets;
  a.R = R;
  a.G = ep ? ep->n_groups : 0;
  a.group = ep ? ep->expert_group : nullptr;
  a.local_group = -1;
  a.group_load = group_load;
  a.sel_mask = sel_mask;
  a.ids = ids ? ids : at<int32_t>(ws, L.ids);
  a.w = w ? w : at<float>(ws, L.w);
  a.stats = reinterpret_cast<int32_t*>(stats);
  a.ledger = reinterpret_cast<int32_t*>(p->ledger);
  a.offsets = at<int32_t>(ws, L.offsets);
  a.perm = at<int32_t>(ws, L.perm);
  a.active = at<int4>(ws, L.active);
  a.counters = at<int32_t>(ws, L.counters);
  a.dense = p->score_mode == XSHARE_SCORE_DENSE ? at<float>(ws, L.dense) : nullptr;
  return a;
}

int n_shared_of(const xshare_shared_experts* shared) { return shared ? shared->n_shared : 0; }

xs::FfnLayout layer_layout(int32_t T, int32_t d, int32_t f, const xshare_route_params* p,
                           const xshare_ep_layout* ep, int n_shared) {
  return xs::ffn_layout(T, p->n_experts, p->top_k, p->score_mode == XSHARE_SCORE_DENSE, d, f,
                        layer_estimate(T, p, ep) + n_shared, n_shared,
                        p->budget_mode == XSHARE_BUDGET_TOTAL);
}

// Router scratch: its fp32 part planes [parts, T, N].
size_t router_planes_bytes(int32_t T, int32_t d, int32_t N) {
  return xs::align256(sizeof(float) * size_t(xs::router_parts(T, d, N)) *
                      size_t(T > 0 ? T : 1) * size_t(N));
}

// xshare_moe_layer's extra scratch: the router planes, then a logits buffer [T, N] used when
// the caller does not take the logits.
size_t layer_router_bytes(int32_t T, int32_t d, int32_t N) {
  return router_planes_bytes(T, d, N) +
         xs::align256(sizeof(float) * size_t(T > 0 ? T : 1) * size_t(N));
}

// Shared experts: 0 <= N_s <= 64 experts of the routed shape, 16-byte aligned; none with a
// local GPU group (a group's share holds routed experts only).
xshare_status check_shared(const xshare_shared_experts* shared, const xshare_ep_layout* ep) {
  if (!shared || shared->n_shared == 0) return XSHARE_OK;
  if (shared->n_shared < 0) return XSHARE_EINVAL;
  if (shared->n_shared > 64) return XSHARE_EUNSUPPORTED;
  if (!shared->w1 || !shared->w3 || !shared->w2) return XSHARE_EINVAL;
  if (!aligned16(shared->w1) || !aligned16(shared->w3) || !aligned16(shared->w2))
    return XSHARE_EINVAL;
  if (ep && ep->local_group >= 0) return XSHARE_EUNSUPPORTED;
  return XSHARE_OK;
}

xshare_status route_common(const float* logits, int32_t T, const int32_t* req_offsets,
                           const int32_t* host_offsets, int32_t R, bool hier,
                           const xshare_route_params* p, uint8_t* sel_mask, int32_t* ids,
                           float* w, xshare_stats* stats, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  xshare_status st = check_params(T, p, hier);
  if (st != XSHARE_OK) return st;
  if (hier) {
    st = check_offsets(T, req_offsets, host_offsets, R);
    if (st != XSHARE_OK) return st;
  }
  if (!sel_mask || (T > 0 && (!logits || !ids || !w))) return XSHARE_EINVAL;
  const xs::RouteLayout L =
      xs::route_layout(T, p->n_experts, p->top_k, p->score_mode == XSHARE_SCORE_DENSE);
  if (!ws || ws_bytes < L.total) return XSHARE_EWORKSPACE;
  const xs::RouteArgs a = route_args(logits, T, p, hier ? req_offsets : nullptr, R, nullptr,
                                     nullptr, sel_mask, ids, w, stats, ws, L);
  return xs::launch_route(a, stream) == hipSuccess ? XSHARE_OK : XSHARE_EHIP;
}

// Routed expert weights of a layer call, by format: bf16 matrices, FP8 E4M3FN codes with
// one fp32 scale per row, or MXFP4 E2M1 codes with one E8M0 scale per 32 inputs.
struct Weights {
  const uint16_t* w1 = nullptr;
  const uint16_t* w3 = nullptr;
  const uint16_t* w2 = nullptr;
  const uint8_t* q1 = nullptr;
  const uint8_t* q3 = nullptr;
  const uint8_t* q2 = nullptr;
  const float* s1 = nullptr;
  const float* s3 = nullptr;
  const float* s2 = nullptr;
  const uint8_t* e1 = nullptr;   // MXFP4 block scales
  const uint8_t* e3 = nullptr;
  const uint8_t* e2 = nullptr;
  int fmt = 0;                   // XSHARE_WEIGHTS_*
  explicit Weights(const xshare_layer_args& a) : fmt(a.weight_format) {
    if (fmt == XSHARE_WEIGHTS_BF16) {
      w1 = static_cast<const uint16_t*>(a.w1);
      w3 = static_cast<const uint16_t*>(a.w3);
      w2 = static_cast<const uint16_t*>(a.w2);
      return;
    }
    q1 = static_cast<const uint8_t*>(a.w1);
    q3 = static_cast<const uint8_t*>(a.w3);
    q2 = static_cast<const uint8_t*>(a.w2);
    if (fmt == XSHARE_WEIGHTS_FP8) {
      s1 = static_cast<const float*>(a.w1_scale);
      s3 = static_cast<const float*>(a.w3_scale);
      s2 = static_cast<const float*>(a.w2_scale);
    } else {
      e1 = static_cast<const uint8_t*>(a.w1_scale);
      e3 = static_cast<const uint8_t*>(a.w3_scale);
      e2 = static_cast<const uint8_t*>(a.w2_scale);
    }
  }
  bool present() const {
    if (fmt == XSHARE_WEIGHTS_FP8) return q1 && q3 && q2 && s1 && s3 && s2;
    if (fmt == XSHARE_WEIGHTS_MXFP4) return q1 && q3 && q2 && e1 && e3 && e2;
    return w1 && w3 && w2;
  }
  bool aligned() const {
    // MXFP4 scale rows are read in pieces of up to 16 bytes
    if (fmt == XSHARE_WEIGHTS_MXFP4 && !(aligned16(e1) && aligned16(e3) && aligned16(e2)))
      return false;
    return fmt != XSHARE_WEIGHTS_BF16 ? (aligned16(q1) && aligned16(q3) && aligned16(q2))
                                      : (aligned16(w1) && aligned16(w3) && aligned16(w2));
  }
};

// Checks of a layer call that do not depend on the workspace; XSHARE_OK if it may run.
xshare_status check_layer(const xshare_layer_args& a) {
  const bool hier = a.req_offsets != nullptr;
  if (hier && a.ep) return XSHARE_EUNSUPPORTED;
  xshare_status st = check_params(a.T, a.params, hier, a.ep != nullptr);
  if (st != XSHARE_OK) return st;
  if (hier) {
    st = check_offsets(a.T, a.req_offsets, a.host_offsets, a.R);
    if (st != XSHARE_OK) return st;
  }
  st = check_ep(a.params->n_experts, a.ep, true);
  if (st != XSHARE_OK) return st;
  st = check_shared(a.shared, a.ep);
  if (st != XSHARE_OK) return st;
  if (a.weight_format != XSHARE_WEIGHTS_BF16 && a.weight_format != XSHARE_WEIGHTS_FP8 &&
      a.weight_format != XSHARE_WEIGHTS_MXFP4)
    return XSHARE_EINVAL;
  if (a.weight_format != XSHARE_WEIGHTS_BF16 && a.shared && a.shared->n_shared > 0)
    return XSHARE_EUNSUPPORTED;
  if (a.d <= 0 || a.f <= 0) return XSHARE_EINVAL;
  if (a.d % xs::kDimAlign != 0 || a.f % xs::kDimAlign != 0) return XSHARE_EUNSUPPORTED;
  const Weights wt(a);
  if (a.T > 0) {
    if (!a.x || !wt.present() || !a.y) return XSHARE_EINVAL;
    if ((a.logits != nullptr) == (a.w_gate != nullptr)) return XSHARE_EINVAL;  // exactly one
  }
  if (!aligned16(a.x) || !wt.aligned() || !aligned16(a.y) || (a.w_gate && !aligned16(a.w_gate)))
    return XSHARE_EINVAL;
  return XSHARE_OK;
}

// Workspace of a layer call (valid arguments): the routing and expert regions, then the
// router's scratch when the logits are computed on the device.
size_t layer_workspace(const xshare_layer_args& a) {
  const xs::FfnLayout L = layer_layout(a.T, a.d, a.f, a.params, a.ep, n_shared_of(a.shared));
  return L.total + (a.w_gate ? layer_router_bytes(a.T, a.d, a.params->n_experts) : 0);
}

// The layer: optional router GEMM (w_gate given: logits computed on the device), selection,
// expert GEMMs (routed and shared), combine.
xshare_status layer_common(const xshare_layer_args& a) {
  if (a.struct_size != sizeof(xshare_layer_args)) return XSHARE_EINVAL;
  xshare_status st = check_layer(a);
  if (st != XSHARE_OK) return st;
  const xshare_route_params* params = a.params;
  const int32_t T = a.T, d = a.d, f = a.f;
  const hipStream_t stream = a.stream;
  const bool hier = a.req_offsets != nullptr;
  const Weights wt(a);
  const int N = params->n_experts, k = params->top_k;
  const int n_shared = n_shared_of(a.shared);
  const int bound = layer_bound(T, params, a.ep);
  const xs::FfnLayout L = layer_layout(T, d, f, params, a.ep, n_shared);
  void* const ws = a.ws;
  if (!ws || a.ws_bytes < layer_workspace(a)) return XSHARE_EWORKSPACE;

  // The selection kernel always writes a mask; keep it in the workspace if not wanted.
  uint8_t* mask = a.sel_mask ? a.sel_mask : at<uint8_t>(ws, L.route.mask);
  auto record = [&](int s) -> bool {
    if (!a.stage_events) return true;
    return hipEventRecord(static_cast<hipEvent_t>(a.stage_events[s]), stream) == hipSuccess;
  };
  if (!record(0)) return XSHARE_EHIP;
  xs::RouteArgs ra = route_args(a.logits, T, params, hier ? a.req_offsets : nullptr, a.R, a.ep,
                                nullptr, mask, a.topk_ids, a.topk_w, a.stats, ws, L.route);
  if (a.ep) ra.local_group = a.ep->local_group;
  if (a.w_gate && T > 0) {
    float* planes = at<float>(ws, L.total);
    float* h = a.logits_out ? a.logits_out
                            : at<float>(ws, L.total + router_planes_bytes(T, d, N));
    const xs::RouterArgs r{a.x, a.w_gate, T, d, N, xs::router_parts(T, d, N), planes, h};
    if (xs::launch_router(r, stream) != hipSuccess) return XSHARE_EHIP;
    ra.logits = h;
  }
  if (xs::launch_route(ra, stream) != hipSuccess || !record(1)) return XSHARE_EHIP;
  if (T == 0) {
    for (int s = 2; s < XSHARE_N_STAGE_EVENTS; ++s)
      if (!record(s)) return XSHARE_EHIP;
    return XSHARE_OK;
  }

  xs::FfnArgs fa{};
  fa.x = a.x;
  fa.w1 = wt.w1;
  fa.w3 = wt.w3;
  fa.w2 = wt.w2;
  fa.q1 = wt.q1;
  fa.q3 = wt.q3;
  fa.q2 = wt.q2;
  fa.s1 = wt.s1;
  fa.s3 = wt.s3;
  fa.s2 = wt.s2;
  fa.e1 = wt.e1;
  fa.e3 = wt.e3;
  fa.e2 = wt.e2;
  fa.wfmt = wt.fmt;
  fa.T = T;
  fa.N = N;
  fa.k = k;
  fa.d = d;
  fa.f = f;
  fa.max_active = bound;
  // the threshold rule's set size is not known before the selection runs
  fa.est_active = params->budget_mode == XSHARE_BUDGET_THRESHOLD
                      ? 0
                      : layer_estimate(T, params, a.ep);
  fa.splits = wt.fmt == XSHARE_WEIGHTS_MXFP4 ? L.q4_splits : L.splits;
  fa.gu_splits = L.gu_splits;
  fa.gu_tail_splits = L.gu_tail_splits;
  fa.slot_base = 0;
  fa.gpart = at<float>(ws, L.gpart);
  fa.G = ra.G;
  fa.group = ra.group;
  fa.local_group = ra.local_group;
  fa.n_shared = n_shared;
  fa.sw1 = n_shared ? a.shared->w1 : nullptr;
  fa.sw3 = n_shared ? a.shared->w3 : nullptr;
  fa.sw2 = n_shared ? a.shared->w2 : nullptr;
  fa.rows = (long)xs::ffn_rows(T, k, n_shared);
  fa.part_rows = fa.rows;
  fa.part_compact = 0;
  fa.offsets = ra.offsets;
  fa.perm = ra.perm;
  fa.active = ra.active;
  fa.counters = ra.counters;
  fa.ids = ra.ids;
  fa.w = ra.w;
  fa.h = at<uint16_t>(ws, L.h);
  fa.yslot = at<float>(ws, L.y);
  fa.y = a.y;
  if (xs::launch_gate_up(fa, stream) != hipSuccess || !record(2)) return XSHARE_EHIP;
  if (xs::launch_down(fa, stream) != hipSuccess || !record(3)) return XSHARE_EHIP;
  if (xs::launch_combine(fa, stream) != hipSuccess || !record(4)) return XSHARE_EHIP;
  return XSHARE_OK;
}

// A layer call of the fixed-signature entry points (no second stream).
xshare_layer_args layer_args(const uint16_t* x, const float* logits, const uint16_t* w_gate,
                             int32_t T, int32_t d, int32_t f, int32_t fmt, const void* w1,
                             const void* w3, const void* w2, const void* s1, const void* s3,
                             const void* s2, const xshare_shared_experts* shared,
                             const xshare_route_params* params, const int32_t* req_offsets,
                             const int32_t* host_offsets, int32_t R, const xshare_ep_layout* ep,
                             uint16_t* y, float* logits_out, uint8_t* sel_mask,
                             int32_t* topk_ids, float* topk_w, xshare_stats* stats, void* ws,
                             size_t ws_bytes, void* const* stage_events, hipStream_t stream) {
  xshare_layer_args a{};
  a.struct_size = sizeof(xshare_layer_args);
  a.T = T;
  a.d = d;
  a.f = f;
  a.x = x;
  a.logits = logits;
  a.w_gate = w_gate;
  a.weight_format = fmt;
  a.w1 = w1;
  a.w3 = w3;
  a.w2 = w2;
  a.w1_scale = s1;
  a.w3_scale = s3;
  a.w2_scale = s2;
  a.params = params;
  a.req_offsets = req_offsets;
  a.host_offsets = host_offsets;
  a.R = R;
  a.ep = ep;
  a.shared = shared;
  a.y = y;
  a.logits_out = logits_out;
  a.sel_mask = sel_mask;
  a.topk_ids = topk_ids;
  a.topk_w = topk_w;
  a.stats = stats;
  a.ws = ws;
  a.ws_bytes = ws_bytes;
  a.stage_events = stage_events;
  a.stream = stream;
  return a;
}

// Scratch of xshare_moe_forward_noalloc: one fixed array per GPU, for callers that cannot
// allocate.  Host code never names the array in a kernel argument or a copy (its host-side
// name is not a device address): each device's address comes from hipGetSymbolAddress, taken
// once per device with that device current, and only that address is passed on.
static __device__ __align__(256) unsigned char scratch[XSHARE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (nullptr, with the HIP error in *err, on failure).
void* scratch_for_current_device(hipError_t* err) {
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

size_t xshare_route_workspace_bytes(int32_t T, const xshare_route_params* params) {
  const bool ep = params && params->budget_mode == XSHARE_BUDGET_PER_GROUP;
  if (check_params(T, params, false, ep) != XSHARE_OK) return 0;
  return xs::route_layout(T, params->n_experts, params->top_k,
                          params->score_mode == XSHARE_SCORE_DENSE)
      .total;
}

size_t xshare_moe_workspace_bytes(int32_t T, int32_t d, int32_t f,
                                  const xshare_route_params* params, const xshare_ep_layout* ep,
                                  const xshare_shared_experts* shared) {
  if (check_params(T, params, false, ep != nullptr) != XSHARE_OK || d <= 0 || f <= 0) return 0;
  if (check_ep(params->n_experts, ep, true) != XSHARE_OK) return 0;
  return layer_layout(T, d, f, params, ep, n_shared_of(shared)).total;
}

size_t xshare_layer_workspace_bytes(int32_t T, int32_t d, int32_t f,
                                    const xshare_route_params* params,
                                    const xshare_ep_layout* ep,
                                    const xshare_shared_experts* shared) {
  const size_t m = xshare_moe_workspace_bytes(T, d, f, params, ep, shared);
  return m == 0 || d % xs::kDimAlign != 0 ? 0 : m + layer_router_bytes(T, d, params->n_experts);
}

xshare_status xshare_route(const float* logits, int32_t T, const xshare_route_params* params,
                           uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                           xshare_stats* stats, void* ws, size_t ws_bytes, hipStream_t stream) {
  return route_common(logits, T, nullptr, nullptr, 0, false, params, sel_mask, topk_ids, topk_w,
                      stats, ws, ws_bytes, stream);
}

xshare_status xshare_select_hier(const float* logits, int32_t T, const int32_t* req_offsets,
                                 const int32_t* host_offsets, int32_t R,
                                 const xshare_route_params* params, uint8_t* sel_mask,
                                 int32_t* topk_ids, float* topk_w, xshare_stats* stats,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  return route_common(logits, T, req_offsets, host_offsets, R, true, params, sel_mask, topk_ids,
                      topk_w, stats, ws, ws_bytes, stream);
}

xshare_status xshare_select_ep(const float* logits, int32_t T, const xshare_route_params* params,
                               const xshare_ep_layout* ep, uint8_t* sel_mask, int32_t* topk_ids,
                               float* topk_w, int32_t* group_load, xshare_stats* stats,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!ep) return XSHARE_EINVAL;
  xshare_status st = check_params(T, params, false, true);
  if (st != XSHARE_OK) return st;
  st = check_ep(params->n_experts, ep, false);
  if (st != XSHARE_OK) return st;
  if (!sel_mask || (T > 0 && (!logits || !topk_ids || !topk_w))) return XSHARE_EINVAL;
  const xs::RouteLayout L = xs::route_layout(T, params->n_experts, params->top_k,
                                             params->score_mode == XSHARE_SCORE_DENSE);
  if (!ws || ws_bytes < L.total) return XSHARE_EWORKSPACE;
  const xs::RouteArgs a = route_args(logits, T, params, nullptr, 0, ep, group_load, sel_mask,
                                     topk_ids, topk_w, stats, ws, L);
  return xs::launch_route(a, stream) == hipSuccess ? XSHARE_OK : XSHARE_EHIP;
}

xshare_status xshare_moe_forward_v2(const xshare_layer_args* args) {
  if (!args) return XSHARE_EINVAL;
  return layer_common(*args);
}

size_t xshare_moe_forward_v2_workspace_bytes(const xshare_layer_args* args) {
  if (!args || args->struct_size != sizeof(xshare_layer_args)) return 0;
  const xshare_layer_args& a = *args;
  if (check_params(a.T, a.params, a.req_offsets != nullptr, a.ep != nullptr) != XSHARE_OK ||
      check_ep(a.params->n_experts, a.ep, true) != XSHARE_OK || a.d <= 0 || a.f <= 0 ||
      a.d % xs::kDimAlign != 0 || a.f % xs::kDimAlign != 0)
    return 0;
  return layer_workspace(a);
}

xshare_status xshare_moe_forward(const uint16_t* x, const float* logits, int32_t T, int32_t d,
                                 int32_t f, const uint16_t* w1, const uint16_t* w3,
                                 const uint16_t* w2, const xshare_route_params* params,
                                 const int32_t* req_offsets, const int32_t* host_offsets,
                                 int32_t R, const xshare_ep_layout* ep,
                                 const xshare_shared_experts* shared, uint16_t* y,
                                 uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                 xshare_stats* stats, void* ws, size_t ws_bytes,
                                 void* const* stage_events, hipStream_t stream) {
  if (T > 0 && !logits) return XSHARE_EINVAL;
  return layer_common(layer_args(x, logits, nullptr, T, d, f, XSHARE_WEIGHTS_BF16, w1, w3, w2,
                                 nullptr, nullptr, nullptr, shared, params, req_offsets,
                                 host_offsets, R, ep, y, nullptr, sel_mask, topk_ids, topk_w,
                                 stats, ws, ws_bytes, stage_events, stream));
}

xshare_status xshare_moe_forward_noalloc(const uint16_t* x, const float* logits, int32_t T,
                                         int32_t d, int32_t f, const uint16_t* w1,
                                         const uint16_t* w3, const uint16_t* w2,
                                         const xshare_route_params* params,
                                         const int32_t* req_offsets,
                                         const int32_t* host_offsets, int32_t R,
                                         const xshare_ep_layout* ep,
                                         const xshare_shared_experts* shared, uint16_t* y,
                                         uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                         xshare_stats* stats, void* const* stage_events,
                                         hipStream_t stream) {
  if (T > 0 && !logits) return XSHARE_EINVAL;
  xshare_layer_args a = layer_args(x, logits, nullptr, T, d, f, XSHARE_WEIGHTS_BF16, w1, w3, w2,
                                   nullptr, nullptr, nullptr, shared, params, req_offsets,
                                   host_offsets, R, ep, y, nullptr, sel_mask, topk_ids, topk_w,
                                   stats, nullptr, 0, stage_events, stream);
  // host checks first (the same as xshare_moe_forward's), then the size limit
  xshare_status st = check_layer(a);
  if (st != XSHARE_OK) return st;
  if (layer_workspace(a) > size_t(XSHARE_NOALLOC_SCRATCH_BYTES)) return XSHARE_EWORKSPACE;
  if (stream) {             // the array used is the current device's
    int cur = 0, sdev = 0;
    if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(stream, &sdev) != hipSuccess)
      return XSHARE_EHIP;
    if (sdev != cur) return XSHARE_EINVAL;
  }
  hipError_t err = hipSuccess;
  a.ws = scratch_for_current_device(&err);
  if (!a.ws) return XSHARE_EHIP;
  a.ws_bytes = size_t(XSHARE_NOALLOC_SCRATCH_BYTES);
  return layer_common(a);
}

xshare_status xshare_moe_forward_fp8(const uint16_t* x, const float* logits, int32_t T,
                                     int32_t d, int32_t f, const uint8_t* w1, const uint8_t* w3,
                                     const uint8_t* w2, const float* w1_scale,
                                     const float* w3_scale, const float* w2_scale,
                                     const xshare_route_params* params,
                                     const int32_t* req_offsets, const int32_t* host_offsets,
                                     int32_t R, const xshare_ep_layout* ep, uint16_t* y,
                                     uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                     xshare_stats* stats, void* ws, size_t ws_bytes,
                                     void* const* stage_events, hipStream_t stream) {
  if (T > 0 && !logits) return XSHARE_EINVAL;
  return layer_common(layer_args(x, logits, nullptr, T, d, f, XSHARE_WEIGHTS_FP8, w1, w3, w2,
                                 w1_scale, w3_scale, w2_scale, nullptr, params, req_offsets,
                                 host_offsets, R, ep, y, nullptr, sel_mask, topk_ids, topk_w,
                                 stats, ws, ws_bytes, stage_events, stream));
}

xshare_status xshare_moe_forward_mxfp4(const uint16_t* x, const float* logits, int32_t T,
                                       int32_t d, int32_t f, const uint8_t* w1,
                                       const uint8_t* w3, const uint8_t* w2,
                                       const uint8_t* w1_scale, const uint8_t* w3_scale,
                                       const uint8_t* w2_scale,
                                       const xshare_route_params* params,
                                       const int32_t* req_offsets, const int32_t* host_offsets,
                                       int32_t R, const xshare_ep_layout* ep, uint16_t* y,
                                       uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                       xshare_stats* stats, void* ws, size_t ws_bytes,
                                       void* const* stage_events, hipStream_t stream) {
  if (T > 0 && !logits) return XSHARE_EINVAL;
  return layer_common(layer_args(x, logits, nullptr, T, d, f, XSHARE_WEIGHTS_MXFP4, w1, w3, w2,
                                 w1_scale, w3_scale, w2_scale, nullptr, params, req_offsets,
                                 host_offsets, R, ep, y, nullptr, sel_mask, topk_ids, topk_w,
                                 stats, ws, ws_bytes, stage_events, stream));
}

xshare_status xshare_moe_layer(const uint16_t* x, const uint16_t* w_gate, int32_t T, int32_t d,
                               int32_t f, const uint16_t* w1, const uint16_t* w3,
                               const uint16_t* w2, const xshare_shared_experts* shared,
                               const xshare_route_params* params, const int32_t* req_offsets,
                               const int32_t* host_offsets, int32_t R,
                               const xshare_ep_layout* ep, uint16_t* y, float* logits_out,
                               uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                               xshare_stats* stats, void* ws, size_t ws_bytes,
                               void* const* stage_events, hipStream_t stream) {
  if (T > 0 && !w_gate) return XSHARE_EINVAL;
  return layer_common(layer_args(x, nullptr, w_gate, T, d, f, XSHARE_WEIGHTS_BF16, w1, w3, w2,
                                 nullptr, nullptr, nullptr, shared, params, req_offsets,
                                 host_offsets, R, ep, y, logits_out, sel_mask, topk_ids, topk_w,
                                 stats, ws, ws_bytes, stage_events, stream));
}

size_t xshare_router_workspace_bytes(int32_t T, int32_t d, int32_t n_experts) {
  if (T < 0 || T > kMaxTokens || d <= 0 || d % xs::kDimAlign != 0 || n_experts < 1 ||
      n_experts > kMaxExperts)
    return 0;
  return router_planes_bytes(T, d, n_experts);
}

xshare_status xshare_router_logits(const uint16_t* x, const uint16_t* w_gate, int32_t T,
                                   int32_t d, int32_t n_experts, float* logits, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
  if (T < 0 || d <= 0 || n_experts < 1) return XSHARE_EINVAL;
  if (T > kMaxTokens || n_experts > kMaxExperts || d % xs::kDimAlign != 0)
    return XSHARE_EUNSUPPORTED;
  if (T == 0) return XSHARE_OK;
  if (!x || !w_gate || !logits || !aligned16(x) || !aligned16(w_gate)) return XSHARE_EINVAL;
  if (!ws || ws_bytes < router_planes_bytes(T, d, n_experts)) return XSHARE_EWORKSPACE;
  const xs::RouterArgs r{x, w_gate, T, d, n_experts, xs::router_parts(T, d, n_experts),
                         static_cast<float*>(ws), logits};
  return xs::launch_router(r, stream) == hipSuccess ? XSHARE_OK : XSHARE_EHIP;
}

size_t xshare_mx_scales_tiled_bytes(int32_t n_mat, int32_t rows, int32_t k) {
  if (n_mat < 0 || rows < 0 || k < 0) return 0;
  return xs::mx_scales_tiled_bytes(n_mat, rows, k);
}

xshare_status xshare_mx_scales_tile(const uint8_t* scales, uint8_t* tiled, int32_t n_mat,
                                    int32_t rows, int32_t k, hipStream_t stream) {
  if (n_mat < 0 || rows < 0 || k < 0 || rows % 16 != 0 || k % 32 != 0) return XSHARE_EINVAL;
  if (n_mat == 0 || rows == 0 || k == 0) return XSHARE_OK;
  if (!scales || !tiled) return XSHARE_EINVAL;
  return xs::launch_mx_scales_tile(scales, tiled, n_mat, rows, k, stream) == hipSuccess
             ? XSHARE_OK
             : XSHARE_EHIP;
}

xshare_status xshare_layer_budgets(int32_t K, int32_t L, int32_t* m) {
  if (L < 1 || K < 0 || !m) return XSHARE_EINVAL;
  const int32_t base = K / L, extra = K % L;
  for (int32_t l = 0; l < L; ++l) m[l] = base + (l < extra ? 1 : 0);
  return XSHARE_OK;
}

const char* xshare_status_string(int32_t status) {
  switch (status) {
    case XSHARE_OK: return "ok";
    case XSHARE_EINVAL: return "invalid argument";
    case XSHARE_EUNSUPPORTED: return "unsupported size";
    case XSHARE_EWORKSPACE: return "workspace too small";
    case XSHARE_EHIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

const char* xshare_version(void) { return "0.1.0"; }

}  // extern "C"
