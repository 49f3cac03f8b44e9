// Internal declarations shared by the HIP translation units of libxshare.so:
// workspace layout and kernel launchers.  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace xs {

constexpr int kMaxExperts = 1024;   // one thread per expert in the selection workgroup
constexpr int kMaxTopK = 32;
constexpr int kMaxTokens = 4096;
constexpr int kMaxAssignments = 8192;  // T * k, staged in LDS by the selection kernel
constexpr int kDimAlign = 32;          // d and f granularity of the expert GEMMs

constexpr size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// Counters written by the selection kernel (device memory, inside the workspace).
enum Counter : int {
  kCntActive = 0,     // number of experts that received >= 1 token
  kCntSelected = 1,
  kCntStatus = 2,     // 0 = ok, 1 = invalid request offsets seen on the device
  kCntCount = 8
};

// Byte offsets of the routing workspace regions.
struct RouteLayout {
  size_t offsets;   // int32 [N + 1]   exclusive prefix of tokens per expert (permuted order)
  size_t perm;      // int32 [T * k]   slot (i * k + r) of each permuted row
  size_t active;    // int32 [N]       active experts, ascending
  size_t counters;  // int32 [kCntCount]
  size_t dense;     // fp32 [T * N]    dense gates (score_mode DENSE only)
  size_t ids;       // int32 [T * k]   refined ids when the caller passes none
  size_t w;         // fp32 [T * k]    refined gates when the caller passes none
  size_t mask;      // uint8 [N]       selected-set mask when the caller passes none
  size_t total;
};

inline RouteLayout route_layout(int T, int N, int k, bool dense) {
  RouteLayout L{};
  size_t tk = size_t(T > 0 ? T : 1) * size_t(k);
  size_t o = 0;
  L.offsets = o;  o += align256(sizeof(int32_t) * (N + 1));
  L.perm = o;     o += align256(sizeof(int32_t) * tk);
  L.active = o;   o += align256(sizeof(int32_t) * N);
  L.counters = o; o += align256(sizeof(int32_t) * kCntCount);
  L.dense = o;    o += dense ? align256(sizeof(float) * size_t(T) * N) : 0;
  L.ids = o;      o += align256(sizeof(int32_t) * tk);
  L.w = o;        o += align256(sizeof(float) * tk);
  L.mask = o;     o += align256(N);
  L.total = o;
  return L;
}

// Upper bound on the experts that receive tokens: never more than the (token, slot) pairs,
// and never more than a total budget.
inline int active_bound(int T, int N, int k, int budget_mode, int budget) {
  int b = N < T * k ? N : T * k;
  if (budget_mode == 0 && budget < b) b = budget;
  return b;
}

// The down GEMM splits its reduction (f) into this many parts when the active experts'
// 32-row output tiles alone would give too few waves to keep HBM busy (few, wide experts).
inline int down_splits(int max_active, int d, int f) {
  const long waves = (long)max_active * (d / 32);
  int s = 1;
  while (s < 8 && waves * s < 2048 && f % (2 * s * 256) == 0) s *= 2;
  return s;
}

struct FfnLayout {
  RouteLayout route;
  int splits;    // K-splits of the down GEMM
  size_t h;      // bf16 [T * k, f]            SwiGLU hidden rows in permuted order
  size_t y;      // fp32 [splits, T * k, d]    per-(token, slot) partial expert outputs
  size_t total;
};

inline FfnLayout ffn_layout(int T, int N, int k, bool dense, int d, int f, int max_active) {
  FfnLayout L{};
  L.route = route_layout(T, N, k, dense);
  L.splits = down_splits(max_active, d, f);
  size_t tk = size_t(T > 0 ? T : 1) * size_t(k);
  size_t o = L.route.total;
  L.h = o; o += align256(sizeof(uint16_t) * tk * size_t(f));
  L.y = o; o += align256(sizeof(float) * size_t(L.splits) * tk * size_t(d));
  L.total = o;
  return L;
}

struct RouteArgs {
  const float* logits;
  int T, N, k, k0, budget, budget_mode, score_mode, m_r;
  const int32_t* req_offsets;  // nullptr: flat Algorithm 2
  int R;
  int G;                       // GPU groups (Algorithms 5-6); 0: no groups
  const int32_t* group;        // [N] group of each expert; nullptr: contiguous blocks of N / G
  int local_group;             // >= 0: only this group's experts are listed as active
  int32_t* group_load;         // nullable [G] output
  uint8_t* sel_mask;
  int32_t* ids;
  float* w;
  int32_t* stats;              // nullable, xshare_stats layout (8 int32)
  int32_t* offsets;
  int32_t* perm;
  int32_t* active;
  int32_t* counters;
  float* dense;
};

hipError_t launch_route(const RouteArgs& a, hipStream_t stream);

struct FfnArgs {
  const uint16_t* x;
  const uint16_t* w1;
  const uint16_t* w3;
  const uint16_t* w2;
  int T, N, k, d, f;
  int max_active;              // host bound on the number of active experts (grid size)
  int splits;                  // K-splits of the down GEMM (partials summed in the combine)
  int G;                       // GPU groups, with `group` and `local_group` as in RouteArgs
  const int32_t* group;
  int local_group;
  const int32_t* offsets;
  const int32_t* perm;
  const int32_t* active;
  const int32_t* counters;
  const int32_t* ids;
  const float* w;
  uint16_t* h;
  float* yslot;
  uint16_t* y;
};

hipError_t launch_gate_up(const FfnArgs& a, hipStream_t stream);
hipError_t launch_down(const FfnArgs& a, hipStream_t stream);
hipError_t launch_combine(const FfnArgs& a, hipStream_t stream);

}  // namespace xs
