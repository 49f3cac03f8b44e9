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
  size_t active;    // int4 [N]        active experts, ascending: {expert, first permuted row,
                    //                 rows, 0}, so a GEMM block finds its work in one load
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
  L.active = o;   o += align256(4 * sizeof(int32_t) * N);
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

// The expert GEMMs split their reduction into this many parts when the experts expected
// to be active would give too few waves to keep HBM busy (few experts, or one GPU group's
// share): gate/up splits d (16 output columns of W1 and W3 per wave), down splits f (32
// output rows of W2 per wave).  Each part stays a multiple of the kernels' K step.  The
// split count only changes speed; the grid always covers the bound on active experts.
#ifndef XS_GATE_UP_MAX_SPLITS
#define XS_GATE_UP_MAX_SPLITS 8
#endif
#ifndef XS_GU_SPLIT_BELOW
#define XS_GU_SPLIT_BELOW 1024
#endif
#ifndef XS_GU_SPLIT_TARGET
#define XS_GU_SPLIT_TARGET 2048
#endif
#ifndef XS_DN_SPLIT_BELOW
#define XS_DN_SPLIT_BELOW 1536
#endif
#ifndef XS_DN_SPLIT_TARGET
#define XS_DN_SPLIT_TARGET 2048
#endif
#ifndef XS_Q4_DN_SPLIT_TARGET
#define XS_Q4_DN_SPLIT_TARGET 4096
#endif
// Splits (a power of two <= max_splits) for a launch of `waves` waves: none at or above
// `below`, else the fewest that reach `target` waves, each part a multiple of `step`.
// Measured on MI355X: gate/up pays for its partials and the finish pass, so it splits only
// below 1024 waves (five DeepSeek experts, 640 waves: 4 splits); down splits below 1536
// waves, to reach 2048 with bf16 and FP8 weights (five DeepSeek experts, 1120 waves: 2
// splits; Mixtral's five, 640 waves: 4) and 4096 with MXFP4 (4 and 8 splits).  With the
// token rows staged in LDS, bf16 and FP8 down run best with fewer parts (a five-expert
// DeepSeek share 141 -> 134 us, FP8 Mixtral down 67 -> 64 us); MXFP4 down, with half the
// weight bytes per wave in flight, kept the larger target (Mixtral down 53 against 61 us).
inline int split_for(long waves, int K, int step, int below, int target, int max_splits = 8) {
  if (waves >= below) return 1;
  int s = 1;
  while (s < max_splits && waves * s < target && K % (2 * s * step) == 0) s *= 2;
  return s;
}
inline int gate_up_splits(int est_active, int d, int f) {
  return split_for((long)est_active * (f / 16), d, 128, XS_GU_SPLIT_BELOW, XS_GU_SPLIT_TARGET,
                   XS_GATE_UP_MAX_SPLITS);
}
// 16-row tiles of W2 per wave of the down GEMM (output rows per wave = 16 * NM), the base
// that the launch doubles for bf16 and FP8 when experts hold several tokens each (the shared
// token operand then serves more weight rows); MXFP4 keeps 2 (its 8-word steps need the
// registers).  The split counts below use the bf16 base for every format, so the workspace
// does not depend on the weight format.
#ifndef XS_DOWN_NM
#define XS_DOWN_NM 2
#endif
#ifndef XS_Q8_DOWN_NM
#define XS_Q8_DOWN_NM 2
#endif
#ifndef XS_Q4_DOWN_NM
#define XS_Q4_DOWN_NM 2
#endif
inline int down_splits(int est_active, int d, int f, bool mxfp4 = false) {
  return split_for((long)est_active * (d / (16 * XS_DOWN_NM)), f, 128, XS_DN_SPLIT_BELOW,
                   mxfp4 ? XS_Q4_DN_SPLIT_TARGET : XS_DN_SPLIT_TARGET);
}

// Hidden and output rows of the expert GEMMs: the T * k routed (token, slot) rows in
// permuted order, then T rows per always-on shared expert (token order).
inline size_t ffn_rows(int T, int k, int n_shared) {
  const size_t t = size_t(T > 0 ? T : 1);
  return t * size_t(k) + size_t(n_shared) * t;
}

// The gate/up launch's last, partly filled round of blocks: when it holds under a quarter
// of the blocks the GPU runs at once and at most XS_GU_TAIL_MAX_SLOTS expert slots, its
// slots are taken out of the launch and run after it split up to XS_GU_TAIL_SPLITS ways
// along d (a lone block streams its weights several times slower than its share of a full
// round).  Only under a total budget, where the active experts usually fill the budget and
// the launch's rounds are known on the host.  The tail's partial planes hold its rows only,
// (slot - first tail slot) * T + t, if within the cap.
#ifndef XS_GU_TAIL_SPLITS
#define XS_GU_TAIL_SPLITS 8
#endif
#ifndef XS_GU_TAIL_MAX_SLOTS
#define XS_GU_TAIL_MAX_SLOTS 4
#endif
#ifndef XS_GU_TAIL_CAP
#define XS_GU_TAIL_CAP (64L << 20)
#endif
inline size_t gu_tail_rows(int T) { return size_t(XS_GU_TAIL_MAX_SLOTS) * size_t(T > 0 ? T : 1); }

struct FfnLayout {
  RouteLayout route;
  int gu_tail_splits;  // K-splits available to the gate/up tail (0: none)
  int gu_splits;  // K-splits of the gate/up GEMM
  int splits;     // K-splits of the down GEMM (bf16 and FP8 weights)
  int q4_splits;  // K-splits of the down GEMM with MXFP4 weights
  size_t gpart;   // fp32 [gu_splits, 2, rows, f] gate and up partial sums (gu_splits > 1),
                  //      or the tail's [gu_tail_splits, 2, gu_tail_rows(T), f]
  size_t h;       // bf16 [rows, 2f]            SwiGLU hidden rows as hi = bf16(H) and
                  //                            lo = bf16(H - hi), interleaved in 8-element
                  //                            chunks: row p holds hi(c..c+7), lo(c..c+7), ...
  size_t y;       // fp32 [max(splits, q4_splits), rows, d]  per-row partial expert outputs
  size_t total;
};

// est_active: experts expected to be active (routed plus shared), for the split counts;
// tail_ok: the gate/up tail may run (a total budget).
inline FfnLayout ffn_layout(int T, int N, int k, bool dense, int d, int f, int est_active,
                            int n_shared, bool tail_ok) {
  FfnLayout L{};
  L.route = route_layout(T, N, k, dense);
  L.gu_splits = gate_up_splits(est_active, d, f);
  L.splits = down_splits(est_active, d, f);
  L.q4_splits = down_splits(est_active, d, f, true);
  const size_t rows = ffn_rows(T, k, n_shared);
  size_t o = L.route.total;
  const size_t tail_plane = sizeof(float) * 2 * gu_tail_rows(T) * size_t(f);
  L.gu_tail_splits = 0;
  if (tail_ok && L.gu_splits == 1 && size_t(XS_GU_TAIL_SPLITS) * tail_plane <= size_t(XS_GU_TAIL_CAP))
    L.gu_tail_splits = XS_GU_TAIL_SPLITS;
  L.gpart = o;
  if (L.gu_splits > 1)
    o += align256(sizeof(float) * 2 * size_t(L.gu_splits) * rows * size_t(f));
  else if (L.gu_tail_splits > 1)
    o += align256(size_t(L.gu_tail_splits) * tail_plane);
  L.h = o; o += align256(sizeof(uint16_t) * rows * 2 * size_t(f));
  const int y_planes = L.splits > L.q4_splits ? L.splits : L.q4_splits;   // any format
  L.y = o; o += align256(sizeof(float) * size_t(y_planes) * rows * size_t(d));
  L.total = o;
  return L;
}

// The router GEMM h = W_g x: waves of 16 router rows (experts) x one part of d, parts of 128
// elements where d allows (one load step per wave, so the whole weight read is in flight at
// once), at most 64 parts and 16 MB of fp32 partial planes [parts, T, N]; a second kernel
// sums the planes in part order.
inline int router_parts(int T, int d, int N) {
  const int q = d / 32;                                   // 32-element chunks of d
  int s = (q % 4 == 0) ? q / 4 : (q % 2 == 0 ? q / 2 : q);
  const long per_plane = 4L * (T > 0 ? T : 1) * N;
  long cap = (16L << 20) / per_plane;
  cap = cap < 1 ? 1 : (cap > 64 ? 64 : cap);
  while (s > cap || q % s != 0) --s;                      // largest divisor of q within the cap
  return s;
}
inline int router_token_groups(int T) {
  const int tiles = (T + 31) / 32;
  return tiles < 64 ? (tiles > 0 ? tiles : 1) : 64;
}

struct RouterArgs {
  const uint16_t* x;           // bf16 [T, d]
  const uint16_t* wg;          // bf16 [N, d]
  int T, d, N, parts;
  float* planes;               // fp32 [parts, T, N]
  float* logits;               // fp32 [T, N]
};

hipError_t launch_router(const RouterArgs& r, hipStream_t stream);   // GEMM, then the sum

struct RouteArgs {
  const float* logits;         // [T, N]
  int T, N, k, k0, budget, budget_mode, score_mode, m_r;
  float tau;                   // threshold mode (budget_mode 3)
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
  int32_t* ledger;             // nullable, xshare_budget_ledger layout (8 int32), accumulated
  int32_t* offsets;
  int32_t* perm;
  int4* active;
  int32_t* counters;
  float* dense;
};

hipError_t launch_route(const RouteArgs& a, hipStream_t stream);

struct FfnArgs {
  const uint16_t* x;
  const uint16_t* w1;          // bf16 weights (nullptr with FP8 weights)
  const uint16_t* w3;
  const uint16_t* w2;
  const uint8_t* q1;           // FP8 / MXFP4 weight codes (nullptr with bf16 weights)
  const uint8_t* q3;
  const uint8_t* q2;
  const float* s1;             // FP8 scales, one per output row: [N, f], [N, f], [N, d]
  const float* s3;
  const float* s2;
  const uint8_t* e1;           // MXFP4 E8M0 block scales, tiled (mx_scales_tile_kernel):
                               //   [N, f/16, G(d), 16, 8], [N, f/16, G(d), 16, 8],
                               //   [N, d/16, G(f), 16, 8] with G(K) = ceil(K / 256)
  const uint8_t* e3;           //   (q1, q3, q2 then hold packed E2M1 codes, two per byte)
  const uint8_t* e2;
  int wfmt;                    // 0 bf16, 1 FP8, 2 MXFP4
  int T, N, k, d, f;
  int max_active;              // host bound on the number of active experts (grid size)
  int est_active;              // experts expected to be active (0: unknown), for launch shapes
  int splits;                  // K-splits of the down GEMM (partials summed in the combine)
  int gu_splits;               // K-splits of the gate/up GEMM (partials summed by finish)
  float* gpart;                // [gu_splits, 2, part_rows, f] when gu_splits > 1 (or the tail's)
  long part_rows;              // rows of one partial plane: rows, or gu_tail_rows(T) in the tail
  int part_compact;            // the tail's partial rows: (slot - slot_base) * T + t
  int gu_tail_splits;          // partial planes available to the gate/up tail (0: none)
  int slot_base;               // first expert slot of this launch (the tail's launch: > 0)
  int G;                       // GPU groups, with `group` and `local_group` as in RouteArgs
  const int32_t* group;
  int local_group;
  int n_shared;                // always-on shared experts (slots after the routed ones)
  const uint16_t* sw1;         // [n_shared, f, d]
  const uint16_t* sw3;
  const uint16_t* sw2;         // [n_shared, d, f]
  long rows;                   // T * k + n_shared * T hidden / output rows
  const int32_t* offsets;
  const int32_t* perm;
  const int4* active;
  const int32_t* counters;
  const int32_t* ids;
  const float* w;
  uint16_t* h;                 // hidden rows, bf16 hi and lo interleaved per 8 elements
  float* yslot;
  uint16_t* y;
};

hipError_t launch_gate_up(const FfnArgs& a, hipStream_t stream);  // + finish if split
// MXFP4 scales [n_mat, rows, K/32] -> tiled [n_mat, rows/16, ceil(K/256), 16, 8]
hipError_t launch_mx_scales_tile(const uint8_t* src, uint8_t* dst, int n_mat, int rows, int K,
                                 hipStream_t stream);
inline size_t mx_scales_tiled_bytes(int n_mat, int rows, int K) {
  return size_t(n_mat) * size_t(rows) * size_t((K + 255) / 256) * 8;
}
hipError_t launch_down(const FfnArgs& a, hipStream_t stream);
hipError_t launch_combine(const FfnArgs& a, hipStream_t stream);

}  // namespace xs
