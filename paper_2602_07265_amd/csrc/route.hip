// Expert selection for one MoE layer and one decode batch (XShare, arXiv 2602.07265):
// router scoring, batch scores, greedy selection (flat Algorithm 2 or per-request +
// batch Algorithms 3-4), refinement, and the token permutation consumed by the expert
// GEMMs.  One workgroup of 1024 threads does all of it: the whole problem is a few
// thousand logits and is latency-, not throughput-bound, so the kernel avoids LDS round
// trips in its inner loops: wave reductions use DPP, rankings compare packed integer keys,
// and for decode-sized batches (T <= 64) a token bitmask per expert turns every
// per-expert gather into popcounts.
//
// Numerics: this translation unit is compiled with -ffp-contract=off; every fp32 step
// of the gates is a separate IEEE round-to-nearest operation in a fixed order, so the
// selected set and the per-token routing are reproducible bit for bit.
#pragma clang fp contract(off)

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace xs {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr uint32_t kNoEntry = 0xFFFFu;   // empty slot of the per-token lists
#ifndef XS_HEAVY_ROWS
#define XS_HEAVY_ROWS 8
#endif
constexpr int kHeavyRows = XS_HEAVY_ROWS;   // active-list class boundary (routed rows)

// exp(x) for x <= 0 in fp32: n = rint(x log2 e); r = (x - n ln2_hi) - n ln2_lo with a
// 15-bit ln2_hi (Cody-Waite: n ln2_hi is exact); p = degree-7 Taylor polynomial of e^r
// (coefficients 1/i!) in Horner form; result p * 2^n.  Below -80 the result is 0.
__device__ __forceinline__ float exp_fixed(float x) {
  constexpr float kLog2e = (float)1.4426950408889634;
  constexpr float kLn2Hi = 0.693145751953125f;
  constexpr float kLn2Lo = (float)(0.6931471805599453 - 0.693145751953125);
  constexpr float c2 = 0.5f;
  constexpr float c3 = (float)(1.0 / 6.0);
  constexpr float c4 = (float)(1.0 / 24.0);
  constexpr float c5 = (float)(1.0 / 120.0);
  constexpr float c6 = (float)(1.0 / 720.0);
  constexpr float c7 = (float)(1.0 / 5040.0);
  if (x < -80.0f) return 0.0f;
  const float n = rintf(x * kLog2e);
  const float r = (x - n * kLn2Hi) - n * kLn2Lo;
  float p = c7;
  p = p * r + c6;
  p = p * r + c5;
  p = p * r + c4;
  p = p * r + c3;
  p = p * r + c2;
  p = p * r + 1.0f;
  p = p * r + 1.0f;
  return ldexpf(p, (int)n);
}

// Order-preserving map of finite fp32 values to uint32 (> 0); 0 marks "no value".
__device__ __forceinline__ uint32_t ord(float h) {
  const uint32_t b = __float_as_uint(h);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float unord(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// One DPP step of a reduction: the value of the lane that Ctrl names, or the reduction's
// identity in rows outside RowMask.  With the identity as the "old" operand the compiler
// folds the move into the reducing instruction (one v_max_u32_dpp / v_min_u32_dpp per step
// instead of two moves and the max).
template <int Ctrl, int RowMask, uint32_t Identity>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)Identity, (int)v, Ctrl, RowMask, 0xF, false);
}

// Wave-wide max / min of a uint32 with DPP (quad swaps, row mirrors, row broadcasts);
// lane 63 ends with the result, which is returned to every lane.
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = max(v, dpp<0xB1, 0xF, 0u>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp<0x4E, 0xF, 0u>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp<0x141, 0xF, 0u>(v));  // row_half_mirror
  v = max(v, dpp<0x140, 0xF, 0u>(v));  // row_mirror
  v = max(v, dpp<0x142, 0xA, 0u>(v));  // row_bcast:15
  v = max(v, dpp<0x143, 0xC, 0u>(v));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
  constexpr uint32_t kId = 0xFFFFFFFFu;
  v = min(v, dpp<0xB1, 0xF, kId>(v));
  v = min(v, dpp<0x4E, 0xF, kId>(v));
  v = min(v, dpp<0x141, 0xF, kId>(v));
  v = min(v, dpp<0x140, 0xF, kId>(v));
  v = min(v, dpp<0x142, 0xA, kId>(v));
  v = min(v, dpp<0x143, 0xC, kId>(v));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

__device__ __forceinline__ float lane_value(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// One round of a wave-wide selection over keys held Q per lane (expert lane + 64 q):
// returns the expert with the largest key, lowest index on equal keys (key 0 = not
// available), removes it from its lane, and reports its key; -1 if nothing is left.
// A second (min-index) reduction over the holders of the largest key finds the expert.
template <int Q>
__device__ __forceinline__ int wave_pick(uint32_t (&key)[Q], int lane, uint32_t& kbest) {
  uint32_t bk = 0;
  uint32_t bj = 0xFFFFFFFFu;
#pragma unroll
  for (int q = 0; q < Q; ++q) {  // strict: the lower q (lower index) wins inside a lane
    const bool up = key[q] > bk;
    bk = up ? key[q] : bk;
    bj = up ? (uint32_t)(lane + 64 * q) : bj;
  }
  kbest = wave_max(bk);
  if (kbest == 0) return -1;
  // the lowest expert index among the holders of the largest key
  const uint32_t jmin = wave_min(bk == kbest ? bj : 0xFFFFFFFFu);
  // the holder lane drops the key: selects, not a branch around the holder lane
  const bool mine = (int)(jmin & 63) == lane;
  const int qsel = (int)(jmin >> 6);
#pragma unroll
  for (int q = 0; q < Q; ++q) key[q] = (mine && q == qsel) ? 0u : key[q];
  return (int)jmin;
}

// Ranks [r0, k) of the available keys; lane r receives rank r as (logit, expert), or
// (-inf, -1) if fewer are available.  Lanes below r0 keep what they hold.
template <int Q>
__device__ __forceinline__ void wave_topk(uint32_t (&key)[Q], int r0, int k, int lane,
                                          float& my_h, int& my_j) {
  if (lane >= r0) {
    my_h = -INFINITY;
    my_j = -1;
  }
  for (int r = r0; r < k; ++r) {
    uint32_t kb;
    const int jb = wave_pick<Q>(key, lane, kb);
    if (jb < 0) break;
    const bool at = lane == r;
    my_h = at ? unord(kb) : my_h;
    my_j = at ? jb : my_j;
  }
}

// Gates of the ranked list held by lanes 0..k-1: e_r = exp(h_r - h_0), Z summed in rank
// order, g_r = e_r / Z (correctly rounded division).
__device__ __forceinline__ float ranked_gate(float my_h, int lane, int k) {
  const float m = lane_value(my_h, 0);
  const float e = lane < k ? exp_fixed(my_h - m) : 0.0f;
  float z = 0.0f;
  for (int r = 0; r < k; ++r) z = z + lane_value(e, r);
  return lane < k ? e / z : 0.0f;
}

// ---- Two tokens per wave: each 32-lane half ranks its own token (lane l of half h holds
//      experts l, l + 32, ... of token 2p + h), so one chain of dependent reductions
//      serves two tokens.  Used where a token's experts fit 8 per lane (N <= 256).

// Max / min over each 32-lane half (lanes 0-31 and 32-63), returned to every lane: four
// DPP steps give every lane its 16-lane row's value, then the two rows of each half
// exchange (v_permlane16_swap pairs rows 0 and 1, and rows 2 and 3).
__device__ __forceinline__ uint32_t half_max(uint32_t v) {
  v = max(v, dpp<0xB1, 0xF, 0u>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp<0x4E, 0xF, 0u>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp<0x141, 0xF, 0u>(v));  // row_half_mirror
  v = max(v, dpp<0x140, 0xF, 0u>(v));  // row_mirror
  const auto s = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return max((uint32_t)s[0], (uint32_t)s[1]);
}
__device__ __forceinline__ uint32_t half_min(uint32_t v) {
  constexpr uint32_t kId = 0xFFFFFFFFu;
  v = min(v, dpp<0xB1, 0xF, kId>(v));
  v = min(v, dpp<0x4E, 0xF, kId>(v));
  v = min(v, dpp<0x141, 0xF, kId>(v));
  v = min(v, dpp<0x140, 0xF, kId>(v));
  const auto s = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return min((uint32_t)s[0], (uint32_t)s[1]);
}

// wave_pick for both halves at once: each half takes its largest key (lowest expert index
// on equal keys), drops it and returns its expert (-1 if the half has no key left or is
// not active this round); kbest receives the half's largest key.  sl: lane within the half.
template <int Q2>
__device__ __forceinline__ int half_pick(uint32_t (&key)[Q2], int sl, bool act,
                                         uint32_t& kbest) {
  uint32_t bk = 0;
  uint32_t bj = 0xFFFFFFFFu;
#pragma unroll
  for (int q = 0; q < Q2; ++q) {  // strict: the lower q (lower index) wins inside a lane
    const bool up = key[q] > bk;
    bk = up ? key[q] : bk;
    bj = up ? (uint32_t)(sl + 32 * q) : bj;
  }
  const uint32_t kb = half_max(bk);
  kbest = kb;
  const bool got = act && kb != 0;
  // the lowest expert index among the half's holders of the largest key
  const uint32_t jb = half_min(got && bk == kb ? bj : 0xFFFFFFFFu);
  const bool mine = got && (int)(jb & 31) == sl;
  const int qsel = (int)(jb >> 5);
#pragma unroll
  for (int q = 0; q < Q2; ++q) key[q] = (mine && q == qsel) ? 0u : key[q];
  return got ? (int)jb : -1;
}

// wave_topk for both halves: ranks [r0, k) of each half's keys (r0 uniform within a half);
// lane sl of a half receives rank sl as (logit, expert).  Lanes below r0 keep what they hold.
template <int Q2>
__device__ __forceinline__ void half_topk(uint32_t (&key)[Q2], int r0, int k, int sl, int h,
                                          float& my_h, int& my_j) {
  if (sl >= r0) {
    my_h = -INFINITY;
    my_j = -1;
  }
  const int rs = min(__builtin_amdgcn_readlane(r0, 0), __builtin_amdgcn_readlane(r0, 32));
  for (int r = rs; r < k; ++r) {
    uint32_t kb;
    const int jb = half_pick<Q2>(key, sl, r >= r0, kb);
    const bool at = jb >= 0 && sl == r;
    my_h = at ? unord(kb) : my_h;
    my_j = at ? jb : my_j;
  }
}

// ranked_gate for both halves: e_r = exp(h_r - h_0), Z summed in rank order, g_r = e_r / Z.
__device__ __forceinline__ float half_gate(float my_h, int sl, int h, int k) {
  const float m = h ? lane_value(my_h, 32) : lane_value(my_h, 0);
  const float e = sl < k ? exp_fixed(my_h - m) : 0.0f;
  float z0 = 0.0f, z1 = 0.0f;
  for (int r = 0; r < k; ++r) {
    z0 = z0 + lane_value(e, r);
    z1 = z1 + lane_value(e, 32 + r);
  }
  const float z = h ? z1 : z0;
  return sl < k ? e / z : 0.0f;
}

// ---- Four tokens per wave: each 16-lane row ranks its own token (lane l of row r holds
//      experts l, l + 16, ... of token 4p + r).  Used where a token's experts fit 8 per lane
//      (N <= 128) and its k ranks fit in a row (k <= 16).

// Max / min over each 16-lane row, returned to every lane of the row (the first four steps
// of half_max).
__device__ __forceinline__ uint32_t row_max(uint32_t v) {
  v = max(v, dpp<0xB1, 0xF, 0u>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp<0x4E, 0xF, 0u>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp<0x141, 0xF, 0u>(v));  // row_half_mirror
  v = max(v, dpp<0x140, 0xF, 0u>(v));  // row_mirror
  return v;
}
__device__ __forceinline__ uint32_t row_min(uint32_t v) {
  constexpr uint32_t kId = 0xFFFFFFFFu;
  v = min(v, dpp<0xB1, 0xF, kId>(v));
  v = min(v, dpp<0x4E, 0xF, kId>(v));
  v = min(v, dpp<0x141, 0xF, kId>(v));
  v = min(v, dpp<0x140, 0xF, kId>(v));
  return v;
}

// The value of `v` in lane 16 r + c for this lane's row r (c uniform).
__device__ __forceinline__ int row_lane(int v, int r, int c) {
  const int v0 = __builtin_amdgcn_readlane(v, c);
  const int v1 = __builtin_amdgcn_readlane(v, 16 + c);
  const int v2 = __builtin_amdgcn_readlane(v, 32 + c);
  const int v3 = __builtin_amdgcn_readlane(v, 48 + c);
  return r < 2 ? (r == 0 ? v0 : v1) : (r == 2 ? v2 : v3);
}

// wave_pick for the four rows at once: each row takes its largest key (lowest expert index
// on equal keys), drops it and returns its expert (-1 if the row has no key left or is not
// active this round); kbest receives the row's largest key.  ql: lane within the row.
template <int Q4>
__device__ __forceinline__ int row_pick(uint32_t (&key)[Q4], int ql, bool act, uint32_t& kbest) {
  uint32_t bk = 0;
  uint32_t bj = 0xFFFFFFFFu;
#pragma unroll
  for (int q = 0; q < Q4; ++q) {  // strict: the lower q (lower index) wins inside a lane
    const bool up = key[q] > bk;
    bk = up ? key[q] : bk;
    bj = up ? (uint32_t)(ql + 16 * q) : bj;
  }
  const uint32_t kb = row_max(bk);
  kbest = kb;
  const bool got = act && kb != 0;
  // the lowest expert index among the row's holders of the largest key: a second row
  // reduction, cheaper than a ballot and a lane read per row
  const uint32_t jb = row_min(got && bk == kb ? bj : 0xFFFFFFFFu);
  const bool mine = got && (int)(jb & 15) == ql;
  const int qsel = (int)(jb >> 4);
#pragma unroll
  for (int q = 0; q < Q4; ++q) key[q] = (mine && q == qsel) ? 0u : key[q];
  return got ? (int)jb : -1;
}

// wave_topk for the four rows: ranks [r0, k) of each row's keys (r0 uniform within a row);
// lane ql of a row receives rank ql as (logit, expert).  Lanes below r0 keep what they hold.
template <int Q4>
__device__ __forceinline__ void row_topk(uint32_t (&key)[Q4], int r0, int k, int ql, int qr,
                                         float& my_h, int& my_j) {
  if (ql >= r0) {
    my_h = -INFINITY;
    my_j = -1;
  }
  const int rs = min(min(__builtin_amdgcn_readlane(r0, 0), __builtin_amdgcn_readlane(r0, 16)),
                     min(__builtin_amdgcn_readlane(r0, 32), __builtin_amdgcn_readlane(r0, 48)));
  for (int r = rs; r < k; ++r) {
    uint32_t kb;
    const int jb = row_pick<Q4>(key, ql, r >= r0, kb);
    const bool at = jb >= 0 && ql == r;
    my_h = at ? unord(kb) : my_h;
    my_j = at ? jb : my_j;
  }
}

// ranked_gate for the four rows: e_r = exp(h_r - h_0), Z summed in rank order, g_r = e_r / Z.
__device__ __forceinline__ float row_gate(float my_h, int ql, int qr, int k) {
  const float m = __int_as_float(row_lane(__float_as_int(my_h), qr, 0));
  const float e = ql < k ? exp_fixed(my_h - m) : 0.0f;
  float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f, z3 = 0.0f;
  for (int r = 0; r < k; ++r) {
    z0 = z0 + lane_value(e, r);
    z1 = z1 + lane_value(e, 16 + r);
    z2 = z2 + lane_value(e, 32 + r);
    z3 = z3 + lane_value(e, 48 + r);
  }
  const float z = qr < 2 ? (qr == 0 ? z0 : z1) : (qr == 2 ? z2 : z3);
  return ql < k ? e / z : 0.0f;
}

// Raw logits of token quad p: lane ql of row qr holds experts ql, ql + 16, ... of token
// 4p + qr (0 beyond the batch or beyond N).
template <int Q4>
__device__ __forceinline__ void load_quad(const RouteArgs& a, int p, int ql, int qr,
                                          float (&raw)[Q4]) {
  const int i = 4 * p + qr;
  const size_t row = (size_t)i * a.N;
#pragma unroll
  for (int q = 0; q < Q4; ++q) {
    const int j = ql + 16 * q;
    raw[q] = (i < a.T && j < a.N) ? a.logits[row + j] : 0.0f;
  }
}

// Raw logits of token pair p: lane sl of half h holds experts sl, sl + 32, ... of token
// 2p + h (0 beyond the batch or beyond N).
template <int Q2>
__device__ __forceinline__ void load_pair(const RouteArgs& a, int p, int sl, int h,
                                          float (&raw)[Q2]) {
  const int i = 2 * p + h;
  const size_t row = (size_t)i * a.N;
#pragma unroll
  for (int q = 0; q < Q2; ++q) {
    const int j = sl + 32 * q;
    raw[q] = (i < a.T && j < a.N) ? a.logits[row + j] : 0.0f;
  }
}

// Raw logits of token i, lane l holding experts l, l + 64, ...
template <int Q>
__device__ __forceinline__ void load_row(const RouteArgs& a, int i, int lane, float (&raw)[Q]) {
  const size_t row = (size_t)i * a.N;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int j = lane + 64 * q;
    raw[q] = j < a.N ? a.logits[row + j] : 0.0f;
  }
}

// Canonicalised logits (h + 0.0 maps -0.0 to +0.0) and their keys.
template <int Q>
__device__ __forceinline__ void row_keys(const float (&raw)[Q], int N, int lane, float (&v)[Q],
                                         uint32_t (&key)[Q]) {
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int j = lane + 64 * q;
    v[q] = raw[q] + 0.0f;
    key[q] = j < N ? ord(v[q]) : 0u;
  }
}

template <int Q>
__device__ __forceinline__ void copy_keys(uint32_t (&dst)[Q], const uint32_t (&src)[Q]) {
#pragma unroll
  for (int q = 0; q < Q; ++q) dst[q] = src[q];
}

// Wave-wide inclusive prefix sum with DPP: shifts by 1, 2, 4 and 8 lanes inside each row
// of 16 (lanes without a source add 0), then each row's total added to the rows above it
// (row_bcast:15 into rows 1 and 3, row_bcast:31 into rows 2 and 3).
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Block-wide exclusive prefix sum of one int per thread; every thread must call it.
__device__ int block_excl_scan(int v, int* s_wsum, int& total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int inc = wave_incl_scan(v);
  if (lane == 63) s_wsum[wave] = inc;
  __syncthreads();
  int pre = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int t = s_wsum[w];
    if (w < wave) pre += t;
    total += t;
  }
  __syncthreads();
  return pre + inc - v;
}

// Per-token list entry: bits 0-9 expert, bits 10-14 rank; kNoEntry = empty.
__device__ __forceinline__ bool entry_is(uint32_t ent, int j) { return (ent & 0x83FFu) == (uint32_t)j; }
__device__ __forceinline__ uint32_t entry_at(const uint4& v, int u) {
  const uint32_t w = u < 2 ? v.x : u < 4 ? v.y : u < 6 ? v.z : v.w;
  return (w >> (16 * (u & 1))) & 0xFFFFu;
}

// Batches of up to this many tokens keep one token bitmask per expert, which turns the
// per-expert gathers (scores, per-request scores, permutation) into popcounts.
constexpr int kOccTokens = 64;

__device__ __forceinline__ uint64_t below(int i) { return i >= 64 ? ~0ull : ((1ull << i) - 1ull); }

// Groups the entries by expert (ascending), tokens ascending inside: s_off[e] is the start
// of expert e's run in s_list, which holds entry indices p = i * k + r.  Needs T <= 64 and
// s_occ zeroed; every thread must call.  Returns this thread's expert count (j = tid < N).
__device__ int group_by_expert(const uint16_t* s_ent, uint64_t* s_occ, int* s_off,
                               uint16_t* s_list, int* s_wsum, int TK, int k, int N, int& total) {
  const int tid = threadIdx.x;
  for (int p = tid; p < TK; p += kThreads) {
    const uint32_t ent = s_ent[p];
    if (ent != kNoEntry) atomicOr(reinterpret_cast<unsigned long long*>(&s_occ[ent & 1023u]),
                                  1ull << (p / k));
  }
  __syncthreads();
  const int cnt = tid < N ? __popcll(s_occ[tid]) : 0;
  const int off = block_excl_scan(cnt, s_wsum, total);
  if (tid < N) s_off[tid] = off;
  if (tid == N - 1) s_off[N] = off + cnt;
  __syncthreads();
  for (int p = tid; p < TK; p += kThreads) {
    const uint32_t ent = s_ent[p];
    if (ent == kNoEntry) continue;
    const int e = (int)(ent & 1023u);
    s_list[s_off[e] + __popcll(s_occ[e] & below(p / k))] = (uint16_t)p;
  }
  __syncthreads();
  return cnt;
}

template <int Q>
__global__ __launch_bounds__(kThreads) void route_kernel(RouteArgs a) {
  __shared__ __align__(16) uint16_t s_ent[kMaxAssignments];  // (token, rank) -> expert | rank
  __shared__ float s_g[kMaxAssignments];                     // vanilla gate of that entry
  __shared__ float s_vh[kMaxAssignments];                    // vanilla logit of that entry
  __shared__ uint16_t s_list[kMaxAssignments];               // entries grouped by expert
  __shared__ __align__(16) uint64_t s_occ[kMaxExperts];      // token bitmask per expert
  __shared__ __align__(16) uint64_t s_key[kMaxExperts];      // greedy keys of the candidates
  __shared__ int s_off[kMaxExperts + 1];
  __shared__ uint8_t s_tier1[kMaxExperts];                   // picked by some request
  __shared__ uint8_t s_sel[kMaxExperts];
  __shared__ uint32_t s_seed[kWaves][2 * kMaxTopK];          // refinement seeds per wave
  __shared__ float s_seed_h[kWaves][2 * kMaxTopK];            //   (and per half of a wave)
  __shared__ int s_wsum[kWaves];
  __shared__ int s_cnt[8];
  __shared__ int s_gload[kMaxExperts];   // GPU groups: warm-up experts per group, then |S| per group
  // GPU groups: candidates per group outside the warm-up set; threshold rule: scores by index
  __shared__ __align__(16) int s_gcand[kMaxExperts];
  // GPU groups: takeable candidates per rank inside their group; threshold rule: scores by rank
  __shared__ __align__(16) int s_hist[kMaxExperts];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int T = a.T, N = a.N, k = a.k, k0 = a.k0;
  const bool dense = a.score_mode == 1;
  const bool hier = a.req_offsets != nullptr;
  const bool ep = a.G > 0;
  const bool occ = T <= kOccTokens;
  const int TK = T * k;
  const int TK8 = (TK + 7) & ~7;

  // tokens per wave whose keys stay in registers (1024 threads allow 128 VGPRs each)
  constexpr int kCache = Q <= 4 ? 4 : (Q <= 8 ? 2 : 1);
  const bool cached = T <= kCache * kWaves;
  // Two tokens per wave (one per half) where a token's experts fit 8 per lane and the batch
  // gives a wave more than one token, except with dense scores (their softmax sums every
  // expert of the token in index order): token pairs p = wave, wave + 16, ..., pair p
  // holding tokens 2p and 2p + 1.  Measured (selection us, one token per wave -> halves):
  // DeepSeek T=32 25.8 -> 25.0, Qwen T=64 34.4 -> 30.7, speculative T=64 40.0 -> 37.5; with
  // at most one token per wave (T <= 16) the half-wave rounds only add: T=8 18.0 -> 19.5.
  // Four tokens per wave (one per 16-lane row) where a token's experts fit 8 per lane, its
  // ranks fit in a row and the batch gives a wave more than two tokens, with every quad's
  // remaining keys kept in registers (token quads p = wave, wave + 16, ...).
  constexpr bool kHalves = Q <= 4;
  constexpr int Q2 = 2 * Q;
  constexpr int kCacheP = Q2 <= 4 ? 4 : (Q2 <= 8 ? 2 : 1);   // pairs per wave in registers
  constexpr bool kQuads = Q <= 2;
  constexpr int Q4 = 4 * Q;
  constexpr int kCacheQ = Q4 <= 4 ? 4 : 2;                    // quads per wave in registers
  const int n_quads = (T + 3) >> 2;
  const bool quads = kQuads && !dense && k <= 16 && T > 2 * kWaves &&
                     n_quads <= kCacheQ * kWaves;
  const bool halves = kHalves && !dense && T > kWaves && !quads;
  const int hh = lane >> 5, sl = lane & 31;
  const int qr = lane >> 4, ql = lane & 15;
  const int n_pairs = (T + 1) >> 1;
  const bool cached_p = n_pairs <= kCacheP * kWaves;
  uint32_t kc[kCache][Q];
  uint32_t kcp[kHalves ? kCacheP : 1][kHalves ? Q2 : 1];
  uint32_t kcq[kQuads ? kCacheQ : 1][kQuads ? Q4 : 1];
  float raw_next[Q];
  float rawp_next[kHalves ? Q2 : 1];
  float rawq_next[kQuads ? Q4 : 1];
  // the wave's first logits row is on its way while the workgroup clears its tables
  if (quads) {
    if constexpr (kQuads)
      if (wave < n_quads) load_quad<Q4>(a, wave, ql, qr, rawq_next);
  } else if (halves) {
    if constexpr (kHalves)
      if (wave < n_pairs) load_pair<Q2>(a, wave, sl, hh, rawp_next);
  } else if (wave < T) {
    load_row<Q>(a, wave, lane, raw_next);
  }

  if (tid < 8) s_cnt[tid] = 0;
  for (int j = tid; j < kMaxExperts; j += kThreads) {
    s_tier1[j] = 0;
    s_occ[j] = 0;
    s_gload[j] = 0;
    s_gcand[j] = 0;
    s_hist[j] = 0;
  }
  for (int p = TK + tid; p < TK8; p += kThreads) s_ent[p] = (uint16_t)kNoEntry;
  __syncthreads();

  // ---- request offsets must be 0 = o_0 < o_1 < ... < o_R = T and every expert's group must
  //      lie in [0, G) (checked in parallel); otherwise the call selects nothing
  if (hier) {
    const int R = a.R;
    for (int r = tid; r < R; r += kThreads) {
      const int lo = a.req_offsets[r], hi = a.req_offsets[r + 1];
      if (!(lo < hi) || lo < 0 || hi > T) atomicOr(&s_cnt[7], 1);
    }
    if (tid == 0 && (a.req_offsets[0] != 0 || a.req_offsets[R] != T)) atomicOr(&s_cnt[7], 1);
  }
  if (ep && a.group)
    for (int jj = tid; jj < N; jj += kThreads)
      if (a.group[jj] < 0 || a.group[jj] >= a.G) atomicOr(&s_cnt[7], 1);
  if (hier || (ep && a.group)) {
    __syncthreads();
    if (s_cnt[7]) {
      for (int j = tid; j < N; j += kThreads) a.sel_mask[j] = 0;
      for (int p = tid; p < TK; p += kThreads) {
        a.ids[p] = -1;
        a.w[p] = 0.0f;
      }
      for (int j = tid; j <= N; j += kThreads) a.offsets[j] = 0;
      if (a.group_load)
        for (int g = tid; g < a.G; g += kThreads) a.group_load[g] = 0;
      if (tid == 0) {
        a.counters[kCntActive] = 0;
        a.counters[kCntSelected] = 0;
        a.counters[kCntStatus] = 1;
        if (a.stats) {
          a.stats[0] = -1;
          for (int s = 1; s < 8; ++s) a.stats[s] = 0;
        }
        if (a.ledger) {
          a.ledger[0] += 1;
          a.ledger[4] += 1;
        }
      }
      return;
    }
  }

  // ---- (a) per token: plain top-k and its gates (Section 2.2); dense softmax if requested.
  //      The next token's row is loaded while the current one is ranked; for batches of
  //      up to four tokens per wave the keys left after the top-k (all experts but the
  //      token's top-k) stay in registers for the refinement.
  // Token i: its plain top-k, gates and entries; `left` receives the keys that remain
  // after the top-k.  The wave's next row is loaded meanwhile.
  auto plain_topk = [&](int i, uint32_t (&left)[Q]) {
    float raw[Q], v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) raw[q] = raw_next[q];
    if (i + kWaves < T) load_row<Q>(a, i + kWaves, lane, raw_next);
    row_keys<Q>(raw, N, lane, v, left);
    float my_h;
    int my_j;
    wave_topk<Q>(left, 0, k, lane, my_h, my_j);
    const float g = ranked_gate(my_h, lane, k);
    if (lane < k) {
      s_ent[i * k + lane] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((lane << 10) | my_j));
      s_g[i * k + lane] = g;
      s_vh[i * k + lane] = my_h;
    }
    if (dense) {
      const float m = lane_value(my_h, 0);
      float e[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) e[q] = (lane + 64 * q < N) ? exp_fixed(v[q] - m) : 0.0f;
      float z = 0.0f;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int lim = min(64, N - 64 * q);
        for (int l = 0; l < lim; ++l) z = z + lane_value(e[q], l);
      }
#pragma unroll
      for (int q = 0; q < Q; ++q)
        if (lane + 64 * q < N) a.dense[(size_t)i * N + lane + 64 * q] = e[q] / z;
    }
  };
  // Token pair p (halves): the plain top-k of both tokens, as plain_topk.
  auto plain_topk_pair = [&](int p, uint32_t (&left)[kHalves ? Q2 : 1]) {
    if constexpr (kHalves) {
      float raw[Q2];
#pragma unroll
      for (int q = 0; q < Q2; ++q) raw[q] = rawp_next[q];
      if (p + kWaves < n_pairs) load_pair<Q2>(a, p + kWaves, sl, hh, rawp_next);
      const int i = 2 * p + hh;
      const bool valid = i < T;
#pragma unroll
      for (int q = 0; q < Q2; ++q)
        left[q] = (valid && sl + 32 * q < N) ? ord(raw[q] + 0.0f) : 0u;
      float my_h;
      int my_j;
      half_topk<Q2>(left, 0, k, sl, hh, my_h, my_j);
      const float g = half_gate(my_h, sl, hh, k);
      if (valid && sl < k) {
        s_ent[i * k + sl] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((sl << 10) | my_j));
        s_g[i * k + sl] = g;
        s_vh[i * k + sl] = my_h;
      }
    }
  };
  // Token quad p (rows): the plain top-k of four tokens, as plain_topk.
  auto plain_topk_quad = [&](int p, uint32_t (&left)[kQuads ? Q4 : 1]) {
    if constexpr (kQuads) {
      float raw[Q4];
#pragma unroll
      for (int q = 0; q < Q4; ++q) raw[q] = rawq_next[q];
      if (p + kWaves < n_quads) load_quad<Q4>(a, p + kWaves, ql, qr, rawq_next);
      const int i = 4 * p + qr;
      const bool valid = i < T;
#pragma unroll
      for (int q = 0; q < Q4; ++q)
        left[q] = (valid && ql + 16 * q < N) ? ord(raw[q] + 0.0f) : 0u;
      float my_h;
      int my_j;
      row_topk<Q4>(left, 0, k, ql, qr, my_h, my_j);
      const float g = row_gate(my_h, ql, qr, k);
      if (valid && ql < k) {
        s_ent[i * k + ql] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((ql << 10) | my_j));
        s_g[i * k + ql] = g;
        s_vh[i * k + ql] = my_h;
      }
    }
  };
  if (quads) {
    if constexpr (kQuads) {
#pragma unroll
      for (int it = 0; it < kCacheQ; ++it)
        if (wave + it * kWaves < n_quads) plain_topk_quad(wave + it * kWaves, kcq[it]);
    }
  } else if (halves) {
    if constexpr (kHalves) {
      if (cached_p) {
#pragma unroll
        for (int it = 0; it < kCacheP; ++it)
          if (wave + it * kWaves < n_pairs) plain_topk_pair(wave + it * kWaves, kcp[it]);
      } else {
        for (int p = wave; p < n_pairs; p += kWaves) {
          uint32_t left[Q2];
          plain_topk_pair(p, left);
        }
      }
    }
  } else if (cached) {
    // compile-time slots keep the cache in registers
#pragma unroll
    for (int it = 0; it < kCache; ++it)
      if (wave + it * kWaves < T) plain_topk(wave + it * kWaves, kc[it]);
  } else {
    for (int i = wave; i < T; i += kWaves) {
      uint32_t left[Q];
      plain_topk(i, left);
    }
  }
  __syncthreads();

  // ---- (b) per expert: batch score (ascending tokens), membership of U and S_0
  const int j = tid;
  float s = 0.0f;
  bool inU = false, inS0 = false;
  if (occ) {
    int total;
    const int cnt = group_by_expert(s_ent, s_occ, s_off, s_list, s_wsum, TK, k, N, total);
    if (j < N) {
      // eight entries' loads, then their adds in token order (the loads do not wait for the
      // sum, so a long list costs one LDS round trip per eight tokens)
      const int o = s_off[j];
      for (int q0 = 0; q0 < cnt; q0 += 8) {
        float gq[8];
        uint32_t eq[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int p = s_list[o + min(q0 + u, cnt - 1)];
          gq[u] = s_g[p];
          eq[u] = s_ent[p];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (q0 + u < cnt) {
            if (!dense) s = s + gq[u];
            if ((int)((eq[u] >> 10) & 31u) < k0) inS0 = true;
          }
        }
      }
      inU = cnt > 0;
    }
  } else if (j < N) {
    const uint4* ents = reinterpret_cast<const uint4*>(s_ent);
    for (int vb = 0; vb < TK8 / 8; ++vb) {
      const uint4 e4 = ents[vb];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t ent = entry_at(e4, u);
        if (entry_is(ent, j)) {
          inU = true;
          if ((int)((ent >> 10) & 31u) < k0) inS0 = true;
          if (!dense) s = s + s_g[vb * 8 + u];
        }
      }
    }
  }
  if (dense && j < N)
    for (int i = 0; i < T; ++i) s = s + a.dense[(size_t)i * N + j];

  // ---- (c) per request (Algorithm 3), one wave per request: S_0(r) plus the m_r best
  //      remaining experts of r under the request's own score
  if (hier && a.m_r > 0) {
    for (int r = wave; r < a.R; r += kWaves) {
      const int lo = a.req_offsets[r], hi = a.req_offsets[r + 1];
      float sr[Q];
      unsigned inUr = 0, inS0r = 0;
#pragma unroll
      for (int q = 0; q < Q; ++q) sr[q] = 0.0f;
      if (occ) {
        const uint64_t range = below(hi) & ~below(lo);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int jq = lane + 64 * q;
          if (jq >= N) continue;
          const uint64_t m = s_occ[jq];
          const int n = __popcll(m & range);
          const int o = s_off[jq] + __popcll(m & below(lo));
          for (int t0 = 0; t0 < n; t0 += 8) {   // loads ahead of the ordered adds, as in (b)
            float gq[8];
            uint32_t eq[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int p = s_list[o + min(t0 + u, n - 1)];
              gq[u] = s_g[p];
              eq[u] = s_ent[p];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              if (t0 + u < n) {
                if ((int)((eq[u] >> 10) & 31u) < k0) inS0r |= 1u << q;
                if (!dense) sr[q] = sr[q] + gq[u];
              }
            }
          }
          if (n > 0) inUr |= 1u << q;
        }
      } else {
        for (int p = lo * k; p < hi * k; ++p) {
          const uint32_t ent = s_ent[p];
          if (ent == kNoEntry || (int)(ent & 63u) != lane) continue;
          const int qe = (int)((ent & 1023u) >> 6);
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            if (q == qe) {
              inUr |= 1u << q;
              if ((int)((ent >> 10) & 31u) < k0) inS0r |= 1u << q;
              if (!dense) sr[q] = sr[q] + s_g[p];
            }
          }
        }
      }
      if (dense)
        for (int i = lo; i < hi; ++i)
#pragma unroll
          for (int q = 0; q < Q; ++q)
            if (lane + 64 * q < N) sr[q] = sr[q] + a.dense[(size_t)i * N + lane + 64 * q];
      uint32_t key[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const bool cand = (lane + 64 * q < N) && (dense || ((inUr >> q) & 1u)) &&
                          !((inS0r >> q) & 1u);
        key[q] = cand ? ord(sr[q]) : 0u;
      }
      for (int t = 0; t < a.m_r; ++t) {
        uint32_t kb;
        const int jb = wave_pick<Q>(key, lane, kb);
        if (jb < 0) break;
        if (lane == 0) s_tier1[jb] = 1;
      }
    }
  }
  __syncthreads();

  // ---- (d) batch greedy (Algorithm 1 with a fixed budget; Algorithm 4's final stage):
  //      order (tier, score desc, index asc), keep the first budget_eff candidates.
  //      Key: (3 - tier) << 42 | ord(score) << 10 | (1023 - j); candidates are compacted
  //      and each counts the candidates ahead of it.
  bool sel = false;
  int n_s0 = 0, n_start = 0, n_u = 0, m_eff = 0, max_load = 0;
  if (!ep) {
    int tier = 3;
    uint64_t mykey = 0;
    if (j < N) {
      const bool cand = dense ? (T > 0) : inU;
      tier = inS0 ? 0 : (s_tier1[j] ? 1 : (cand ? 2 : 3));
      if (tier < 3)
        mykey = ((uint64_t)(3 - tier) << 42) | ((uint64_t)ord(s) << 10) | (uint64_t)(1023 - j);
      if (tier == 0) atomicAdd(&s_cnt[1], 1);
      if (tier <= 1) atomicAdd(&s_cnt[2], 1);
      if (inU) atomicAdd(&s_cnt[3], 1);
    }
    int n_cand = 0;
    const int cpos = block_excl_scan(mykey != 0 ? 1 : 0, s_wsum, n_cand);
    if (mykey != 0) s_key[cpos] = mykey;
    if (tid == 0 && (n_cand & 1)) s_key[n_cand] = 0;
    __syncthreads();
    n_s0 = s_cnt[1];
    n_start = s_cnt[2];
    n_u = s_cnt[3];
    int rank = 0;
    if (mykey != 0) {
      const ulonglong2* keys2 = reinterpret_cast<const ulonglong2*>(s_key);
      const int n2 = (n_cand + 1) >> 1;
      for (int jj = 0; jj < n2; ++jj) {
        const ulonglong2 kk = keys2[jj];
        rank += (kk.x > mykey) + (kk.y > mykey);
      }
    }
    if (a.budget_mode == 3) {
      // Algorithm 1's threshold rule: the starting set (ranks below n_start) and then the
      // candidates in rank order join while f(S) < tau * f(E).  One thread replays the fp32
      // sums in the stated order: f(E) over every expert in index order, f(S) in rank order.
      float* const by_index = reinterpret_cast<float*>(s_gcand);
      float* const by_rank = reinterpret_cast<float*>(s_hist);
      if (j < N) by_index[j] = s;
      if (j >= N && j < ((N + 3) & ~3)) by_index[j] = 0.0f;   // pad to whole float4s
      if (mykey != 0) by_rank[rank] = s;
      __syncthreads();
      if (tid == 0) {
        // sequential fp32 sums; 16-byte LDS reads keep the loads ahead of the adds
        const float4* e4 = reinterpret_cast<const float4*>(by_index);
        float f_E = 0.0f;
#pragma unroll 4
        for (int q = 0; q < (N + 3) / 4; ++q) {
          const float4 v = e4[q];
          f_E = f_E + v.x;
          f_E = f_E + v.y;
          f_E = f_E + v.z;
          f_E = f_E + v.w;
        }
        const float target = a.tau * f_E;
        float f_S = 0.0f;
        for (int r = 0; r < n_start; ++r) f_S = f_S + by_rank[r];
        int m = n_start;
        while (m < n_cand && f_S < target) f_S = f_S + by_rank[m++];
        s_cnt[6] = m;
      }
      __syncthreads();
      m_eff = max(s_cnt[6], min(k, n_cand));
    } else {
      const int base = a.budget_mode == 0 ? a.budget : n_start + a.budget;
      m_eff = max(min(base, n_cand), min(k, n_cand));
    }
    sel = mykey != 0 && rank < m_eff;
  } else {
    // GPU groups (Algorithms 5 and 6).  Group g can take a_g = m_g - |S_0 on g| experts
    // (m_g caps every group's load, Eq. (5)), one per round, best first; its candidate of
    // rank r (score desc, index asc, among its candidates outside S_0) is taken in round
    // r + 1 if r < a_g.  The loop stops after the fewest rounds R that bring |S| to m_g * G,
    // or when no group can take more; so S = S_0 plus every takeable candidate of rank < R,
    // and R follows from a prefix count of the takeable candidates by rank.
    const int G = a.G, m_g = a.budget;
    const int gj = j < N ? (a.group ? a.group[j] : j / (N / G)) : 0;
    const bool cand = j < N && (dense ? (T > 0) : inU);
    const bool pick = cand && !inS0;
    if (j < N) {
      if (inS0) {
        atomicAdd(&s_gload[gj], 1);
        atomicAdd(&s_cnt[1], 1);
      }
      if (pick) atomicAdd(&s_gcand[gj], 1);
      if (inU) atomicAdd(&s_cnt[3], 1);
      if (cand) atomicAdd(&s_cnt[5], 1);
    }
    // key: group << 44 | ord(score) << 10 | (1023 - j); the rank counts the group's keys above
    const uint64_t pkey =
        pick ? ((uint64_t)gj << 44) | ((uint64_t)ord(s) << 10) | (uint64_t)(1023 - j) : 0;
    int n_pick = 0;
    const int ppos = block_excl_scan(pick ? 1 : 0, s_wsum, n_pick);
    if (pick) s_key[ppos] = pkey;
    if (tid == 0 && (n_pick & 1)) s_key[n_pick] = 0;
    __syncthreads();
    int rank = 0;
    bool takeable = false;
    if (pick) {
      const ulonglong2* keys2 = reinterpret_cast<const ulonglong2*>(s_key);
      const uint64_t mine = (uint64_t)gj;
      const int n2 = (n_pick + 1) >> 1;
      for (int jj = 0; jj < n2; ++jj) {
        const ulonglong2 kk = keys2[jj];
        rank += ((kk.x >> 44) == mine && kk.x > pkey) + ((kk.y >> 44) == mine && kk.y > pkey);
      }
      takeable = rank < m_g - s_gload[gj];
      if (takeable) atomicAdd(&s_hist[rank], 1);
    }
    __syncthreads();
    n_s0 = s_cnt[1];
    n_u = s_cnt[3];
    const int n_cand = s_cnt[5];
    const int need = m_g * G - n_s0;          // picks the rounds must reach
    static_assert(kThreads == kMaxExperts, "one rank of s_hist per thread");
    const int at_rank = s_hist[tid];
    int n_take = 0;
    const int before = block_excl_scan(at_rank, s_wsum, n_take);
    if (need > 0 && before < need && before + at_rank >= need) s_cnt[6] = tid + 1;
    __syncthreads();
    const int rounds = need <= 0 ? 0 : (n_take < need ? kMaxExperts : s_cnt[6]);
    sel = inS0 || (takeable && rank < rounds);
    if (sel) atomicAdd(&s_cnt[2], 1);
    __syncthreads();
    // fewer than k experts: the best remaining candidates join regardless of group
    const int n_loop = s_cnt[2], want = min(k, n_cand);
    if (n_loop < want) {
      const bool rest = cand && !sel;
      const uint64_t fkey = rest ? ((uint64_t)ord(s) << 10) | (uint64_t)(1023 - j) : 0;
      int n_rest = 0;
      const int fpos = block_excl_scan(rest ? 1 : 0, s_wsum, n_rest);
      if (rest) s_key[fpos] = fkey;
      if (tid == 0 && (n_rest & 1)) s_key[n_rest] = 0;
      __syncthreads();
      if (rest) {
        const ulonglong2* keys2 = reinterpret_cast<const ulonglong2*>(s_key);
        int r2 = 0;
        const int n2 = (n_rest + 1) >> 1;
        for (int jj = 0; jj < n2; ++jj) {
          const ulonglong2 kk = keys2[jj];
          r2 += (kk.x > fkey) + (kk.y > fkey);
        }
        sel = r2 < want - n_loop;
      }
    }
    // Load_g(S) and MaxLoad(S) (Section 5.1)
    if (tid < G) s_gload[tid] = 0;
    __syncthreads();
    if (sel) atomicAdd(&s_gload[gj], 1);
    __syncthreads();
    if (tid < G) {
      if (a.group_load) a.group_load[tid] = s_gload[tid];
      atomicMax(&s_cnt[0], s_gload[tid]);
    }
    n_start = n_s0;
    m_eff = min(m_g * G, N);
  }
  if (j < N) {
    s_sel[j] = sel;
    a.sel_mask[j] = sel;
    if (sel) atomicAdd(&s_cnt[4], 1);
  }
  __syncthreads();
  if (ep) max_load = s_cnt[0];

  // ---- (e) refinement: every token to its top-k inside S, gates renormalised (Section 3.4).
  //      The token's plain top-k experts that are in S are its first refined ranks (in
  //      their order); only the remaining ranks are searched, among the other experts.
  // Token i: `key` holds its keys without its plain top-k.
  auto refine = [&](int i, uint32_t (&key)[Q]) {
    const uint32_t vent = lane < k ? (uint32_t)s_ent[i * k + lane] : kNoEntry;
    const int vid = vent == kNoEntry ? -1 : (int)(vent & 1023u);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int jq = lane + 64 * q;
      if (jq >= N || !s_sel[jq]) key[q] = 0;
    }
    const bool keep = vid >= 0 && s_sel[vid];
    const uint64_t kept = __ballot(keep);
    const int m = __popcll(kept);
    if (keep) {
      const int dst = __popcll(kept & below(lane));
      s_seed[wave][dst] = (uint32_t)vid;
      s_seed_h[wave][dst] = s_vh[i * k + lane];
    }
    float my_h = -INFINITY;
    int my_j = -1;
    if (lane < m) {
      my_j = (int)s_seed[wave][lane];
      my_h = s_seed_h[wave][lane];
    }
    wave_topk<Q>(key, m, k, lane, my_h, my_j);
    const float g = ranked_gate(my_h, lane, k);
    if (lane < k) {
      a.ids[i * k + lane] = my_j;
      a.w[i * k + lane] = g;
      s_ent[i * k + lane] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((lane << 10) | my_j));
    }
  };
  // Token pair p (halves): as refine, each half with its own token and seeds.
  auto refine_pair = [&](int p, uint32_t (&key)[kHalves ? Q2 : 1]) {
    if constexpr (kHalves) {
      const int i = 2 * p + hh;
      const bool valid = i < T;
      const uint32_t vent = (valid && sl < k) ? (uint32_t)s_ent[i * k + sl] : kNoEntry;
      const int vid = vent == kNoEntry ? -1 : (int)(vent & 1023u);
#pragma unroll
      for (int q = 0; q < Q2; ++q) {
        const int jq = sl + 32 * q;
        if (jq >= N || !s_sel[jq]) key[q] = 0;
      }
      const bool keep = vid >= 0 && s_sel[vid];
      const uint64_t kept = __ballot(keep);
      const uint32_t kh = hh ? (uint32_t)(kept >> 32) : (uint32_t)kept;
      const int m = __popc(kh);
      if (keep) {
        const int dst = __popc(kh & ((1u << sl) - 1u));
        s_seed[wave][hh * kMaxTopK + dst] = (uint32_t)vid;
        s_seed_h[wave][hh * kMaxTopK + dst] = s_vh[i * k + sl];
      }
      float my_h = -INFINITY;
      int my_j = -1;
      if (sl < m) {
        my_j = (int)s_seed[wave][hh * kMaxTopK + sl];
        my_h = s_seed_h[wave][hh * kMaxTopK + sl];
      }
      half_topk<Q2>(key, m, k, sl, hh, my_h, my_j);
      const float g = half_gate(my_h, sl, hh, k);
      if (valid && sl < k) {
        a.ids[i * k + sl] = my_j;
        a.w[i * k + sl] = g;
        s_ent[i * k + sl] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((sl << 10) | my_j));
      }
    }
  };
  // Token quad p (rows): as refine, each row with its own token and seeds.
  auto refine_quad = [&](int p, uint32_t (&key)[kQuads ? Q4 : 1]) {
    if constexpr (kQuads) {
      const int i = 4 * p + qr;
      const bool valid = i < T;
      const uint32_t vent = (valid && ql < k) ? (uint32_t)s_ent[i * k + ql] : kNoEntry;
      const int vid = vent == kNoEntry ? -1 : (int)(vent & 1023u);
#pragma unroll
      for (int q = 0; q < Q4; ++q) {
        const int jq = ql + 16 * q;
        if (jq >= N || !s_sel[jq]) key[q] = 0;
      }
      const bool keep = vid >= 0 && s_sel[vid];
      const uint64_t kept = __ballot(keep);
      const uint32_t kq = (uint32_t)(kept >> (16 * qr)) & 0xFFFFu;
      const int m = __popc(kq);
      if (keep) {
        const int dst = __popc(kq & ((1u << ql) - 1u));
        s_seed[wave][qr * 16 + dst] = (uint32_t)vid;
        s_seed_h[wave][qr * 16 + dst] = s_vh[i * k + ql];
      }
      float my_h = -INFINITY;
      int my_j = -1;
      if (ql < m) {
        my_j = (int)s_seed[wave][qr * 16 + ql];
        my_h = s_seed_h[wave][qr * 16 + ql];
      }
      row_topk<Q4>(key, m, k, ql, qr, my_h, my_j);
      const float g = row_gate(my_h, ql, qr, k);
      if (valid && ql < k) {
        a.ids[i * k + ql] = my_j;
        a.w[i * k + ql] = g;
        s_ent[i * k + ql] = (uint16_t)(my_j < 0 ? kNoEntry : (uint32_t)((ql << 10) | my_j));
      }
    }
  };
  if (quads) {
    if constexpr (kQuads) {
#pragma unroll
      for (int it = 0; it < kCacheQ; ++it)
        if (wave + it * kWaves < n_quads) refine_quad(wave + it * kWaves, kcq[it]);
    }
  } else if (halves) {
    if constexpr (kHalves) {
      if (cached_p) {
#pragma unroll
        for (int it = 0; it < kCacheP; ++it)
          if (wave + it * kWaves < n_pairs) refine_pair(wave + it * kWaves, kcp[it]);
      } else {
        if (wave < n_pairs) load_pair<Q2>(a, wave, sl, hh, rawp_next);
        for (int p = wave; p < n_pairs; p += kWaves) {
          float raw[Q2];
          uint32_t key[Q2];
#pragma unroll
          for (int q = 0; q < Q2; ++q) raw[q] = rawp_next[q];
          if (p + kWaves < n_pairs) load_pair<Q2>(a, p + kWaves, sl, hh, rawp_next);
          const int i = 2 * p + hh;
          const bool valid = i < T;
#pragma unroll
          for (int q = 0; q < Q2; ++q)
            key[q] = (valid && sl + 32 * q < N) ? ord(raw[q] + 0.0f) : 0u;
          const uint32_t vent = (valid && sl < k) ? (uint32_t)s_ent[i * k + sl] : kNoEntry;
          const int vid = vent == kNoEntry ? -1 : (int)(vent & 1023u);
          for (int r = 0; r < k; ++r) {   // the plain top-k is not searched again
            const int v0 = __builtin_amdgcn_readlane(vid, r);
            const int v1 = __builtin_amdgcn_readlane(vid, 32 + r);
            const int vr = hh ? v1 : v0;
            const bool drop = vr >= 0 && (vr & 31) == sl;
#pragma unroll
            for (int q = 0; q < Q2; ++q) key[q] = (drop && q == (vr >> 5)) ? 0u : key[q];
          }
          refine_pair(p, key);
        }
      }
    }
  } else if (cached) {
#pragma unroll
    for (int it = 0; it < kCache; ++it)
      if (wave + it * kWaves < T) refine(wave + it * kWaves, kc[it]);
  } else {
    if (wave < T) load_row<Q>(a, wave, lane, raw_next);
    for (int i = wave; i < T; i += kWaves) {
      float raw[Q], v[Q];
      uint32_t key[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) raw[q] = raw_next[q];
      if (i + kWaves < T) load_row<Q>(a, i + kWaves, lane, raw_next);
      row_keys<Q>(raw, N, lane, v, key);
      const uint32_t vent = lane < k ? (uint32_t)s_ent[i * k + lane] : kNoEntry;
      const int vid = vent == kNoEntry ? -1 : (int)(vent & 1023u);
      for (int r = 0; r < k; ++r) {     // the plain top-k is not searched again
        const int vr = __builtin_amdgcn_readlane(vid, r);
        if (vr >= 0 && (vr & 63) == lane) {
#pragma unroll
          for (int q = 0; q < Q; ++q)
            if (q == (vr >> 6)) key[q] = 0;
        }
      }
      refine(i, key);
    }
  }
  __syncthreads();

  // ---- (f) permutation: rows grouped by expert (ascending), tokens ascending inside
  int cnt = 0, total = 0, off = 0;
  if (occ) {
    for (int jj = tid; jj < kMaxExperts; jj += kThreads) s_occ[jj] = 0;
    __syncthreads();
    cnt = group_by_expert(s_ent, s_occ, s_off, s_list, s_wsum, TK, k, N, total);
    if (j < N) {
      off = s_off[j];
      for (int q = 0; q < cnt; ++q) a.perm[off + q] = s_list[off + q];
    }
  } else {
    if (j < N) {
      const uint4* ents = reinterpret_cast<const uint4*>(s_ent);
      for (int vb = 0; vb < TK8 / 8; ++vb) {
        const uint4 e4 = ents[vb];
#pragma unroll
        for (int u = 0; u < 8; ++u) cnt += entry_is(entry_at(e4, u), j);
      }
    }
    off = block_excl_scan(cnt, s_wsum, total);
    if (j < N && cnt > 0) {
      const uint4* ents = reinterpret_cast<const uint4*>(s_ent);
      int pos = off;
      for (int vb = 0; vb < TK8 / 8; ++vb) {
        const uint4 e4 = ents[vb];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (entry_is(entry_at(e4, u), j)) a.perm[pos++] = vb * 8 + u;
      }
    }
  }
  // with a local GPU group only that group's experts are listed for the expert GEMMs
  const bool listed = j < N && cnt > 0 &&
                      (a.local_group < 0 ||
                       (a.group ? a.group[j] : j / (N / a.G)) == a.local_group);
  // The active list puts experts with more than kHeavyRows routed rows first (in expert
  // order), then the others: their GEMM blocks run longest, so they start first instead of
  // trailing the launch.  One scan counts both classes (16 bits each).
  const bool heavy = listed && cnt > kHeavyRows;
  int packed_total = 0;
  const int packed = block_excl_scan(listed ? (heavy ? 1 : (1 << 16)) : 0, s_wsum, packed_total);
  const int n_heavy = packed_total & 0xFFFF;
  const int n_active = n_heavy + (packed_total >> 16);
  const int arank = heavy ? (packed & 0xFFFF) : n_heavy + (packed >> 16);
  if (j < N) {
    a.offsets[j] = off;
    if (j == N - 1) a.offsets[N] = off + cnt;
    if (listed) a.active[arank] = make_int4(j, off, cnt, 0);
  }
  if (tid == 0) {
    a.counters[kCntActive] = n_active;
    a.counters[kCntSelected] = s_cnt[4];
    a.counters[kCntStatus] = 0;
    if (a.stats) {
      a.stats[0] = s_cnt[4];
      a.stats[1] = n_active;
      a.stats[2] = n_u;
      a.stats[3] = n_s0;
      a.stats[4] = n_start;
      a.stats[5] = m_eff;
      a.stats[6] = max_load;
      a.stats[7] = 0;
    }
    if (a.ledger) {   // running totals over the layers of a pass (global budget K)
      a.ledger[0] += 1;
      a.ledger[1] += s_cnt[4];
      a.ledger[2] += n_active;
      a.ledger[3] += n_u;
      a.ledger[5] = max(a.ledger[5], s_cnt[4]);
    }
  }
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t stream) {
  const dim3 grid(1), block(kThreads);
  if (a.N <= 64)
    hipLaunchKernelGGL(route_kernel<1>, grid, block, 0, stream, a);
  else if (a.N <= 128)
    hipLaunchKernelGGL(route_kernel<2>, grid, block, 0, stream, a);
  else if (a.N <= 256)
    hipLaunchKernelGGL(route_kernel<4>, grid, block, 0, stream, a);
  else if (a.N <= 512)
    hipLaunchKernelGGL(route_kernel<8>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(route_kernel<16>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace xs
