// Expert selection for one MoE layer and one decode batch (XShare, arXiv 2602.07265):
// router scoring, batch scores, greedy selection (flat Algorithm 2 or per-request +
// batch Algorithms 3-4), refinement, and the token permutation consumed by the expert
// GEMMs.  One workgroup of 1024 threads does all of it: the whole problem is a few
// thousand logits and is latency-, not throughput-bound.
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

// Ranking key: larger value first, lower expert index first on equal values.
__device__ __forceinline__ bool better(float ha, int ja, float hb, int jb) {
  return ha > hb || (ha == hb && ja < jb);
}

__device__ __forceinline__ void wave_argmax(float& h, int& j) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ho = __shfl_xor(h, off, 64);
    const int jo = __shfl_xor(j, off, 64);
    if (better(ho, jo, h, j)) {
      h = ho;
      j = jo;
    }
  }
}

__device__ __forceinline__ float lane_value(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Lane l holds the logits of experts l, l+64, ..., canonicalised (h + 0.0 maps -0.0 to +0.0).
template <int Q>
__device__ __forceinline__ void load_row(const float* row, int N, int lane, float (&v)[Q]) {
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int j = lane + 64 * q;
    v[q] = j < N ? row[j] + 0.0f : -INFINITY;
  }
}

// The k best entries whose bit is set in `allowed` (bit q <-> expert lane + 64 q).
// Lane r < k receives rank r: (value, expert) or (-inf, -1) if fewer than k are allowed.
template <int Q>
__device__ __forceinline__ void wave_topk(const float (&v)[Q], unsigned allowed, int k, int lane,
                                          float& my_h, int& my_j) {
  unsigned avail = allowed;
  my_h = -INFINITY;
  my_j = -1;
  for (int r = 0; r < k; ++r) {
    float bh = -INFINITY;
    int bj = INT_MAX;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int j = lane + 64 * q;
      if (((avail >> q) & 1u) && better(v[q], j, bh, bj)) {
        bh = v[q];
        bj = j;
      }
    }
    wave_argmax(bh, bj);
    if (bj != INT_MAX && (bj & 63) == lane) avail &= ~(1u << (bj >> 6));
    if (lane == r) {
      my_h = bh;
      my_j = bj == INT_MAX ? -1 : bj;
    }
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

// Block-wide exclusive prefix sum of one int per thread; every thread must call it.
__device__ int block_excl_scan(int v, int* s_wsum, int& total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(inc, off, 64);
    if (lane >= off) inc += y;
  }
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

template <int Q>
__global__ __launch_bounds__(kThreads) void route_kernel(RouteArgs a) {
  __shared__ uint16_t s_id[kMaxAssignments];   // per (token, rank): vanilla, later refined expert
  __shared__ float s_g[kMaxAssignments];       // per (token, rank): vanilla gate
  __shared__ float s_score[kMaxExperts];       // batch score s_j
  __shared__ float s_rscore[kMaxExperts];      // per-request score s^r_j
  __shared__ uint8_t s_tier[kMaxExperts];
  __shared__ uint8_t s_cand[kMaxExperts];
  __shared__ uint8_t s_sel[kMaxExperts];
  __shared__ int s_wsum[kWaves];
  __shared__ int s_cnt[8];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int T = a.T, N = a.N, k = a.k, k0 = a.k0;
  const bool dense = a.score_mode == 1;
  const bool hier = a.req_offsets != nullptr;
  const int TK = T * k;

  if (tid < 8) s_cnt[tid] = 0;
  __syncthreads();

  // ---- request offsets must be 0 = o_0 < o_1 < ... < o_R = T (checked in parallel)
  if (hier) {
    const int R = a.R;
    for (int r = tid; r < R; r += kThreads) {
      const int lo = a.req_offsets[r], hi = a.req_offsets[r + 1];
      if (!(lo < hi) || lo < 0 || hi > T) atomicOr(&s_cnt[7], 1);
    }
    if (tid == 0 && (a.req_offsets[0] != 0 || a.req_offsets[R] != T)) atomicOr(&s_cnt[7], 1);
    __syncthreads();
    if (s_cnt[7]) {
      for (int j = tid; j < N; j += kThreads) a.sel_mask[j] = 0;
      for (int p = tid; p < TK; p += kThreads) {
        a.ids[p] = -1;
        a.w[p] = 0.0f;
      }
      for (int j = tid; j <= N; j += kThreads) a.offsets[j] = 0;
      if (tid == 0) {
        a.counters[kCntActive] = 0;
        a.counters[kCntSelected] = 0;
        a.counters[kCntStatus] = 1;
        if (a.stats) {
          a.stats[0] = -1;
          for (int s = 1; s < 8; ++s) a.stats[s] = 0;
        }
      }
      return;
    }
  }

  // ---- (a) per token: plain top-k, its gates (Section 2.2); dense softmax if requested
  for (int i = wave; i < T; i += kWaves) {
    float v[Q];
    load_row<Q>(a.logits + (size_t)i * N, N, lane, v);
    unsigned all = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (lane + 64 * q < N) all |= 1u << q;
    float my_h;
    int my_j;
    wave_topk<Q>(v, all, k, lane, my_h, my_j);
    const float g = ranked_gate(my_h, lane, k);
    if (lane < k) {
      s_id[i * k + lane] = (uint16_t)my_j;
      s_g[i * k + lane] = g;
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
  }
  __syncthreads();

  // ---- (b) per expert: batch score, membership of U and S_0 (Eq. (2), Algorithm 2)
  const int j = tid;
  float s = 0.0f;
  bool inU = false, inS0 = false;
  if (j < N) {
    for (int i = 0; i < T; ++i) {
      for (int r = 0; r < k; ++r) {
        if (s_id[i * k + r] == j) {
          inU = true;
          if (r < k0) inS0 = true;
          if (!dense) s = s + s_g[i * k + r];
        }
      }
      if (dense) s = s + a.dense[(size_t)i * N + j];
    }
  }

  // ---- (c) per request (Algorithm 3): S_0(r) plus the m_r best remaining experts of r
  bool tier1 = false;
  if (hier && a.m_r > 0) {
    for (int r = 0; r < a.R; ++r) {
      const int lo = a.req_offsets[r], hi = a.req_offsets[r + 1];
      float sr = 0.0f;
      bool inUr = false, inS0r = false;
      if (j < N) {
        for (int i = lo; i < hi; ++i) {
          for (int q = 0; q < k; ++q) {
            if (s_id[i * k + q] == j) {
              inUr = true;
              if (q < k0) inS0r = true;
              if (!dense) sr = sr + s_g[i * k + q];
            }
          }
          if (dense) sr = sr + a.dense[(size_t)i * N + j];
        }
        s_rscore[j] = sr;
        s_cand[j] = (dense || inUr) && !inS0r;
      }
      __syncthreads();
      if (j < N && s_cand[j]) {
        int rank = 0;
        for (int jj = 0; jj < N && rank < a.m_r; ++jj)
          if (s_cand[jj] && better(s_rscore[jj], jj, sr, j)) ++rank;
        if (rank < a.m_r) tier1 = true;
      }
      __syncthreads();
    }
  }

  // ---- (d) batch greedy (Algorithm 1 with a fixed budget; Algorithm 4's final stage):
  //      order (tier, score desc, index asc), keep the first budget_eff candidates.
  int tier = 3;
  if (j < N) {
    const bool cand = dense ? (T > 0) : inU;
    tier = inS0 ? 0 : (tier1 ? 1 : (cand ? 2 : 3));
    s_tier[j] = (uint8_t)tier;
    s_score[j] = s;
    if (tier < 3) atomicAdd(&s_cnt[0], 1);
    if (tier == 0) atomicAdd(&s_cnt[1], 1);
    if (tier <= 1) atomicAdd(&s_cnt[2], 1);
    if (inU) atomicAdd(&s_cnt[3], 1);
  }
  __syncthreads();
  const int n_cand = s_cnt[0], n_s0 = s_cnt[1], n_start = s_cnt[2], n_u = s_cnt[3];
  const int base = a.budget_mode == 0 ? a.budget : n_start + a.budget;
  const int m_eff = max(min(base, n_cand), min(k, n_cand));
  bool sel = false;
  if (j < N && tier < 3) {
    int rank = 0;
    for (int jj = 0; jj < N && rank < m_eff; ++jj) {
      const int tj = s_tier[jj];
      if (tj < tier || (tj == tier && better(s_score[jj], jj, s, j))) ++rank;
    }
    sel = rank < m_eff;
  }
  if (j < N) {
    s_sel[j] = sel;
    a.sel_mask[j] = sel;
    if (sel) atomicAdd(&s_cnt[4], 1);
  }
  __syncthreads();

  // ---- (e) refinement: every token to its top-k inside S, gates renormalised (Section 3.4)
  for (int i = wave; i < T; i += kWaves) {
    float v[Q];
    load_row<Q>(a.logits + (size_t)i * N, N, lane, v);
    unsigned allowed = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int jq = lane + 64 * q;
      if (jq < N && s_sel[jq]) allowed |= 1u << q;
    }
    float my_h;
    int my_j;
    wave_topk<Q>(v, allowed, k, lane, my_h, my_j);
    const float g = ranked_gate(my_h, lane, k);
    if (lane < k) {
      a.ids[i * k + lane] = my_j;
      a.w[i * k + lane] = g;
      s_id[i * k + lane] = (uint16_t)my_j;
    }
  }
  __syncthreads();

  // ---- (f) permutation: rows grouped by expert (ascending), tokens ascending inside
  int cnt = 0;
  if (j < N)
    for (int p = 0; p < TK; ++p) cnt += s_id[p] == j;
  int total = 0;
  const int off = block_excl_scan(cnt, s_wsum, total);
  int n_active = 0;
  const int arank = block_excl_scan(cnt > 0 ? 1 : 0, s_wsum, n_active);
  if (j < N) {
    a.offsets[j] = off;
    if (j == N - 1) a.offsets[N] = off + cnt;
    if (cnt > 0) a.active[arank] = j;
    int pos = off;
    for (int p = 0; p < TK && pos < off + cnt; ++p)
      if (s_id[p] == j) a.perm[pos++] = p;
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
      a.stats[6] = 0;
      a.stats[7] = 0;
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
