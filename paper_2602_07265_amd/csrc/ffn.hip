// Expert FFNs of the selected experts only (SwiGLU, nn.Linear [out, in] weights, bf16):
//   gate/up:  H[p, :] = silu(x_i W1_e^T) * (x_i W3_e^T)      for every permuted row p = (i, r)
//   down:     Y[i*k + r, :] = H[p, :] W2_e^T
// H is kept as hi = bf16(H) and lo = bf16(H - hi) (about 16 significant bits): with H in
// bf16 alone its rounding moved large outputs across a bf16 rounding boundary of y.  The two
// are interleaved in 8-element chunks, so a token's hi and lo for one k-range share a cache
// line.  The down GEMM feeds both to one MFMA: 8 tokens per 16-row tile, hi rows 0-7 and lo
// rows 8-15, summed after the reduction.
//   combine:  y_i = sum_r w_ir Y[i*k + r, :]  (rank order, fp32) -> bf16
// Always-on shared experts (Section 2.1) are extra slots after the routed ones, with all T
// tokens; their output rows are added after the routed terms with weight 1.  The router
// GEMM h = W_g x uses the same wave pass with the router rows as weights.
//
// Decode batches give an expert 1..T tokens, so each weight element is used a few times:
// the GEMMs are bound by streaming the selected experts' weights from HBM.  Each wave owns
// 16 weight rows and the whole reduction dimension; weights go from HBM straight into the
// B operand of v_mfma_f32_16x16x32_bf16 (lane (n, g) loads 16 contiguous bytes of row n per
// MFMA, so a wave reads 16 rows x 32*U contiguous elements per step), tokens form the M
// dimension (16 per tile, up to two tiles per pass), accumulation is fp32.  The block's
// four waves share the expert and its token rows, which the block stages in LDS one step
// at a time (block_pass); the next step's loads are issued before the current step's
// MFMAs (register double buffering).  The per-wave passes (wave_pass*) serve the router
// GEMM and the shapes the staged pass does not take.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "internal.h"
#include "xshare.h"

namespace xs {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;       // 4 waves
constexpr int kWaves = kBlock / 64;
constexpr int kCols = 16;         // weight rows (output columns) per wave
constexpr int kTiles = 2;         // 16-token tiles per pass over the weights

// Block timeline of the expert GEMMs, in a profiling build only (XS_BLOCK_TIMES 1, the
// library libxshare_timeline.so): thread 0 of every block of a gate/up and a down launch
// stamps its start and end, and every block of a persistent down launch its start and the
// end of each unit, from the 100 MHz global clock (s_memrealtime), by block id; each launch
// overwrites the entries of its blocks.  xshare_block_times copies them out.
#ifndef XS_BLOCK_TIMES
#define XS_BLOCK_TIMES 0
#endif
constexpr int kTimeSeqStride = XSHARE_TIME_SEQ_STRIDE;  // a block's start, then 32 unit ends
#if XS_BLOCK_TIMES
constexpr int kTimeBlocks = XSHARE_TIME_BLOCKS;         // stamped blocks of a grid launch
constexpr int kTimeSeqBlocks = XSHARE_TIME_SEQ_BLOCKS;  // stamped persistent down blocks
__device__ unsigned long long xs_times_gu[2 * kTimeBlocks];
__device__ unsigned long long xs_times_dn[2 * kTimeBlocks];
__device__ unsigned long long xs_times_seq[kTimeSeqBlocks * kTimeSeqStride];
__device__ __forceinline__ unsigned block_id3() {
  return (blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
}
#define XS_TIME(arr, idx, lim)                                                          \
  do {                                                                                  \
    if (threadIdx.x == 0 && (idx) < (lim)) arr[idx] = __builtin_amdgcn_s_memrealtime(); \
  } while (0)
#else
#define XS_TIME(arr, idx, lim) \
  do {                         \
  } while (0)
#endif

__device__ __forceinline__ bf16x8 load8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

__device__ __forceinline__ floatx4 mfma(const bf16x8& a, const bf16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t to_bf16(float v) {
  uint32_t b = __float_as_uint(v);
  b += 0x7FFFu + ((b >> 16) & 1u);  // round to nearest even
  return (uint16_t)(b >> 16);
}

__device__ __forceinline__ float from_bf16(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// 8 FP8 E4M3FN codes (two words, element order = byte order) -> 8 bf16.  The hardware
// conversion gives fp32; an E4M3 value has at most 4 significant bits, so its upper 16 bits
// are the exact bf16 (v_perm_b32 gathers the upper halves of two floats).
__device__ __forceinline__ bf16x8 fp8x8_to_bf16(uint2 v) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8((int)v.x, false);
  const f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8((int)v.x, true);
  const f32x2 c = __builtin_amdgcn_cvt_pk_f32_fp8((int)v.y, false);
  const f32x2 d = __builtin_amdgcn_cvt_pk_f32_fp8((int)v.y, true);
  u32x4 r;
  r.x = __builtin_amdgcn_perm(__float_as_uint(a.y), __float_as_uint(a.x), 0x07060302u);
  r.y = __builtin_amdgcn_perm(__float_as_uint(b.y), __float_as_uint(b.x), 0x07060302u);
  r.z = __builtin_amdgcn_perm(__float_as_uint(c.y), __float_as_uint(c.x), 0x07060302u);
  r.w = __builtin_amdgcn_perm(__float_as_uint(d.y), __float_as_uint(d.x), 0x07060302u);
  return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ uint2 load_q8(const uint8_t* p) {
  return *reinterpret_cast<const uint2*>(p);
}

// Weight formats of the expert GEMMs.
constexpr int kBf16 = 0;   // bf16
constexpr int kFp8 = 1;    // OCP FP8 E4M3FN codes, one fp32 scale per output row
constexpr int kMx4 = 2;    // MXFP4: E2M1 codes, two per byte, one E8M0 scale per 32 elements

// 8U packed E2M1 codes of one lane and step (U words, 8 elements each, low nibble first).
template <int U>
struct Q4 {
  uint32_t w[U];
};
template <int U>
__device__ __forceinline__ Q4<U> load_q4(const uint8_t* p) {
  Q4<U> r;
  if constexpr (U == 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 v = *reinterpret_cast<const uint4*>(p + 16 * i);
      r.w[4 * i] = v.x;
      r.w[4 * i + 1] = v.y;
      r.w[4 * i + 2] = v.z;
      r.w[4 * i + 3] = v.w;
    }
  } else if constexpr (U == 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint4 w = *reinterpret_cast<const uint4*>(p + 16);
    r.w[0] = v.x;
    r.w[1] = v.y;
    r.w[2] = v.z;
    r.w[3] = v.w;
    r.w[4] = w.x;
    r.w[5] = w.y;
    r.w[6] = w.z;
    r.w[7] = w.w;
  } else if constexpr (U == 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    r.w[0] = v.x;
    r.w[1] = v.y;
    r.w[2] = v.z;
    r.w[3] = v.w;
  } else if constexpr (U == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    r.w[0] = v.x;
    r.w[1] = v.y;
  } else {
    r.w[0] = *reinterpret_cast<const uint32_t*>(p);
  }
  return r;
}

// E8M0 scale byte -> 2^(e - 127) as fp32 (e = 0 is the subnormal 2^-127).
__device__ __forceinline__ float e8m0_scale(uint32_t e) {
  return e ? __uint_as_float(e << 23) : __uint_as_float(0x00400000u);
}

// 8 E2M1 codes (one word) times their block scale -> 8 bf16.  The conversion (one byte, two
// elements, per instruction; low nibble first) multiplies by a power of two, so the result
// is exact for scales that keep the weights in bf16's normal range.
__device__ __forceinline__ bf16x8 fp4x8_to_bf16(uint32_t w, float scale) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 0);
  const bf16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 1);
  const bf16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 2);
  const bf16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 3);
  bf16x8 r;
  r[0] = p0[0];
  r[1] = p0[1];
  r[2] = p1[0];
  r[3] = p1[1];
  r[4] = p2[0];
  r[5] = p2[1];
  r[6] = p3[0];
  r[7] = p3[1];
  return r;
}

// Stores v = H[p, c] as hi = bf16(v) and lo = bf16(v - hi) in the interleaved rows of 2f
// elements: hi at 16 (c / 8) + c % 8, lo 8 elements further.
__device__ __forceinline__ void store_hilo(uint16_t* h2, size_t p, int c, int f, float v) {
  const uint16_t h = to_bf16(v);
  uint16_t* const at = h2 + p * 2 * (size_t)f + 2 * (c & ~7) + (c & 7);
  at[0] = h;
  at[8] = to_bf16(v - from_bf16(h));
}

// One pass of a wave over the reduction dimension K for up to kTiles token tiles:
// acc[m][rt] += A_rt (16 x K) * B_m^T (K x 16) for the NM weight matrices B_m.
// `arow[rt]` points at the token row this lane feeds (a duplicate of a valid row for
// padding lanes, whose output rows are discarded; duplicate addresses coalesce, which
// measured faster than masking those lanes), `brow[m]` at the weight row of this lane's
// column;
// both already offset by this lane's group position g * 8U.  Weight loads (HBM) run one
// step ahead; token loads (L2-resident) are issued either one step ahead too (ADBL) or
// at the top of their own step, which halves their register footprint.
// AS: element stride of the token rows per k (2 for the interleaved hi / lo rows, whose
// 8-element chunks alternate).
#ifndef XS_KMAP
#define XS_KMAP 1
#endif
// Reduction offsets of the bf16 passes: MFMA u of a step and lane group g.  With XS_KMAP 1
// the four lane groups of one MFMA read 32 contiguous elements, so one load instruction
// touches half as many cache lines as with 0 (each lane's U MFMAs on 8U contiguous
// elements); measured 0.3-1.2 % faster.  A and B use the same map, so the sum is the same.
__device__ __forceinline__ constexpr int kstep(int u) { return XS_KMAP ? 32 * u : 8 * u; }
template <int U>
__device__ __forceinline__ constexpr int klane(int g) { return XS_KMAP ? 8 * g : 8 * U * g; }

template <int U, int NM, bool ADBL, int TL = kTiles, int AS = 1>
__device__ __forceinline__ void wave_pass(const uint16_t* const (&arow)[TL], int nt,
                                          const uint16_t* const (&brow)[NM], int K,
                                          floatx4 (&acc)[NM][TL], int k_first = 0) {
  constexpr int KB = 32 * U;
  bf16x8 b[NM][U], x[TL][U];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int u = 0; u < U; ++u) b[m][u] = load8(brow[m] + k_first + kstep(u));
  if (ADBL) {
#pragma unroll
    for (int rt = 0; rt < TL; ++rt)
      if (rt < nt)
#pragma unroll
        for (int u = 0; u < U; ++u) x[rt][u] = load8(arow[rt] + AS * (k_first + kstep(u)));
  }

  int kb = k_first;
  for (int s = 0; s < K; s += KB) {
    bf16x8 nb[NM][U], nx[ADBL ? TL : 1][U];
    const bool more = s + KB < K;
    int kn = kb + KB;
    if (kn >= K) kn -= K;
    // Token loads of this step go out before the next step's weight loads: loads complete
    // in issue order, so waiting for the tokens then leaves the weight prefetch in flight.
    if (!ADBL) {
#pragma unroll
      for (int rt = 0; rt < TL; ++rt)
        if (rt < nt)
#pragma unroll
          for (int u = 0; u < U; ++u) x[rt][u] = load8(arow[rt] + AS * (kb + kstep(u)));
    }
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) nb[m][u] = load8(brow[m] + kn + kstep(u));
      if (ADBL) {
#pragma unroll
        for (int rt = 0; rt < TL; ++rt)
          if (rt < nt)
#pragma unroll
            for (int u = 0; u < U; ++u) nx[rt][u] = load8(arow[rt] + AS * (kn + kstep(u)));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rt = 0; rt < TL; ++rt)
        if (rt < nt)
#pragma unroll
          for (int m = 0; m < NM; ++m) acc[m][rt] = mfma(x[rt][u], b[m][u], acc[m][rt]);
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) b[m][u] = nb[m][u];
      if (ADBL) {
#pragma unroll
        for (int rt = 0; rt < TL; ++rt)
#pragma unroll
          for (int u = 0; u < U; ++u) x[rt][u] = nx[ADBL ? rt : 0][u];
      }
    }
    kb = kn;
  }
}

// wave_pass with FP8 weights: the B operand comes from E4M3 codes (8 bytes per lane and
// MFMA), prefetched one step ahead as raw bytes and converted to bf16 just before use.
template <int U, int NM, int TL = kTiles, int AS = 1>
__device__ __forceinline__ void wave_pass_q8(const uint16_t* const (&arow)[TL], int nt,
                                             const uint8_t* const (&brow)[NM], int K,
                                             floatx4 (&acc)[NM][TL], int k_first = 0) {
  constexpr int KB = 32 * U;
  uint2 b[NM][U];
  bf16x8 x[TL][U];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int u = 0; u < U; ++u) b[m][u] = load_q8(brow[m] + k_first + 8 * u);
  int kb = k_first;
  for (int s = 0; s < K; s += KB) {
    uint2 nb[NM][U];
    const bool more = s + KB < K;
    int kn = kb + KB;
    if (kn >= K) kn -= K;
#pragma unroll
    for (int rt = 0; rt < TL; ++rt)       // tokens first: see wave_pass
      if (rt < nt)
#pragma unroll
        for (int u = 0; u < U; ++u) x[rt][u] = load8(arow[rt] + AS * (kb + 8 * u));
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) nb[m][u] = load_q8(brow[m] + kn + 8 * u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const bf16x8 bv = fp8x8_to_bf16(b[m][u]);
#pragma unroll
        for (int rt = 0; rt < TL; ++rt)
          if (rt < nt) acc[m][rt] = mfma(x[rt][u], bv, acc[m][rt]);
      }
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) b[m][u] = nb[m][u];
    }
    kb = kn;
  }
}

// MXFP4 block scales in the tiled layout (xshare_mx_scales_tile): per matrix of R rows and K
// inputs, [R / 16][G][16 rows][8 bytes] with G = ceil(K / 256) granules of 8 blocks of 32
// inputs, so the scale bytes of one 16-row weight tile over 256 inputs are one 128-byte
// piece, read once and whole: the byte of row r and block c sits at ((r / 16) G + c / 8) 128
// + (r % 16) 8 + c % 8.  mx_row: where row r's bytes of its tile start (granule 0).
__device__ __forceinline__ int mx_granules(int K) { return (K + 255) >> 8; }
__device__ __forceinline__ const uint8_t* mx_row(const uint8_t* mat, int r, int G) {
  return mat + (size_t)(r >> 4) * G * 128 + (r & 15) * 8;
}
// The scale bytes of a lane whose step starts at input k (8U inputs: one block for U <= 4,
// two for U = 8, four for U = 16; a lane's blocks share one granule since k is a multiple of
// 8U), from its row `row` (mx_row).
template <int U>
__device__ __forceinline__ uint32_t load_mx_scales(const uint8_t* row, int k) {
  const int c = k >> 5;
  const uint8_t* const p = row + ((c >> 3) << 7) + (c & 7);
  if constexpr (U >= 16)
    return *reinterpret_cast<const uint32_t*>(p);
  else if constexpr (U == 8)
    return *reinterpret_cast<const uint16_t*>(p);
  else
    return *p;
}

// wave_pass with MXFP4 weights: per step a lane loads 4U bytes of codes (its 8U elements)
// and their scale bytes, one step ahead; the codes become bf16, scaled, just before use.
// `brow[m]` points at the codes of this lane's first element, `srow[m]` at its row's tiled
// scales (mx_row); `kl`: this lane's first input (absolute, for the scale bytes).
template <int U, int NM, int TL = kTiles, int AS = 1>
__device__ __forceinline__ void wave_pass_q4(const uint16_t* const (&arow)[TL], int nt,
                                             const uint8_t* const (&brow)[NM],
                                             const uint8_t* const (&srow)[NM], int kl, int K,
                                             floatx4 (&acc)[NM][TL], int k_first = 0) {
  static_assert(U == 1 || U == 2 || U == 4 || U == 8, "1, 2, 4 or 8 words per lane and step");
  constexpr int KB = 32 * U;
  Q4<U> b[NM];
  uint32_t e[NM];
  bf16x8 x[TL][U];
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    b[m] = load_q4<U>(brow[m] + k_first / 2);
    e[m] = load_mx_scales<U>(srow[m], kl + k_first);
  }
  int kb = k_first;
  for (int s = 0; s < K; s += KB) {
    Q4<U> nb[NM];
    uint32_t ne[NM];
    const bool more = s + KB < K;
    int kn = kb + KB;
    if (kn >= K) kn -= K;
#pragma unroll
    for (int rt = 0; rt < TL; ++rt)       // tokens first: see wave_pass
      if (rt < nt)
#pragma unroll
        for (int u = 0; u < U; ++u) x[rt][u] = load8(arow[rt] + AS * (kb + 8 * u));
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        nb[m] = load_q4<U>(brow[m] + kn / 2);
        ne[m] = load_mx_scales<U>(srow[m], kl + kn);
      }
    }
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const float sc0 = e8m0_scale(e[m] & 0xFFu);
      const float sc1 = U == 8 ? e8m0_scale((e[m] >> 8) & 0xFFu) : sc0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bf16x8 bv = fp4x8_to_bf16(b[m].w[u], u < 4 ? sc0 : sc1);
#pragma unroll
        for (int rt = 0; rt < TL; ++rt)
          if (rt < nt) acc[m][rt] = mfma(x[rt][u], bv, acc[m][rt]);
      }
    }
    if (more) {
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        b[m] = nb[m];
        e[m] = ne[m];
      }
    }
    kb = kn;
  }
}

// Token rows staged in LDS.  With tokens loaded per wave (wave_pass*), every wave of a block
// gathers the same token rows again, as half-line loads; with MXFP4 weights (a quarter of
// bf16's bytes) these were as many load instructions as the weights', or more.  In both
// expert GEMMs the four waves of a block share the expert, the token rows and the reduction
// range: this pass has the block load each step's token rows once, coalesced (16 bytes per
// thread, P threads per row), into a double-buffered LDS tile, and the waves read their A
// operands from it.  The loads of step s + 1 (tokens, then weights) are issued before the
// MFMAs of step s, with no branch around them, so the wait before the LDS write covers the
// token loads only and the weight loads stay in flight across the barrier.  One barrier per
// step: the writes into the other buffer come after this step's reads of it were fenced by
// the previous barrier.
//   gate/up (kDown false): staged rows are x rows, 16 per MFMA tile (lane row n).
//   down (kDown true): staged rows are H rows (hi and lo chunks interleaved, two elements
//   per k), 8 per tile: lanes n < 8 read token n's hi chunk, lanes n >= 8 its lo chunk.
constexpr int kStageRows = 32;            // token rows per pass
template <int U, bool kDown>
struct Stage {
  static constexpr int KB = 32 * U;                  // reduction elements per step
  static constexpr int AS = kDown ? 2 : 1;           // staged elements per reduction element
  static constexpr int P = AS * KB / 8;              // 16-byte pieces per row and step
  static_assert(P * kStageRows >= kBlock, "256 threads cover at most the 32 rows of a step");
  static constexpr int TR = kDown ? 8 : 16;          // token rows per MFMA tile
  // LDS row stride (elements): the rows of one A read start 16 B (x) or 32 B (H, whose lo
  // lanes read 16 B past their hi lanes) apart modulo 256 B, so they fall in distinct banks
  static constexpr int LS = AS * KB + (kDown ? 16 : 8);
  static constexpr int kElems = 2 * kStageRows * LS; // both buffers
};

// One lane's weights of one step for one 16-row tile, by format: where they are (w: this
// lane's first element; sc: MXFP4 scale bytes), the registers that hold them, their loads
// for step s and the B operand of MFMA u.  `koff(g, u)`: the reduction offset, within a
// step, of lane group g's elements in MFMA u (the A operand reads the same).
template <int kW, int U>
struct WTile;
template <int U>
struct WTile<kBf16, U> {
  using GV = uint32_t;
  struct Ptr { const uint16_t* w; };
  struct Regs { bf16x8 w[U]; };
  __device__ static constexpr int koff(int g, int u) { return kstep(u) + klane<U>(g); }
  __device__ static Regs load(const Ptr& p, int s) {
    Regs r;
#pragma unroll
    for (int u = 0; u < U; ++u) r.w[u] = load8(p.w + s + kstep(u));
    return r;
  }
  __device__ static bf16x8 operand(const Regs& r, int u) { return r.w[u]; }
};
template <int U>
struct WTile<kFp8, U> {
  using GV = uint32_t;
  struct Ptr { const uint8_t* w; };
  struct Regs { uint2 w[U]; };
  __device__ static constexpr int koff(int g, int u) { return 8 * U * g + 8 * u; }
  __device__ static Regs load(const Ptr& p, int s) {
    Regs r;
#pragma unroll
    for (int u = 0; u < U; ++u) r.w[u] = load_q8(p.w + s + 8 * u);
    return r;
  }
  __device__ static bf16x8 operand(const Regs& r, int u) { return fp8x8_to_bf16(r.w[u]); }
};
template <int U>
struct WTile<kMx4, U> {
  // w: this lane's codes; sc: its row's tiled scales (mx_row); k: its first input (absolute)
  struct Ptr { const uint8_t* w; const uint8_t* sc; int k; };
  // scale bytes (block u / 4 in byte u / 4) in a type no wider than their load: a widening
  // at the end of a step would wait for the load
  using E = typename std::conditional<(U > 8), uint32_t, uint16_t>::type;
  struct Regs { Q4<U> q; E e; };
  __device__ static constexpr int koff(int g, int u) { return 8 * U * g + 8 * u; }
  __device__ static Regs load(const Ptr& p, int s) {
    Regs r;
    r.q = load_q4<U>(p.w + s / 2);
    r.e = (E)load_mx_scales<U>(p.sc, p.k + s);
    return r;
  }
  __device__ static bf16x8 operand(const Regs& r, int u) {
    const uint32_t e = r.e;
    return fp4x8_to_bf16(r.q.w[u], e8m0_scale((e >> (8 * (u >> 2))) & 0xFFu));
  }
};

// NT: token tiles of the pass (R <= TR * NT rows); NL: loads per thread and step, at least
// ceil(R * P / 256) (pieces beyond R * P repeat the last one).  Staged row r (r < R) is
// x[tok[r] * ld ...], x already offset to this block's reduction range.  acc[m][rt] as in
// wave_pass (gate/up) or the down pass.
template <int kW, int U, bool kDown, int NM, int NT, int NL, int TA>
__device__ __forceinline__ void block_pass(const uint16_t* x, size_t ld, const int* tok, int R,
                                           const typename WTile<kW, U>::Ptr (&wp)[NM], int K,
                                           int k_first, floatx4 (&acc)[NM][TA], uint16_t* lds) {
  using S = Stage<U, kDown>;
  using WT = WTile<kW, U>;
  constexpr int KB = S::KB;
  static_assert(NT <= TA && S::TR * NT <= kStageRows, "tiles of the pass");
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int t = threadIdx.x, lane = t & 63;
  const int n = lane & 15, g = lane >> 4;
  const uint16_t* src[NL];   // this thread's pieces: global source and LDS offset
  int wofs[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int q = min(t + i * kBlock, R * S::P - 1);
    const int row = q / S::P, piece = q % S::P;
    src[i] = x + (size_t)tok[row] * ld + piece * 8;
    wofs[i] = row * S::LS + piece * 8;
  }
  int rofs[NT];              // this lane's A rows (padding lanes repeat the last token row)
#pragma unroll
  for (int rt = 0; rt < NT; ++rt)
    rofs[rt] = kDown ? min(8 * rt + (n & 7), R - 1) * S::LS + (n & 8)
                     : min(16 * rt + n, R - 1) * S::LS;

  u32x4 v[NL];
  typename WT::Regs b[NM];
#pragma unroll
  for (int i = 0; i < NL; ++i) v[i] = *reinterpret_cast<const u32x4*>(src[i] + S::AS * k_first);
#pragma unroll
  for (int m = 0; m < NM; ++m) b[m] = WT::load(wp[m], k_first);
#pragma unroll
  for (int i = 0; i < NL; ++i) *reinterpret_cast<u32x4*>(lds + wofs[i]) = v[i];
  __syncthreads();

  // MFMAs of one step from LDS buffer `cur`
  auto step = [&](const uint16_t* cur) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ka = S::AS * WT::koff(g, u);
      bf16x8 xa[NT];
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) xa[rt] = *reinterpret_cast<const bf16x8*>(cur + rofs[rt] + ka);
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const bf16x8 bv = WT::operand(b[m], u);
#pragma unroll
        for (int rt = 0; rt < NT; ++rt) acc[m][rt] = mfma(xa[rt], bv, acc[m][rt]);
      }
    }
  };
  int buf = 0;
  // loads of step kn, MFMAs of the step before it, then kn's tokens into the other buffer
  auto advance = [&](int kn) {
#pragma unroll
    for (int i = 0; i < NL; ++i) v[i] = *reinterpret_cast<const u32x4*>(src[i] + S::AS * kn);
    typename WT::Regs nb[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) nb[m] = WT::load(wp[m], kn);
    step(lds + buf * kStageRows * S::LS);
    uint16_t* const nxt = lds + (buf ^ 1) * kStageRows * S::LS;
#pragma unroll
    for (int i = 0; i < NL; ++i) *reinterpret_cast<u32x4*>(nxt + wofs[i]) = v[i];
#pragma unroll
    for (int m = 0; m < NM; ++m) b[m] = nb[m];
    __syncthreads();
    buf ^= 1;
  };
  // the pass starts at step k_first and wraps around (two plain loops: a wrap test inside
  // one loop measured slower)
  for (int kn = k_first + KB; kn < K; kn += KB) advance(kn);
  for (int kn = 0; kn < k_first; kn += KB) advance(kn);
  step(lds + buf * kStageRows * S::LS);
  __syncthreads();                         // the block's next pass rewrites both buffers
}

// The staged pass over R token rows, by block-uniform instance: the fewest tiles that hold
// R rows and the loads per thread that the largest R of that tile count needs.
template <int kW, int U, bool kDown, int NM, int TA>
__device__ __forceinline__ void staged_pass(const uint16_t* x, size_t ld, const int* tok,
                                               int R, const typename WTile<kW, U>::Ptr (&wp)[NM],
                                               int K, int k_first, floatx4 (&acc)[NM][TA],
                                               uint16_t* lds) {
  using S = Stage<U, kDown>;
  constexpr int TR = S::TR;
  constexpr int L1 = (TR * S::P + kBlock - 1) / kBlock, L2 = (2 * TR * S::P + kBlock - 1) / kBlock;
  if constexpr (TA == 2) {          // gate/up: up to two 16-row tiles
    constexpr int L1h = (TR / 2 * S::P + kBlock - 1) / kBlock;
    constexpr int L2h = (3 * TR / 2 * S::P + kBlock - 1) / kBlock;
    if (R <= TR / 2)
      block_pass<kW, U, kDown, NM, 1, L1h, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    else if (R <= TR)
      block_pass<kW, U, kDown, NM, 1, L1, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    else if (R <= 3 * TR / 2)
      block_pass<kW, U, kDown, NM, 2, L2h, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    else
      block_pass<kW, U, kDown, NM, 2, L2, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
  } else {                          // down: up to four 8-token tiles
    static_assert(TA == 2 || TA == 4, "two or four 8-token tiles");
    if (R <= TR) {
      block_pass<kW, U, kDown, NM, 1, L1, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    } else if (TA == 2 || R <= 2 * TR) {
      block_pass<kW, U, kDown, NM, 2, L2, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    } else if constexpr (TA == 4) {
      constexpr int L3 = (3 * TR * S::P + kBlock - 1) / kBlock;
      constexpr int L4 = (4 * TR * S::P + kBlock - 1) / kBlock;
      if (R <= 3 * TR)
        block_pass<kW, U, kDown, NM, 3, L3, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
      else
        block_pass<kW, U, kDown, NM, 4, L4, TA>(x, ld, tok, R, wp, K, k_first, acc, lds);
    }
  }
}

// Unroll (32-element k-groups per step) and token-operand buffering of the two GEMMs.
#ifndef XS_GATE_UP_U
#define XS_GATE_UP_U 4
#endif
#ifndef XS_GATE_UP_ADBL
#define XS_GATE_UP_ADBL 1
#endif
#ifndef XS_DOWN_U
#define XS_DOWN_U 2
#endif
#ifndef XS_DOWN_ADBL
#define XS_DOWN_ADBL 0
#endif
#ifndef XS_Q8_GATE_UP_U
#define XS_Q8_GATE_UP_U 4
#endif
#ifndef XS_Q8_DOWN_U
#define XS_Q8_DOWN_U 4
#endif
// gate/up launches whose grid keeps at least this many blocks with two column tiles per
// wave use two (measured: DeepSeek T=32 gate/up -1 % bf16, -5 % FP8, -10 % MXFP4; a grid
// half that size, as at T=8, ran 10-14 % slower).
// bf16 and FP8 down launches use twice the base tiles per wave when the routed rows are at
// least XS_DN_WIDE_TOKENS per expected expert and the grid keeps XS_DN_WIDE_MIN_BLOCKS blocks
// (measured on DeepSeek T=32 and the speculative batch: bf16 down -1.6 % and -3 %, FP8 -10 %
// and -13 %; with 1-3 tokens per expert, as at T=8, wide waves ran 4-20 % slower).
#ifndef XS_DN_WIDE_TOKENS
#define XS_DN_WIDE_TOKENS 4
#endif
#ifndef XS_DN_WIDE_MIN_BLOCKS
#define XS_DN_WIDE_MIN_BLOCKS 768
#endif
#ifndef XS_GU_CT2_MIN_BLOCKS
#define XS_GU_CT2_MIN_BLOCKS 768
#endif
#ifndef XS_Q4_GU_CT2_MIN_BLOCKS
#define XS_Q4_GU_CT2_MIN_BLOCKS XS_GU_CT2_MIN_BLOCKS
#endif
#ifndef XS_Q4_GATE_UP_U
#define XS_Q4_GATE_UP_U 8
#endif
// Unroll of one-tile gate/up launches (small grids), twice the two-tile one for bf16:
// twice the weight bytes in flight per wave where there are fewer waves.  Same-box A/B:
// bf16 DeepSeek T=32 M=24 gate/up 246 -> 237 us, Mixtral 232 -> 215, T=8 239 -> 234.  FP8
// at 8 words gained on Mixtral and lost on Qwen and T=8.  MXFP4 gained from 16 words while
// every step read its scales; with scales read once per four steps, 8 words are ahead
// (DeepSeek T=8 M=24 gate/up 76.2 -> 74.5 us, Mixtral 69.1 -> 67.1 us).
#ifndef XS_GATE_UP_U1
#define XS_GATE_UP_U1 8
#endif
#ifndef XS_Q8_GATE_UP_U1
#define XS_Q8_GATE_UP_U1 XS_Q8_GATE_UP_U
#endif
// FP8 gate/up instances of up to 4 words a step held to 3 waves per SIMD (168 registers, no
// spills; left alone the compiler kept 2).  Same-box A/B, gate/up us (2 -> 3 waves):
// DeepSeek T=32 M=48 252.0 -> 246.6, speculative 335.5 -> 331.8, T=8 M=24 127.0 -> 124.5,
// Qwen 32.9 -> 32.4, Mixtral 137.8 -> 135.0.  Not kept at 3 waves: the two-tile MXFP4
// gate/up (72 bytes spilled; DeepSeek T=32 138 -> 152 us) and the 32-row FP8 down (no
// change).
#ifndef XS_Q8_GU_W3
#define XS_Q8_GU_W3 1
#endif
#ifndef XS_Q4_GATE_UP_U1
#define XS_Q4_GATE_UP_U1 8
#endif
#ifndef XS_Q4_DOWN_U
#define XS_Q4_DOWN_U 8
#endif
#ifndef XS_Q4_DN_WIDE
#define XS_Q4_DN_WIDE 1
#endif
#ifndef XS_Q4_DOWN_ROT
#define XS_Q4_DOWN_ROT 0
#endif
// K steps between the starts of consecutive down waves (blocks, when the pass is staged):
// one with bf16 weights (per wave: DeepSeek T=32 down 270 -> 263 us; per block, staged:
// 266 -> 258 us, speculative 358 -> 351 us); none with FP8, where it measured no gain.
#ifndef XS_DOWN_ROT
#define XS_DOWN_ROT 1
#endif
#ifndef XS_Q8_DOWN_ROT
#define XS_Q8_DOWN_ROT 0
#endif
// Expert slots from which the down grid keeps each slot's column blocks on one XCD (with
// fewer, whole XCDs would idle: five experts left three of eight without work).
#ifndef XS_DOWN_XCD_SLOTS
#define XS_DOWN_XCD_SLOTS 16
#endif
static_assert(XS_DOWN_XCD_SLOTS >= 8, "at least one slot per XCD");
#ifndef XS_DOWN_TL
#define XS_DOWN_TL 4                 // 8-token (hi + lo) tiles per pass of the down GEMM
#endif
// Seven 16-row W2 tiles per wave (448 output rows per block, one block per CU) for the bf16
// down GEMM when that grid is a whole number of rounds: at d = 7168 the DeepSeek layer's 48
// slots give 768 blocks, three rounds, where 64-row waves leave 2.6 rounds of 512.  With
// U = 4 a wave keeps 28 KB of weights in flight.  Same-box A/B, down us (64-row waves ->
// seven tiles): DeepSeek T=32 M=48 256 -> 245, iid logits 257 -> 245, speculative 347 ->
// 333; M=96 (six rounds against 5.25) 464 -> 464; at U = 2 M=48 ran 260, and on grids
// that leave a partial round the seven tiles lose (M=24 138 -> 148, the layer with its
// shared expert 262 -> 295).  FP8 gained nothing (DeepSeek 137 -> 136, speculative 188 ->
// 191) and MXFP4 lost (81 -> 85 us), so they keep their waves.
#ifndef XS_DOWN_NM7
#define XS_DOWN_NM7 1
#endif
#ifndef XS_DOWN_NM7_U
#define XS_DOWN_NM7_U 4
#endif
// The seven-tile bf16 down launch as a persistent grid (down_seq_kernel).  Same-box A/B,
// down us (grid of rounds -> persistent): DeepSeek T=32 M=48 246.0 / 245.8 -> 243.5 / 242.5,
// speculative 333.2 / 334.9 -> 331.9 / 333.1.  With 2 waves per SIMD (FP8 and bf16 64- and
// 32-row waves) it lost: FP8 DeepSeek T=32 137.4 -> 147.0, bf16 T=8 M=24 130 -> 133.5 (a
// CU's second block already overlaps the first one's start there), so only this launch
// takes it.
#ifndef XS_DOWN_SEQ
#define XS_DOWN_SEQ 1
#endif


#ifndef XS_DOWN_WAVES_PER_EU
#define XS_DOWN_WAVES_PER_EU 2       // waves per SIMD of the staged down instances (3: spills)
#endif

// Formats whose GEMMs stage the token rows in LDS (bit kW of each mask; all three by
// default).  Same-box A/B against per-wave token loads, gate/up and down (us):
//   bf16  DeepSeek T=32 M=48  469 / 262 -> 460 / 258   M=24  250 / 165 -> 245 / 138
//         Qwen M=32            64 /  40 ->  53 /  32   DeepSeek T=8  236 / 132 -> 237 / 132
//   FP8   DeepSeek T=32 M=48  249 / 147 -> 249 / 138   speculative  371 / 209 -> 329 / 189
//   MXFP4 DeepSeek T=32 M=48  193 / 142 -> 170 /  99   Qwen M=32     44 /  32 ->  25 /  19
// A staged down pass rotates its start by block, not by wave (the waves of a block share
// one token step).
#ifndef XS_STAGE_GATE_UP
#define XS_STAGE_GATE_UP 7
#endif
#ifndef XS_STAGE_DOWN
#define XS_STAGE_DOWN 7
#endif
constexpr bool stage_gate_up(int kW, int U) { return ((XS_STAGE_GATE_UP >> kW) & 1) && U >= 2; }
constexpr bool stage_down(int kW) { return (XS_STAGE_DOWN >> kW) & 1; }

// Work of grid row `slot` of the expert GEMMs: the always-on shared experts first (all T
// tokens, rows T*k + s*T + t; their blocks are the longest, so they start first and do
// not trail the launch), then the routed active experts (their tokens' rows in permuted
// order).  False for rows beyond both.  `e` is the shared or the routed expert.
struct SlotWork {
  int e, p0, te;
  bool shared;
};

__device__ __forceinline__ bool slot_work(const FfnArgs& a, int slot, SlotWork& w) {
  if (slot < a.n_shared) {
    w.e = slot;
    w.p0 = a.T * a.k + slot * a.T;
    w.te = a.T;
    w.shared = true;
    return true;
  }
  const int r = slot - a.n_shared;
  // both loads are issued together; the record is used only below the count
  const int n_active = a.counters[kCntActive];
  const int4 rec = a.active[r < a.N ? r : 0];
  if (r >= n_active) return false;
  w.e = rec.x;
  w.p0 = rec.y;
  w.te = rec.z;
  w.shared = false;
  return true;
}

// The slot's bf16 weight matrix (routed or shared), or its FP8 codes (routed only).
__device__ __forceinline__ const uint16_t* slot_w(const FfnArgs& a, const SlotWork& w,
                                                  const uint16_t* routed,
                                                  const uint16_t* shared) {
  return (w.shared ? shared : routed) + (size_t)w.e * a.f * a.d;
}
__device__ __forceinline__ const uint8_t* slot_q(const FfnArgs& a, const SlotWork& w,
                                                 const uint8_t* codes) {
  return codes + (size_t)w.e * a.f * a.d;
}

// kSplit: the block covers one part of the reduction (blockIdx.z) and writes fp32 gate and
// up partials; otherwise it covers all of d and writes H directly.
// CT: column tiles (16 weight rows of W1 and of W3 each) per wave; with two, one token load
// feeds four weight tiles instead of two, at the cost of registers and of half as many
// blocks (the launch takes two only for grids that stay large).
// The MXFP4 one-tile instance is held to 168 registers (3 waves per SIMD): left alone the
// compiler took 175 and 2 waves, and DeepSeek T=8 gate/up ran 14 % slower.  So are the FP8
// instances of up to 4 words a step (XS_Q8_GU_W3).
template <int U, bool kSplit, int kW, int CT>
__global__ __attribute__((amdgpu_waves_per_eu((kW == kMx4 && CT == 1) ||
                                               (kW == kFp8 && U <= 4 && XS_Q8_GU_W3) ? 3 : 1)))
__launch_bounds__(kBlock) void gate_up_kernel(FfnArgs a) {
  constexpr int NM = 2 * CT;                   // weight tiles: W1 and W3 of each column tile
  SlotWork sw;
  if (!slot_work(a, a.slot_base + blockIdx.y, sw)) return;
  XS_TIME(xs_times_gu, 2 * block_id3(), 2u * kTimeBlocks);
  const int p0 = sw.p0, te = sw.te;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j0 = (blockIdx.x * kWaves + wave) * kCols * CT;
  // a staged pass needs the whole block: a wave past f stays for the staging and the
  // barriers (its columns are clamped into range and its stores skipped)
  constexpr bool kStaged = stage_gate_up(kW, U);
  if (!kStaged && j0 >= a.f) return;
  const int n = lane & 15, g = lane >> 4;
  const int d = a.d, f = a.f;
  const int Kg = kSplit ? d / a.gu_splits : d;   // this block's part of the reduction
  const size_t kbase = kSplit ? (size_t)blockIdx.z * Kg : 0;
  const size_t k0 = kbase + (size_t)(kW == kBf16 ? klane<U>(g) : g * 8 * U);
  const size_t plane = (size_t)a.part_rows * f;   // one fp32 partial plane [part_rows, f]
  int col[CT];                                 // this lane's column of each tile (< f)
  float sc[NM];                                // FP8 per-row scales (else 1)
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    col[ct] = min(j0 + 16 * ct, f - 16) + n;
    sc[2 * ct] = kW == kFp8 ? a.s1[(size_t)sw.e * f + col[ct]] : 1.0f;
    sc[2 * ct + 1] = kW == kFp8 ? a.s3[(size_t)sw.e * f + col[ct]] : 1.0f;
  }

  for (int c0 = 0; c0 < te; c0 += 16 * kTiles) {
    const int nt = min(kTiles, (te - c0 + 15) / 16);
    const uint16_t* arow[kTiles];
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt) {
      const int t = min(c0 + rt * 16 + n, te - 1);
      const int tok = sw.shared ? t : a.perm[p0 + t] / a.k;
      arow[rt] = a.x + (size_t)tok * d + k0;
    }
    floatx4 acc[NM][kTiles];
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int rt = 0; rt < kTiles; ++rt) acc[m][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    if constexpr (kStaged) {
      typename WTile<kW, U>::Ptr wp[NM];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const size_t wrow = (size_t)col[ct] * d + k0;
        if constexpr (kW == kBf16) {
          wp[2 * ct].w = slot_w(a, sw, a.w1, a.sw1) + wrow;
          wp[2 * ct + 1].w = slot_w(a, sw, a.w3, a.sw3) + wrow;
        } else if constexpr (kW == kFp8) {
          wp[2 * ct].w = slot_q(a, sw, a.q1) + wrow;
          wp[2 * ct + 1].w = slot_q(a, sw, a.q3) + wrow;
        } else {        // row col of the expert: d / 2 code bytes; its tiled scale row
          const size_t r = (size_t)sw.e * f + col[ct];
          const int G = mx_granules(d);
          const size_t emat = (size_t)sw.e * f * G * 8;     // the expert's scale matrix
          wp[2 * ct] = {a.q1 + r * (d / 2) + k0 / 2, mx_row(a.e1 + emat, col[ct], G), (int)k0};
          wp[2 * ct + 1] = {a.q3 + r * (d / 2) + k0 / 2, mx_row(a.e3 + emat, col[ct], G),
                            (int)k0};
        }
      }
      __shared__ __align__(16) uint16_t stage[Stage<U, false>::kElems];
      __shared__ int s_tok[kStageRows];
      const int R = min(kStageRows, te - c0);
      if (threadIdx.x < R)
        s_tok[threadIdx.x] = sw.shared ? c0 + threadIdx.x : a.perm[p0 + c0 + threadIdx.x] / a.k;
      __syncthreads();
      staged_pass<kW, U, false, NM, kTiles>(a.x + kbase, d, s_tok, R, wp, Kg, 0, acc, stage);
    } else if constexpr (kW == kFp8) {
      const uint8_t* brow[NM];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const size_t wrow = (size_t)col[ct] * d + k0;
        brow[2 * ct] = slot_q(a, sw, a.q1) + wrow;
        brow[2 * ct + 1] = slot_q(a, sw, a.q3) + wrow;
      }
      wave_pass_q8<U, NM>(arow, nt, brow, Kg, acc);
    } else if constexpr (kW == kMx4) {
      // row col of the expert: d / 2 code bytes; its tiled scale row
      const uint8_t* brow[NM];
      const uint8_t* srow[NM];
      const int G = mx_granules(d);
      const size_t emat = (size_t)sw.e * f * G * 8;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const size_t r = (size_t)sw.e * f + col[ct];
        brow[2 * ct] = a.q1 + r * (d / 2) + k0 / 2;
        brow[2 * ct + 1] = a.q3 + r * (d / 2) + k0 / 2;
        srow[2 * ct] = mx_row(a.e1 + emat, col[ct], G);
        srow[2 * ct + 1] = mx_row(a.e3 + emat, col[ct], G);
      }
      wave_pass_q4<U, NM>(arow, nt, brow, srow, (int)k0, Kg, acc);
    } else {
      const uint16_t* brow[NM];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const size_t wrow = (size_t)col[ct] * d + k0;
        brow[2 * ct] = slot_w(a, sw, a.w1, a.sw1) + wrow;
        brow[2 * ct + 1] = slot_w(a, sw, a.w3, a.sw3) + wrow;
      }
      wave_pass<U, NM, XS_GATE_UP_ADBL != 0>(arow, nt, brow, Kg, acc);
    }
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt) {
      if (rt >= nt) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = c0 + rt * 16 + 4 * g + i;
        if (t < te) {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            if (j0 + 16 * ct >= f) break;
            const float h1 = acc[2 * ct][rt][i] * sc[2 * ct];
            const float h3 = acc[2 * ct + 1][rt][i] * sc[2 * ct + 1];
            if (!kSplit) {
              store_hilo(a.h, p0 + t, col[ct], f, h1 / (1.0f + __expf(-h1)) * h3);
            } else {
              // the tail's planes hold its slots' rows only
              const size_t prow = a.part_compact ? (size_t)blockIdx.y * a.T + t : (size_t)(p0 + t);
              const size_t at = prow * f + col[ct];
              float* const part = a.gpart + 2 * blockIdx.z * plane;
              part[at] = h1;
              part[plane + at] = h3;
            }
          }
        }
      }
    }
  }
  XS_TIME(xs_times_gu, 2 * block_id3() + 1, 2u * kTimeBlocks);
}

// NM: 16-row W2 tiles per wave (the launch picks it per weight format and batch shape).
// Staged down instances are held to 2 waves per SIMD: left alone the compiler took 1 for the
// 64-row bf16 and FP8 instances (FP8 DeepSeek T=32 down 166 -> 138 us with the hint).
// TL: token tiles per pass, 8 tokens each (hi and lo rows).
template <int U, int kW, int NM, int TL = XS_DOWN_TL>
__global__ __attribute__((amdgpu_waves_per_eu(stage_down(kW) && NM <= 4 ? XS_DOWN_WAVES_PER_EU
                                                                          : 1)))
__launch_bounds__(kBlock) void down_kernel(FfnArgs a) {
  // (bx, slot): this block's column block and expert slot.  In grids of at least
  // XS_DOWN_XCD_SLOTS slots, with `live` slots holding work (shared, then active), all
  // column blocks of slot y < 8 * (live / 8) run on XCD y mod 8 (the dispatcher deals
  // consecutive workgroups to the 8 XCDs in turn), so one L2 serves the slot's H rows to
  // all of them; the blocks of the other slots keep the plain order, which spreads the
  // last live % 8 slots over all XCDs.
  int bx = blockIdx.x, slot = blockIdx.y;
  if (gridDim.y >= XS_DOWN_XCD_SLOTS) {
    const int L = blockIdx.x + gridDim.x * blockIdx.y;
    const int live = a.n_shared + a.counters[kCntActive];   // <= gridDim.y
    if (L < (int)gridDim.x * (live & ~7)) {
      const int s = L >> 3;
      slot = (L & 7) + 8 * (s / gridDim.x);
      bx = s % gridDim.x;
    }
  }
  SlotWork sw;
  if (!slot_work(a, slot, sw)) return;
  XS_TIME(xs_times_dn, 2 * block_id3(), 2u * kTimeBlocks);
  const int p0 = sw.p0, te = sw.te;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = (bx * kWaves + wave) * kCols * NM;
  // a staged pass needs the whole block (see gate_up_kernel)
  constexpr bool kStaged = stage_down(kW);
  if (!kStaged && n0 >= a.d) return;
  const int n = lane & 15, g = lane >> 4;
  const int d = a.d, f = a.f;
  const int Ks = f / a.splits;                 // this block's part of the reduction
  const size_t k0 = (size_t)blockIdx.z * Ks + (size_t)(kW == kBf16 ? klane<U>(g) : g * 8 * U);
  float* const ypart = a.yslot + (size_t)blockIdx.z * a.rows * d;
  const int lo_off = n < 8 ? 0 : 8;                    // A rows 0-7: hi, rows 8-15: lo
  size_t wrow[NM];
  int rowm[NM];
  float sc[NM];                                        // FP8 per-row scales (else 1)
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    rowm[m] = min(n0 + 16 * m, d - 16) + n;
    wrow[m] = (size_t)rowm[m] * f + k0;
    sc[m] = kW == kFp8 ? a.s2[(size_t)sw.e * d + rowm[m]] : 1.0f;
  }

  for (int c0 = 0; c0 < te; c0 += 8 * TL) {
    const int nt = min(TL, (te - c0 + 7) / 8);
    const uint16_t* arow[TL];
#pragma unroll
    for (int rt = 0; rt < TL; ++rt) {
      const int t = min(c0 + rt * 8 + (n & 7), te - 1);
      arow[rt] = a.h + (size_t)(p0 + t) * 2 * f + 2 * k0 + lo_off;
    }
    floatx4 acc[NM][TL];
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int rt = 0; rt < TL; ++rt) acc[m][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    // Consecutive waves start their pass over K one step apart (and wrap around): W2 rows
    // are f elements apart, often a power of two, so waves that stepped through K in the
    // same order would read the same offsets of every row at the same time.
    const int rot = kW == kBf16 ? XS_DOWN_ROT : (kW == kFp8 ? XS_Q8_DOWN_ROT : XS_Q4_DOWN_ROT);
    const int k_first = (int)(((bx * kWaves + wave) * rot) % (Ks / (32 * U))) * 32 * U;
    if constexpr (kStaged) {
      static_assert(TL == 2 || TL == 4, "the staged pass takes two or four 8-token tiles");
      typename WTile<kW, U>::Ptr wp[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        if constexpr (kW == kBf16) {
          wp[m].w = slot_w(a, sw, a.w2, a.sw2) + wrow[m];
        } else if constexpr (kW == kFp8) {
          wp[m].w = slot_q(a, sw, a.q2) + wrow[m];
        } else {         // f / 2 code bytes of row rowm; its tiled scale row
          const size_t r = (size_t)sw.e * d + rowm[m];
          const int G = mx_granules(f);
          wp[m] = {a.q2 + r * (f / 2) + k0 / 2,
                   mx_row(a.e2 + (size_t)sw.e * d * G * 8, rowm[m], G), (int)k0};
        }
      }
      __shared__ __align__(16) uint16_t stage[Stage<U, true>::kElems];
      __shared__ int s_tok[kStageRows];
      const int R = min(8 * TL, te - c0);
      if (threadIdx.x < R) s_tok[threadIdx.x] = p0 + c0 + threadIdx.x;   // H rows
      __syncthreads();
      // staged: consecutive blocks, not waves, start their pass `rot` steps apart
      const int kb_first = (int)((bx * rot) % (Ks / (32 * U))) * 32 * U;
      staged_pass<kW, U, true, NM, TL>(a.h + 2 * (size_t)blockIdx.z * Ks, 2 * (size_t)f, s_tok, R,
                                       wp, Ks, kb_first, acc, stage);
    } else if constexpr (kW == kFp8) {
      const uint8_t* brow[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) brow[m] = slot_q(a, sw, a.q2) + wrow[m];
      wave_pass_q8<U, NM, TL, 2>(arow, nt, brow, Ks, acc, k_first);
    } else if constexpr (kW == kMx4) {
      const uint8_t* brow[NM];
      const uint8_t* srow[NM];
      const int G = mx_granules(f);
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const size_t r = (size_t)sw.e * d + rowm[m];      // f / 2 code bytes; tiled scale row
        brow[m] = a.q2 + r * (f / 2) + k0 / 2;
        srow[m] = mx_row(a.e2 + (size_t)sw.e * d * G * 8, rowm[m], G);
      }
      wave_pass_q4<U, NM, TL, 2>(arow, nt, brow, srow, (int)k0, Ks, acc, k_first);
    } else {
      const uint16_t* brow[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) brow[m] = slot_w(a, sw, a.w2, a.sw2) + wrow[m];
      wave_pass<U, NM, XS_DOWN_ADBL != 0, TL, 2>(arow, nt, brow, Ks, acc, k_first);
    }
#pragma unroll
    for (int rt = 0; rt < TL; ++rt) {
      if (rt >= nt) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // lanes g = 0, 1 hold the hi rows of tokens 4g + i, lanes 32 above them the lo rows
        float v[NM];
#pragma unroll
        for (int m = 0; m < NM; ++m)
          v[m] = (acc[m][rt][i] + __shfl_xor(acc[m][rt][i], 32, 64)) * sc[m];
        const int t = c0 + rt * 8 + 4 * g + i;
        if (g < 2 && t < te) {
          // routed rows go to their (token, slot) row, shared rows keep their own
          float* yrow = ypart + (size_t)(sw.shared ? p0 + t : a.perm[p0 + t]) * d;
#pragma unroll
          for (int m = 0; m < NM; ++m)
            if (n0 + 16 * m < d) yrow[n0 + 16 * m + n] = v[m];
        }
      }
    }
  }
  XS_TIME(xs_times_dn, 2 * block_id3() + 1, 2u * kTimeBlocks);
}

// ---- Persistent down GEMM, for launches of whole rounds with one block per CU (the
// seven-tile bf16 waves).  Such a launch runs its rounds in lock step: the blocks of a round
// stream the same bytes, so they end together, and every CU then spends the next block's
// start (dispatch, its slot record, then the first weight loads) with no reads in flight, at
// the same moment.  Here the grid holds one block per CU and each block walks a fixed list
// of work units: units b, b + G, b + 2G, ... (G blocks), a unit being one column block of
// one expert slot, taken in passes of up to 8 * TL token rows.  The block reads its units'
// slot records once, into LDS; the first step's loads of its next pass are issued in the
// last step of the current one, so a CU's weight stream does not drain between units.  The
// MFMAs always cover TL token tiles (one code path for every pass; rows past the pass repeat
// its last row and are not stored).  Units map to (slot, column block) as in down_kernel's
// grid, so with G a multiple of 8 every unit of a slot below 8 * (live / 8) runs on the XCD
// of that slot.  Blocks share nothing: no counters, no flags, no block waits for another.
constexpr int kSeqUnits = 32;     // units per block of a persistent launch, at most
static_assert(kTimeSeqStride == 1 + kSeqUnits, "a stamp per unit of a persistent block");

__device__ __forceinline__ void down_unit(int L, int CB, int live, bool xcd, int& slot, int& bx) {
  if (xcd && L < CB * (live & ~7)) {
    const int s = L >> 3;
    slot = (L & 7) + 8 * (s / CB);
    bx = s % CB;
  } else {
    slot = L / CB;
    bx = L % CB;
  }
}

// Lane state of one pass that its loads need: weight pointers, token pieces and the pass's
// first reduction step.
template <int kW, int U, int NM, int NLM>
struct DnLoads {
  typename WTile<kW, U>::Ptr wp[NM];
  const uint16_t* src[NLM];
  int wofs[NLM];
  int kb;
};

// A pass: unit record {expert | shared << 30, first permuted row, rows, column block} and
// the pass's first row.
struct DnPass {
  int4 rec;
  int c0;
  __device__ int e() const { return rec.x & 0x3FFFFFFF; }
  __device__ bool shared() const { return (rec.x >> 30) & 1; }
};

template <int kW, int U, int NM, int NLM, int TL>
__device__ __forceinline__ void dn_loads(const FfnArgs& a, const DnPass& ps, int wave, int n,
                                         size_t kl, int nsteps, int rot,
                                         DnLoads<kW, U, NM, NLM>& L) {
  using S = Stage<U, true>;
  const int d = a.d, f = a.f;
  const int bx = ps.rec.w, p0 = ps.rec.y, te = ps.rec.z;
  const int n0 = (bx * kWaves + wave) * kCols * NM;
  const size_t ebase = (size_t)ps.e() * d * f;
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    const size_t wrow = (size_t)(min(n0 + 16 * m, d - 16) + n) * f + kl;
    if constexpr (kW == kBf16) L.wp[m].w = (ps.shared() ? a.sw2 : a.w2) + ebase + wrow;
    else L.wp[m].w = a.q2 + ebase + wrow;
  }
  const int R = max(1, min(8 * TL, te - ps.c0));
#pragma unroll
  for (int i = 0; i < NLM; ++i) {
    const int q = min((int)threadIdx.x + i * kBlock, R * S::P - 1);
    const int row = q / S::P, piece = q % S::P;
    L.src[i] = a.h + (size_t)(p0 + ps.c0 + row) * 2 * f + piece * 8;
    L.wofs[i] = row * S::LS + piece * 8;
  }
  L.kb = ((bx * rot) % nsteps) * S::KB;
}

template <int U, int kW, int NM, int TL>
__global__ __attribute__((amdgpu_waves_per_eu(NM <= 4 ? XS_DOWN_WAVES_PER_EU : 1)))
__launch_bounds__(kBlock) void down_seq_kernel(FfnArgs a) {
  using S = Stage<U, true>;
  using WT = WTile<kW, U>;
  static_assert(kW != kMx4, "bf16 and FP8 weights");
  constexpr int KB = S::KB;
  constexpr int NLM = (TL * S::TR * S::P + kBlock - 1) / kBlock;
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n = lane & 15, g = lane >> 4;
  const int d = a.d, f = a.f;
  const int CB = (d + kWaves * kCols * NM - 1) / (kWaves * kCols * NM);
  const int live = a.n_shared + a.counters[kCntActive];
  const int units = live * CB;
  const int G = (int)gridDim.x;
  const int nu = (int)blockIdx.x < units ? min((units - (int)blockIdx.x + G - 1) / G, kSeqUnits) : 0;
  if (nu == 0) return;   // uniform: the whole block leaves before any barrier
  XS_TIME(xs_times_seq, blockIdx.x * kTimeSeqStride, (unsigned)(kTimeSeqBlocks * kTimeSeqStride));
  const bool xcd = a.max_active + a.n_shared >= XS_DOWN_XCD_SLOTS;
  const int nsteps = f / KB;                    // unsplit: the launch takes one K part
  const int rot = kW == kBf16 ? XS_DOWN_ROT : XS_Q8_DOWN_ROT;
  const size_t kl = (size_t)(kW == kBf16 ? klane<U>(g) : g * 8 * U);

  // the block's unit records, one thread each
  __shared__ int4 s_rec[kSeqUnits];
  if (tid < nu) {
    int slot, bx;
    down_unit((int)blockIdx.x + tid * G, CB, live, xcd, slot, bx);
    SlotWork sw;
    const bool ok = slot_work(a, slot, sw);   // slot < live: always work
    s_rec[tid] = ok ? make_int4(sw.e | (sw.shared ? 1 << 30 : 0), sw.p0, sw.te, bx)
                    : make_int4(0, 0, 0, bx);
  }
  __syncthreads();

  int j = 0;                                    // current unit
  DnPass cur{s_rec[0], 0};
  __shared__ __align__(16) uint16_t lds[S::kElems];
  DnLoads<kW, U, NM, NLM> L;
  dn_loads<kW, U, NM, NLM, TL>(a, cur, wave, n, kl, nsteps, rot, L);

  u32x4 v[NLM];
  typename WT::Regs b[NM];
#pragma unroll
  for (int i = 0; i < NLM; ++i) v[i] = *reinterpret_cast<const u32x4*>(L.src[i] + S::AS * L.kb);
#pragma unroll
  for (int m = 0; m < NM; ++m) b[m] = WT::load(L.wp[m], L.kb);
#pragma unroll
  for (int i = 0; i < NLM; ++i) *reinterpret_cast<u32x4*>(lds + L.wofs[i]) = v[i];
  __syncthreads();

  floatx4 acc[NM][TL];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int rt = 0; rt < TL; ++rt) acc[m][rt] = floatx4{0.f, 0.f, 0.f, 0.f};

  int buf = 0;
  // MFMAs of one step from LDS buffer `buf`: all TL tiles (rows past the pass repeat its last
  // row; their sums are not stored), so every pass runs the same code
  auto mfma_step = [&](const int (&rofs)[TL]) {
    const uint16_t* const cl = lds + buf * kStageRows * S::LS;
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      const int ka = S::AS * WT::koff(g, uu);
      bf16x8 xa[TL];
#pragma unroll
      for (int rt = 0; rt < TL; ++rt) xa[rt] = *reinterpret_cast<const bf16x8*>(cl + rofs[rt] + ka);
#pragma unroll
      for (int rt = 0; rt < TL; ++rt)
#pragma unroll
        for (int m = 0; m < NM; ++m) acc[m][rt] = mfma(xa[rt], WT::operand(b[m], uu), acc[m][rt]);
    }
  };
  while (true) {
    const int te = cur.rec.z, p0 = cur.rec.y;
    const int R = max(1, min(8 * TL, te - cur.c0));
    const int nt = (R + 7) >> 3;
    const int n0 = (cur.rec.w * kWaves + wave) * kCols * NM;
    int rofs[TL];
#pragma unroll
    for (int rt = 0; rt < TL; ++rt) rofs[rt] = min(8 * rt + (n & 7), R - 1) * S::LS + (n & 8);
    // every step but the last: loads of the next step, MFMAs of this one
    for (int ks = 0; ks < nsteps - 1; ++ks) {
      int kn = L.kb + KB;
      if (kn >= f) kn -= f;
#pragma unroll
      for (int i = 0; i < NLM; ++i) v[i] = *reinterpret_cast<const u32x4*>(L.src[i] + S::AS * kn);
      typename WT::Regs nb[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) nb[m] = WT::load(L.wp[m], kn);
      mfma_step(rofs);
      uint16_t* const nl = lds + (buf ^ 1) * kStageRows * S::LS;
#pragma unroll
      for (int i = 0; i < NLM; ++i) *reinterpret_cast<u32x4*>(nl + L.wofs[i]) = v[i];
#pragma unroll
      for (int m = 0; m < NM; ++m) b[m] = nb[m];
      __syncthreads();
      buf ^= 1;
      L.kb = kn;
    }
    // the last step: the loads of the block's next pass (the unit's next rows, else its next
    // unit; after the block's last pass the same loads again), then this step's MFMAs and the
    // pass's epilogue
    DnPass nxt = cur;
    int jn = j;
    bool has_nxt = true;
    if (cur.c0 + 8 * TL < te) {
      nxt.c0 += 8 * TL;
    } else {
      jn = j + 1;
      has_nxt = jn < nu;
      if (has_nxt) nxt = DnPass{s_rec[jn], 0};
    }
    DnLoads<kW, U, NM, NLM> Ln = L;
    if (has_nxt) dn_loads<kW, U, NM, NLM, TL>(a, nxt, wave, n, kl, nsteps, rot, Ln);
    int yrow[TL][4];
#pragma unroll
    for (int rt = 0; rt < TL; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = max(0, min(cur.c0 + rt * 8 + 4 * (g & 1) + i, te - 1));
        yrow[rt][i] = cur.shared() ? p0 + t : a.perm[p0 + t];
      }
    float sc[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m)
      sc[m] = kW == kFp8 ? a.s2[(size_t)cur.e() * d + min(n0 + 16 * m, d - 16) + n] : 1.0f;
#pragma unroll
    for (int i = 0; i < NLM; ++i) v[i] = *reinterpret_cast<const u32x4*>(Ln.src[i] + S::AS * Ln.kb);
    typename WT::Regs nb[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) nb[m] = WT::load(Ln.wp[m], Ln.kb);
    mfma_step(rofs);
    // lanes g = 0, 1 hold the hi rows of tokens 4g + i, lanes 32 above them the lo rows;
    // routed rows go to their (token, slot) row, shared rows keep their own
#pragma unroll
    for (int rt = 0; rt < TL; ++rt) {
      if (rt >= nt) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float o[NM];
#pragma unroll
        for (int m = 0; m < NM; ++m)
          o[m] = (acc[m][rt][i] + __shfl_xor(acc[m][rt][i], 32, 64)) * sc[m];
        const int t = cur.c0 + rt * 8 + 4 * g + i;
        if (g < 2 && t < te) {
          float* const yr = a.yslot + (size_t)yrow[rt][i] * d;
#pragma unroll
          for (int m = 0; m < NM; ++m)
            if (n0 + 16 * m < d) yr[n0 + 16 * m + n] = o[m];
        }
      }
    }
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int rt = 0; rt < TL; ++rt) acc[m][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    uint16_t* const nl = lds + (buf ^ 1) * kStageRows * S::LS;
#pragma unroll
    for (int i = 0; i < NLM; ++i) *reinterpret_cast<u32x4*>(nl + Ln.wofs[i]) = v[i];
#pragma unroll
    for (int m = 0; m < NM; ++m) b[m] = nb[m];
    __syncthreads();
    buf ^= 1;
    if (jn != j)
      XS_TIME(xs_times_seq, blockIdx.x * kTimeSeqStride + 1 + j,
              (unsigned)(kTimeSeqBlocks * kTimeSeqStride));
    if (!has_nxt) break;
    cur = nxt;
    j = jn;
    L = Ln;
  }
}

// Sums the gate and up partials of hidden element c..c+3 of partial row `prow` in split
// order, then H[hrow] = silu(gate) * up as bf16 hi and lo.
__device__ __forceinline__ void finish_row(const FfnArgs& a, size_t prow, size_t hrow, int c) {
  const size_t plane = (size_t)a.part_rows * a.f;
  const size_t at = prow * a.f + c;
  float4 gs = *reinterpret_cast<const float4*>(a.gpart + at);
  float4 us = *reinterpret_cast<const float4*>(a.gpart + plane + at);
  for (int z = 1; z < a.gu_splits; ++z) {
    const float4 gz = *reinterpret_cast<const float4*>(a.gpart + 2 * z * plane + at);
    const float4 uz = *reinterpret_cast<const float4*>(a.gpart + (2 * z + 1) * plane + at);
    gs.x += gz.x; gs.y += gz.y; gs.z += gz.z; gs.w += gz.w;
    us.x += uz.x; us.y += uz.y; us.z += uz.z; us.w += uz.w;
  }
  store_hilo(a.h, hrow, c + 0, a.f, gs.x / (1.0f + __expf(-gs.x)) * us.x);
  store_hilo(a.h, hrow, c + 1, a.f, gs.y / (1.0f + __expf(-gs.y)) * us.y);
  store_hilo(a.h, hrow, c + 2, a.f, gs.z / (1.0f + __expf(-gs.z)) * us.z);
  store_hilo(a.h, hrow, c + 3, a.f, gs.w / (1.0f + __expf(-gs.w)) * us.w);
}

// Split gate/up reduction: H for every hidden row from its partials.  Block row y takes
// hidden rows y, y + gridDim.y, ... (the grid keeps at most 65535 rows); routed rows beyond
// the routed count, and rows whose expert the GEMMs did not cover (another GPU group's),
// are skipped.
__global__ __launch_bounds__(kBlock) void gate_up_finish_kernel(FfnArgs a) {
  const int c = (blockIdx.x * kBlock + threadIdx.x) * 4;
  if (c >= a.f) return;
  for (long p = blockIdx.y; p < a.rows; p += gridDim.y) {
    const bool shared_row = p >= (long)a.T * a.k;
    if (!shared_row && p >= a.offsets[a.N]) continue;
    if (!shared_row && a.local_group >= 0) {
      const int e = a.ids[a.perm[p]];
      if ((a.group ? a.group[e] : e / (a.N / a.G)) != a.local_group) continue;
    }
    finish_row(a, (size_t)p, (size_t)p, c);
  }
}

// The finish pass of the gate/up tail: block row y is partial row y of the tail's compact
// planes, token y % T of slot slot_base + y / T (at most T rows a slot: a token takes an
// expert once; a shared expert takes every token).
__global__ __launch_bounds__(kBlock) void gate_up_tail_finish_kernel(FfnArgs a) {
  SlotWork sw;
  if (!slot_work(a, a.slot_base + blockIdx.y / a.T, sw)) return;
  const int t = blockIdx.y % a.T;
  if (t >= sw.te) return;
  const int c = (blockIdx.x * kBlock + threadIdx.x) * 4;
  if (c >= a.f) return;
  finish_row(a, blockIdx.y, (size_t)(sw.p0 + t), c);
}

__global__ __launch_bounds__(kBlock) void combine_kernel(FfnArgs a) {
  const int i = blockIdx.y;
  const int c = (blockIdx.x * kBlock + threadIdx.x) * 4;
  if (c >= a.d) return;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  // kR ranks at a time: their ids, weights and rows are loaded together (the rows of the
  // ranks that turn out unused, empty slots and other GPU groups' experts, hold stale
  // values and are left out of the sums), so a group costs one round trip; the sums keep
  // rank order and, per rank, split order
  constexpr int kR = 8;
  for (int r0 = 0; r0 < a.k; r0 += kR) {
    int e[kR];
    float wr[kR];
    float4 v[kR];
#pragma unroll
    for (int j = 0; j < kR; ++j) {
      const bool in = r0 + j < a.k;
      e[j] = in ? a.ids[i * a.k + r0 + j] : -1;
      wr[j] = in ? a.w[i * a.k + r0 + j] : 0.0f;
      v[j] = *reinterpret_cast<const float4*>(a.yslot +
                                              (size_t)(i * a.k + min(r0 + j, a.k - 1)) * a.d + c);
    }
    bool use[kR];
#pragma unroll
    for (int j = 0; j < kR; ++j)
      use[j] = e[j] >= 0 &&   // another GPU group's terms of y_i are left out
               (a.local_group < 0 ||
                (a.group ? a.group[e[j]] : e[j] / (a.N / a.G)) == a.local_group);
    for (int s = 1; s < a.splits; ++s) {   // partial sums of a split reduction, in order
#pragma unroll
      for (int j = 0; j < kR; ++j) {
        if (!use[j]) continue;
        const float4 u = *reinterpret_cast<const float4*>(
            a.yslot + ((size_t)s * a.rows + i * a.k + r0 + j) * a.d + c);
        v[j].x += u.x;
        v[j].y += u.y;
        v[j].z += u.z;
        v[j].w += u.w;
      }
    }
#pragma unroll
    for (int j = 0; j < kR; ++j) {
      if (!use[j]) continue;
      acc[0] += wr[j] * v[j].x;
      acc[1] += wr[j] * v[j].y;
      acc[2] += wr[j] * v[j].z;
      acc[3] += wr[j] * v[j].w;
    }
  }
  for (int sh = 0; sh < a.n_shared; ++sh) {  // shared experts, weight 1, after the routed terms
    const size_t row = (size_t)a.T * a.k + (size_t)sh * a.T + i;
    float4 v = *reinterpret_cast<const float4*>(a.yslot + row * a.d + c);
    for (int s = 1; s < a.splits; ++s) {
      const float4 u = *reinterpret_cast<const float4*>(
          a.yslot + ((size_t)s * a.rows + row) * a.d + c);
      v.x += u.x;
      v.y += u.y;
      v.z += u.z;
      v.w += u.w;
    }
    acc[0] += v.x;
    acc[1] += v.y;
    acc[2] += v.z;
    acc[3] += v.w;
  }
  const uint32_t lo = (uint32_t)to_bf16(acc[0]) | ((uint32_t)to_bf16(acc[1]) << 16);
  const uint32_t hi = (uint32_t)to_bf16(acc[2]) | ((uint32_t)to_bf16(acc[3]) << 16);
  *reinterpret_cast<uint2*>(a.y + (size_t)i * a.d + c) = make_uint2(lo, hi);
}

// Router GEMM h = W_g x: each wave owns 16 router rows (experts) and part blockIdx.z of d,
// for the token tiles of blockIdx.y; fp32 results go to that part's plane.
template <int U>
__global__ __launch_bounds__(kBlock) void router_kernel(RouterArgs r) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j0 = (blockIdx.x * kWaves + wave) * kCols;
  if (j0 >= r.N) return;
  const int n = lane & 15, g = lane >> 4;
  const int Kp = r.d / r.parts;
  const size_t k0 = (size_t)blockIdx.z * Kp + (size_t)klane<U>(g);
  const uint16_t* const brow[1] = {r.wg + (size_t)min(j0 + n, r.N - 1) * r.d + k0};
  float* const out = r.planes + (size_t)blockIdx.z * r.T * r.N;
  for (int c0 = blockIdx.y * 16 * kTiles; c0 < r.T; c0 += gridDim.y * 16 * kTiles) {
    const int nt = min(kTiles, (r.T - c0 + 15) / 16);
    const uint16_t* arow[kTiles];
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt)
      arow[rt] = r.x + (size_t)min(c0 + rt * 16 + n, r.T - 1) * r.d + k0;
    floatx4 acc[1][kTiles];
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt) acc[0][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    wave_pass<U, 1, true>(arow, nt, brow, Kp, acc);
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt) {
      if (rt >= nt) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = c0 + rt * 16 + 4 * g + i;
        if (t < r.T && j0 + n < r.N) out[(size_t)t * r.N + j0 + n] = acc[0][rt][i];
      }
    }
  }
}

// logits = sum of the router's part planes, in part order.
__global__ __launch_bounds__(kBlock) void router_sum_kernel(RouterArgs r) {
  const size_t idx = (size_t)blockIdx.x * kBlock + threadIdx.x;
  const size_t plane = (size_t)r.T * r.N;
  if (idx >= plane) return;
  float v = r.planes[idx];
  int z = 1;
  for (; z + 8 <= r.parts; z += 8) {   // eight loads in flight, then the adds in order
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = r.planes[(z + u) * plane + idx];
#pragma unroll
    for (int u = 0; u < 8; ++u) v = v + t[u];
  }
  for (; z < r.parts; ++z) v = v + r.planes[z * plane + idx];
  r.logits[idx] = v;
}

int unroll_for(int K, int want);

// Column tiles per wave: two if the expected active blocks stay enough with them.
bool gu_two_tiles(const FfnArgs& a, int kW, unsigned splits) {
  const long min_blocks = kW == kMx4 ? XS_Q4_GU_CT2_MIN_BLOCKS : XS_GU_CT2_MIN_BLOCKS;
  return (long)((a.f + 2 * kWaves * kCols - 1) / (2 * kWaves * kCols)) *
             (a.est_active + a.n_shared) * splits >= min_blocks;
}

// Blocks of the unsplit gate/up instance the GPU runs at once (cached per instance; one
// device type).
template <int U, int kW, int CT>
int resident_blocks() {
  static std::atomic<int> cached{0};   // callers on several threads may fill it at once
  int r = cached.load(std::memory_order_relaxed);
  if (r == 0) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, gate_up_kernel<U, false, kW, CT>,
                                                     kBlock, 0) != hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    r = per_cu * cus;
    cached.store(r, std::memory_order_relaxed);
  }
  return r;
}

// An unsplit gate/up launch of grid (B, S): when its last round of blocks holds slots
// S_main .. S - 1 and under a quarter of the resident blocks, those slots run after the
// main launch, split `ts` ways along d (partials, then their finish pass).  Returns ts (1:
// no tail launch) and S_main.
template <int U>
int gu_tail_split(const FfnArgs& a, dim3 grid, int resident, int& s_main) {
  s_main = (int)grid.y;
  if (a.gu_tail_splits < 2 || a.slot_base != 0 || resident <= 0 || a.T <= 0) return 1;
  const long B = grid.x, S = grid.y;
  const long rounds = S * B / resident;
  if (rounds < 1) return 1;
  const long main_slots = rounds * resident / B;
  const long tail = S - main_slots;
  if (tail <= 0 || 4 * tail * B > resident || tail > XS_GU_TAIL_MAX_SLOTS) return 1;
  if (tail * a.T > 65535) return 1;                 // the finish pass's grid rows
  int ts = 1;
  while (2 * ts <= a.gu_tail_splits && a.d % (2 * ts * 32 * U) == 0 &&
         tail * B * 2 * ts <= resident)
    ts *= 2;
  if (ts < 2) return 1;
  s_main = (int)main_slots;
  return ts;
}

template <int U, int kW, int CT>
void launch_gu_tail(const FfnArgs& a, dim3 grid, int s_main, int ts, hipStream_t stream) {
  FfnArgs t = a;
  t.slot_base = s_main;
  t.gu_splits = ts;
  t.part_rows = (long)gu_tail_rows(a.T);     // compact planes: (slot - s_main) * T + t
  t.part_compact = 1;
  const int tail = (int)grid.y - s_main;
  const dim3 g(grid.x, tail, ts), block(kBlock);
  hipLaunchKernelGGL((gate_up_kernel<U, true, kW, CT>), g, block, 0, stream, t);
  const dim3 fg((a.f + kBlock * 4 - 1) / (kBlock * 4), tail * a.T);
  hipLaunchKernelGGL(gate_up_tail_finish_kernel, fg, block, 0, stream, t);
}

// An unsplit launch, with its last round's slots split off when that pays (see
// gu_tail_split).
template <int U, int kW, int CT>
void launch_gu_unsplit(const FfnArgs& a, dim3 grid, dim3 block, hipStream_t stream) {
  int s_main = 0;
  const int ts = gu_tail_split<U>(a, grid, resident_blocks<U, kW, CT>(), s_main);
  const dim3 g(grid.x, s_main, grid.z);
  if (s_main > 0) hipLaunchKernelGGL((gate_up_kernel<U, false, kW, CT>), g, block, 0, stream, a);
  if (ts > 1) launch_gu_tail<U, kW, CT>(a, grid, s_main, ts, stream);
}

template <int U, int kW>
void launch_gu(const FfnArgs& a, bool split, bool two, dim3 grid, dim3 block,
               hipStream_t stream) {
  if (two) grid.x = (a.f + 2 * kWaves * kCols - 1) / (2 * kWaves * kCols);
  if constexpr (U <= 8) {   // U = 16: one-tile launches only
    if (split && two) {
      hipLaunchKernelGGL((gate_up_kernel<U, true, kW, 2>), grid, block, 0, stream, a);
      return;
    }
    if (two) {
      launch_gu_unsplit<U, kW, 2>(a, grid, block, stream);
      return;
    }
  }
  if (split)
    hipLaunchKernelGGL((gate_up_kernel<U, true, kW, 1>), grid, block, 0, stream, a);
  else
    launch_gu_unsplit<U, kW, 1>(a, grid, block, stream);
}

// Unroll U (a power of two dividing K / 32; at most u2 for two-tile launches, u1 for
// one-tile launches, 16 only for MXFP4) for weight format kW.
template <int kW>
void launch_gu_fmt(const FfnArgs& a, int K, int u2, int u1, bool split, dim3 grid, dim3 block,
                   hipStream_t stream) {
  const bool two = gu_two_tiles(a, kW, grid.z);
  const int u = unroll_for(K, two ? u2 : u1);
  if constexpr (kW == kMx4 && (XS_Q4_GATE_UP_U == 16 || XS_Q4_GATE_UP_U1 == 16)) {
    if (u == 16) {
      launch_gu<16, kW>(a, split, false, grid, block, stream);
      return;
    }
  }
  if (u >= 8)
    launch_gu<8, kW>(a, split, two, grid, block, stream);
  else if (u == 4)
    launch_gu<4, kW>(a, split, two, grid, block, stream);
  else if (u == 2)
    launch_gu<2, kW>(a, split, two, grid, block, stream);
  else
    launch_gu<1, kW>(a, split, two, grid, block, stream);
}
// Blocks of the down instance (unroll u) that the GPU runs at once (cached per instance).
template <int U, int kW, int NM, int TL>
int down_resident_u() {
  static std::atomic<int> cached{0};
  int r = cached.load(std::memory_order_relaxed);
  if (r == 0) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, down_kernel<U, kW, NM, TL>, kBlock,
                                                     0) != hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    r = per_cu * cus;
    cached.store(r, std::memory_order_relaxed);
  }
  return r;
}
template <int kW, int NM, int TL = XS_DOWN_TL>
int down_resident(int u) {
  if (u == 8) return down_resident_u<8, kW, NM, TL>();
  if (u >= 4) return down_resident_u<4, kW, NM, TL>();
  if (u == 2) return down_resident_u<2, kW, NM, TL>();
  return down_resident_u<1, kW, NM, TL>();
}

template <int kW, int NM, int TL = XS_DOWN_TL>
void launch_down_fmt(const FfnArgs& a, int u, hipStream_t stream) {
  const int cols = kWaves * kCols * NM;
  const int slots = a.max_active + a.n_shared;
  const dim3 grid((a.d + cols - 1) / cols, slots, a.splits), block(kBlock);
  if (u == 8) {
    hipLaunchKernelGGL((down_kernel<8, kW, NM, TL>), grid, block, 0, stream, a);
    return;
  }
  if (u >= 4)
    hipLaunchKernelGGL((down_kernel<4, kW, NM, TL>), grid, block, 0, stream, a);
  else if (u == 2)
    hipLaunchKernelGGL((down_kernel<2, kW, NM, TL>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((down_kernel<1, kW, NM, TL>), grid, block, 0, stream, a);
}

// The persistent down launch (down_seq_kernel): one block per resident slot, rounded up to a
// multiple of 8 (one XCD per slot's units) and to at least the unit bound / kSeqUnits.
// False if the instance's residency is unknown.
template <int U, int kW, int NM, int TL = XS_DOWN_TL>
bool launch_down_seq(const FfnArgs& a, hipStream_t stream) {
  static std::atomic<int> cached{0};
  int r = cached.load(std::memory_order_relaxed);
  if (r == 0) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, down_seq_kernel<U, kW, NM, TL>,
                                                     kBlock, 0) != hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        per_cu <= 0)
      return false;
    r = per_cu * cus;
    cached.store(r, std::memory_order_relaxed);
  }
  const int CB = (a.d + kWaves * kCols * NM - 1) / (kWaves * kCols * NM);
  const long max_units = (long)(a.max_active + a.n_shared) * CB;
  long G = std::max<long>(r, (max_units + kSeqUnits - 1) / kSeqUnits);
  G = (G + 7) & ~7L;
  hipLaunchKernelGGL((down_seq_kernel<U, kW, NM, TL>), dim3((unsigned)G), dim3(kBlock), 0, stream,
                     a);
  return true;
}

int unroll_for(int K, int want) {
  for (int u = want; u > 1; u >>= 1)
    if (K % (32 * u) == 0) return u;
  return 1;
}

}  // namespace

hipError_t launch_gate_up(const FfnArgs& a, hipStream_t stream) {
  const int cols = kWaves * kCols;            // one column tile per wave; launch_gu may take two
  const dim3 grid((a.f + cols - 1) / cols, a.max_active + a.n_shared, a.gu_splits),
      block(kBlock);
  const bool split = a.gu_splits > 1;
  const int K = a.d / a.gu_splits;
  if (a.wfmt == kFp8)
    launch_gu_fmt<kFp8>(a, K, XS_Q8_GATE_UP_U, XS_Q8_GATE_UP_U1, split, grid, block, stream);
  else if (a.wfmt == kMx4)
    launch_gu_fmt<kMx4>(a, K, XS_Q4_GATE_UP_U, XS_Q4_GATE_UP_U1, split, grid, block, stream);
  else
    launch_gu_fmt<kBf16>(a, K, XS_GATE_UP_U, XS_GATE_UP_U1, split, grid, block, stream);
  if (split) {
    const dim3 fgrid((a.f + kBlock * 4 - 1) / (kBlock * 4), (unsigned)std::min(a.rows, 65535L));
    hipLaunchKernelGGL(gate_up_finish_kernel, fgrid, block, 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_down(const FfnArgs& a, hipStream_t stream) {
  const int K = a.f / a.splits;
  const long est = a.est_active + a.n_shared;
  if (a.wfmt == kMx4) {
    // twice the rows per wave (twice the weight bytes in flight) over 16-token passes, when
    // experts hold 8 rows or fewer on average (an expert past 16 rows reads its weights
    // once per pass) and the grid stays large.  Same-box A/B: DeepSeek T=32 M=48 down
    // 98.5 -> 93.6 us, speculative 135.6 -> 127.2 us; at T=8 (672 blocks) 50.6 -> 53.2 us.
    const int wcols = kWaves * kCols * 2 * XS_Q4_DOWN_NM;
    const bool wide = XS_Q4_DN_WIDE && est > 0 && (long)a.T * a.k <= 8 * est &&
                      (long)((a.d + wcols - 1) / wcols) * est * a.splits >= XS_DN_WIDE_MIN_BLOCKS;
    if (wide)
      launch_down_fmt<kMx4, 2 * XS_Q4_DOWN_NM, 2>(a, unroll_for(K, XS_Q4_DOWN_U), stream);
    else
      launch_down_fmt<kMx4, XS_Q4_DOWN_NM>(a, unroll_for(K, XS_Q4_DOWN_U), stream);
    return hipGetLastError();
  }
  // bf16 and FP8: twice the rows per wave (one token load feeding twice the weight tiles)
  // pays when experts hold several tokens each and the grid stays large, or fills whole
  // rounds of the blocks the GPU runs at once: the Qwen-MoE shape at M=64 (512 wide blocks,
  // one round) ran down 53.6 -> 45.8 us wide, while 672 wide blocks (DeepSeek T=32 M=24,
  // 1.3 rounds) ran 137 -> 158 us.
  const int nm = a.wfmt == kFp8 ? XS_Q8_DOWN_NM : XS_DOWN_NM;
  const long wide_blocks =
      (long)((a.d + kWaves * kCols * 2 * nm - 1) / (kWaves * kCols * 2 * nm)) * est * a.splits;
  bool wide = est > 0 && (long)a.T * a.k >= XS_DN_WIDE_TOKENS * est &&
              wide_blocks >= XS_DN_WIDE_MIN_BLOCKS;
  if (!wide && est > 0 && (long)a.T * a.k >= XS_DN_WIDE_TOKENS * est) {
    const int r = a.wfmt == kFp8
                      ? down_resident<kFp8, 2 * XS_Q8_DOWN_NM>(unroll_for(K, XS_Q8_DOWN_U))
                      : down_resident<kBf16, 2 * XS_DOWN_NM>(unroll_for(K, XS_DOWN_U));
    wide = r > 0 && wide_blocks >= r && wide_blocks % r == 0;
  }
#if XS_DOWN_NM7
  // bf16: seven tiles per wave where that grid fills whole rounds (see XS_DOWN_NM7); not
  // for one GPU group's share, whose expected count (the group's experts under plain top-k)
  // overstates its live slots: the plain top-k share of DeepSeek T=32 (about 12 live of 32
  // slots) ran down 296 us with 64-row waves and 324 us with seven tiles
  if (a.wfmt == kBf16 && est > 0 && a.local_group < 0 &&
      (long)a.T * a.k >= XS_DN_WIDE_TOKENS * est) {
    const long b7 = (long)((a.d + kWaves * kCols * 7 - 1) / (kWaves * kCols * 7)) * est * a.splits;
    const int u7 = unroll_for(K, XS_DOWN_NM7_U);
    const int r7 = down_resident<kBf16, 7>(u7);
    if (r7 > 0 && b7 >= r7 && b7 % r7 == 0) {
#if XS_DOWN_SEQ
      if (a.splits == 1 && u7 == 4 && launch_down_seq<4, kBf16, 7>(a, stream))
        return hipGetLastError();
#endif
      launch_down_fmt<kBf16, 7>(a, u7, stream);
      return hipGetLastError();
    }
  }
#endif
  if (a.wfmt == kFp8) {
    if (wide)
      launch_down_fmt<kFp8, 2 * XS_Q8_DOWN_NM>(a, unroll_for(K, XS_Q8_DOWN_U), stream);
    else
      launch_down_fmt<kFp8, XS_Q8_DOWN_NM>(a, unroll_for(K, XS_Q8_DOWN_U), stream);
  } else {
    if (wide)
      launch_down_fmt<kBf16, 2 * XS_DOWN_NM>(a, unroll_for(K, XS_DOWN_U), stream);
    else
      launch_down_fmt<kBf16, XS_DOWN_NM>(a, unroll_for(K, XS_DOWN_U), stream);
  }
  return hipGetLastError();
}

hipError_t launch_router(const RouterArgs& r, hipStream_t stream) {
  const dim3 grid((r.N + kWaves * kCols - 1) / (kWaves * kCols), router_token_groups(r.T),
                  r.parts),
      block(kBlock);
  switch (unroll_for(r.d / r.parts, 4)) {
    case 4: hipLaunchKernelGGL(router_kernel<4>, grid, block, 0, stream, r); break;
    case 2: hipLaunchKernelGGL(router_kernel<2>, grid, block, 0, stream, r); break;
    default: hipLaunchKernelGGL(router_kernel<1>, grid, block, 0, stream, r); break;
  }
  const size_t n = (size_t)r.T * r.N;
  hipLaunchKernelGGL(router_sum_kernel, dim3((unsigned)((n + kBlock - 1) / kBlock)), block, 0,
                     stream, r);
  return hipGetLastError();
}

// MXFP4 scales [n_mat, rows, K / 32] -> the tiled layout [n_mat, rows / 16, G, 16, 8] (G =
// ceil(K / 256)); bytes past the last block of a row are 127 (scale 1), never read.
__global__ __launch_bounds__(kBlock) void mx_scales_tile_kernel(const uint8_t* src, uint8_t* dst,
                                                                long total, int rows, int K) {
  const long i = (long)blockIdx.x * kBlock + threadIdx.x;
  if (i >= total) return;
  const int G = (K + 255) >> 8, nb = K >> 5;
  const long per_mat = (long)rows * G * 8;
  const long mat = i / per_mat;
  const int r = (int)(i % per_mat);
  const int tile = r / (G * 128), in_tile = r % (G * 128);
  const int gran = in_tile >> 7, row = tile * 16 + ((in_tile >> 3) & 15);
  const int c = gran * 8 + (in_tile & 7);
  dst[i] = c < nb ? src[(mat * rows + row) * nb + c] : (uint8_t)127;
}

hipError_t launch_mx_scales_tile(const uint8_t* src, uint8_t* dst, int n_mat, int rows, int K,
                                 hipStream_t stream) {
  const long total = (long)n_mat * rows * ((K + 255) / 256) * 8;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(mx_scales_tile_kernel, dim3((unsigned)((total + kBlock - 1) / kBlock)),
                     dim3(kBlock), 0, stream, src, dst, total, rows, K);
  return hipGetLastError();
}

hipError_t launch_combine(const FfnArgs& a, hipStream_t stream) {
  const dim3 grid((a.d + kBlock * 4 - 1) / (kBlock * 4), a.T), block(kBlock);
  hipLaunchKernelGGL(combine_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace xs

// The block timeline of the last gate/up, down and persistent down launches (a profiling
// build); XSHARE_EUNSUPPORTED in the product build.  With `clear` the stamps are zeroed after
// the copy (hipMemsetAsync: a measurement call, not for graph capture).
extern "C" xshare_status xshare_block_times(uint64_t* gate_up, uint64_t* down,
                                            uint64_t* down_units, int32_t clear,
                                            hipStream_t stream) {
#if XS_BLOCK_TIMES
  if (!gate_up || !down || !down_units) return XSHARE_EINVAL;
  void* src[3] = {nullptr, nullptr, nullptr};
  if (hipGetSymbolAddress(&src[0], HIP_SYMBOL(xs::xs_times_gu)) != hipSuccess ||
      hipGetSymbolAddress(&src[1], HIP_SYMBOL(xs::xs_times_dn)) != hipSuccess ||
      hipGetSymbolAddress(&src[2], HIP_SYMBOL(xs::xs_times_seq)) != hipSuccess)
    return XSHARE_EHIP;
  uint64_t* dst[3] = {gate_up, down, down_units};
  const size_t bytes[3] = {sizeof(xs::xs_times_gu), sizeof(xs::xs_times_dn),
                           sizeof(xs::xs_times_seq)};
  for (int i = 0; i < 3; ++i) {
    if (hipMemcpyAsync(dst[i], src[i], bytes[i], hipMemcpyDeviceToDevice, stream) != hipSuccess)
      return XSHARE_EHIP;
    if (clear && hipMemsetAsync(src[i], 0, bytes[i], stream) != hipSuccess) return XSHARE_EHIP;
  }
  return XSHARE_OK;
#else
  (void)gate_up;
  (void)down;
  (void)down_units;
  (void)clear;
  (void)stream;
  return XSHARE_EUNSUPPORTED;
#endif
}
