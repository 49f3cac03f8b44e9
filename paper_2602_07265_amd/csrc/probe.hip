// Streaming-read probe: the HBM read rate a plain coalesced kernel reaches on this GPU, the
// practical ceiling against which the expert GEMMs' weight streams are read (decode is bound
// by reading expert weights, Section 2.3).  Measurement only; not part of the layer.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "xshare.h"

namespace {

constexpr int kProbeBlock = 256;

// 16-byte pieces [begin, end) of the buffer, U loads in flight per thread: consecutive lanes
// read consecutive pieces, a block's threads cover `stride` pieces per load; every piece is
// folded into one word, written only when it equals `magic` (never, for the caller's magic),
// which keeps the loads without a store per thread.
template <int U>
__device__ __forceinline__ void read_range(const uint4* p, size_t i, size_t end, size_t stride,
                                           uint32_t* sink, uint32_t magic) {
  uint32_t acc = 0;
  for (; i + (U - 1) * stride < end; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < end; i += stride) {
    const uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == magic) sink[0] = acc;
}

// kChunk false: the whole grid strides through the buffer together (pieces i, i + grid
// threads, ...).  kChunk true: block b reads its own contiguous chunk of about n16 / blocks
// pieces, its threads striding through it.
template <int U, bool kChunk>
__global__ __launch_bounds__(kProbeBlock) void stream_read_kernel(const uint4* p, size_t n16,
                                                                  uint32_t* sink,
                                                                  uint32_t magic) {
  if (kChunk) {
    const size_t b0 = n16 * blockIdx.x / gridDim.x, b1 = n16 * (blockIdx.x + 1) / gridDim.x;
    read_range<U>(p, b0 + threadIdx.x, b1, kProbeBlock, sink, magic);
  } else {
    read_range<U>(p, (size_t)blockIdx.x * kProbeBlock + threadIdx.x, n16,
                  (size_t)gridDim.x * kProbeBlock, sink, magic);
  }
}

}  // namespace

extern "C" xshare_status xshare_probe_stream_read(const void* buf, size_t bytes, int32_t blocks,
                                                  int32_t mode, uint32_t* sink,
                                                  hipStream_t stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(buf) & 15u) != 0 || blocks < 1 || mode < 0 || mode > 3)
    return XSHARE_EINVAL;
  const dim3 grid((unsigned)blocks), block(kProbeBlock);
  const uint4* p = static_cast<const uint4*>(buf);
  const size_t n16 = bytes / 16;
  const uint32_t magic = 0x9E3779B9u;
  switch (mode) {
    case 0: hipLaunchKernelGGL((stream_read_kernel<4, false>), grid, block, 0, stream, p, n16, sink, magic); break;
    case 1: hipLaunchKernelGGL((stream_read_kernel<8, false>), grid, block, 0, stream, p, n16, sink, magic); break;
    case 2: hipLaunchKernelGGL((stream_read_kernel<4, true>), grid, block, 0, stream, p, n16, sink, magic); break;
    default: hipLaunchKernelGGL((stream_read_kernel<8, true>), grid, block, 0, stream, p, n16, sink, magic); break;
  }
  return hipGetLastError() == hipSuccess ? XSHARE_OK : XSHARE_EHIP;
}
