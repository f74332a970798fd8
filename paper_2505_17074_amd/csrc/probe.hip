// Diagnostics for gfx950: the device's plain streaming read rate, the
// ceiling the verify kernels' HBM rates are compared with beside the vendor
// peak.  Each thread keeps eight coalesced 16-byte loads in flight, with the
// non-temporal hint (as the attention kernel's K/V stream: about 12 % faster
// than plain loads over 2 GiB); each work-group writes one word (an XOR of
// what it read) so that no load is dropped.  The words mean nothing.
#include "sv_internal.h"

namespace sv {
namespace {

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_read(const u32x4v* __restrict__ src, size_t n16, uint32_t* out) {
  __shared__ uint32_t red[4];
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4v v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = __builtin_nontemporal_load(src + i + k * stride);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  }
  for (; i < n16; i += stride) {
    const u32x4v v = __builtin_nontemporal_load(src + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* out, int blocks, hipStream_t s) {
  stream_read<<<blocks, 256, 0, s>>>(static_cast<const u32x4v*>(src), bytes / 16, out);
  return hipGetLastError();
}

}  // namespace sv
