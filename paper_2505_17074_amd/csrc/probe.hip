// Diagnostics for gfx950, not on the verify path.
//
// The device's plain streaming read rate, the ceiling the verify kernels'
// HBM rates are compared with beside the vendor peak (stream_read), and the
// acceptance kernels' floor (floor_stream, floor_chain; below).
//
// stream_read: each thread keeps eight coalesced 16-byte loads in flight, with the
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

// The acceptance floor: the acceptance kernels' memory traffic and dependent
// round trips with none of their arithmetic.
//
// floor_stream (grid rows x chunks of 4096 entries, 256 threads) reads every
// entry of the given rows once with 16-byte loads, as the row-statistics
// kernel does, and writes one word per work-group; work-group 0 also clears
// the tickets, as the row-statistics kernel does for the decision kernel.
__global__ __launch_bounds__(256) void floor_stream(const char* __restrict__ rows, int64_t row_bytes, int64_t v_bytes,
                                                    int64_t chunk_bytes, int nch, int B, uint32_t* sink,
                                                    int32_t* tickets) {
  __shared__ uint32_t red[4];
  const int r = blockIdx.x / nch, c = blockIdx.x % nch;
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < B; i += 256) tickets[i] = 0;
  const char* row = rows + (int64_t)r * row_bytes;
  const int64_t c0 = (int64_t)c * chunk_bytes, c1 = min(c0 + chunk_bytes, v_bytes);
  // up to four 16-byte loads per thread in flight (a 16 KB chunk), issued before use
  u32x4v v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t o = c0 + ((int64_t)k * 256 + threadIdx.x) * 16;
    v[k] = o + 16 <= c1 ? *reinterpret_cast<const u32x4v*>(row + o) : u32x4v{0u, 0u, 0u, 0u};
  }
  uint32_t acc = 0u;
#pragma unroll
  for (int k = 0; k < 4; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

// floor_chain (grid B x chunks, 256 threads): the decision kernel's chain of
// dependent round trips, each a load whose address comes from the one before:
//   1. a word of the stream's output for the request (its table);
//   2. a word chosen by it (the rows' normalisers and the test operands);
//   3. a chunk of a row chosen by that (the chosen row's chunk), summed;
//   4. the sum handed over: an agent-scope store, then a ticket, and the
//      request's last work-group goes on (the mass publication);
//   5. that work-group reads the request's published sums (the masses);
//   6. and a chunk chosen by them (the sampler's chunk), then one word out.
__global__ __launch_bounds__(256) void floor_chain(const char* __restrict__ rows, int64_t row_bytes, int64_t v_bytes,
                                                   int64_t chunk_bytes, int nch, int rows_per_req,
                                                   const uint32_t* sink, int32_t* tickets, uint64_t* sums,
                                                   uint32_t* out) {
  __shared__ uint32_t red[4];
  __shared__ int s_last;
  __shared__ uint32_t s_pick;
  const int i = blockIdx.x / nch, c = blockIdx.x % nch;
  const int64_t r0 = (int64_t)i * rows_per_req;
  auto chunk_xor = [&](int64_t r, int64_t ch) -> uint32_t {
    const char* row = rows + r * row_bytes;
    const int64_t c0 = ch * chunk_bytes, c1 = min(c0 + chunk_bytes, v_bytes);
    u32x4v v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t o = c0 + ((int64_t)k * 256 + threadIdx.x) * 16;
      v[k] = o + 16 <= c1 ? *reinterpret_cast<const u32x4v*>(row + o) : u32x4v{0u, 0u, 0u, 0u};
    }
    uint32_t acc = 0u;
#pragma unroll
    for (int k = 0; k < 4; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
    for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    return red[0] ^ red[1] ^ red[2] ^ red[3];
  };
  const uint32_t a = sink[r0 * nch + c];                                   // 1
  const uint32_t b = sink[(r0 + (int64_t)(a % (uint32_t)rows_per_req)) * nch + c];   // 2
  const uint32_t m = chunk_xor(r0 + (int64_t)(b % (uint32_t)rows_per_req), c);        // 3
  if (threadIdx.x == 0) {                                                  // 4
    __hip_atomic_store(sums + (int64_t)i * nch + c, (uint64_t)m | 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    s_last = __hip_atomic_fetch_add(tickets + i, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nch - 1;
  }
  __syncthreads();
  if (!s_last) return;
  if (threadIdx.x == 0) {                                                  // 5
    uint64_t x = 0;
    for (int k = 0; k < nch; ++k)
      x ^= __hip_atomic_load(sums + (int64_t)i * nch + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_pick = (uint32_t)(x % (uint64_t)nch);
  }
  __syncthreads();
  const uint32_t w = chunk_xor(r0 + (int64_t)(s_pick % (uint32_t)rows_per_req), s_pick);   // 6
  if (threadIdx.x == 0) out[i] = w;
}

}  // namespace

hipError_t launch_accept_floor(const void* rows, int64_t row_bytes, int64_t v_bytes, int64_t chunk_bytes, int nch,
                               int num_rows, int B, uint32_t* sink, int32_t* tickets, uint64_t* sums, uint32_t* out,
                               hipStream_t s) {
  const char* r = static_cast<const char*>(rows);
  const int rows_per_req = num_rows / B;           // request i's row choices stay in [i rpr, (i + 1) rpr)
  floor_stream<<<(unsigned)((int64_t)num_rows * nch), 256, 0, s>>>(r, row_bytes, v_bytes, chunk_bytes, nch, B, sink,
                                                                   tickets);
  floor_chain<<<(unsigned)((int64_t)B * nch), 256, 0, s>>>(r, row_bytes, v_bytes, chunk_bytes, nch, rows_per_req, sink,
                                                          tickets, sums, out);
  return hipGetLastError();
}

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* out, int blocks, hipStream_t s) {
  stream_read<<<blocks, 256, 0, s>>>(static_cast<const u32x4v*>(src), bytes / 16, out);
  return hipGetLastError();
}

}  // namespace sv
