// Speculative acceptance and final sample for gfx950.
//
// Three launches, each streaming what it needs once:
//   acc_rowstats     every target-logit row in 4096-entry chunks: chunk max
//                    and chunk sum of exp(l - max)          grid Nq x nch
//   acc_decide_mass  per (request, chunk): fold the chunk stats of the rows
//                    the tests need, run the acceptance tests (one lane per
//                    draft node), walk to the deepest accepted node, then
//                    the chunk's mass of the final-sample weights
//                      w = max(0, p - q)  (residual, node with children)
//                      w = p              (extra token, leaf / all accepted)
//                                                           grid B x nch
//   acc_select       per request: prefix over chunk masses, pick the chunk
//                    holding u * total, block scan inside it, smallest token
//                    id whose cumulative weight exceeds the target   grid B
// exp(l - max) is evaluated per entry in fp32 (expf, ~1 ulp), but every sum
// -- the softmax normaliser Z, chunk masses, prefixes and the in-chunk scan --
// is accumulated in fp64, and p = e / Z and the residual are formed in fp64.
// The sampled token then follows the exact inverse CDF except where u * S
// lies within ~1e-8 (probability mass) of a cumulative boundary.
#include "sv_internal.h"

namespace sv {
namespace {

__device__ __forceinline__ float ld(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t* p, int64_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

// Block-wide reductions over 256 threads (4 waves); `red` holds 4 values.
__device__ __forceinline__ float block_max(float x, float* red) {
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ __forceinline__ double block_sum(double x, double* red) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// 16-byte vector loads of VW = 16 / sizeof(T) entries, padded past V.
template <typename T>
__device__ __forceinline__ void load_vec(const T* row, int v, int V, float pad, float* out) {
  constexpr int VW = 16 / sizeof(T);
  if (v + VW <= V) {
    const uint4 u = *reinterpret_cast<const uint4*>(row + v);
    if constexpr (sizeof(T) == 4) {
      out[0] = __uint_as_float(u.x);
      out[1] = __uint_as_float(u.y);
      out[2] = __uint_as_float(u.z);
      out[3] = __uint_as_float(u.w);
    } else {
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        out[2 * k] = __uint_as_float(w[k] << 16);
        out[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < VW; ++k) out[k] = (v + k < V) ? ld(row, v + k) : pad;
  }
}

// This thread's 16 entries of chunk `base`, interleaved across the block so
// every vector load instruction is fully coalesced (order-free reductions).
template <typename T>
__device__ __forceinline__ void load16_coalesced(const T* row, int base, int V, float pad, float* x) {
  constexpr int VW = 16 / sizeof(T);
#pragma unroll
  for (int j = 0; j < 16 / VW; ++j) load_vec(row, base + j * kAccThreads * VW + threadIdx.x * VW, V, pad, x + j * VW);
}

// This thread's 16 CONSECUTIVE entries [base + 16 tid, +16): token order is
// thread order, as the inverse-CDF scan needs.
template <typename T>
__device__ __forceinline__ void load16_contiguous(const T* row, int base, int V, float pad, float* x) {
  constexpr int VW = 16 / sizeof(T);
#pragma unroll
  for (int j = 0; j < 16 / VW; ++j) load_vec(row, base + 16 * threadIdx.x + j * VW, V, pad, x + j * VW);
}

template <typename T>
__global__ __launch_bounds__(kAccThreads) void acc_rowstats(AccParams p) {
  __shared__ float redf[4];
  __shared__ double redd[4];
  const int row = blockIdx.x / p.nch, c = blockIdx.x % p.nch;
  const T* lp = static_cast<const T*>(p.logits) + (int64_t)row * p.l_st;
  float x[16];
  load16_coalesced(lp, c * kAccChunk, p.V, -INFINITY, x);
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < 16; ++k) m = fmaxf(m, x[k]);
  m = block_max(m, redf);
  double s = 0.0;
#pragma unroll
  for (int k = 0; k < 16; ++k) s += (double)expf(x[k] - m);
  s = block_sum(s, redd);
  if (threadIdx.x == 0) p.rowstats[(int64_t)row * p.nch + c] = ChunkStat{s, m, 0.f};
}

// Fold the chunk stats of one row into (M, Z) in fixed chunk order.
__device__ __forceinline__ void fold_row(const AccParams& p, int row, float* M_out, double* Z_out) {
  const ChunkStat* st = p.rowstats + (int64_t)row * p.nch;
  float M = -INFINITY;
  for (int c = 0; c < p.nch; ++c) M = fmaxf(M, st[c].m);
  double Z = 0.0;
  for (int c = 0; c < p.nch; ++c) Z += st[c].s * exp((double)st[c].m - (double)M);
  *M_out = M;
  *Z_out = Z;
}

__device__ __forceinline__ int node_parent(const AccParams& p, int n) {
  return p.tree ? p.topo->parent[n] : n - 1;
}
__device__ __forceinline__ int node_depth(const AccParams& p, int n) {
  return p.tree ? p.topo->depth[n] : n;
}
__device__ __forceinline__ int node_qrank(const AccParams& p, int n, int N) {
  return p.tree ? p.topo->qrank[n] : (n < N - 1 ? n : -1);
}

// Final-sample weight of one entry: residual max(0, p - q) or p itself.
__device__ __forceinline__ double final_weight(float l, float q, float M, double invZ, bool residual) {
  const double pv = (double)expf(l - M) * invZ;
  return residual ? fmax(0.0, pv - (double)q) : pv;
}

template <typename T>
__global__ __launch_bounds__(kAccThreads) void acc_decide_mass(AccParams p) {
  __shared__ double redd[4];
  __shared__ Decision s_dec;
  const int i = blockIdx.x / p.nch, c = blockIdx.x % p.nch;
  const ReqInfo rq = p.reqs[i];
  const int N = rq.nq;
  const T* L = static_cast<const T*>(p.logits);
  const T* Q = static_cast<const T*>(p.probs);

  if (threadIdx.x < 64) {
    // one lane per non-root node: the test of Eq. (1) against its parent's rows
    const int n = threadIdx.x;
    bool pass = false;
    if (n >= 1 && n < N) {
      const int par = node_parent(p, n);
      const int row = rq.q0 + par;
      float M;
      double Z;
      fold_row(p, row, &M, &Z);
      const int x = p.tokens[rq.q0 - i + n - 1];
      const double px = exp((double)ld(L, (int64_t)row * p.l_st + x) - (double)M) / Z;
      const int qr = rq.d0 + node_qrank(p, par, N);
      const double qx = (double)ld(Q, (int64_t)qr * p.p_st + x);
      const double u = (double)p.uniforms[rq.q0 + n - 1];
      pass = u * qx < px;
    }
    const unsigned long long passmask = __ballot(pass);
    if (n == 0) {
      uint32_t accepted = 1u;   // bit per node
      int best = 0;
      for (int m = 1; m < N; ++m) {
        const int par = node_parent(p, m);
        if (((accepted >> par) & 1u) && ((passmask >> m) & 1ull)) {
          accepted |= 1u << m;
          if (node_depth(p, m) > node_depth(p, best)) best = m;
        }
      }
      const int qrank = node_qrank(p, best, N);
      Decision d;
      d.node = best;
      d.row = rq.q0 + best;
      d.qrow = qrank >= 0 ? rq.d0 + qrank : -1;
      d.len = node_depth(p, best);
      fold_row(p, d.row, &d.M, &d.Z);
      d.pad = 0.f;
      s_dec = d;
    }
  }
  __syncthreads();
  const Decision d = s_dec;
  const double invZ = 1.0 / d.Z;
  const bool residual = d.qrow >= 0;
  float x[16], q[16];
  load16_coalesced(L + (int64_t)d.row * p.l_st, c * kAccChunk, p.V, -INFINITY, x);
  if (residual) load16_coalesced(Q + (int64_t)d.qrow * p.p_st, c * kAccChunk, p.V, 0.f, q);
  double s = 0.0;
#pragma unroll
  for (int k = 0; k < 16; ++k) s += final_weight(x[k], residual ? q[k] : 0.f, d.M, invZ, residual);
  s = block_sum(s, redd);
  if (threadIdx.x == 0) {
    p.masses[(int64_t)i * p.nch + c] = s;
    if (c == 0) p.decision[i] = d;
  }
}

template <typename T>
__global__ __launch_bounds__(kAccThreads) void acc_select(AccParams p) {
  __shared__ double redd[4];
  __shared__ double s_mass[kAccMaxChunks];
  __shared__ double s_tsum[kAccThreads];
  __shared__ double s_tot, s_base, s_target;
  __shared__ int s_chunk;
  __shared__ int s_cand[4], s_last[4];
  const int i = blockIdx.x;
  const int tid = threadIdx.x;
  const Decision d = p.decision[i];
  const double invZ = 1.0 / d.Z;
  const T* L = static_cast<const T*>(p.logits) + (int64_t)d.row * p.l_st;
  const T* Q = static_cast<const T*>(p.probs) + (int64_t)(d.qrow >= 0 ? d.qrow : 0) * p.p_st;
  const float u = p.uniforms[p.reqs[i].q0 + p.reqs[i].nq - 1];
  const double* masses = p.masses + (int64_t)i * p.nch;

  if (tid == 0) {
    double tot = 0.0;
    for (int c = 0; c < p.nch; ++c) tot += masses[c];
    s_tot = tot;
  }
  __syncthreads();
  // zero residual mass (reachable only through rounding): sample from p itself
  const bool fallback = !(s_tot > 0.0);
  const bool residual = d.qrow >= 0 && !fallback;
  if (!fallback) {
    for (int c = tid; c < p.nch; c += kAccThreads) s_mass[c] = masses[c];
  } else {
    for (int c = 0; c < p.nch; ++c) {
      float x[16];
      load16_coalesced(L, c * kAccChunk, p.V, -INFINITY, x);
      double s = 0.0;
#pragma unroll
      for (int k = 0; k < 16; ++k) s += final_weight(x[k], 0.f, d.M, invZ, false);
      s = block_sum(s, redd);
      if (tid == 0) s_mass[c] = s;
    }
  }
  __syncthreads();
  if (tid == 0) {
    double tot = 0.0;
    for (int c = 0; c < p.nch; ++c) tot += s_mass[c];
    const double target = (double)u * tot;
    double cum = 0.0;
    int chosen = -1, last_pos = 0;
    for (int c = 0; c < p.nch; ++c) {
      if (s_mass[c] > 0.0) last_pos = c;
      if (chosen < 0) {
        if (cum + s_mass[c] > target) chosen = c;
        else cum += s_mass[c];
      }
    }
    if (chosen < 0) {   // target rounded past the total: last chunk with mass
      chosen = last_pos;
      cum = 0.0;
      for (int c = 0; c < chosen; ++c) cum += s_mass[c];
    }
    s_chunk = chosen;
    s_base = cum;
    s_target = target;
  }
  __syncthreads();
  const int c = s_chunk;
  float x[16], q[16];
  double w[16];
  load16_contiguous(L, c * kAccChunk, p.V, -INFINITY, x);
  if (residual) load16_contiguous(Q, c * kAccChunk, p.V, 0.f, q);
  double tsum = 0.0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    w[k] = final_weight(x[k], residual ? q[k] : 0.f, d.M, invZ, residual);
    tsum += w[k];
  }
  // exclusive prefix of the per-thread sums, in thread (= token) order
  s_tsum[tid] = tsum;
  __syncthreads();
  if (tid < 64) {
    const double a0 = s_tsum[4 * tid], a1 = s_tsum[4 * tid + 1], a2 = s_tsum[4 * tid + 2];
    const double lsum = ((a0 + a1) + a2) + s_tsum[4 * tid + 3];
    double incl = lsum;
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(incl, o);
      if (tid >= o) incl += y;
    }
    double ex = incl - lsum;
    s_tsum[4 * tid] = ex;
    ex += a0;
    s_tsum[4 * tid + 1] = ex;
    ex += a1;
    s_tsum[4 * tid + 2] = ex;
    ex += a2;
    s_tsum[4 * tid + 3] = ex;
  }
  __syncthreads();
  double run = s_base + s_tsum[tid];
  const double target = s_target;
  int cand = 0x7fffffff, lastpos = -1;
  const int v0 = c * kAccChunk + 16 * tid;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    run += w[k];
    if (w[k] > 0.0) {
      lastpos = v0 + k;
      if (cand == 0x7fffffff && run > target) cand = v0 + k;
    }
  }
  // smallest crossing token, else the chunk's last positive weight
  for (int o = 32; o >= 1; o >>= 1) {
    cand = min(cand, __shfl_xor(cand, o));
    lastpos = max(lastpos, __shfl_xor(lastpos, o));
  }
  if ((tid & 63) == 0) {
    s_cand[tid >> 6] = cand;
    s_last[tid >> 6] = lastpos;
  }
  __syncthreads();
  if (tid == 0) {
    int best = min(min(s_cand[0], s_cand[1]), min(s_cand[2], s_cand[3]));
    if (best == 0x7fffffff) best = max(max(s_last[0], s_last[1]), max(s_last[2], s_last[3]));
    p.next_tok[i] = best;
    p.acc_len[i] = d.len;
    if (p.acc_node) p.acc_node[i] = d.node;
  }
}

}  // namespace

hipError_t launch_accept(const AccParams& p, hipStream_t s) {
  dim3 block(kAccThreads);
  if (p.bf16) {
    acc_rowstats<uint16_t><<<dim3(p.Nq * p.nch), block, 0, s>>>(p);
    acc_decide_mass<uint16_t><<<dim3(p.B * p.nch), block, 0, s>>>(p);
    acc_select<uint16_t><<<dim3(p.B), block, 0, s>>>(p);
  } else {
    acc_rowstats<float><<<dim3(p.Nq * p.nch), block, 0, s>>>(p);
    acc_decide_mass<float><<<dim3(p.B * p.nch), block, 0, s>>>(p);
    acc_select<float><<<dim3(p.B), block, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace sv
