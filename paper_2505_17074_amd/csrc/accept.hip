// Speculative acceptance and final sample for gfx950.
//
// Two launches, each streaming what it needs once:
//   acc_rowstats       target-logit rows in 4096-entry chunks: chunk max and
//                      chunk sum of exp(l - max), 32 KB of a row per
//                      work-group                    grid Nq x ceil(nch / SUB)
//                      (independent tree rule: only the rows of nodes with
//                      children, grid B x inner nodes x nch)
//   acc_decide_select  per (request, chunk): fold the chunk stats of the
//                      request's rows, run the acceptance tests (one lane per
//                      draft node), walk to the deepest accepted node, then
//                      the final sample's weights
//                        w = max(0, p - q)  (residual, node with children):
//                            each chunk's mass, published
//                        w = p              (extra token, leaf / all accepted):
//                            chunk masses from the row's chunk statistics
//                            (a tree leaf's taken here first)
//                      the request's last work-group to check in then takes
//                      the prefix over chunk masses, picks the chunk holding
//                      u * total, scans inside it and emits the smallest
//                      token id whose cumulative weight exceeds the target
//                                                            grid B x nch
// exp(l - max) is evaluated per entry in fp32 (exp_rel, ~1 ulp), but every sum
// -- the softmax normaliser Z, chunk masses, prefixes and the in-chunk scan --
// is accumulated in fp64, and p = e / Z and the residual are formed in fp64.
// The sampled token then follows the exact inverse CDF except where u * S
// lies within ~1e-8 (probability mass) of a cumulative boundary.
#include <algorithm>
#include <climits>

#include "sv_internal.h"

// Sub-chunks (4096 entries) per row-statistics work-group, by logit dtype.
#ifndef SV_RS_SUB_F32
#define SV_RS_SUB_F32 1
#endif
#ifndef SV_RS_SUB_BF16
#define SV_RS_SUB_BF16 1
#endif
// Cache policy of the row-statistics loads: 1 = non-temporal hint.
#ifndef SV_RS_NT
#define SV_RS_NT 0
#endif

namespace sv {
namespace {

// Diagnostic builds only (-DSV_ACC_TRACE): per work-group phase timestamps
// of the acceptance kernels on the device's constant-rate clock, read back
// by sv_acc_trace_copy, for measuring where a kernel's time goes.
#ifdef SV_ACC_TRACE
constexpr int kTraceBlocks = 16384, kTracePhases = 8;
__device__ unsigned long long g_acc_trace[2][kTraceBlocks][kTracePhases];
#define SV_TRACE(kern, k)                                                         \
  do {                                                                            \
    if (threadIdx.x == 0 && blockIdx.x < kTraceBlocks)                            \
      g_acc_trace[kern][blockIdx.x][k] = wall_clock64();                          \
  } while (0)
#else
#define SV_TRACE(kern, k) ((void)0)
#endif

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

// One 16-byte word of a row as stored (VW entries; entries past V hold
// pad's bit pattern), and entry e of such a word.
template <typename T>
__device__ __forceinline__ uint4 load_raw(const T* row, int v, int V, float pad) {
  constexpr int VW = 16 / sizeof(T);
  if (v + VW <= V) return *reinterpret_cast<const uint4*>(row + v);
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < VW; ++e) {
    const uint32_t b = __float_as_uint(v + e < V ? ld(row, v + e) : pad);
    if constexpr (sizeof(T) == 4) w[e] = b;
    else w[e >> 1] |= (b >> 16) << (16 * (e & 1));
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}
template <typename T>
__device__ __forceinline__ float entry(const uint4& r, int e) {
  if constexpr (sizeof(T) == 4) {
    return __uint_as_float(e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w);
  } else {
    const uint32_t w = (e >> 1) == 0 ? r.x : (e >> 1) == 1 ? r.y : (e >> 1) == 2 ? r.z : r.w;
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
  }
}

// load_vec with the row-statistics kernel's cache policy.
template <typename T>
__device__ __forceinline__ void load_vec_rs(const T* row, int v, int V, float pad, float* out) {
  if constexpr (SV_RS_NT) {
    constexpr int VW = 16 / sizeof(T);
    if (v + VW <= V) {
      typedef uint32_t u4v __attribute__((ext_vector_type(4)));
      const u4v u = __builtin_nontemporal_load(reinterpret_cast<const u4v*>(row + v));
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
      return;
    }
  }
  load_vec(row, v, V, pad, out);
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
struct RowGeo {
  static constexpr int VW = 16 / sizeof(T);                 // entries per 16-byte load
  static constexpr int LPS = kAccChunk / (kAccThreads * VW);  // loads per thread per sub-chunk
  static constexpr int SUB = sizeof(T) == 4 ? SV_RS_SUB_F32 : SV_RS_SUB_BF16;   // sub-chunks per work-group
};

template <typename T>
__global__ __launch_bounds__(kAccThreads) void acc_rowstats(AccParams p) {
  using RG = RowGeo<T>;
  constexpr int VW = RG::VW, LPS = RG::LPS, SUB = RG::SUB;
  __shared__ float redf[SUB][4];
  __shared__ double redd[SUB][4];
  const int nwg = (p.nch + SUB - 1) / SUB;                 // work-groups per row
  const int su = blockIdx.x / nwg, c0 = (blockIdx.x % nwg) * SUB;
  // Under the independent tree rule only the rows of nodes with children:
  // their normalisers enter the tests, while a leaf's row is needed only when
  // that leaf is chosen, and the decision kernel then takes its statistics.
  // Every request has the tree's `nodes` rows there, so the row is arithmetic.
  int row = su;
  if (p.tree == 1 && !p.all_stats) {
    const int ni = p.topo.n_inner;
    row = (ni > 0 && su < p.B * ni) ? (su / ni) * p.topo.nodes + p.topo.inner[su % ni] : -1;
  }
  const T* lp = static_cast<const T*>(p.logits) + (int64_t)max(row, 0) * p.l_st;
  SV_TRACE(0, 0);
  // the first B work-groups (the grid has at least B of them) bring request
  // blockIdx.x's entry of the staged table into device memory and clear its
  // ticket, for the decision kernel that follows on the stream
  uint4 rq_half;
  const bool copier = blockIdx.x < p.B && threadIdx.x < 2;
  if (copier) rq_half = reinterpret_cast<const uint4*>(p.reqs_src + blockIdx.x)[threadIdx.x];
  // Sub-chunk c0 + s is loads s*LPS .. s*LPS + LPS-1: thread t holds entries
  // (c0+s)*4096 + j*256*VW + t*VW + e, the decision kernel's layout of a chunk,
  // so both kernels reduce a chunk in the same order (bit-identical statistics).
  float x[SUB][LPS * VW];
  if (row >= 0) {
#pragma unroll
    for (int sc = 0; sc < SUB; ++sc)
#pragma unroll
      for (int j = 0; j < LPS; ++j)
        load_vec_rs(lp, (c0 + sc) * kAccChunk + j * kAccThreads * VW + threadIdx.x * VW, p.V, -INFINITY,
                    x[sc] + j * VW);
  }
  if (copier) {
    reinterpret_cast<uint4*>(p.reqs + blockIdx.x)[threadIdx.x] = rq_half;
    if (threadIdx.x == 0) p.tickets[blockIdx.x] = 0;
  }
  // per-request trees: the same work-groups copy the node table
  if (p.per_req && blockIdx.x < p.B)
    for (int x = blockIdx.x * kAccThreads + threadIdx.x; x < p.nodes_n16; x += p.B * kAccThreads)
      reinterpret_cast<uint4*>(p.nodes)[x] = reinterpret_cast<const uint4*>(p.nodes_src)[x];
  if (row < 0) return;              // uniform: a work-group kept for the copy only
  const int wv = threadIdx.x >> 6;
  float m[SUB];
#pragma unroll
  for (int sc = 0; sc < SUB; ++sc) {
    m[sc] = -INFINITY;
#pragma unroll
    for (int k = 0; k < LPS * VW; ++k) m[sc] = fmaxf(m[sc], x[sc][k]);
    for (int o = 32; o >= 1; o >>= 1) m[sc] = fmaxf(m[sc], __shfl_xor(m[sc], o));
  }
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int sc = 0; sc < SUB; ++sc) redf[sc][wv] = m[sc];
  __syncthreads();
  SV_TRACE(0, 1);
  double sm[SUB];
#pragma unroll
  for (int sc = 0; sc < SUB; ++sc) {
    m[sc] = fmaxf(fmaxf(redf[sc][0], redf[sc][1]), fmaxf(redf[sc][2], redf[sc][3]));
    sm[sc] = 0.0;
#pragma unroll
    for (int k = 0; k < LPS * VW; ++k) sm[sc] += (double)exp_rel(x[sc][k], m[sc]);
    for (int o = 32; o >= 1; o >>= 1) sm[sc] += __shfl_xor(sm[sc], o);
  }
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int sc = 0; sc < SUB; ++sc) redd[sc][wv] = sm[sc];
  __syncthreads();
  if (threadIdx.x < SUB) {
    const int sc = threadIdx.x;
    const double tot = (redd[sc][0] + redd[sc][1]) + (redd[sc][2] + redd[sc][3]);
    if (c0 + sc < p.nch) p.rowstats[(int64_t)row * p.nch + c0 + sc] = ChunkStat{tot, m[sc], 0.f};
  }
  SV_TRACE(0, 2);
}

__device__ __forceinline__ int node_parent(const AccParams& p, int n) {
  return p.tree ? p.topo.parent[n] : n - 1;
}
__device__ __forceinline__ int node_depth(const AccParams& p, int n) {
  return p.tree ? p.topo.depth[n] : n;
}
__device__ __forceinline__ int node_qrank(const AccParams& p, int n, int N) {
  return p.tree ? p.topo.qrank[n] : (n < N - 1 ? n : -1);
}

// Node n of request rq: its parent, depth, draft-row rank (nodes with
// children) and its parent's draft-row rank, from the request's node-table
// entry (per-request trees), the shared tree or the chain.
struct NodeRec {
  int par, dep, qr, pq;
};
__device__ __forceinline__ NodeRec node_rec(const AccParams& p, const NodeInfo* nodes, const ReqInfo& rq, int n) {
  NodeRec r;
  if (p.per_req) {
    const NodeInfo e = nodes[rq.node0 + n];
    r.par = e.parent;
    r.dep = e.depth;
    r.qr = e.qrank;
    r.pq = e.pqrank;
  } else {
    r.par = node_parent(p, n);
    r.dep = node_depth(p, n);
    r.qr = node_qrank(p, n, rq.nq);
    r.pq = n > 0 ? node_qrank(p, r.par, rq.nq) : -1;
  }
  return r;
}

// Final-sample weight of one entry: residual max(0, p - q) or p itself.
__device__ __forceinline__ double final_weight(float l, float q, float M, double invZ, bool residual) {
  const double pv = (double)exp_rel(l, M) * invZ;
  return residual ? fmax(0.0, pv - (double)q) : pv;
}

// Device-scope (all XCDs) publication of the chunk masses between the
// work-groups of one request.  The hand-over rests on how gfx950 executes
// agent-scope accesses rather than on a release/acquire pair:
//   * an agent-scope store (sc1) is written through this XCD's L2 to the
//     device coherence point, and its vmcnt completes only once it is there;
//   * the publishing wave waits for that completion (s_waitcnt 0) before its
//     ticket, an agent-scope atomic performed at the coherence point;
//   * an agent-scope load (sc1) is served from the coherence point, never
//     from a stale line of the reader's L2, and the sampler issues its loads
//     only after its own ticket returned the last count (after the other
//     publishers' tickets, hence after their stores completed).
// Only the masses (and a leaf's chunk statistics) cross, all written and
// read this way.  A release/acquire ticket would write back and invalidate
// the whole L2 of the XCD at every work-group's hand-over; measured, that
// lengthens the ragged GQA step from 182 to 222 us, since the attention
// running beside the acceptance loses its L2 every time.
__device__ __forceinline__ void store_dev(double* p, double v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), __double_as_longlong(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double load_dev(const double* p) {
  return __longlong_as_double(__hip_atomic_load(reinterpret_cast<const unsigned long long*>(p), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT));
}

// Per (request i, chunk c):
//   fold the chunk statistics of the request's rows that have them (one wave
//   per row, fixed reduction order) into fp64 (M, Z); run the tests of
//   Eq. (1) (one lane per draft node, against its parent's rows); walk to the
//   deepest accepted node.  The final sample then weighs the chosen row by
//   * the residual max(0, p - q) when the node has children (a draft row):
//     every work-group publishes its chunk's mass of it;
//   * p itself at a leaf or when every draft is accepted: chunk c's mass is
//     s_c * exp(m_c - M) from the row's chunk statistics (max m_c, sum s_c of
//     exp(l - m_c)).  Under the independent tree rule a leaf's row has none
//     yet, and each work-group takes its chunk's here with the row-statistics
//     kernel's arithmetic; otherwise only chunk 0's work-group goes on.
//   The last of the request's work-groups to check in (a device-scope ticket)
//   samples: prefix over the chunk masses, the chunk holding u * total, an
//   fp64 scan inside it (for p, in that chunk's units exp(l - m_c)), the
//   smallest token id whose cumulative weight exceeds the target.
// TILES: the statistics are the LM head's per-tile ones (p.tiles), folded
// here; otherwise the row-statistics kernel's chunk statistics.  A separate
// build, so the verify path keeps the smaller register footprint (80 VGPRs
// against 96 with the tile fold's held loads: 6 waves per SIMD instead of 5
// beside the attention).
template <typename T, bool TILES>
__global__ __launch_bounds__(kAccThreads) void acc_decide_select(AccParams p) {
  __shared__ double redd[4];
  __shared__ float redf[4];
  __shared__ float s_M[kMaxNodes];
  __shared__ double s_Z[kMaxNodes];
  __shared__ Decision s_dec;
  __shared__ int s_last;
  __shared__ double s_mass[kAccMaxChunks];
  __shared__ float s_mc[kAccMaxChunks];
  __shared__ double s_tsum[kAccThreads];
  __shared__ double s_tot, s_base, s_target;
  __shared__ float s_mrow, s_mcc;
  __shared__ int s_chunk;
  __shared__ int s_cand[4], s_last_pos[4];
  __shared__ int s_par[kMaxNodes], s_dep[kMaxNodes], s_qr[kMaxNodes];
  const int i = blockIdx.x / p.nch, c = blockIdx.x % p.nch;
  const int tid = threadIdx.x, wv = tid >> 6, ln = tid & 63;
  SV_TRACE(1, 0);
  const ReqInfo rq = p.reqs[i];
  const int N = rq.nq;
  const T* L = static_cast<const T*>(p.logits);
  const T* Q = static_cast<const T*>(p.probs);

  // Loads the tests need that do not depend on the row statistics, issued
  // first: each non-root node's token, the parent row's logit and draft
  // probability at it, and its uniform.
  const int n = tid;
  const bool tester = n >= 1 && n < N;      // lanes of wave 0 only (N <= 32)
  int par = 0;
  float lx = 0.f, qx = 0.f, un = 0.f;
  if (n < N) {
    const NodeRec nr = node_rec(p, p.nodes, rq, n);
    s_par[n] = nr.par;
    s_dep[n] = nr.dep;
    s_qr[n] = nr.qr;
    if (tester) {
      par = nr.par;
      // an out-of-range id (the caller's contract) is clamped: no read leaves the row
      const int x = min(max(p.tokens[rq.q0 - i + n - 1], 0), p.V - 1);
      lx = ld(L, (int64_t)(rq.q0 + par) * p.l_st + x);
      qx = ld(Q, (int64_t)(rq.d0 + nr.pq) * p.p_st + x);
      un = p.uniforms[rq.q0 + n - 1];
    }
  }

  // (M, Z) of every row of the request that has chunk statistics (after the
  // LM head, its tile statistics: the same fold over 16 times as many entries)
  // A row of at most 64 * kHeld tile statistics is loaded whole into
  // registers before any is used (one round trip); chunk statistics (at
  // most a few per lane) and longer rows take two passes.
  constexpr int kHeld = 8;
  const int nst = TILES ? p.ntiles : p.nch;
  for (int r = wv; r < N; r += kAccThreads / 64) {
    if (p.tree == 1 && !p.all_stats && p.topo.qrank[r] < 0) continue;     // a leaf's row: none yet
    const ChunkStat* st = (TILES ? p.tiles : p.rowstats) + (int64_t)(rq.q0 + r) * nst;
    float m = -INFINITY;
    double z = 0.0;
    if (TILES && nst <= 64 * kHeld) {
      float hm[kHeld];
      double hs[kHeld];
#pragma unroll
      for (int j = 0; j < kHeld; ++j) {
        hm[j] = -INFINITY;
        hs[j] = 0.0;
        if (ln + 64 * j < nst) {
          hm[j] = st[ln + 64 * j].m;
          hs[j] = st[ln + 64 * j].s;
        }
      }
#pragma unroll
      for (int j = 0; j < kHeld; ++j) m = fmaxf(m, hm[j]);
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
#pragma unroll
      for (int j = 0; j < kHeld; ++j)
        if (ln + 64 * j < nst) z += hs[j] * exp((double)hm[j] - (double)m);
    } else {
      for (int k = ln; k < nst; k += 64) m = fmaxf(m, st[k].m);
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
      for (int k = ln; k < nst; k += 64) z += st[k].s * exp((double)st[k].m - (double)m);
    }
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    if (ln == 0) {
      s_M[r] = m;
      s_Z[r] = z;
    }
  }
  __syncthreads();
  SV_TRACE(1, 1);

  if (tid < 64) {
    // one lane per non-root node: the test of Eq. (1) against its parent's rows
    bool pass = false;
    if (tester) {
      const double px = exp((double)lx - (double)s_M[par]) / s_Z[par];
      pass = (double)un * (double)qx < px;
    }
    const unsigned long long passmask = __ballot(pass);
    if (n == 0) {
      uint32_t accepted = 1u;   // bit per node
      int best = 0;
      for (int m = 1; m < N; ++m) {
        const int par = s_par[m];
        if (((accepted >> par) & 1u) && ((passmask >> m) & 1ull)) {
          accepted |= 1u << m;
          if (s_dep[m] > s_dep[best]) best = m;
        }
      }
      const int qrank = s_qr[best];
      Decision d;
      d.node = best;
      d.row = rq.q0 + best;
      d.qrow = qrank >= 0 ? rq.d0 + qrank : -1;
      d.len = s_dep[best];
      d.M = qrank >= 0 ? s_M[best] : 0.f;      // the residual's normaliser (a node with children)
      d.Z = qrank >= 0 ? s_Z[best] : 1.0;
      d.pad = 0.f;
      s_dec = d;
    }
  }
  __syncthreads();
  SV_TRACE(1, 2);
  const Decision d = s_dec;
  const double invZ = 1.0 / d.Z;
  bool residual = d.qrow >= 0;
  // a leaf's row under the independent rule over a shared tree has no statistics yet
  const bool own_stats = !residual && p.tree == 1 && !p.all_stats;
  const T* Lr = L + (int64_t)d.row * p.l_st;
  const T* Qr = Q + (int64_t)(d.qrow >= 0 ? d.qrow : 0) * p.p_st;
  ChunkStat* rst = p.rowstats + (int64_t)d.row * p.nch;
  if (!residual && !own_stats) {
    // p with the row's statistics at hand: one work-group samples
    if (c != 0) return;
    if (tid == 0) s_last = 1;
  } else {
    float x[16], q[16];
    load16_coalesced(Lr, c * kAccChunk, p.V, -INFINITY, x);
    if (residual) load16_coalesced(Qr, c * kAccChunk, p.V, 0.f, q);
    double sm = 0.0;
    float m = 0.f;
    if (residual) {
#pragma unroll
      for (int k = 0; k < 16; ++k) sm += final_weight(x[k], q[k], d.M, invZ, true);
      sm = block_sum(sm, redd);
    } else {
      // this chunk's statistics of the leaf's row, as the row-statistics kernel takes them
      m = -INFINITY;
#pragma unroll
      for (int k = 0; k < 16; ++k) m = fmaxf(m, x[k]);
      m = block_max(m, redf);
#pragma unroll
      for (int k = 0; k < 16; ++k) sm += (double)exp_rel(x[k], m);
      sm = block_sum(sm, redd);
    }
    SV_TRACE(1, 3);
    if (tid == 0) {
      if (residual) {
        if (p.nch == 1) s_mass[0] = sm;
        else store_dev(p.masses + (int64_t)i * p.nch + c, sm);
      } else {
        store_dev(&rst[c].s, sm);
        __hip_atomic_store(reinterpret_cast<uint32_t*>(&rst[c].m), __float_as_uint(m), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
      if (p.nch == 1) {
        s_last = 1;
      } else {
        __builtin_amdgcn_s_waitcnt(0);     // the stores have reached the device coherence point
        const int t = __hip_atomic_fetch_add(p.tickets + i, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = (t == p.nch - 1);
      }
      SV_TRACE(1, 4);
    }
  }
  __syncthreads();
  if (!s_last) return;              // uniform: another work-group of the request samples

  // ---- the request's sampler
  if (residual) {
    if (p.nch > 1)
      for (int k = tid; k < p.nch; k += kAccThreads) s_mass[k] = load_dev(p.masses + (int64_t)i * p.nch + k);
    __syncthreads();
    if (tid == 0) {
      double tot = 0.0;
      for (int k = 0; k < p.nch; ++k) tot += s_mass[k];
      s_tot = tot;
    }
    __syncthreads();
    // zero residual mass (reachable only through rounding): sample from p
    // itself, whose row (a node with children) has its statistics
    residual = s_tot > 0.0;
  }
  if (!residual) {
    // the chosen row's chunk statistics (device-scope loads: a leaf's were
    // written by this kernel's work-groups), masses in units of exp(M)
    if constexpr (TILES) {
      // after the LM head: each chunk's statistics folded from its tiles,
      // one tile per thread and a chunk's tiles on consecutive lanes; kQ
      // tiles per thread are loaded before any is used
      static_assert(kLmhTilesPerChunk <= 64 && (kLmhTilesPerChunk & (kLmhTilesPerChunk - 1)) == 0,
                    "a chunk's tiles fold inside one wave");
      constexpr int kQ = 4;
      const ChunkStat* ts = p.tiles + (int64_t)d.row * p.ntiles;
      for (int j0 = 0; j0 < p.ntiles; j0 += kQ * kAccThreads) {
        float tm[kQ];
        double tsm[kQ];
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
          const int j = j0 + q * kAccThreads + tid;
          tm[q] = -INFINITY;
          tsm[q] = 0.0;
          if (j < p.ntiles) {
            tm[q] = ts[j].m;
            tsm[q] = ts[j].s;
          }
        }
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
          const int j = j0 + q * kAccThreads + tid;
          float m = tm[q];
          for (int o = kLmhTilesPerChunk / 2; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
          double sum = j < p.ntiles ? tsm[q] * exp((double)tm[q] - (double)m) : 0.0;
          for (int o = kLmhTilesPerChunk / 2; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
          const int k = j / kLmhTilesPerChunk;
          if (j % kLmhTilesPerChunk == 0 && k < p.nch) {
            s_mass[k] = sum;
            s_mc[k] = m;
          }
        }
      }
    } else {
      for (int k = tid; k < p.nch; k += kAccThreads) {
        s_mass[k] = load_dev(&rst[k].s);
        s_mc[k] = __uint_as_float(__hip_atomic_load(reinterpret_cast<const uint32_t*>(&rst[k].m), __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT));
      }
    }
    __syncthreads();
    if (tid == 0) {
      float mx = -INFINITY;
      for (int k = 0; k < p.nch; ++k) mx = fmaxf(mx, s_mc[k]);
      double tot = 0.0;
      for (int k = 0; k < p.nch; ++k) {
        s_mass[k] = s_mass[k] * exp((double)s_mc[k] - (double)mx);
        tot += s_mass[k];
      }
      s_tot = tot;
      s_mrow = mx;                  // the row's max M
    }
    __syncthreads();
  }
  SV_TRACE(1, 5);
  const float u = p.uniforms[rq.q0 + N - 1];
  if (tid == 0) {
    const double tot = s_tot;
    const double target = (double)u * tot;
    double cum = 0.0;
    int chosen = -1, last_pos = 0;
    for (int k = 0; k < p.nch; ++k) {
      if (s_mass[k] > 0.0) last_pos = k;
      if (chosen < 0) {
        if (cum + s_mass[k] > target) chosen = k;
        else cum += s_mass[k];
      }
    }
    if (chosen < 0) {   // target rounded past the total: last chunk with mass
      chosen = last_pos;
      cum = 0.0;
      for (int k = 0; k < chosen; ++k) cum += s_mass[k];
    }
    s_chunk = chosen;
    if (residual) {
      s_mcc = 0.f;
      s_base = cum;
      s_target = target;
    } else {
      // the scan below runs in the chunk's own units exp(l - m_c)
      const float mc = s_mc[chosen];
      s_mcc = mc;
      s_base = 0.0;
      s_target = (target - cum) / exp((double)mc - (double)s_mrow);
    }
  }
  __syncthreads();
  SV_TRACE(1, 6);
  const int cc = s_chunk;
  const float mcc = s_mcc;
  float x[16], q[16];
  double w[16];
  load16_contiguous(Lr, cc * kAccChunk, p.V, -INFINITY, x);
  if (residual) load16_contiguous(Qr, cc * kAccChunk, p.V, 0.f, q);
  double tsum = 0.0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    w[k] = residual ? final_weight(x[k], q[k], d.M, invZ, true) : (double)exp_rel(x[k], mcc);
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
  const int v0 = cc * kAccChunk + 16 * tid;
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
    s_last_pos[tid >> 6] = lastpos;
  }
  __syncthreads();
  if (tid == 0) {
    int best = min(min(s_cand[0], s_cand[1]), min(s_cand[2], s_cand[3]));
    if (best == 0x7fffffff) best = max(max(s_last_pos[0], s_last_pos[1]), max(s_last_pos[2], s_last_pos[3]));
    p.next_tok[i] = best;
    p.acc_len[i] = d.len;
    if (p.acc_node) p.acc_node[i] = d.node;
  }
  SV_TRACE(1, 7);
}

// Sequential sibling verification over a token tree (SpecInfer's multi-step
// speculative sampling), C 1024-thread work-groups per request, each holding
// a contiguous slice of the vocabulary (whole 1024 x VW-entry chunks).  At
// the current node the children (BFS order) are tested against a running
// target distribution p', evaluated per token as
//   p'_0(v) = exp(l(v) - M) / Z,   p'_{j+1}(v) = max(0, p'_j(v) - q(v)) / S_{j+1},
// where S_{j+1} is the vocabulary sum of max(0, p'_j - q): each work-group
// takes its slice's part in one coalesced fp64 pass (16-byte loads, several
// chunks in flight), and the parts are exchanged (below) and added in slice
// order, so every work-group holds the same S and takes the same decisions;
// S is applied as its reciprocal (within an ulp of the division), and a zero
// sum, reachable only through rounding, leaves p' as it is.  Each child's
// test inputs (token, the parent row's logit and draft probability there,
// uniform) do not depend on the walk and are loaded up front.  The first
// accepted child becomes the current node; when none is, or the node is a
// leaf, the final token is the smallest id whose cumulative p' exceeds u *
// (its total): the slices' totals are exchanged, and the work-group whose
// slice holds the target scans it and writes the outputs.
//
// Exchange j of a request: each work-group writes its value with an
// agent-scope store, waits for it to complete, adds one to the request's
// counter (cleared by the row-statistics kernel before this launch), and
// waits until the counter reaches (j + 1) C before reading the C values
// with agent-scope loads (the acceptance's hand-over argument).  The
// request's work-groups are consecutive in the grid and dispatched in order,
// so every one the waiters depend on is resident or already dispatched ahead
// of them (a CPU model of the protocol checks this).  The wait is bounded:
// past kSeqSpinLimit polls the work-group gives up and writes -1 outputs.
constexpr int kSeqThreads = 1024;
constexpr int kSeqSpinLimit = 1 << 18;

template <int NW>
__device__ __forceinline__ double block_sum_n(double x, double* red) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < NW; ++w) s += red[w];
  return s;
}

// U block-wide fp64 sums at once (one pair of barriers), each in a fixed order.
template <int NW, int U>
__device__ __forceinline__ void block_sum_u(double (&x)[U], double* red) {
#pragma unroll
  for (int u = 0; u < U; ++u)
    for (int o = 32; o >= 1; o >>= 1) x[u] += __shfl_xor(x[u], o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int u = 0; u < U; ++u) red[u * NW + (threadIdx.x >> 6)] = x[u];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < U; ++u) {
    double s = 0.0;
    for (int w = 0; w < NW; ++w) s += red[u * NW + w];
    x[u] = s;
  }
}

// Exchange j of request i among its C work-groups: this one's (x, y) in,
// all C pairs out (in LDS, valid after the call for every thread).  Returns
// false if the wait gave up.
__device__ __forceinline__ bool seq_exchange(const AccParams& p, int i, int c, int C, int j, double x, int y,
                                             double* xs, int* ys, int* s_ok) {
  if (C == 1) {
    if (threadIdx.x == 0) {
      xs[0] = x;
      ys[0] = y;
    }
    __syncthreads();
    return true;
  }
  if (threadIdx.x == 0) {
    SeqSlot* base = p.seq_slots + ((int64_t)i * kMaxNodes + j) * C;
    store_dev(&base[c].x, x);
    __hip_atomic_store(&base[c].y, y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);     // both stores have reached the device coherence point
    __hip_atomic_fetch_add(p.tickets + i, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int want = (j + 1) * C;
    int ok = 1;
    for (int spins = 0; __hip_atomic_load(p.tickets + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < want;) {
      __builtin_amdgcn_s_sleep(2);
      if (++spins > kSeqSpinLimit) {
        ok = 0;
        break;
      }
    }
    for (int cc = 0; cc < C; ++cc) {
      xs[cc] = load_dev(&base[cc].x);
      ys[cc] = __hip_atomic_load(&base[cc].y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    *s_ok = ok;
  }
  __syncthreads();
  return *s_ok != 0;
}

template <typename T>
__global__ __launch_bounds__(kSeqThreads) void acc_tree_seq(AccParams p) {
  constexpr int NW = kSeqThreads / 64;
  constexpr int VW = 16 / sizeof(T);            // entries per 16-byte load
  constexpr int CH = kSeqThreads * VW;          // entries per chunk
  constexpr int UNR = 2;                        // chunks whose loads are in flight together
  __shared__ float s_M[kMaxNodes];
  __shared__ double s_Z[kMaxNodes];
  __shared__ double s_iS[kMaxNodes];           // 1 / S_j at the current node
  __shared__ float s_lx[kMaxNodes], s_qx[kMaxNodes], s_u[kMaxNodes];
  __shared__ double redd[NW];
  __shared__ double s_redu[NW * 4];              // U <= 4 sums at once (UNR and the resident RES)
  __shared__ int s_v;
  __shared__ double s_chunk[kAccMaxChunks * kAccChunk / (kSeqThreads * 4)];
  __shared__ double s_wtot[NW];
  __shared__ double s_run, s_target;
  __shared__ int s_pos[NW];
  __shared__ int s_pick;
  __shared__ int s_par[kMaxNodes], s_dep[kMaxNodes], s_qr[kMaxNodes];
  __shared__ double s_xs[kSeqMaxGroups];
  __shared__ int s_ys[kSeqMaxGroups];
  __shared__ int s_ok;
  SV_TRACE(1, 0);
  const int C = p.seq_groups;
  const int i = blockIdx.x / C, c = blockIdx.x % C;
  const int tid = threadIdx.x, wv = tid >> 6, ln = tid & 63;
  const ReqInfo rq = p.reqs[i];
  const int N = rq.nq;
  const T* L = static_cast<const T*>(p.logits);
  const T* Q = static_cast<const T*>(p.probs);
  // this work-group's chunks [ch0, ch1) of the vocabulary
  const int nchunk = (p.V + CH - 1) / CH;
  const int ch0 = (int)((int64_t)c * nchunk / C), ch1 = (int)((int64_t)(c + 1) * nchunk / C);

  // every child's test inputs, which do not depend on the walk: its token,
  // its parent's logit and draft probability there, and its uniform
  if (tid < N) {
    const NodeRec nr = node_rec(p, p.nodes, rq, tid);
    s_par[tid] = nr.par;
    s_dep[tid] = nr.dep;
    s_qr[tid] = nr.qr;
    if (tid >= 1) {
      const int x = min(max(p.tokens[rq.q0 - i + tid - 1], 0), p.V - 1);
      s_lx[tid] = ld(L + (int64_t)(rq.q0 + nr.par) * p.l_st, x);
      s_qx[tid] = nr.pq >= 0 ? ld(Q + (int64_t)(rq.d0 + nr.pq) * p.p_st, x) : 0.f;
      s_u[tid] = p.uniforms[rq.q0 + tid - 1];
    }
  }
  // (M, Z) of every row of the request, as in the decision kernel
  for (int r = wv; r < N; r += NW) {
    const ChunkStat* st = p.rowstats + (int64_t)(rq.q0 + r) * p.nch;
    float m = -INFINITY;
    for (int k = ln; k < p.nch; k += 64) m = fmaxf(m, st[k].m);
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    double z = 0.0;
    for (int k = ln; k < p.nch; k += 64) z += st[k].s * exp((double)st[k].m - (double)m);
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    if (ln == 0) {
      s_M[r] = m;
      s_Z[r] = z;
    }
  }
  __syncthreads();
  SV_TRACE(1, 1);

  int node = 0, k = 0, xj = 0;                 // current node, rejections at it, exchanges so far (uniform)
  const T* Lr = L;
  const T* Qr = Q;
  bool has_q = false;
  float M = 0.f;
  double invZ = 1.0;
  auto give_up = [&]() {
    if (tid == 0 && c == 0) {
      p.acc_len[i] = -1;
      p.next_tok[i] = -1;
      if (p.acc_node) p.acc_node[i] = -1;
    }
  };
  // running distribution at a token from its logit l and draft probability q
  auto prun = [&](float l, float q) -> double {
    double x = (double)exp_rel(l, M) * invZ;
    for (int j = 0; j < k; ++j) x = fmax(0.0, x - (double)q) * s_iS[j];
    return x;
  };
  // this thread's VW entries starting at v: logits (-inf past V) and draft
  // probabilities (0 past V, or everywhere for a node without a draft row)
  auto load = [&](int v, float* l, float* q) {
    load_vec(Lr, v, p.V, -INFINITY, l);
    if (has_q) load_vec(Qr, v, p.V, 0.f, q);
    else
      for (int e = 0; e < VW; ++e) q[e] = 0.f;
  };
  // A slice of at most RES chunks stays in registers while the walk is at a
  // node: loaded as the node is entered (in flight during its first test),
  // it serves every normaliser pass and the final sample there; longer
  // slices, and bf16 rows (whose unpacked entries would not fit the register
  // budget), are streamed per pass.  Both read the entries in the same order.
  constexpr int RES = 2;
  const bool resident = sizeof(T) == 4 && ch1 - ch0 <= RES;
  uint4 rl[RES], rqv[RES];
#pragma unroll
  for (int r = 0; r < RES; ++r) rl[r] = rqv[r] = make_uint4(0u, 0u, 0u, 0u);
  auto load_resident = [&]() {
    if (!resident) return;
#pragma unroll
    for (int r = 0; r < RES; ++r) {
      if (ch0 + r < ch1) {
        const int v = (ch0 + r) * CH + tid * VW;
        rl[r] = load_raw(Lr, v, p.V, -INFINITY);
        rqv[r] = has_q ? load_raw(Qr, v, p.V, 0.f) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };
  for (;;) {
    M = s_M[node];
    invZ = 1.0 / s_Z[node];
    Lr = L + (int64_t)(rq.q0 + node) * p.l_st;
    const int qr = s_qr[node];
    has_q = qr >= 0;
    Qr = Q + (int64_t)(rq.d0 + (has_q ? qr : 0)) * p.p_st;
    load_resident();
    k = 0;
    int next = -1;
    for (int cn = node + 1; cn < N && next < 0; ++cn) {
      if (s_par[cn] != node) continue;
      const float qx = s_qx[cn];
      const double px = prun(s_lx[cn], qx);
      if ((double)s_u[cn] * (double)qx < px) {
        next = cn;
        break;
      }
      // rejected: this slice's part of the normaliser of max(0, p' - q),
      // UNR chunks' loads in flight, then the parts of all slices
      double part = 0.0;
      if (resident) {
#pragma unroll
        for (int r = 0; r < RES; ++r)
          if (ch0 + r < ch1)
#pragma unroll
            for (int e = 0; e < VW; ++e) {
              const float q = entry<T>(rqv[r], e);
              part += fmax(0.0, prun(entry<T>(rl[r], e), q) - (double)q);
            }
      }
      for (int b = ch0 * CH; !resident && b < ch1 * CH; b += CH * UNR) {
        float l[UNR][VW], q[UNR][VW];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          if (b + u * CH < ch1 * CH) {
            load(b + u * CH + tid * VW, l[u], q[u]);
          } else {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
              l[u][e] = -INFINITY;
              q[u][e] = 0.f;
            }
          }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u)
#pragma unroll
          for (int e = 0; e < VW; ++e) part += fmax(0.0, prun(l[u][e], q[u][e]) - (double)q[u][e]);
      }
      part = block_sum_n<NW>(part, redd);
      if (!seq_exchange(p, i, c, C, xj++, part, 0, s_xs, s_ys, &s_ok)) return give_up();
      double S = 0.0;
      for (int cc = 0; cc < C; ++cc) S += s_xs[cc];
      if (S > 0.0) {
        if (tid == 0) s_iS[k] = 1.0 / S;
        __syncthreads();
        ++k;
      }
    }
    if (next < 0) break;
    node = next;
  }
  SV_TRACE(1, 2);

  // The final token from p' at `node`.  This slice's chunk totals (block
  // sums) and its last id with positive weight; the slices' totals and last
  // ids exchanged; the slice holding u * total (its running sum from the
  // slices before it) walks its chunk totals, the chosen chunk's per-thread
  // sums and that thread's entries in token order, so every boundary comes
  // from one sequence of fp64 sums.
  int last = -1;
  if (resident) {
    double part[RES];
#pragma unroll
    for (int r = 0; r < RES; ++r) {
      part[r] = 0.0;
      if (ch0 + r < ch1)
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const double w = prun(entry<T>(rl[r], e), entry<T>(rqv[r], e));
          part[r] += w;
          if (w > 0.0) last = (ch0 + r) * CH + tid * VW + e;
        }
    }
    block_sum_u<NW, RES>(part, s_redu);
    if (tid == 0)
#pragma unroll
      for (int r = 0; r < RES; ++r)
        if (ch0 + r < ch1) s_chunk[ch0 + r] = part[r];
    __syncthreads();
  }
  for (int c0 = ch0; !resident && c0 < ch1; c0 += UNR) {
    float l[UNR][VW], q[UNR][VW];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      if (c0 + u < ch1) {
        load((c0 + u) * CH + tid * VW, l[u], q[u]);
      } else {
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          l[u][e] = -INFINITY;
          q[u][e] = 0.f;
        }
      }
    }
    double part[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      part[u] = 0.0;
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        const double w = prun(l[u][e], q[u][e]);
        part[u] += w;
        if (w > 0.0) last = (c0 + u) * CH + tid * VW + e;
      }
    }
    block_sum_u<NW, UNR>(part, s_redu);
    if (tid == 0)
#pragma unroll
      for (int u = 0; u < UNR; ++u)
        if (c0 + u < ch1) s_chunk[c0 + u] = part[u];
    __syncthreads();                   // s_redu is reused by the next pass
  }
  for (int o = 32; o >= 1; o >>= 1) last = max(last, __shfl_xor(last, o));
  if (ln == 0) s_pos[wv] = last;
  __syncthreads();
  SV_TRACE(1, 3);
  double slice = 0.0;
  int slice_last = -1;
  if (tid == 0) {
    for (int ch = ch0; ch < ch1; ++ch) slice += s_chunk[ch];
    for (int w = 0; w < NW; ++w) slice_last = max(slice_last, s_pos[w]);
  }
  if (!seq_exchange(p, i, c, C, xj++, slice, slice_last, s_xs, s_ys, &s_ok)) return give_up();
  // the slice that holds the target writes the outputs; if none does (the
  // target rounded to or past the total), the last slice with positive weight
  // writes its last such id
  double total = 0.0;
  for (int cc = 0; cc < C; ++cc) total += s_xs[cc];
  const double target = (double)p.uniforms[rq.q0 + N - 1] * total;
  int owner = -1, fallback = -1;
  double before = 0.0, before_owner = 0.0;
  for (int cc = 0; cc < C; ++cc) {
    if (owner < 0 && s_xs[cc] > 0.0 && before + s_xs[cc] > target) {
      owner = cc;
      before_owner = before;
    }
    before += s_xs[cc];
    if (s_ys[cc] >= 0) fallback = cc;
  }
  const int writer = owner >= 0 ? owner : (fallback >= 0 ? fallback : 0);
  SV_TRACE(1, 4);
  if (c != writer) return;
  if (tid == 0) {
    const double t = target;
    double run = owner >= 0 ? before_owner : 0.0;
    int pick = -1;
    if (owner >= 0)
      for (int ch = ch0; ch < ch1 && pick < 0; ++ch) {
        if (run + s_chunk[ch] > t) pick = ch;
        else run += s_chunk[ch];
      }
    s_pick = pick;
    s_run = run;
    s_target = t;
  }
  __syncthreads();
  SV_TRACE(1, 5);
  // Inside the chosen chunk: each thread's sum of its VW entries, a prefix
  // over the threads (a scan in each wave, then the waves' totals), and the
  // thread whose range holds the target scans its own entries.
  if (tid == 0) s_v = INT_MAX;
  if (s_pick >= 0) {
    const int vb = s_pick * CH + tid * VW;
    float l[VW], q[VW];
    if (resident) {
      const int pr = s_pick - ch0;
#pragma unroll
      for (int r = 0; r < RES; ++r)
        if (r == pr)
#pragma unroll
          for (int e = 0; e < VW; ++e) {
            l[e] = entry<T>(rl[r], e);
            q[e] = entry<T>(rqv[r], e);
          }
    } else {
      load(vb, l, q);
    }
    double w[VW];
    double part = 0.0;
#pragma unroll
    for (int e = 0; e < VW; ++e) {
      w[e] = prun(l[e], q[e]);
      part += w[e];
    }
    double incl = part;
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(incl, o);
      if (ln >= o) incl += y;
    }
    if (ln == 63) s_wtot[wv] = incl;
    __syncthreads();
    double cum = s_run;
    for (int ww = 0; ww < wv; ++ww) cum += s_wtot[ww];
    cum += incl - part;                   // before this thread's entries
    const double t = s_target;
    if (part > 0.0 && cum <= t && cum + part > t) {
      // one thread in exact arithmetic; should rounding let two ranges
      // straddle the target, the smaller id wins, whatever their order
      int v = -1;
      for (int e = 0; e < VW && v < 0; ++e) {
        cum += w[e];
        if (cum > t) v = vb + e;
      }
      if (v >= 0) atomicMin(&s_v, v);
    }
  }
  __syncthreads();
  int v = s_v == INT_MAX ? -1 : s_v;
  if (tid == 0) {
    // a target at or past this slice's total (rounding): its last id with positive weight
    if (v < 0) v = s_ys[c];
    p.acc_len[i] = s_dep[node];
    p.next_tok[i] = v;
    if (p.acc_node) p.acc_node[i] = node;
  }
  SV_TRACE(1, 7);
}

// One work-group: every request's draft tokens, their draft probabilities
// and the uniforms, against the caller's contract (debug builds of a call).
template <typename T>
__global__ __launch_bounds__(kAccThreads) void acc_validate(AccParams p, uint32_t* flag) {
  if (threadIdx.x == 0) *flag = 0u;
  __syncthreads();
  uint32_t bad = 0u;
  const T* Q = static_cast<const T*>(p.probs);
  for (int i = threadIdx.x; i < p.B; i += kAccThreads) {
    const ReqInfo rq = p.reqs_src[i];   // runs before the row statistics make the device copy
    for (int n = 0; n < rq.nq; ++n) {
      const float u = p.uniforms[rq.q0 + n];
      if (!(u >= 0.f && u < 1.f)) bad |= 2u;
      if (n == 0) continue;
      const int x = p.tokens[rq.q0 - i + n - 1];
      if (x < 0 || x >= p.V) {
        bad |= 1u;
        continue;
      }
      const float qx = ld(Q, (int64_t)(rq.d0 + node_rec(p, p.nodes_src, rq, n).pq) * p.p_st + x);
      if (!(qx > 0.f)) bad |= 4u;
    }
  }
  if (bad) atomicOr(flag, bad);
}

// Chunk statistics from the LM head's tile statistics: thread t of the grid
// folds the kLmhTilesPerChunk tiles of one (row, chunk) in tile order into
// (max, sum of exp(l - max)), max over the tiles' maxima and the tiles' sums
// rescaled in fp64.  The first B work-groups also make the device copies of
// the request and node tables and clear the tickets, as the row-statistics
// kernel does on the unfused path.
__global__ __launch_bounds__(kAccThreads) void acc_foldstats(AccParams p, const ChunkStat* tiles, int ntiles) {
  if (blockIdx.x < p.B) {
    if (threadIdx.x < 2)
      reinterpret_cast<uint4*>(p.reqs + blockIdx.x)[threadIdx.x] =
          reinterpret_cast<const uint4*>(p.reqs_src + blockIdx.x)[threadIdx.x];
    if (threadIdx.x == 0) p.tickets[blockIdx.x] = 0;
    if (p.per_req)
      for (int x = blockIdx.x * kAccThreads + threadIdx.x; x < p.nodes_n16; x += p.B * kAccThreads)
        reinterpret_cast<uint4*>(p.nodes)[x] = reinterpret_cast<const uint4*>(p.nodes_src)[x];
  }
  const int64_t idx = (int64_t)blockIdx.x * kAccThreads + threadIdx.x;
  if (idx >= (int64_t)p.Nq * p.nch) return;
  const int row = (int)(idx / p.nch), c = (int)(idx % p.nch);
  const int t0 = c * kLmhTilesPerChunk, t1 = min(t0 + kLmhTilesPerChunk, ntiles);
  const ChunkStat* ts = tiles + (int64_t)row * ntiles;
  float m = -INFINITY;
  for (int t = t0; t < t1; ++t) m = fmaxf(m, ts[t].m);
  double sum = 0.0;
  for (int t = t0; t < t1; ++t) sum += ts[t].s * exp((double)ts[t].m - (double)m);
  p.rowstats[idx] = ChunkStat{sum, m, 0.f};
}

}  // namespace

hipError_t launch_foldstats(const AccParams& p, const ChunkStat* tiles, int ntiles, hipStream_t s) {
  const int64_t n = (int64_t)p.Nq * p.nch;
  const dim3 grid((unsigned)std::max<int64_t>((n + kAccThreads - 1) / kAccThreads, p.B));
  acc_foldstats<<<grid, dim3(kAccThreads), 0, s>>>(p, tiles, ntiles);
  return hipGetLastError();
}

#ifdef SV_ACC_TRACE
extern "C" __attribute__((visibility("default"))) int sv_acc_trace_copy(void* dst, size_t bytes) {
  return (int)hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_acc_trace), bytes);
}
#endif

hipError_t launch_accept_validate(const AccParams& p, uint32_t* flag, hipStream_t s) {
  if (p.bf16) acc_validate<uint16_t><<<1, kAccThreads, 0, s>>>(p, flag);
  else acc_validate<float><<<1, kAccThreads, 0, s>>>(p, flag);
  return hipGetLastError();
}

hipError_t launch_rowstats(const AccParams& p, hipStream_t s) {
  dim3 block(kAccThreads);
  // independent tree rule: the rows of nodes with children (at least B work-groups)
  const int64_t rows = (p.tree == 1 && !p.all_stats) ? (int64_t)p.B * p.topo.n_inner : (int64_t)p.Nq;
  if (p.bf16) {
    constexpr int SUB = RowGeo<uint16_t>::SUB;
    const dim3 grid((unsigned)std::max<int64_t>(rows * ((p.nch + SUB - 1) / SUB), p.B));
    acc_rowstats<uint16_t><<<grid, block, 0, s>>>(p);
  } else {
    constexpr int SUB = RowGeo<float>::SUB;
    const dim3 grid((unsigned)std::max<int64_t>(rows * ((p.nch + SUB - 1) / SUB), p.B));
    acc_rowstats<float><<<grid, block, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_decide(const AccParams& p, hipStream_t s) {
  dim3 block(kAccThreads);
  if (p.tree == 2) {                       // sequential sibling verification
    const dim3 grid((unsigned)(p.B * p.seq_groups));
    if (p.bf16) acc_tree_seq<uint16_t><<<grid, dim3(kSeqThreads), 0, s>>>(p);
    else acc_tree_seq<float><<<grid, dim3(kSeqThreads), 0, s>>>(p);
    return hipGetLastError();
  }
  const dim3 grid((unsigned)(p.B * p.nch));
  if (p.tiles) {
    if (p.bf16) acc_decide_select<uint16_t, true><<<grid, block, 0, s>>>(p);
    else acc_decide_select<float, true><<<grid, block, 0, s>>>(p);
  } else {
    if (p.bf16) acc_decide_select<uint16_t, false><<<grid, block, 0, s>>>(p);
    else acc_decide_select<float, false><<<grid, block, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_accept(const AccParams& p, hipStream_t s, hipEvent_t mid) {
  hipError_t e = launch_rowstats(p, s);
  if (e != hipSuccess) return e;
  if (mid && (e = hipEventRecord(mid, s)) != hipSuccess) return e;
  return launch_decide(p, s);
}

}  // namespace sv
