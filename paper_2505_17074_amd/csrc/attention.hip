// Verify attention for gfx950: split-KV partial kernels and the split combine.
//
// Each work item is one KV range [kb, ke) of one (request, KV head, group of
// query heads).  Its query rows are the group's heads times the request's
// n_i verify positions; every row sees the request's cached positions plus
// its own ancestors-or-self inside the verify block (causal for a chain).
// Scores and the online softmax run in fp32; the running max is kept in log2
// units (scores pre-multiplied by scale * log2 e) so exp2 is one v_exp_f32.
#include "sv_internal.h"

namespace sv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ float wave_max(float x) {
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// Visibility of KV position t (relative to the request's first KV row) to a
// query whose node has ancestor mask `anc`; ctx = cached positions.
__device__ __forceinline__ bool visible(int t, int ctx, uint32_t anc) {
  return t < ctx || ((anc >> (t - ctx)) & 1u);
}

// ---------------------------------------------------------------------------
// bf16 MFMA path.  One wave per work item, all query rows of the item in NR
// tiles of 16.  Per 32-key tile:
//   S^T[key, row] = K[key, :] . Q[row, :]      v_mfma_f32_16x16x32_bf16, K as A
//   online softmax over keys (fp32, log2 domain)
//   O^T[e, row]  += V^T[e, key] . P^T[key, row] with P = hi + lo in two bf16
//                   parts, so P's rounding stays near fp32 (error ~2^-17)
// The 16 MFMA A-rows of key tile kt hold keys 8*(m>>2) + 4*kt + (m&3): the
// C layout then leaves lane group g holding keys 8g..8g+7 of its query row,
// which is exactly the B operand the PV product needs, with no data movement.
// V is staged through a wave-private LDS tile and read back transposed
// (8 keys of one column per lane).
// ---------------------------------------------------------------------------
template <int D, int NR>
__global__ __launch_bounds__(64) void attn_split_mfma(AttnParams p) {
  constexpr int KS = D / 32;       // QK k-steps
  constexpr int ET = D / 16;       // PV column tiles
  constexpr int VCH = D / 16;      // 16-byte V chunks per lane per tile
  constexpr int PITCH = D + 2;     // LDS row pitch (bf16): odd dword count, conflict-free columns
  __shared__ uint16_t vt[32 * PITCH];

  const int lane = threadIdx.x;
  const int c16 = lane & 15, grp = lane >> 4;
  const AttnItem it = p.items[blockIdx.x];
  const ReqInfo rq = p.reqs[it.req];
  const int n = rq.nq;
  const int R = it.nheads * n;
  const int ctx = rq.ctx;
  const uint16_t* __restrict__ Kb =
      static_cast<const uint16_t*>(p.k) + (int64_t)rq.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;
  const uint16_t* __restrict__ Vb =
      static_cast<const uint16_t*>(p.v) + (int64_t)rq.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;

  bf16x8 qop[NR][KS];
  uint32_t anc[NR];
#pragma unroll
  for (int rt = 0; rt < NR; ++rt) {
    const int r = rt * 16 + c16;
    if (r < R) {
      const int hh = r / n, j = r - hh * n;
      const uint16_t* qp = static_cast<const uint16_t*>(p.q) + (int64_t)(rq.q0 + j) * p.q_st +
                           (int64_t)(it.head_lo + hh) * p.q_sh + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qop[rt][ks] = *reinterpret_cast<const bf16x8*>(qp + ks * 32);
      anc[rt] = p.topo->anc[j];
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qop[rt][ks] = bf16x8{};
      anc[rt] = 0u;
    }
  }

  f32x4 o[NR][ET];
  float m_run[NR], l_run[NR];
#pragma unroll
  for (int rt = 0; rt < NR; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.f;
#pragma unroll
    for (int et = 0; et < ET; ++et) o[rt][et] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int nrt = (R + 15) >> 4;   // active row tiles (wave-uniform)

  for (int t0 = it.kb; t0 < it.ke; t0 += 32) {
    // K operands straight from HBM in MFMA A layout (16 B per lane per k-step)
    bf16x8 kop[2][KS];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int key = min(t0 + 8 * (c16 >> 2) + 4 * kt + (c16 & 3), it.ke - 1);
      const uint16_t* kp = Kb + (int64_t)key * p.kv_st + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kop[kt][ks] = *reinterpret_cast<const bf16x8*>(kp + ks * 32);
    }
    // V tile, coalesced: consecutive lanes read consecutive 16 B of a key row
    uint4 vraw[VCH];
#pragma unroll
    for (int c = 0; c < VCH; ++c) {
      const int chunk = c * 64 + lane;
      const int key = min(t0 + chunk / (D / 8), it.ke - 1);
      vraw[c] = *reinterpret_cast<const uint4*>(Vb + (int64_t)key * p.kv_st + (chunk % (D / 8)) * 8);
    }
    __syncthreads();   // previous tile's transposed reads are done
#pragma unroll
    for (int c = 0; c < VCH; ++c) {
      const int chunk = c * 64 + lane;
      uint32_t* dst = reinterpret_cast<uint32_t*>(vt + (chunk / (D / 8)) * PITCH + (chunk % (D / 8)) * 8);
      dst[0] = vraw[c].x;
      dst[1] = vraw[c].y;
      dst[2] = vraw[c].z;
      dst[3] = vraw[c].w;
    }
    __syncthreads();
    bf16x8 vop[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et) {
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        const uint16_t bits = vt[(8 * grp + m) * PITCH + et * 16 + c16];
        vop[et][m] = __builtin_bit_cast(__bf16, bits);
      }
    }

#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      if (rt >= nrt) break;
      f32x4 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[kt][ks], qop[rt][ks], acc, 0, 0, 0);
        s[kt] = acc;
      }
      float sv[8];
      float mloc = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 8 * grp + 4 * kt + i;
          float x = s[kt][i] * p.scale_log2;
          if (t >= it.ke || !visible(t, ctx, anc[rt])) x = -INFINITY;
          sv[kt * 4 + i] = x;
          mloc = fmaxf(mloc, x);
        }
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run[rt], mloc);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run[rt] - m_use);
      float psum = 0.f;
      bf16x8 phi, plo;
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const float pv = exp2f(sv[x] - m_use);
        psum += pv;
        const __bf16 h = static_cast<__bf16>(pv);
        phi[x] = h;
        plo[x] = static_cast<__bf16>(pv - static_cast<float>(h));
      }
      l_run[rt] = l_run[rt] * alpha + psum;
      m_run[rt] = m_new;
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        o[rt][et] *= alpha;
        o[rt][et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[et], phi, o[rt][et], 0, 0, 0);
        o[rt][et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[et], plo, o[rt][et], 0, 0, 0);
      }
    }
  }

#pragma unroll
  for (int rt = 0; rt < NR; ++rt) {
    float l = l_run[rt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int r = rt * 16 + c16;
    if (r >= R) continue;
    const int hh = r / n, j = r - hh * n, h = it.head_lo + hh;
    if (it.seg < 0) {
      const float inv = 1.f / l;
      float* op = p.out + ((int64_t)(rq.q0 + j) * p.Hq + h) * D + 4 * grp;
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        const f32x4 v = o[rt][et] * inv;
        *reinterpret_cast<float4*>(op + et * 16) = make_float4(v[0], v[1], v[2], v[3]);
      }
    } else {
      const int64_t pr = (int64_t)rq.part0 + ((int64_t)it.seg * n + j) * p.Hq + h;
      float* op = p.part_o + pr * D + 4 * grp;
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        const f32x4 v = o[rt][et];
        *reinterpret_cast<float4*>(op + et * 16) = make_float4(v[0], v[1], v[2], v[3]);
      }
      if (grp == 0) p.part_ml[pr] = make_float2(m_run[rt], l);
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 (or widened bf16) VALU path: one 256-thread work-group per item,
// 64-key tiles staged in LDS.  Used for fp32 inputs, whose products the bf16
// matrix cores cannot take without rounding.
// Rows per item <= kValuRows(D) = 4096 / D, 16 output values per thread.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ float load_elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_split_valu(AttnParams p) {
  constexpr int TK = 64;
  constexpr int RV = 4096 / D;           // max rows per item
  constexpr int OPT = RV * D / 256;      // outputs per thread (16)
  __shared__ float qs[RV][D + 1];
  __shared__ float ks[TK][D + 1];
  __shared__ float vs[TK][D];
  __shared__ float ps[RV][TK];
  __shared__ float alpha_s[RV];
  __shared__ float ml_s[RV][2];

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const AttnItem it = p.items[blockIdx.x];
  const ReqInfo rq = p.reqs[it.req];
  const int n = rq.nq;
  const int R = it.nheads * n;
  const int ctx = rq.ctx;
  const T* Kb = static_cast<const T*>(p.k) + (int64_t)rq.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;
  const T* Vb = static_cast<const T*>(p.v) + (int64_t)rq.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;

  for (int x = tid; x < RV * D; x += 256) {
    const int r = x / D, e = x % D;
    float val = 0.f;
    if (r < R) {
      const int hh = r / n, j = r - hh * n;
      val = load_elem<T>(static_cast<const T*>(p.q),
                         (int64_t)(rq.q0 + j) * p.q_st + (int64_t)(it.head_lo + hh) * p.q_sh + e);
    }
    qs[r][e] = val;
  }
  for (int r = tid; r < RV; r += 256) {
    ml_s[r][0] = -INFINITY;
    ml_s[r][1] = 0.f;
  }
  float o[OPT];
#pragma unroll
  for (int x = 0; x < OPT; ++x) o[x] = 0.f;

  for (int t0 = it.kb; t0 < it.ke; t0 += TK) {
    __syncthreads();
    for (int x = tid; x < TK * D; x += 256) {
      const int t = x / D, e = x % D;
      const int key = min(t0 + t, it.ke - 1);
      ks[t][e] = load_elem<T>(Kb, (int64_t)key * p.kv_st + e);
      vs[t][e] = load_elem<T>(Vb, (int64_t)key * p.kv_st + e);
    }
    __syncthreads();
    const int t = t0 + lane;
    for (int r = wv; r < R; r += 4) {
      float s = 0.f;
#pragma unroll 8
      for (int e = 0; e < D; ++e) s += qs[r][e] * ks[lane][e];
      const int j = r % n;
      s *= p.scale_log2;
      if (t >= it.ke || !visible(t, ctx, p.topo->anc[j])) s = -INFINITY;
      const float m_old = ml_s[r][0];
      const float m_new = fmaxf(m_old, wave_max(s));
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float pv = exp2f(s - m_use);
      const float psum = wave_sum(pv);
      ps[r][lane] = pv;
      if (lane == 0) {
        const float a = exp2f(m_old - m_use);
        alpha_s[r] = a;
        ml_s[r][0] = m_new;
        ml_s[r][1] = ml_s[r][1] * a + psum;
      }
    }
    __syncthreads();
#pragma unroll
    for (int x = 0; x < OPT; ++x) {
      const int idx = tid + 256 * x;
      const int r = idx / D, e = idx % D;
      if (r < R) {
        float acc = o[x] * alpha_s[r];
#pragma unroll 8
        for (int tt = 0; tt < TK; ++tt) acc += ps[r][tt] * vs[tt][e];
        o[x] = acc;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int x = 0; x < OPT; ++x) {
    const int idx = tid + 256 * x;
    const int r = idx / D, e = idx % D;
    if (r >= R) continue;
    const int hh = r / n, j = r - hh * n, h = it.head_lo + hh;
    if (it.seg < 0) {
      p.out[((int64_t)(rq.q0 + j) * p.Hq + h) * D + e] = o[x] / ml_s[r][1];
    } else {
      const int64_t pr = (int64_t)rq.part0 + ((int64_t)it.seg * n + j) * p.Hq + h;
      p.part_o[pr * D + e] = o[x];
      if (e == 0) p.part_ml[pr] = make_float2(ml_s[r][0], ml_s[r][1]);
    }
  }
}

// ---------------------------------------------------------------------------
// Split combine: one wave per (query row, head) of a request with nseg > 1.
//   O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, splits in fixed order.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void attn_combine(AttnParams p) {
  constexpr int PER = D / 64;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= (int64_t)p.Nq * p.Hq) return;
  const int qrow = (int)(row / p.Hq), h = (int)(row % p.Hq);
  const ReqInfo rq = p.reqs[p.row_req[qrow]];
  if (rq.nseg <= 1) return;
  const int j = qrow - rq.q0, n = rq.nq;
  float M = -INFINITY;
  for (int s = 0; s < rq.nseg; ++s)
    M = fmaxf(M, p.part_ml[rq.part0 + ((int64_t)s * n + j) * p.Hq + h].x);
  float acc[PER];
#pragma unroll
  for (int x = 0; x < PER; ++x) acc[x] = 0.f;
  float L = 0.f;
  for (int s = 0; s < rq.nseg; ++s) {
    const int64_t pr = rq.part0 + ((int64_t)s * n + j) * p.Hq + h;
    const float2 ml = p.part_ml[pr];
    const float w = (ml.x == -INFINITY) ? 0.f : exp2f(ml.x - M);
    L += ml.y * w;
#pragma unroll
    for (int x = 0; x < PER; ++x) acc[x] += w * p.part_o[pr * D + lane + 64 * x];
  }
  const float inv = 1.f / L;
#pragma unroll
  for (int x = 0; x < PER; ++x) p.out[((int64_t)qrow * p.Hq + h) * D + lane + 64 * x] = acc[x] * inv;
}

template <int D>
hipError_t launch_mfma(const AttnParams& p, int nr, hipStream_t s) {
  dim3 grid(p.n_items), block(64);
  switch (nr) {
    case 1: attn_split_mfma<D, 1><<<grid, block, 0, s>>>(p); break;
    case 2: attn_split_mfma<D, 2><<<grid, block, 0, s>>>(p); break;
    case 3: attn_split_mfma<D, 3><<<grid, block, 0, s>>>(p); break;
    case 4: attn_split_mfma<D, 4><<<grid, block, 0, s>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int max_rows_per_item(int dtype_bf16, int D) { return dtype_bf16 ? 64 : 4096 / D; }

hipError_t launch_attention(const AttnParams& p, int dtype_bf16, int nr_max, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (p.n_items > 0) {
    if (dtype_bf16) {
      e = (p.D == 64) ? launch_mfma<64>(p, nr_max, s) : launch_mfma<128>(p, nr_max, s);
    } else {
      dim3 grid(p.n_items), block(256);
      if (p.D == 64) attn_split_valu<float, 64><<<grid, block, 0, s>>>(p);
      else attn_split_valu<float, 128><<<grid, block, 0, s>>>(p);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
  }
  return e;
}

hipError_t launch_combine(const AttnParams& p, hipStream_t s) {
  const int64_t rows = (int64_t)p.Nq * p.Hq;
  dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (p.D == 64) attn_combine<64><<<grid, block, 0, s>>>(p);
  else attn_combine<128><<<grid, block, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace sv
