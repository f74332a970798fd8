// The target model's LM head for the verify step (gfx950): the verify
// positions' logits, logits = hidden . weight^T, the forward that produces
// the target distributions of Eq. (1) (Sec. 2.2), with the softmax
// statistics of every (row, 256-entry tile) taken in the epilogue so that
// the acceptance never re-reads the logits for its normalisers.
//
// hidden [M, K] and weight [V, K] (one row per vocabulary entry, the linear
// layer's layout) are bf16 and both contiguous along K, so the operands of
// v_mfma_f32_16x16x32_bf16 are plain 16-byte row reads: lane l takes row
// l % 16, k = 8 (l / 16) .. +7 of a 16-row block, for the A (hidden) and the
// B (weight) operand alike, and holds C[4 (l / 16) + i][l % 16].
//
// A work-group (4 waves) computes a tile of 16 MB rows x 256 vocabulary
// entries: wave w owns entries 64 w .. 64 w + 63 (four 16-column blocks) of
// every row block.  32-k slices of the hidden rows and the weight rows
// stream HBM -> LDS through an NS-stage ring of direct buffer -> LDS
// transfers (the attention kernel's ring); the hidden rows are re-read by
// every vocabulary tile (they stay in L2), each weight byte is read by the
// work-groups of its vocabulary tile, which are launched together on one
// XCD so that only the first of them reads it from HBM.
#include "sv_internal.h"

#include <algorithm>

namespace sv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kRowB = 64;            // bytes of one 32-k row slice in LDS
#ifndef SV_LMH_WAVES
#define SV_LMH_WAVES 8
#endif
#ifndef SV_LMH_MAXROWS
#define SV_LMH_MAXROWS 128
#endif
constexpr int kLmhWaves = SV_LMH_WAVES;   // waves per work-group
constexpr int kLmhThreads = 64 * kLmhWaves;
constexpr int kLmhCB = kLmhNT / (16 * kLmhWaves);   // 16-column blocks per wave

template <int N>
__device__ __forceinline__ void lmh_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void lmh_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// 16-byte chunk c of LDS row r sits at chunk c ^ swz(r): the 16 rows one
// quarter-wave reads (a 16-row block, one chunk each) fall on 16 distinct
// 4-bank groups.
__device__ __forceinline__ int lmh_swz(int r) { return (r >> 2) & 3; }

template <int MB>
struct LmhGeo {
  static constexpr int RA = 16 * MB;                  // hidden rows per tile
  static constexpr int ROWS = RA + kLmhNT;            // LDS rows per stage
  static constexpr int STAGE = ROWS * kRowB;
  static constexpr int XF = ROWS / 16;                // 1 KB transfers per stage (16 rows each)
  static constexpr int PER = (XF + kLmhWaves - 1) / kLmhWaves;   // per wave (padded with repeats)
};

// Ring depth by row blocks: weight-streaming shapes (few rows) keep more
// stages in flight; the LDS also holds the epilogue's reductions.
template <int MB>
struct LmhStages {
  // as many stages as 144 KB of LDS holds, at most 6
  static constexpr int fit = (144 * 1024) / LmhGeo<MB>::STAGE;
  static constexpr int value = fit < 6 ? fit : 6;
};

template <int MB, int NS, bool BF16OUT>
__global__ __launch_bounds__(kLmhThreads) void lmh_gemm(LmhParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using G = LmhGeo<MB>;
  constexpr int PER = G::PER;
  __shared__ __attribute__((aligned(1024))) char lds[NS * G::STAGE];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15, grp = lane >> 4;

  // block -> (row tile, vocabulary tile): the row tiles of one vocabulary
  // tile are 8 blocks apart (one XCD of the round-robin dispatch) and within
  // one window of 8 * m_tiles blocks, so they run together and share that
  // tile's weight rows in the XCD's L2
  const int T = p.m_tiles;
  const int g = blockIdx.x / (8 * T), r8 = blockIdx.x % (8 * T);
  const int mt = r8 / 8, nt = g * 8 + (r8 % 8);
  if (nt >= p.ntiles) return;                       // uniform: past the vocabulary
  const int m0 = mt * G::RA, n0 = nt * kLmhNT;
  const int mrows = min(G::RA, p.M - m0), ncols = min(kLmhNT, p.V - n0);
  if (mrows <= 0) return;
  // buffer resources over this tile's rows: loads past them read zeros
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.hidden + (int64_t)m0 * p.h_st), 0, (uint32_t)(mrows * p.h_st * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.weight + (int64_t)n0 * p.w_st), 0, (uint32_t)(ncols * p.w_st * 2), 0x00020000);
  // this lane's byte offset in each of its transfers (the k slice's start is soffset)
  uint32_t off[PER];
  bool isw[PER];
  int dst[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int j = (w + kLmhWaves * q) % G::XF;       // transfer index (repeats pad the last wave)
    const int row = 16 * j + lane / 4;               // LDS row of this lane's chunk
    const int chunk = (lane & 3) ^ lmh_swz(row);     // global chunk that lands at LDS chunk lane & 3
    isw[q] = row >= G::RA;
    const int grow = isw[q] ? row - G::RA : row;
    off[q] = (uint32_t)grow * (uint32_t)((isw[q] ? p.w_st : p.h_st) * 2) + (uint32_t)chunk * 16u;
    dst[q] = j * 1024;
  }
  auto issue = [&](int stage, int t) {
    char* base = lds + stage * G::STAGE;
    const uint32_t soff = (uint32_t)t * 64u;          // 32 bf16 of k per slice
#pragma unroll
    for (int q = 0; q < PER; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isw[q] ? rw : rh, (lds_void_t*)(base + dst[q]), 16, off[q], soff, 0,
                                               0);
  };

  constexpr int CB = kLmhCB;
  f32x4 acc[MB][CB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // LDS read offsets (stage 0) of this lane's A rows and B rows
  uint32_t aoff[MB], boff[CB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) {
    const int row = 16 * rb + l16;
    aoff[rb] = row * kRowB + ((grp ^ lmh_swz(row)) * 16);
  }
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int row = G::RA + 16 * CB * w + 16 * cb + l16;
    boff[cb] = row * kRowB + ((grp ^ lmh_swz(row)) * 16);
  }

  const int nk = p.K / 32;
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) issue(st, st);
  for (int t = 0; t < nk; ++t) {
    const int stage = t % NS;
    // this wave's transfers of slice t have landed (later ones may still fly)
    if (t + NS - 2 < nk) lmh_wait_vm<PER * (NS - 2)>();
    else lmh_wait_vm<0>();
    lmh_barrier();                  // everyone's have; stage (t - 1) % NS is free
    if (t + NS - 1 < nk) issue((t + NS - 1) % NS, t + NS - 1);
    const char* sb = lds + stage * G::STAGE;
    bf16x8 bop[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) bop[cb] = *reinterpret_cast<const bf16x8*>(sb + boff[cb]);
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      const bf16x8 aop = *reinterpret_cast<const bf16x8*>(sb + aoff[rb]);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[cb], acc[rb][cb], 0, 0, 0);
    }
  }
  lmh_wait_vm<0>();
  __syncthreads();                  // the ring is no longer read: reuse its LDS

  // Epilogue.  The logits are stored (fp32, or rounded to bf16), and the
  // statistics of each row over the tile's 256 entries are taken on the
  // stored values: the maximum, then the sum of exp(l - max) in fp64, lane
  // sums in column-block order, then across the 16 lanes of a row by an xor
  // butterfly, then across the four waves in wave order.
  constexpr int NW = kLmhWaves;
  float* red_m = reinterpret_cast<float*>(lds);                     // [NW][RA]
  double* red_s = reinterpret_cast<double*>(lds + NW * G::RA * 4);  // [NW][RA]
  float val[MB][CB][4];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int col = 16 * CB * w + 16 * cb + l16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * rb + 4 * grp + i;
        float v = acc[rb][cb][i];
        if constexpr (BF16OUT) {
          const uint32_t u = __float_as_uint(v);
          const uint16_t b = (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);   // round to nearest even
          v = __uint_as_float((uint32_t)b << 16);
          if (row < mrows && col < ncols)
            static_cast<uint16_t*>(p.out)[(int64_t)(m0 + row) * p.o_st + n0 + col] = b;
        } else {
          if (row < mrows && col < ncols) static_cast<float*>(p.out)[(int64_t)(m0 + row) * p.o_st + n0 + col] = v;
        }
        val[rb][cb][i] = col < ncols ? v : -INFINITY;
      }
    }
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = val[rb][0][i];
#pragma unroll
      for (int cb = 1; cb < CB; ++cb) m = fmaxf(m, val[rb][cb][i]);
      for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
      if (l16 == 0) red_m[w * G::RA + 16 * rb + 4 * grp + i] = m;
    }
  __syncthreads();
  auto row_max = [&](int row) {
    float m = red_m[row];
#pragma unroll
    for (int x = 1; x < NW; ++x) m = fmaxf(m, red_m[x * G::RA + row]);
    return m;
  };
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * rb + 4 * grp + i;
      const float m = row_max(row);
      double sm = 0.0;
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) sm += (double)exp_rel(val[rb][cb][i], m);
      for (int o = 1; o < 16; o <<= 1) sm += __shfl_xor(sm, o);
      if (l16 == 0) red_s[w * G::RA + row] = sm;
    }
  __syncthreads();
  for (int row = threadIdx.x; row < mrows; row += kLmhThreads) {
    double sm = red_s[row];
#pragma unroll
    for (int x = 1; x < NW; ++x) sm += red_s[x * G::RA + row];
    p.tiles[(int64_t)(m0 + row) * p.ntiles + nt] = ChunkStat{sm, row_max(row), 0.f};
  }
#endif
}

template <int MB>
hipError_t launch_mb(const LmhParams& p, hipStream_t s) {
  const int groups = (p.ntiles + 7) / 8;
  const dim3 grid((unsigned)(groups * 8 * p.m_tiles));
  constexpr int NS = LmhStages<MB>::value;
  if (p.out_bf16) lmh_gemm<MB, NS, true><<<grid, dim3(kLmhThreads), 0, s>>>(p);
  else lmh_gemm<MB, NS, false><<<grid, dim3(kLmhThreads), 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

int lmh_row_blocks(int M) {
  const int tiles = (M + SV_LMH_MAXROWS - 1) / SV_LMH_MAXROWS;
  const int rows = (M + tiles - 1) / tiles;
  return (rows + 15) / 16;
}

hipError_t launch_lmh(const LmhParams& p, hipStream_t s) {
  switch (lmh_row_blocks(p.M)) {
    case 1: return launch_mb<1>(p, s);
    case 2: return launch_mb<2>(p, s);
    case 3: return launch_mb<3>(p, s);
    case 4: return launch_mb<4>(p, s);
    case 5: return launch_mb<5>(p, s);
    case 6: return launch_mb<6>(p, s);
    case 7: return launch_mb<7>(p, s);
    case 8: return launch_mb<8>(p, s);
#if SV_LMH_MAXROWS > 128
    case 9: return launch_mb<9>(p, s);
    case 10: return launch_mb<10>(p, s);
#endif
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sv
