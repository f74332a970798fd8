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
// A work-group (WR x WC = 4 x 2 waves, two per SIMD) computes a tile of
// 16 RB WR rows x 256 vocabulary entries; wave (wr, wc) owns row blocks
// RB wr .. RB wr + RB - 1 and column blocks CB wc .. CB wc + CB - 1 (CB =
// 16 / WC), so each slice of k is read from LDS (RB + CB) times per wave
// instead of once per row block and column block.  64-k slices of the hidden
// rows and the weight rows (one 128-byte cache line per row) stream L2 ->
// LDS through an NS-stage ring of direct buffer -> LDS transfers (the
// attention kernel's ring); all of a slice's operands are read into
// registers before its MFMAs.
//
// What bounds it: every CU fetches its operand lines from L2 at a roughly
// fixed rate (its vector L1 keeps a bounded number of misses in flight), so
// the time goes with the cache lines a CU fetches per slice, hidden rows +
// 256 weight rows, and with the rounds of work-groups over the CUs.  Tall
// tiles fetch fewer lines per flop but fill the LDS with fewer ring stages;
// lmh_geometry() picks the tile height per shape from that cost, and the row
// tiles of one vocabulary tile run together on one XCD, so that each weight
// line comes from HBM once and the hidden rows stay in L2.
#include "sv_internal.h"

#include <algorithm>
#include <type_traits>

namespace sv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

#ifndef SV_LMH_KS
#define SV_LMH_KS 2
#endif
#ifndef SV_LMH_HOIST
#define SV_LMH_HOIST 1
#endif
constexpr int kKS = SV_LMH_KS;       // 32-k halves per slice
constexpr int kRowB = 64 * kKS;      // bytes of one row slice in LDS
static_assert(kKS == 1 || kKS == 2, "32- or 64-k slices");
#ifndef SV_LMH_WR
#define SV_LMH_WR 4
#endif
#ifndef SV_LMH_WC
#define SV_LMH_WC 2
#endif
#ifndef SV_LMH_MAXRB
#define SV_LMH_MAXRB 4
#endif
#ifndef SV_LMH_MAXNS
#define SV_LMH_MAXNS 4
#endif
constexpr int kWR = SV_LMH_WR;       // waves along the rows
constexpr int kWC = SV_LMH_WC;       // waves along the vocabulary tile
constexpr int kLmhWaves = kWR * kWC;
constexpr int kLmhThreads = 64 * kLmhWaves;
constexpr int kCB = kLmhNT / (16 * kWC);   // 16-column blocks per wave
static_assert(kCB * 16 * kWC == kLmhNT, "the waves' column blocks tile the vocabulary tile");

template <int N>
__device__ __forceinline__ void lmh_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void lmh_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// 16-byte chunk c of LDS row r sits at chunk c ^ swz(r): the 8 rows that 8
// consecutive lanes read (one chunk each) cover all 32 banks (128-byte rows:
// one row per bank sweep; 64-byte rows: two).
__device__ __forceinline__ int lmh_swz(int r) { return kKS == 2 ? (r & 7) : ((r >> 1) & 3); }

template <int RB>
struct LmhGeo {
  static constexpr int RA = 16 * RB * kWR;            // hidden rows per tile
  static constexpr int ROWS = RA + kLmhNT;            // LDS rows per stage
  static constexpr int STAGE = ROWS * kRowB;
  static constexpr int XF = ROWS * kRowB / 1024;      // 1 KB transfers per stage
  static constexpr int PER = (XF + kLmhWaves - 1) / kLmhWaves;   // per wave (padded with repeats)
  // ring depth: as many stages as 144 KB of LDS holds, at most SV_LMH_MAXNS
  static constexpr int FIT = (144 * 1024) / STAGE;
  static constexpr int NS = FIT < SV_LMH_MAXNS ? FIT : SV_LMH_MAXNS;
  static_assert(NS >= 2, "two stages at least");
};

template <int RB, bool BF16OUT>
// one work-group per CU (its ring fills the LDS): 8 waves are 2 per SIMD
__global__ __launch_bounds__(kLmhThreads) __attribute__((amdgpu_waves_per_eu(kLmhWaves / 4, kLmhWaves / 4))) void lmh_gemm(LmhParams p) {
#if defined(__HIP_DEVICE_COMPILE__)
  using G = LmhGeo<RB>;
  constexpr int PER = G::PER, NS = G::NS, CB = kCB;
  __shared__ __attribute__((aligned(1024))) char lds[NS * G::STAGE];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = w / kWC, wc = w % kWC;
  const int l16 = lane & 15, grp = lane >> 4;

  // block -> (row tile, vocabulary tile): the row tiles of one vocabulary
  // tile are 8 blocks apart (one XCD of the round-robin dispatch) and within
  // one window of 8 * m_tiles blocks, so they run together and share that
  // tile's weight rows in the XCD's L2
  // the decision kernel's inputs the row-statistics kernel would otherwise
  // prepare (every work-group may take part; the grid can be smaller than B)
  for (int b = blockIdx.x; b < p.B; b += gridDim.x) {
    if (threadIdx.x < 2)
      reinterpret_cast<uint4*>(p.reqs + b)[threadIdx.x] = reinterpret_cast<const uint4*>(p.reqs_src + b)[threadIdx.x];
    if (threadIdx.x == 0) p.tickets[b] = 0;
  }
  for (int x = blockIdx.x * kLmhThreads + threadIdx.x; x < p.nodes_n16; x += gridDim.x * kLmhThreads)
    reinterpret_cast<uint4*>(p.nodes)[x] = reinterpret_cast<const uint4*>(p.nodes_src)[x];
  const int T = p.m_tiles;
  const int g = blockIdx.x / (8 * T), r8 = blockIdx.x % (8 * T);
  const int mt = r8 / 8, nt = g * 8 + (r8 % 8);
  if (nt >= p.ntiles) return;                       // uniform: past the vocabulary
  const int m0 = mt * p.tile_rows, n0 = nt * kLmhNT;
  const int mrows = min(p.tile_rows, p.M - m0), ncols = min(kLmhNT, p.V - n0);
  if (mrows <= 0) return;
  // buffer resources over this tile's rows: loads past them read zeros
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.hidden + (int64_t)m0 * p.h_st), 0, (uint32_t)(mrows * p.h_st * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.weight + (int64_t)n0 * p.w_st), 0, (uint32_t)(ncols * p.w_st * 2), 0x00020000);
  // this lane's byte offset in each of its transfers (the k slice's start is
  // soffset): transfer j fills 1 KB of LDS rows from row (1024 / kRowB) j on,
  // lane l the 16 bytes at LDS chunk l % (kRowB / 16) of row (1024 / kRowB) j
  // + l / (kRowB / 16)
  uint32_t off[PER];
  bool isw[PER];
  int dst[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int j = (w + kLmhWaves * q) % G::XF;       // transfer index (repeats pad the last waves)
    constexpr int CPR = kRowB / 16;                  // chunks per row
    const int row = (1024 / kRowB) * j + lane / CPR; // LDS row of this lane's chunk
    const int chunk = (lane % CPR) ^ lmh_swz(row);   // global chunk that lands at LDS chunk lane % CPR
    isw[q] = row >= G::RA;
    const int grow = isw[q] ? row - G::RA : row;
    off[q] = (uint32_t)grow * (uint32_t)((isw[q] ? p.w_st : p.h_st) * 2) + (uint32_t)chunk * 16u;
    dst[q] = j * 1024;
  }
  auto issue = [&](int stage, int t) {
    char* base = lds + stage * G::STAGE;
    const uint32_t soff = (uint32_t)t * kRowB;        // 32 kKS bf16 of k per slice
#pragma unroll
    for (int q = 0; q < PER; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isw[q] ? rw : rh, (lds_void_t*)(base + dst[q]), 16, off[q], soff, 0,
                                               0);
  };

  f32x4 acc[RB][CB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // LDS read offsets in a stage: a 16-row block starts at a multiple of 16,
  // so swz(row) = swz(l16) and the chunk of k half h is (4 h + grp) ^ swz(l16)
  uint32_t ch[kKS];
#pragma unroll
  for (int h = 0; h < kKS; ++h) ch[h] = (uint32_t)(((4 * h + grp) ^ lmh_swz(l16)) * 16);
  const uint32_t abase = (uint32_t)(16 * RB * wr + l16) * kRowB;
  const uint32_t bbase = (uint32_t)(G::RA + 16 * CB * wc + l16) * kRowB;

  const int nk = (p.K + 32 * kKS - 1) / (32 * kKS);
  const int nfull = p.K / (32 * kKS);               // 64-k slices, K % 64 == 32: the last one holds 32 k only
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) issue(st, st);
  auto slice = [&](int t, auto full_c) {
    constexpr bool FULL = decltype(full_c)::value;
    const int stage = t % NS;
    // this wave's transfers of slice t have landed (later ones may still fly)
    if (t + NS - 2 < nk) lmh_wait_vm<PER * (NS - 2)>();
    else lmh_wait_vm<0>();
    lmh_barrier();                  // everyone's have; stage (t - 1) % NS is free
    if (t + NS - 1 < nk) issue((t + NS - 1) % NS, t + NS - 1);
    const char* sb = lds + stage * G::STAGE;
    constexpr int NH = FULL ? kKS : 1;
    bf16x8 a[kKS][RB], b[kKS][CB];
    auto rd = [&](int h) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) b[h][cb] = *reinterpret_cast<const bf16x8*>(sb + bbase + cb * 16 * kRowB + ch[h]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) a[h][rb] = *reinterpret_cast<const bf16x8*>(sb + abase + rb * 16 * kRowB + ch[h]);
    };
    auto mm = [&](int h) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[h][rb], b[h][cb], acc[rb][cb], 0, 0, 0);
    };
#if SV_LMH_HOIST
    // every read of the slice is issued before its first MFMA
#pragma unroll
    for (int h = 0; h < NH; ++h) rd(h);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int h = 0; h < NH; ++h) mm(h);
#else
    // one 32-k half at a time: its operands into registers, then its MFMAs
    // (the other wave on the SIMD covers the reads' latency)
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      rd(h);
      __builtin_amdgcn_sched_barrier(0);
      mm(h);
      __builtin_amdgcn_sched_barrier(0);
    }
#endif
  };
  for (int t = 0; t < nfull; ++t) slice(t, std::true_type{});
  if (nk > nfull) slice(nfull, std::false_type{});
  lmh_wait_vm<0>();
  __syncthreads();                  // the ring is no longer read: reuse its LDS

  // Epilogue.  The logits are stored (fp32, or rounded to bf16), and the
  // statistics of each row over the tile's 256 entries are taken on the
  // stored values: the maximum, then the sum of exp(l - max) in fp64, lane
  // sums in column-block order, then across the 16 lanes of a row by an xor
  // butterfly, then across the WC waves of the row in wave order.
  float* red_m = reinterpret_cast<float*>(lds);                      // [WC][RA]
  double* red_s = reinterpret_cast<double*>(lds + kWC * G::RA * 4);  // [WC][RA]
  float val[RB][CB][4];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int col = 16 * CB * wc + 16 * cb + l16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * (RB * wr + rb) + 4 * grp + i;
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
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float m = val[rb][0][i];
#pragma unroll
      for (int cb = 1; cb < CB; ++cb) m = fmaxf(m, val[rb][cb][i]);
      for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
      if (l16 == 0) red_m[wc * G::RA + 16 * (RB * wr + rb) + 4 * grp + i] = m;
    }
  __syncthreads();
  auto row_max = [&](int row) {
    float m = red_m[row];
#pragma unroll
    for (int x = 1; x < kWC; ++x) m = fmaxf(m, red_m[x * G::RA + row]);
    return m;
  };
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * (RB * wr + rb) + 4 * grp + i;
      const float m = row_max(row);
      double sm = 0.0;
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) sm += (double)exp_rel(val[rb][cb][i], m);
      for (int o = 1; o < 16; o <<= 1) sm += __shfl_xor(sm, o);
      if (l16 == 0) red_s[wc * G::RA + row] = sm;
    }
  __syncthreads();
  for (int row = threadIdx.x; row < mrows; row += kLmhThreads) {
    double sm = red_s[row];
#pragma unroll
    for (int x = 1; x < kWC; ++x) sm += red_s[x * G::RA + row];
    p.tiles[(int64_t)(m0 + row) * p.ntiles + nt] = ChunkStat{sm, row_max(row), 0.f};
  }
#endif
}

template <int RB>
hipError_t launch_rb(const LmhParams& p, hipStream_t s) {
  const int groups = (p.ntiles + 7) / 8;
  const dim3 grid((unsigned)(groups * 8 * p.m_tiles));
  if (p.out_bf16) lmh_gemm<RB, true><<<grid, dim3(kLmhThreads), 0, s>>>(p);
  else lmh_gemm<RB, false><<<grid, dim3(kLmhThreads), 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

// Tile height for M rows and ntiles vocabulary tiles.  Every CU fetches
// its operands from L2 at a fixed rate of cache lines, so a launch costs
// about (rounds of work-groups over the CUs) x (lines per k slice: the
// tile's hidden rows + 256 weight rows); the height with the lowest cost
// wins (ties: the lower one, fewer idle MFMAs), and its row tiles are
// balanced (rows past M read as zeros and cost no line).
LmhGeometry lmh_geometry(int M, int ntiles, int cus) {
  LmhGeometry best{};
  int64_t best_cost = -1;
  for (int rb = 1; rb <= SV_LMH_MAXRB; ++rb) {
    const int ra = 16 * kWR * rb;
    const int m_tiles = (M + ra - 1) / ra;
    const int rows = (M + m_tiles - 1) / m_tiles;
    const int64_t groups = (int64_t)m_tiles * ntiles;
    const int64_t cost = ((groups + cus - 1) / cus) * (int64_t)(rows + kLmhNT);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = LmhGeometry{rb, rows, m_tiles};
    }
  }
  return best;
}

hipError_t launch_lmh(const LmhParams& p, hipStream_t s) {
  if (p.M < 1 || p.tile_rows < 1 || p.tile_rows > 16 * kWR * p.rb || p.m_tiles != (p.M + p.tile_rows - 1) / p.tile_rows)
    return hipErrorInvalidValue;
  switch (p.rb) {
    case 1: return launch_rb<1>(p, s);
    case 2: return launch_rb<2>(p, s);
#if SV_LMH_MAXRB >= 3
    case 3: return launch_rb<3>(p, s);
#endif
#if SV_LMH_MAXRB >= 4
    case 4: return launch_rb<4>(p, s);
#endif
#if SV_LMH_MAXRB >= 8
    case 5: return launch_rb<5>(p, s);
    case 6: return launch_rb<6>(p, s);
    case 7: return launch_rb<7>(p, s);
    case 8: return launch_rb<8>(p, s);
#endif
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sv
