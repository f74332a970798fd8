// Verify attention for gfx950: split-KV partial kernels and the split combine.
//
// Each work item is one KV range [kb, ke) of one (request, KV head, group of
// query heads).  Its query rows are the group's heads times the request's
// n_i verify positions; every row sees the request's cached positions plus
// its own ancestors-or-self inside the verify block (causal for a chain).
// Scores and the online softmax run in fp32; the running max is kept in log2
// units (scores pre-multiplied by scale * log2 e) so exp2 is one v_exp_f32.
#include "sv_attn.h"

#include <algorithm>
#include <atomic>
#include <climits>
#include <type_traits>

namespace sv {
namespace {

// Diagnostic builds only (-DSV_ATTN_TRACE): per work-group timestamps of the
// bf16 split kernel on the device's constant-rate clock (start, first tile
// landed, stream done, end), its hardware placement and its key count, kept
// in registers and written at the end (a store inside the ring loop would
// count among the ring's outstanding transfers), read back by
// sv_attn_trace_copy.
#ifdef SV_ATTN_TRACE
constexpr int kAttnTraceBlocks = 65536;
__device__ unsigned long long g_attn_trace[kAttnTraceBlocks][6];
#endif

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// The last p.mirror_wg work-groups of the split kernel copy the staged
// request table and row map into device memory for the split combine (one
// 16-byte unit per thread and pass).  Each work-group reads its own item from
// the staged block directly, so nothing else of the plan is copied.
__device__ __forceinline__ void mirror_plan(const AttnParams& p) {
  const int k = (int)blockIdx.x - ((int)gridDim.x - p.mirror_wg);
  if (k < 0) return;
  const int step = p.mirror_wg * (int)blockDim.x;
  for (int x = k * (int)blockDim.x + (int)threadIdx.x; x < p.mirror_n16; x += step) p.mirror_dst[x] = p.mirror_src[x];
}

// ---------------------------------------------------------------------------
// bf16 MFMA path.  One work-group of W waves per work item; wave w owns query
// rows 16w .. 16w+15 of the item (W = row tiles).  The waves share 32-key K
// and V tiles that stream HBM -> LDS through an NS-stage ring of direct
// global_load_lds_dwordx4 transfers (no register staging).  Every transfer
// reads whole key rows with consecutive lanes and lands in LDS in lane order;
// the 16-byte chunks of row r are XOR-swizzled (swk for K, swv for V) so that
// both reads below are bank-conflict free and every lane's read addresses
// are one per-lane base plus compile-time offsets.  Per tile and wave:
//   S^T[key, row] = K[key, :] . Q[row, :]   v_mfma_f32_16x16x32_bf16, K as A
//                                            (A rows: ds_read_b128)
//   online softmax over keys (fp32, log2 domain)
//   O^T[e, row]  += V^T[e, key] . P^T[key, row]   with P = hi + lo in two
//                   bf16 parts, so P's rounding stays near fp32 (~2^-17)
// The 16 MFMA A-rows of key tile kt hold keys 8*(m>>2) + 4*kt + (m&3): the
// C layout then leaves lane group g holding keys 8g..8g+7 of its query row,
// which is exactly the B operand of the PV product, with no data movement.
// The V^T A operand comes from two ds_read_b64_tr_b16 per 16 columns: in a
// 16-lane group, lane i receives element i&3 of source lane 4j + (i>>2) as
// its element j, so source lane s pointing at key row 8g + 4h + (s>>2),
// columns 16e + 4(s&3) .. +3 hands lane i the keys 8g + 4h + 0..3 of column
// 16e + i.  The item's output is staged through LDS and written as rows.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;
// Ring depth (tiles in LDS) by waves per work-group, as measured.  A 4-stage
// ring (64 KB) keeps two work-groups of one to three waves per compute unit
// with three tiles each in flight.  A 5-wave work-group loses its second slot
// per compute unit once it holds 56 KB of LDS (long-context GQA 28% slower),
// so W = 5 stays at three stages (48 KB); W = 4 measured 1-2% faster at three.
#ifndef SV_WPE_W34
#define SV_WPE_W34 1
#endif
// Cache policy of the K/V tile transfers: the buffer instructions'
// cachepolicy immediate, bit 1 = nt, the non-temporal (streaming) hint.  Every
// K/V byte is read exactly once per call, and with the hint the tile stream
// runs 10-14 % faster on every workload measured (a plain read kernel over
// 2 GiB: 5.9 TB/s without, 6.6 TB/s with it); sc1 alone changes nothing.
#ifndef SV_KV_CPOL
#define SV_KV_CPOL 2
#endif

#ifndef SV_NS_W1
#define SV_NS_W1 4
#endif
#ifndef SV_NS_W2
#define SV_NS_W2 4
#endif
#ifndef SV_NS_W3
#define SV_NS_W3 4
#endif
#ifndef SV_NS_W4
#define SV_NS_W4 3
#endif
#ifndef SV_WPE_W5
#define SV_WPE_W5 4
#endif
#ifndef SV_NS_W5
#define SV_NS_W5 3
#endif
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

template <int D>
struct Geo {
  static constexpr int CH = D / 8;                  // 16-byte chunks per row
  static constexpr int RPI = 64 / CH;               // rows per 1 KB transfer
  static constexpr int IPM = 32 / RPI;              // transfers per 32-row matrix
  static constexpr int ROWB = D * 2;                // bytes of one LDS row
  static constexpr int MAT = 32 * ROWB;             // bytes of one K (or V) tile
  static constexpr int STAGE = 2 * MAT;
};

// K rows: distinct over the 16 rows of one quarter-wave A read.
template <int D>
__device__ __forceinline__ int swk(int r) {
  if constexpr (D == 128) return (r & 3) | (((r >> 3) & 3) << 2);
  else return ((r >> 1) & 1) | (((r >> 3) & 3) << 1);
}
// V rows: even (keeps 32-byte column pairs together), distinct pair slots over
// the 8 rows of one half-wave transpose read.
template <int D>
__device__ __forceinline__ int swv(int r) {
  if constexpr (D == 128) return 2 * ((r & 3) | (((r >> 3) & 1) << 2));
  else return 2 * (((r >> 1) & 1) | (((r >> 3) & 1) << 1));
}

// vmcnt(n) for gfx950 (expcnt and lgkmcnt left at "no wait")
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// f(integral_constant<int, I>) for I = B .. E-1, in order.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Work-group barrier for the tile ring.  __syncthreads() is a release fence at
// work-group scope, which the compiler implements for a kernel with LDS-bound
// transfers by waiting for all of them (vmcnt(0)), draining the ring.  Here the
// caller has already waited for the transfers the next tile needs; the barrier
// only has to order LDS accesses, and the memory clobber keeps the compiler
// from moving loads or stores across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// A tile's transfers are dealt round-robin over the waves: wave w issues
// transfers w, w + W, ... < NI, PER of them when w < FULL, else PER - 1 (an
// uneven split issues no padding transfer; each wave waits on its own count).
template <int D, int W>
struct Xfer {
  static constexpr int NI = 2 * Geo<D>::IPM;        // transfers per tile (K then V)
  static constexpr int PER = (NI + W - 1) / W;      // per wave, at most
  static constexpr int FULL = NI - (PER - 1) * W;   // waves that issue PER
  static constexpr bool EVEN = NI % W == 0;         // every wave issues PER
};

// Byte offset, inside a tile, of the global chunk lane `lane` moves in
// transfer j (tile row row_in_tile * row_bytes + swizzled chunk).
template <int D>
__device__ __forceinline__ uint32_t xfer_offset(int j, int lane, int row_bytes, int* row_in_tile) {
  using G = Geo<D>;
  const bool isv = j >= G::IPM;
  const int jj = isv ? j - G::IPM : j;
  const int row = jj * G::RPI + lane / G::CH;
  const int chunk = (lane % G::CH) ^ (isv ? swv<D>(row) : swk<D>(row));
  *row_in_tile = row;
  return (uint32_t)row * (uint32_t)row_bytes + (uint32_t)chunk * 16u;
}

template <int D, int W>
struct XferPlan {
  uint32_t off[Xfer<D, W>::PER];    // per-lane byte offset inside the tile
};

// Wave w's transfers of the tile starting at key t0 into `stage`, as
// buffer_load_dwordx4 ... lds with the tile start in soffset and each lane's
// precomputed offset in voffset.  Tiles that reach past ke clamp their rows
// to ke - 1 (in bounds, masked later).
template <int D, int W>
__device__ __forceinline__ void issue_tile(char* stage, __amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                           int row_bytes, int t0, int ke, int w, int lane,
                                           const XferPlan<D, W>& X) {
  using G = Geo<D>;
  if (t0 + 32 <= ke) {                // wave-uniform: the whole tile is inside the item
    const uint32_t soff = (uint32_t)t0 * (uint32_t)row_bytes;
#pragma unroll
    for (int q = 0; q < Xfer<D, W>::PER; ++q) {
      if constexpr (!Xfer<D, W>::EVEN)
        if (w + q * W >= Xfer<D, W>::NI) break;     // wave-uniform: this wave's last is done
      const int j = w + q * W;
      const bool isv = j >= G::IPM;
      const int jj = isv ? j - G::IPM : j;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isv ? rv : rk, (lds_void_t*)(stage + (isv ? G::MAT : 0) + jj * 1024),
                                               16, X.off[q], soff, 0, SV_KV_CPOL);
    }
  } else {
#pragma unroll
    for (int q = 0; q < Xfer<D, W>::PER; ++q) {
      if constexpr (!Xfer<D, W>::EVEN)
        if (w + q * W >= Xfer<D, W>::NI) break;     // wave-uniform: this wave's last is done
      const int j = w + q * W;
      const bool isv = j >= G::IPM;
      const int jj = isv ? j - G::IPM : j;
      int row;
      const uint32_t full = xfer_offset<D>(j, lane, row_bytes, &row);
      const uint32_t chunk_bytes = full - (uint32_t)row * (uint32_t)row_bytes;
      const int key = min(t0 + row, ke - 1);       // >= kb >= 0: items are never empty
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isv ? rv : rk, (lds_void_t*)(stage + (isv ? G::MAT : 0) + jj * 1024),
                                               16, (uint32_t)key * (uint32_t)row_bytes + chunk_bytes, 0u, 0, SV_KV_CPOL);
    }
  }
}

template <int D>
struct RowTile {
  bf16x8 q[D / 32];
  f32x4 o[D / 16];
  uint32_t koff[D / 32];   // A-row read offsets (key tile 0; tile 1 is +4 rows)
  uint32_t voff[D / 16];   // transpose-read offsets (keys 8g + 0..3; +4 rows for 4..7)
  uint32_t anc;
  float m, l;
};

// Tile compute on ring stage SOFF / STAGE (a compile-time byte offset into
// `ring`), so every LDS read of the stage carries its offset as an immediate
// and the per-lane address registers are shared by all stages.
template <int D, int SOFF>
__device__ __forceinline__ void compute_tile(const char* ring, RowTile<D>& S, int t0, int ke, int ctx,
                                             float scale_log2, int lane) {
  using G = Geo<D>;
  const char* stage = ring + SOFF;
  constexpr int KS = D / 32, ET = D / 16;
  const int grp = lane >> 4;
  f32x4 s[2];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(stage + S.koff[ks] + kt * 4 * G::ROWB);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, S.q[ks], acc, 0, 0, 0);
    }
    s[kt] = acc;
  }
  // Scores in log2 units.  The exponent reference S.m trails the running max
  // by at most kLazy: it moves (and O, l are rescaled) only when a score
  // exceeds it by more than that, so p <= 2^kLazy and the common tile leaves
  // the accumulators to the matrix cores alone.
  constexpr float kLazy = 8.f;
  float sv[8];
  if (t0 + 32 <= min(ke, ctx)) {      // wave-uniform: every key visible to every row
#pragma unroll
    for (int x = 0; x < 8; ++x) sv[x] = s[x >> 2][x & 3] * scale_log2;
  } else {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 8 * grp + 4 * kt + i;
        const float x = s[kt][i] * scale_log2;
        sv[kt * 4 + i] = (t >= ke || !visible(t, ctx, S.anc)) ? -INFINITY : x;
      }
    }
  }
  // this lane's largest score (a masked -inf never wins over a finite one)
  const float mloc0 = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                            fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
  if (__any(mloc0 > S.m + kLazy)) {   // wave-uniform
    float mloc = fmaxf(mloc0, __shfl_xor(mloc0, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(S.m, mloc);
    // exp2 of a non-positive argument; S.m = -inf gives 0
    const float alpha = (m_new == S.m) ? 1.f : __builtin_amdgcn_exp2f(S.m - m_new);
    S.l *= alpha;
#pragma unroll
    for (int et = 0; et < ET; ++et) S.o[et] *= alpha;
    S.m = m_new;
  }
  const float m_use = (S.m == -INFINITY) ? 0.f : S.m;
  // p = 2^(score - m) <= 2^kLazy with the hardware exp2 (arguments are at most
  // kLazy; results below the normal range flush to zero, negligible against l >= 1
  // once a row has a finite score).  p is split into bf16 hi + lo so the PV
  // products keep about 16 significant bits of p.
  float pv[8];
  float psum = 0.f;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    pv[x] = __builtin_amdgcn_exp2f(sv[x] - m_use);
    psum += pv[x];
  }
  S.l += psum;
  uint32_t hw[4], lw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 h2 = __builtin_convertvector((f32x2){pv[2 * i], pv[2 * i + 1]}, bf16x2);
    hw[i] = __builtin_bit_cast(uint32_t, h2);
    const float h0 = __uint_as_float(hw[i] << 16), h1 = __uint_as_float(hw[i] & 0xffff0000u);
    lw[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){pv[2 * i] - h0, pv[2 * i + 1] - h1}, bf16x2));
  }
  const bf16x8 phi = __builtin_bit_cast(bf16x8, (u32x4){hw[0], hw[1], hw[2], hw[3]});
  const bf16x8 plo = __builtin_bit_cast(bf16x8, (u32x4){lw[0], lw[1], lw[2], lw[3]});
  // V^T operands by transposing LDS reads, in groups of VG column tiles.  The
  // reads are issued from inline assembly with their own lgkmcnt waits: the
  // compiler's builtin for this read makes it wait for every outstanding
  // LDS-bound transfer (vmcnt(0)), which would serialise the ring.
  // The stage's V offset goes into the instructions' 16-bit immediate where
  // it fits (S.voff holds the ring's LDS address plus the lane offset).
  constexpr int VOFF = SOFF + G::MAT;
  constexpr bool IMM = VOFF + 4 * G::ROWB <= 65535;
  const uint32_t vadd = IMM ? 0u : (uint32_t)VOFF;
  constexpr int I0 = IMM ? VOFF : 0;
  constexpr int VG = 4;
#pragma unroll
  for (int e0 = 0; e0 < ET; e0 += VG) {
    s16x4 lo[VG], hi[VG];
#pragma unroll
    for (int e = 0; e < VG; ++e) {
      const uint32_t a = S.voff[e0 + e] + vadd;
      asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%3\n\tds_read_b64_tr_b16 %1, %2 offset:%4"
                   : "=&v"(lo[e]), "=&v"(hi[e])   // early clobber: the address is read twice
                   : "v"(a), "i"(I0), "i"(I0 + 4 * G::ROWB));
    }
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(lo[0]), "+v"(hi[0]), "+v"(lo[1]), "+v"(hi[1]), "+v"(lo[2]), "+v"(hi[2]), "+v"(lo[3]),
                   "+v"(hi[3]));
#pragma unroll
    for (int e = 0; e < VG; ++e) {
      const bf16x8 vop = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo[e], hi[e], 0, 1, 2, 3, 4, 5, 6, 7));
      S.o[e0 + e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, phi, S.o[e0 + e], 0, 0, 0);
      S.o[e0 + e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, plo, S.o[e0 + e], 0, 0, 0);
    }
  }
}

template <int D, int W, int NS>
struct AttnLds {
  static constexpr int RING = NS * Geo<D>::STAGE;
  static constexpr int OUT = W * 16 * (D + 4) * 4;  // fp32 output staging, padded rows
  static constexpr int BYTES = RING > OUT ? RING : OUT;
};

// Register budget by waves per work-group.  A 5-wave work-group is placed only
// where every SIMD can take two of its waves, so a second one per compute unit
// needs <= 128 registers (measured: long-context GQA 17% faster).  Bounding
// 3-4 waves to 168 (three work-groups per compute unit) measured neutral.
template <int W>
struct WavesPerEu {
  static constexpr int value = W == 5 ? SV_WPE_W5 : (W >= 3 ? SV_WPE_W34 : 1);
};

// Agent-scope (all XCDs) stores of two floats for the fused combine's
// hand-over (the combine reads them with agent-scope loads).  On gfx950 such a store is written through to the
// device coherence point and completes (vmcnt) only once it is there; such a
// load reads from that point, never a stale line of this XCD's L2.  A piece
// checks in only after its stores have completed, and the last piece loads
// the partials only after its check-in returned, so it reads every piece's.
// (Release/acquire fences would write back and invalidate the whole L2 of
// the XCD at every piece's end: measured 80% slower on long-context GQA.)
__device__ __forceinline__ void st_dev2(float* p, float a, float b) {
  const unsigned long long v = (unsigned long long)__float_as_uint(a) | ((unsigned long long)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival of one piece of a split stream on the stream's counter
// ((call tag << 32) | arrivals so far): a counter holding another tag starts
// over.  Returns whether this piece is the stream's last (the total-th).
// Every failed exchange means another piece's succeeded in between, so the
// loop ends after at most `total` tries; the bound only guards that.
__device__ __forceinline__ bool arrive_last(unsigned long long* ctr, uint32_t tag, int total) {
  unsigned long long old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  unsigned long long nw = 0;
  for (int tries = 0; tries <= total + 1; ++tries) {
    nw = ((uint32_t)(old >> 32) == tag) ? old + 1 : (((unsigned long long)tag << 32) | 1ull);
    if (__hip_atomic_compare_exchange_strong(ctr, &old, nw, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return (uint32_t)nw == (uint32_t)total;
  }
  return false;
}

// Work-group 0 starts this call's count on the claim word at `base` as soon
// as the kernel starts (unless a claim has started it already).  The first
// round holds every work-group the device keeps resident at once, so claims
// begin only once a first-round work-group has finished, and each is then a
// single fetch-and-add.  (When many work-groups claim at once on a word that
// still holds another call's value, each exchange loop below succeeds for
// one of them at a time: a burst of k claims would cost about k^2 exchanges.
// So a claim that meets another call's value first waits for this start.)
__device__ __forceinline__ void claim_start(unsigned long long* ctr, uint32_t tag, int base, int bound) {
  unsigned long long old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int tries = 0; tries <= bound + 1 && (uint32_t)(old >> 32) != tag; ++tries)
    if (__hip_atomic_compare_exchange_strong(ctr, &old, ((unsigned long long)tag << 32) | (uint32_t)base,
                                             __ATOMIC_RELAXED, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
      break;
}

// The next unclaimed item (work-groups at or above p.first_round): one
// fetch-and-add on the claim word ((call tag << 32) | next item).  A word
// still holding another call's value (or anything else) was only bumped by
// it.  The claim then polls the word (kClaimPolls reads, a short sleep
// apart, roughly 100 us in all) for work-group 0's start of this call's count
// and claims again once it is there; work-group 0 was dispatched first, so
// it is running.  Should the polls run out, the exchange loop starts the
// count at `base` itself, or takes the next item if another work-group has
// started it meanwhile.  Every failed exchange means another work-group's
// succeeded in between, so the loop ends after at most `bound` tries; the
// bound only guards that.
constexpr int kClaimPolls = 64;
__device__ __forceinline__ int claim_item(unsigned long long* ctr, uint32_t tag, int base, int bound) {
  unsigned long long old = __hip_atomic_fetch_add(ctr, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if ((uint32_t)(old >> 32) == tag) return (int)(uint32_t)old;
  for (int i = 0; i < kClaimPolls; ++i) {
    __builtin_amdgcn_s_sleep(16);
    old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(old >> 32) == tag) {
      old = __hip_atomic_fetch_add(ctr, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return (int)(uint32_t)old;          // the tag, once there, stays for the call
    }
  }
  old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int tries = 0; tries <= bound + 1; ++tries) {
    const unsigned long long nw =
        ((uint32_t)(old >> 32) == tag) ? old + 1 : (((unsigned long long)tag << 32) | (uint32_t)(base + 1));
    if (__hip_atomic_compare_exchange_strong(ctr, &old, nw, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return (int)((uint32_t)nw - 1u);
  }
  return INT_MAX;
}

// The split combine of one stream (rows = heads x verify positions of one
// request, KV head and head group), by the work-group of its last piece:
//   O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,  M = max_s m_s,
// the pieces summed in index order.  Every (row, piece) pair's (m, l) comes
// into LDS at once; the rows' weights replace the maxima there, beside the
// rows' 1 / L.  Then each thread takes 16-byte column groups of two rows at
// a time, eight pieces' loads in flight.  The partials are read with
// agent-scope buffer loads (sc1) from the request's block of partial rows.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr int kCpolAgent = 16;        // the sc1 bit of a buffer instruction's cache policy
template <int D>
__device__ __forceinline__ void combine_stream(const AttnParams& p, const AttnItem& it, char* lds) {
  const int n = it.nq, R = it.nheads * n, nseg = it.nseg;
  const int nth = (int)blockDim.x, tid = (int)threadIdx.x;
  const int blk_rows = nseg * n * p.Hq;   // the request's partial rows (the host keeps the bytes < 2^31)
  const __amdgpu_buffer_rsrc_t ro =
      __builtin_amdgcn_make_buffer_rsrc((void*)(p.part_o + (int64_t)it.part0 * D), 0, blk_rows * D * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rm =
      __builtin_amdgcn_make_buffer_rsrc((void*)(p.part_ml + it.part0), 0, blk_rows * 8, 0x00020000);
  auto lrow = [&](int r, int sg) -> int {
    const int hh = r / n, j = r - hh * n;
    return (sg * n + j) * p.Hq + it.head_lo + hh;
  };
  float2* mlw = reinterpret_cast<float2*>(lds);     // [R][nseg]: (m, l), then (weight, l)
  float* invl = reinterpret_cast<float*>(mlw + R * nseg);
  for (int x = tid; x < R * nseg; x += nth) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rm, lrow(x / nseg, x % nseg) * 8, 0, kCpolAgent);
    mlw[x] = make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
  }
  __syncthreads();
  for (int r = tid; r < R; r += nth) {
    float2* row = mlw + r * nseg;
    float M = -INFINITY;
    for (int sg = 0; sg < nseg; ++sg) M = fmaxf(M, row[sg].x);
    float L = 0.f;
    for (int sg = 0; sg < nseg; ++sg) {
      const float w = (row[sg].x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(row[sg].x - M);
      row[sg].x = w;
      L += row[sg].y * w;
    }
    invl[r] = 1.f / L;
  }
  __syncthreads();
  constexpr int Q = D / 4;                      // 16-byte column groups per row
  const int units = R * Q;
  for (int u0 = tid; u0 < units; u0 += 2 * nth) {
    const int u1 = min(u0 + nth, units - 1);    // a repeat of a valid unit when past the end
    const int r0 = u0 / Q, c0 = (u0 % Q) * 4, r1 = u1 / Q, c1 = (u1 % Q) * 4;
    float4 a0 = make_float4(0.f, 0.f, 0.f, 0.f), a1 = a0;
#pragma unroll 8
    for (int sg = 0; sg < nseg; ++sg) {
      const u32x4 v0 = __builtin_amdgcn_raw_buffer_load_b128(ro, (lrow(r0, sg) * D + c0) * 4, 0, kCpolAgent);
      const u32x4 v1 = __builtin_amdgcn_raw_buffer_load_b128(ro, (lrow(r1, sg) * D + c1) * 4, 0, kCpolAgent);
      const float w0 = mlw[r0 * nseg + sg].x, w1 = mlw[r1 * nseg + sg].x;
      a0.x += w0 * __uint_as_float(v0.x); a0.y += w0 * __uint_as_float(v0.y);
      a0.z += w0 * __uint_as_float(v0.z); a0.w += w0 * __uint_as_float(v0.w);
      a1.x += w1 * __uint_as_float(v1.x); a1.y += w1 * __uint_as_float(v1.y);
      a1.z += w1 * __uint_as_float(v1.z); a1.w += w1 * __uint_as_float(v1.w);
    }
    auto store = [&](int r, int c, float4 a) {
      const int hh = r / n, j = r - hh * n;
      const float sc = invl[r];
      *reinterpret_cast<float4*>(p.out + ((int64_t)(it.q0 + j) * p.Hq + it.head_lo + hh) * D + c) =
          make_float4(a.x * sc, a.y * sc, a.z * sc, a.w * sc);
    };
    store(r0, c0, a0);
    if (u0 + nth < units) store(r1, c1, a1);
  }
}

// PG: paged KV cache.  A tile (32 keys, 32-aligned) never straddles a page
// (pages hold a multiple of 32 tokens), so each tile's transfers take a buffer
// resource based at its page, built from the block table entry (a
// wave-uniform load, clamped into the pool, issued one ring step ahead of its
// use); everything else is the packed path's code.
template <int D, int W, int NS, int PG>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(WavesPerEu<W>::value)))
void attn_split_mfma(AttnParams p) {
#if defined(__HIP_DEVICE_COMPILE__)   // the host pass needs the signature only
  using G = Geo<D>;
  constexpr int ET = D / 16, KS = D / 32;
  constexpr int PER = Xfer<D, W>::PER;
  static_assert(NS >= 2, "ring depth");
  __shared__ __attribute__((aligned(1024))) char lds[AttnLds<D, W, NS>::BYTES];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c16 = lane & 15, grp = lane >> 4;
#ifdef SV_ATTN_TRACE
  unsigned long long tr_start = wall_clock64(), tr_first = 0, tr_done = 0;
#endif
  int idx = blockIdx.x;
  if (idx == 0 && p.first_round < (int)gridDim.x && threadIdx.x == 0)
    claim_start(p.claim, p.call_tag, p.first_round, (int)gridDim.x);
  if (idx >= p.first_round) {
    __shared__ int s_item;
    if (threadIdx.x == 0) {
      s_item = claim_item(p.claim, p.call_tag, p.first_round, (int)gridDim.x);
      // The last of the grid's claims: every other one has been made, so no
      // one touches the word again in this call.  Leave it as work-group 0
      // would start it, so that a replay of this launch with the same tag (a
      // captured graph) claims from the first round again.
      if (s_item == (int)gridDim.x - 1)
        __hip_atomic_store(p.claim, ((unsigned long long)p.call_tag << 32) | (uint32_t)p.first_round,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    idx = __builtin_amdgcn_readfirstlane(s_item);
  }
  mirror_plan(p);
  if (idx >= p.n_items) return;       // uniform: every item is taken
  const AttnItem it = p.items[idx];
  const int n = it.nq;
  const int R = it.nheads * n;
  const int ctx = it.ctx;
  const int row_bytes = (int)(p.kv_st * 2);
  const char* Kb = static_cast<const char*>(p.k) + ((int64_t)it.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh) * 2;
  const char* Vb = static_cast<const char*>(p.v) + ((int64_t)it.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh) * 2;
  const int ntiles = (it.ke - it.kb + 31) / 32;
  // byte range of this request's rows for this KV head (the host keeps it < 2^31)
  const int range = (it.ctx + it.nq) * row_bytes;
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)Kb, 0, range, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)Vb, 0, range, 0x00020000);
  RowTile<D> S;
  // This lane's B operand of the score product straight from HBM: query row
  // 16w + c16 (padding rows repeat the item's row 0), columns 32ks + 8grp ..
  // +7.  These loads are older than every tile transfer, so the wait after
  // the ring's prologue below covers them without draining the ring.
  {
    int rr = w * 16 + c16;
    if (rr >= R) rr = 0;
    const int hh = rr / n, j = rr - hh * n;
    const char* src = static_cast<const char*>(p.q) +
                      ((int64_t)(it.q0 + j) * p.q_st + (int64_t)(it.head_lo + hh) * p.q_sh) * 2 + grp * 16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) S.q[ks] = *reinterpret_cast<const bf16x8*>(src + ks * 64);
  }

  XferPlan<D, W> X;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    int row;
    X.off[q] = xfer_offset<D>((w + q * W) % Xfer<D, W>::NI, lane, row_bytes, &row);
  }

  // paged: this KV head's slice of page 0 of each pool, the item's block
  // table row, and tile t's page id (tiles past the item's end re-read its
  // last tile, as in the packed path)
  const char* Kh = static_cast<const char*>(p.k) + (int64_t)it.kvh * p.kv_sh * 2;
  const char* Vh = static_cast<const char*>(p.v) + (int64_t)it.kvh * p.kv_sh * 2;
  // The block table is read through the constant address space with a
  // wave-uniform index, so the page ids come in by scalar loads: a vector
  // load would count among the ring's outstanding transfers, and its
  // consumer's wait would drain the whole ring every tile.
  typedef __attribute__((address_space(4))) const int32_t cint32_t;
  const cint32_t* btr = PG ? (const cint32_t*)(p.bt + (int64_t)it.req * p.bt_stride) : nullptr;
  const int last_t0 = it.kb + 32 * (ntiles - 1);
  // (generic lambdas: instantiated only in the device pass, like the ring loop's)
  auto page_of = [&](auto t) -> int {
    const int t0 = min(it.kb + 32 * t, last_t0);
    const int idx = __builtin_amdgcn_readfirstlane(t0 / p.page_tokens);
    const int pg = btr[idx];
    return __builtin_amdgcn_readfirstlane(min(max(pg, 0), p.num_pages - 1));
  };
  // PG 2: one descriptor per item over this KV head's slice of the pools
  // (whose byte offsets fit 32 bits); a key at logical position t of page pg
  // is physical key pg * page_tokens + (t - page start) from the slice's base
  // (page_bytes = page_tokens * row_bytes)
  const uint32_t pool_range = PG == 2 ? (uint32_t)(p.pool_bytes - (int64_t)it.kvh * p.kv_sh * 2) : 0u;
  const __amdgpu_buffer_rsrc_t qk = __builtin_amdgcn_make_buffer_rsrc((void*)Kh, 0, pool_range, 0x00020000);
  const __amdgpu_buffer_rsrc_t qv = __builtin_amdgcn_make_buffer_rsrc((void*)Vh, 0, pool_range, 0x00020000);
  auto issue = [&](char* stage, auto t, int pg) {
    if constexpr (PG == 2) {
      const int t0 = min(it.kb + 32 * t, last_t0);
      const int base = t0 - t0 % p.page_tokens;          // the page's first logical key
      const int pk0 = pg * p.page_tokens;                // the page's first physical key
      issue_tile<D, W>(stage, qk, qv, row_bytes, pk0 + (t0 - base), pk0 + (it.ke - base), w, lane, X);
    } else if constexpr (PG == 1) {
      const int t0 = min(it.kb + 32 * t, last_t0);
      const int base = t0 - t0 % p.page_tokens;          // the page's first logical key
      const int64_t pb = (int64_t)pg * p.page_bytes;
      const int prange = p.page_tokens * row_bytes;
      const __amdgpu_buffer_rsrc_t pk = __builtin_amdgcn_make_buffer_rsrc((void*)(Kh + pb), 0, prange, 0x00020000);
      const __amdgpu_buffer_rsrc_t pv = __builtin_amdgcn_make_buffer_rsrc((void*)(Vh + pb), 0, prange, 0x00020000);
      issue_tile<D, W>(stage, pk, pv, row_bytes, t0 - base, it.ke - base, w, lane, X);
    } else {
      (void)pg;
      issue_tile<D, W>(stage, rk, rv, row_bytes, it.kb + 32 * t, it.ke, w, lane, X);
    }
  };

  const int row_node = (w * 16 + c16 < R) ? (w * 16 + c16) % n : -1;   // this lane's verify node
  {
    // A uniform loop over the kernel-argument table: each entry is pinned to a
    // scalar register so the selection cannot become a per-lane vector load.
    // (Per-request trees read their request's masks after the prologue.)
    uint32_t anc = 0u;
    if (!p.per_req) {
      for (int jj = 0; jj < min(n, kMaxNodes); ++jj) {
        uint32_t a = p.anc[jj];
        asm volatile("" : "+s"(a));
        anc = (row_node == jj) ? a : anc;
      }
    }
    S.anc = anc;
    S.m = -INFINITY;
    S.l = 0.f;
#pragma unroll
    for (int et = 0; et < ET; ++et) S.o[et] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int rk0 = 8 * (c16 >> 2) + (c16 & 3);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) S.koff[ks] = rk0 * G::ROWB + (((ks * 4 + grp) ^ swk<D>(rk0)) * 16);
    const int rv0 = 8 * grp + (c16 >> 2);
    const uint32_t ring_lds = (uint32_t)(uintptr_t)lds;
#pragma unroll
    for (int et = 0; et < ET; ++et)
      S.voff[et] = ring_lds + rv0 * G::ROWB + (((2 * et + ((c16 & 3) >> 1)) ^ swv<D>(rv0)) * 16) + (c16 & 1) * 8;
  }
  const bool active = w * 16 < R;     // wave-uniform: this wave has query rows

  // The ring's first NS-1 tiles, issued whatever the item's length so that
  // the transfer count behind each wave's query loads is fixed (a tile
  // past the item's end re-reads its last key row, in bounds, and is never
  // computed).  The query loads are older than these transfers: wait for them
  // alone, and hand the registers through an empty asm so that no later use
  // inherits a wait on the ring.
#pragma unroll
  for (int st = 0; st < NS - 1; ++st) issue(lds + st * G::STAGE, st, PG ? page_of(st) : 0);
  // this wave's transfers per tile: PER, or PER - 1 on the last waves of an uneven split
  const bool full_wave = Xfer<D, W>::EVEN || w < Xfer<D, W>::FULL;
  if (full_wave) wait_vm<PER * (NS - 1)>();
  else wait_vm<(PER - 1) * (NS - 1)>();
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(S.q[ks]));
  if (p.per_req) {
    // Per-request trees: this request's ancestor masks from its node-table
    // entries, by scalar loads (constant address space, wave-uniform
    // indices) issued while the ring's first tiles are in flight; the first
    // tile's barrier waits for them.
    typedef __attribute__((address_space(4))) const uint32_t cu32_t;
    const cu32_t* na = (const cu32_t*)(p.nodes + it.node0);
    uint32_t anc = 0u;
    for (int jj = 0; jj < min(n, kMaxNodes); ++jj) {
      const uint32_t a = na[2 * jj];             // NodeInfo::anc, the first of its two words
      anc = (row_node == jj) ? a : anc;
    }
    S.anc = anc;
  }

  for (int tb = 0; tb < ntiles; tb += NS) {
    bool stop = false;
    static_for<0, NS>([&](auto stc) {             // stage index is a compile-time constant
      constexpr int st = decltype(stc)::value;
      const int t = tb + st;
      if (stop || t >= ntiles) {
        stop = true;
        return;
      }
      // paged: the page of the tile issued below, loaded before the waits
      // (the barrier's lgkmcnt wait covers it)
      const int pg_next = (PG && t + NS - 1 < ntiles) ? page_of(t + NS - 1) : 0;
      // this wave's transfers of tile t have landed: NS-2 later tiles may still
      // be in flight, none in the item's last NS-2 tiles (over-waiting there)
      if (t + NS - 2 >= ntiles) wait_vm<0>();
      else if (full_wave) wait_vm<PER * (NS - 2)>();
      else wait_vm<(PER - 1) * (NS - 2)>();
      ring_barrier();                 // everyone's have landed; stage (t-1) % NS is free
#ifdef SV_ATTN_TRACE
      if (t == 0) tr_first = wall_clock64();
#endif
      if (t + NS - 1 < ntiles) issue(lds + ((st + NS - 1) % NS) * G::STAGE, t + NS - 1, pg_next);
      if (active) compute_tile<D, st * G::STAGE>(lds, S, it.kb + 32 * t, it.ke, ctx, p.scale_log2, lane);
    });
  }
  wait_vm<0>();
  __syncthreads();                    // ring no longer read: reuse it for the output
#ifdef SV_ATTN_TRACE
  tr_done = wall_clock64();
#endif

  // row sums across the four lane groups; stage O^T into row-major LDS
  float l = S.l;
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  float* ost = reinterpret_cast<float*>(lds) + w * 16 * (D + 4);
  const float scale = it.seg < 0 ? 1.f / l : 1.f;
#pragma unroll
  for (int et = 0; et < ET; ++et) {
    const f32x4 v = S.o[et] * scale;
    *reinterpret_cast<float4*>(ost + c16 * (D + 4) + et * 16 + 4 * grp) = make_float4(v[0], v[1], v[2], v[3]);
  }
  // output row of query row r (rows outside the destination are never written)
  auto out_row = [&](int r) -> int64_t {
    const int hh = r / n, j = r - hh * n, h = it.head_lo + hh;
    const int64_t o = it.seg < 0 ? (int64_t)(it.q0 + j) * p.Hq + h
                                 : (int64_t)it.part0 + ((int64_t)it.seg * n + j) * p.Hq + h;
    const int64_t lim = it.seg < 0 ? (int64_t)p.Nq * p.Hq : (int64_t)p.n_parts;
    return (r < R && o >= 0 && o < lim) ? o : -1;
  };
  const int64_t o0 = out_row(w * 16 + c16);
  // The fused combine's partials are written through to the device coherence
  // point (agent-scope stores) for the stream's last piece, which may run on
  // another XCD, to read back the same way.
  const bool publish = it.seg >= 0 && p.fused;
  if (it.seg >= 0 && grp == 0 && o0 >= 0) {
    if (publish) st_dev2(reinterpret_cast<float*>(p.part_ml + o0), S.m, l);
    else p.part_ml[o0] = make_float2(S.m, l);
  }
  __syncthreads();
  // whole-row writes: D/4 lanes per row, 64*4/D rows per pass
  constexpr int LPR = D / 4, RPP = 64 / LPR;
  const int e4 = (lane % LPR) * 4;
#pragma unroll
  for (int pass = 0; pass < 16 / RPP; ++pass) {
    const int rl = pass * RPP + lane / LPR;
    const int64_t o = out_row(w * 16 + rl);
    if (o < 0) continue;
    const float4 v = *reinterpret_cast<const float4*>(ost + rl * (D + 4) + e4);
    float* dst = (it.seg < 0 ? p.out : p.part_o) + o * D + e4;
    if (publish) {
      st_dev2(dst, v.x, v.y);
      st_dev2(dst + 2, v.z, v.w);
    } else {
      *reinterpret_cast<float4*>(dst) = v;
    }
  }
#ifdef SV_ATTN_TRACE
  if (threadIdx.x == 0 && blockIdx.x < kAttnTraceBlocks) {
    unsigned hw = 0, xcc = 0;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    g_attn_trace[blockIdx.x][0] = tr_start;
    g_attn_trace[blockIdx.x][1] = tr_first;
    g_attn_trace[blockIdx.x][2] = tr_done;
    g_attn_trace[blockIdx.x][3] = wall_clock64();
    g_attn_trace[blockIdx.x][4] = ((unsigned long long)xcc << 32) | hw;
    g_attn_trace[blockIdx.x][5] = (unsigned long long)(it.ke - it.kb);
  }
#endif
  if (publish) {
    // Check in on the stream's counter once this work-group's partial stores
    // have completed; the stream's last piece combines.
    // (the flag lives in the ring's LDS, read by no one after the stores above)
    volatile int* s_last = reinterpret_cast<volatile int*>(lds);
    wait_vm<0>();
    __syncthreads();
    if (threadIdx.x == 0) {
      const bool last = arrive_last(p.counters + it.stream, p.call_tag, it.nseg);
      // every piece of the stream has arrived: back to no arrivals under this
      // tag, so that a replay with the same tag (a captured graph) counts again
      if (last)
        __hip_atomic_store(p.counters + it.stream, (unsigned long long)p.call_tag << 32, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      *s_last = last ? 1 : 0;
    }
    __syncthreads();
    if (!*s_last) return;
    __syncthreads();                  // everyone has read the flag before the combine reuses the LDS
    combine_stream<D>(p, it, lds);
  }
#endif
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
  mirror_plan(p);
  const int n = it.nq;
  const int R = it.nheads * n;
  const int ctx = it.ctx;
  const T* Kb = static_cast<const T*>(p.k) + (int64_t)it.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;
  const T* Vb = static_cast<const T*>(p.v) + (int64_t)it.kv0 * p.kv_st + (int64_t)it.kvh * p.kv_sh;

  for (int x = tid; x < RV * D; x += 256) {
    const int r = x / D, e = x % D;
    float val = 0.f;
    if (r < R) {
      const int hh = r / n, j = r - hh * n;
      val = load_elem<T>(static_cast<const T*>(p.q),
                         (int64_t)(it.q0 + j) * p.q_st + (int64_t)(it.head_lo + hh) * p.q_sh + e);
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
      const uint32_t anc = p.per_req ? p.nodes[it.node0 + j].anc : p.anc[j];
      if (t >= it.ke || !visible(t, ctx, anc)) s = -INFINITY;
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
      p.out[((int64_t)(it.q0 + j) * p.Hq + h) * D + e] = o[x] / ml_s[r][1];
    } else {
      const int64_t pr = (int64_t)it.part0 + ((int64_t)it.seg * n + j) * p.Hq + h;
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
  // One wave per (query row, head) of a split request, four per work-group.
  // Lane s holds partial s's running max and sum (64 partials per pass); the
  // log-sum-exp weights reach the other lanes by shuffle.  The column sums
  // take the partial rows eight at a time (a short last group is padded with
  // a repeated row of weight zero), and the first eight rows are requested
  // together with the (max, sum) pairs, since they do not depend on the
  // weights, so a request of up to eight pieces costs one round trip.  Fixed
  // order throughout (bit-reproducible).
  constexpr int PER = D / 64, G8 = 8;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= (int64_t)p.Nq * p.Hq) return;
  const int qrow = (int)(row / p.Hq), h = (int)(row % p.Hq);
  const ReqInfo rq = p.reqs[p.row_req[qrow]];
  if (rq.nseg <= 1) return;           // written directly by the split kernel
  const int j = qrow - rq.q0, n = rq.nq, nseg = rq.nseg;
  auto prow = [&](int sg) -> int64_t { return rq.part0 + ((int64_t)sg * n + j) * p.Hq + h; };
  auto load_group = [&](int k, float (&v)[G8][PER]) {
#pragma unroll
    for (int u = 0; u < G8; ++u)
#pragma unroll
      for (int x = 0; x < PER; ++x) v[u][x] = p.part_o[prow(min(k + u, nseg - 1)) * D + lane + 64 * x];
  };
  float v[G8][PER];
  load_group(0, v);
  float2 ml0 = make_float2(-INFINITY, 0.f);
  if (lane < nseg) ml0 = p.part_ml[prow(lane)];
  float M = ml0.x;
  for (int sg = 64 + lane; sg < nseg; sg += 64) M = fmaxf(M, p.part_ml[prow(sg)].x);
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  float acc[PER], L = 0.f;
#pragma unroll
  for (int x = 0; x < PER; ++x) acc[x] = 0.f;
  for (int s0 = 0; s0 < nseg; s0 += 64) {
    const float2 ml = s0 == 0 ? ml0 : (s0 + lane < nseg ? p.part_ml[prow(s0 + lane)] : make_float2(-INFINITY, 0.f));
    float w = 0.f;
    if (s0 + lane < nseg) {
      w = (ml.x == -INFINITY) ? 0.f : exp2f(ml.x - M);
      L += ml.y * w;
    }
    const int cnt = min(64, nseg - s0);
    for (int k = 0; k < cnt; k += G8) {
      if (s0 + k > 0) load_group(s0 + k, v);
#pragma unroll
      for (int u = 0; u < G8; ++u) {
        const float wu = __shfl(w, min(k + u, 63));
        if (k + u < cnt) {
#pragma unroll
          for (int x = 0; x < PER; ++x) acc[x] += wu * v[u][x];
        }
      }
    }
  }
  for (int o = 32; o >= 1; o >>= 1) L += __shfl_xor(L, o);
  const float inv = 1.f / L;
#pragma unroll
  for (int x = 0; x < PER; ++x) p.out[((int64_t)qrow * p.Hq + h) * D + lane + 64 * x] = acc[x] * inv;
}

template <int D, int PG>
hipError_t launch_mfma(const AttnParams& p, int nr, hipStream_t s) {
  const dim3 grid(p.grid);
  switch (nr) {
    case 1: attn_split_mfma<D, 1, SV_NS_W1, PG><<<grid, dim3(64), 0, s>>>(p); break;
    case 2: attn_split_mfma<D, 2, SV_NS_W2, PG><<<grid, dim3(128), 0, s>>>(p); break;
    case 3: attn_split_mfma<D, 3, SV_NS_W3, PG><<<grid, dim3(192), 0, s>>>(p); break;
    case 4: attn_split_mfma<D, 4, SV_NS_W4, PG><<<grid, dim3(256), 0, s>>>(p); break;
    case 5: attn_split_mfma<D, 5, SV_NS_W5, PG><<<grid, dim3(320), 0, s>>>(p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

#ifdef SV_ATTN_TRACE
extern "C" __attribute__((visibility("default"))) int sv_attn_trace_copy(void* dst, size_t bytes) {
  return (int)hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_attn_trace), bytes);
}
#endif

int max_rows_per_item(int dtype_bf16, int D) { return dtype_bf16 ? 80 : 4096 / D; }

int attn_lds_bytes(int D, int nr) {
  auto bytes = [&](auto d) -> int {
    constexpr int DD = decltype(d)::value;
    switch (nr) {
      case 1: return AttnLds<DD, 1, SV_NS_W1>::BYTES;
      case 2: return AttnLds<DD, 2, SV_NS_W2>::BYTES;
      case 3: return AttnLds<DD, 3, SV_NS_W3>::BYTES;
      case 4: return AttnLds<DD, 4, SV_NS_W4>::BYTES;
      case 5: return AttnLds<DD, 5, SV_NS_W5>::BYTES;
      default: return 0;
    }
  };
  return D == 64 ? bytes(std::integral_constant<int, 64>{}) : bytes(std::integral_constant<int, 128>{});
}

int attn_resident_per_cu(int D, int nr, int paged) {
  // per (D, waves, paged) build, asked once: the device's own placement
  static std::atomic<int> cache[2][5][3] = {};
  if ((D != 64 && D != 128) || nr < 1 || nr > 5) return 0;
  if (paged < 0 || paged > 2) return 0;
  std::atomic<int>& slot = cache[D == 128][nr - 1][paged];
  int v = slot.load(std::memory_order_relaxed);
  if (v != 0) return v > 0 ? v : 0;
  auto ask = [](auto kern, int threads) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, threads, 0) != hipSuccess) {
      (void)hipGetLastError();
      return -1;
    }
    return n > 0 ? n : -1;
  };
  auto by_build = [&](auto d, auto pg) -> int {
    constexpr int DD = decltype(d)::value;
    constexpr int PP = decltype(pg)::value;
    switch (nr) {
      case 1: return ask(attn_split_mfma<DD, 1, SV_NS_W1, PP>, 64);
      case 2: return ask(attn_split_mfma<DD, 2, SV_NS_W2, PP>, 128);
      case 3: return ask(attn_split_mfma<DD, 3, SV_NS_W3, PP>, 192);
      case 4: return ask(attn_split_mfma<DD, 4, SV_NS_W4, PP>, 256);
      default: return ask(attn_split_mfma<DD, 5, SV_NS_W5, PP>, 320);
    }
  };
  using I64 = std::integral_constant<int, 64>;
  using I128 = std::integral_constant<int, 128>;
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  v = D == 64 ? (paged == 2 ? by_build(I64{}, P2{}) : paged == 1 ? by_build(I64{}, P1{}) : by_build(I64{}, P0{}))
              : (paged == 2 ? by_build(I128{}, P2{}) : paged == 1 ? by_build(I128{}, P1{}) : by_build(I128{}, P0{}));
  slot.store(v, std::memory_order_relaxed);
  return v > 0 ? v : 0;
}

hipError_t launch_attention(const AttnParams& p, int dtype_bf16, int nr_max, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (p.n_items > 0) {
    if (dtype_bf16 && p.bt) {
      e = p.pool32 ? ((p.D == 64) ? launch_mfma<64, 2>(p, nr_max, s) : launch_mfma<128, 2>(p, nr_max, s))
                   : ((p.D == 64) ? launch_mfma<64, 1>(p, nr_max, s) : launch_mfma<128, 1>(p, nr_max, s));
    } else if (dtype_bf16) {
      e = (p.D == 64) ? launch_mfma<64, 0>(p, nr_max, s) : launch_mfma<128, 0>(p, nr_max, s);
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
