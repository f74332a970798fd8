// Internal layout shared by the host planner and the gfx950 kernels: the
// acceptance, LM head and no-allocation declarations.  The request tables
// (sv_common.h) and the attention declarations (sv_attn.h) come with it.
#pragma once

#include "../../include/specverify.h"
#include "sv_attn.h"

namespace sv {

constexpr int kAccChunk = 4096;        // vocabulary entries per acceptance work-group
constexpr int kAccThreads = 256;

// Tree / chain topology tables (one per step).
struct Topo {
  uint32_t anc[kMaxNodes];    // ancestors-or-self bit mask of each node
  int32_t parent[kMaxNodes];  // -1 for the root
  int32_t qrank[kMaxNodes];   // draft-probability row of a node with children, else -1
  int32_t depth[kMaxNodes];
  int32_t inner[kMaxNodes];   // the nodes with children, in BFS order (tree mode)
  int32_t nodes;              // tree nodes (tree mode) or 0 (chain)
  int32_t n_inner;            // nodes with children (tree mode)
  int32_t pad[2];
};

// Acceptance scratch: per (row, vocabulary chunk) max and fp64 sum of exp.
struct ChunkStat {
  double s;
  float m;
  float pad;
};

// One value a work-group of the sequential sibling kernel hands the other
// work-groups of its request at one exchange.
struct SeqSlot {
  double x;
  int32_t y;
  int32_t pad;
};
constexpr int kSeqMaxGroups = 8;       // work-groups per request, at most

// Per request: the accepted node, the row the final token is drawn from, its
// draft row (-1: the extra token is drawn from p itself) and normaliser.
struct Decision {
  int32_t node, row, qrow, len;
  float M;      // row max
  float pad;
  double Z;     // sum of exp(l - M), fp64
};

struct AccParams {
  const void* logits;
  const void* probs;
  int64_t l_st, p_st;
  const int32_t* tokens;
  const float* uniforms;
  int32_t* acc_len;
  int32_t* next_tok;
  int32_t* acc_node;
  const ReqInfo* reqs_src;   // request table where the host staged it (mapped pinned memory)
  ReqInfo* reqs;             // [B] device copy, written by the row-statistics kernel
  ChunkStat* rowstats;   // [Nq, nch]; under the independent tree rule the row-statistics
                         // kernel fills the rows of nodes with children only, and the
                         // decision kernel a chosen leaf's row
  double* masses;        // [B, nch] final-sample weight mass per chunk
  int32_t* tickets;      // [B] chunk masses published per request (zeroed by the row-statistics kernel)
  int32_t V, nch, B, Nq;
  int32_t tree;        // 1 = tree mode
  int32_t bf16;
  Topo topo;           // kernel arguments: node tables without a memory round trip
  // per-request trees (per_req = 1): the node table where the host staged it,
  // and the device copy the row-statistics kernel makes (nodes_n16 16-byte units)
  const NodeInfo* nodes_src;
  NodeInfo* nodes;
  int32_t per_req;
  int32_t nodes_n16;
  int32_t all_stats;   // every row has chunk statistics before the decision kernel runs
  // sequential sibling rule: work-groups per request, and their exchange
  // slots [B, kMaxNodes, seq_groups]
  int32_t seq_groups;
  SeqSlot* seq_slots;
  // after the LM head (tiles != nullptr): the decision kernel folds the GEMM's
  // per-(row, kLmhNT-entry tile) statistics itself [Nq, ntiles], and rowstats
  // is not written
  const ChunkStat* tiles;
  int32_t ntiles;
};

constexpr int kAccMaxChunks = 1024;    // vocabularies up to 4M entries

// The target model's LM head, logits = hidden . weight^T, with the softmax
// statistics of each (row, kLmhNT-entry tile) taken in the epilogue.
constexpr int kLmhNT = 256;            // vocabulary entries per work-group and statistics tile
constexpr int kLmhTilesPerChunk = kAccChunk / kLmhNT;
struct LmhParams {
  const uint16_t* hidden;   // [M, K] bf16, row stride h_st elements
  const uint16_t* weight;   // [V, K] bf16, row stride w_st elements
  int64_t h_st, w_st;
  void* out;                // [M, V] logits (fp32, or bf16 when out_bf16), row stride o_st elements
  int64_t o_st;
  ChunkStat* tiles;         // [M, ntiles] per-tile (sum of exp(l - max), max)
  int32_t M, K, V, ntiles;
  int32_t m_tiles;          // row tiles of tile_rows rows (the last one may be shorter)
  int32_t tile_rows;        // <= the kernel's tile height 64 rb
  int32_t rb;               // 16-row blocks per wave: tile height 64 rb
  int32_t out_bf16;
  // the row-statistics kernel's other duties for the decision kernel that
  // follows: the request table's device copy (and the node table's, per-request
  // trees) and cleared tickets, done by the first work-groups
  const ReqInfo* reqs_src;
  ReqInfo* reqs;
  int32_t* tickets;
  const NodeInfo* nodes_src;
  NodeInfo* nodes;
  int32_t nodes_n16;
  int32_t B;
};
struct LmhGeometry {
  int32_t rb, tile_rows, m_tiles;
};
constexpr int kLmhMaxTileRows = 256;   // 16 x waves along the rows x row blocks per wave, at most
// The tile height and row tiles for M rows, ntiles vocabulary tiles and cus
// compute units.
LmhGeometry lmh_geometry(int M, int ntiles, int cus);
hipError_t launch_lmh(const LmhParams& p, hipStream_t s);
// Chunk statistics [Nq, nch] (the decision kernel's input) folded from the
// LM head's tile statistics, plus the row-statistics kernel's other duties
// (the request and node tables' device copies, cleared tickets).
hipError_t launch_foldstats(const AccParams& p, const ChunkStat* tiles, int ntiles, hipStream_t s);

// exp(x - m) for x <= m (a logit against a maximum): the hardware base-2
// exponential of (x - m) log2 e.  Its error is about an ulp of the result
// plus the roundings of x - m and of the product, the same order as the
// library expf, in three instructions instead of a dozen.  Every kernel that
// takes softmax statistics of logits evaluates exp(l - m) through this one
// function, so a statistic and the entries it summarises are always computed
// alike.
__device__ __forceinline__ float exp_rel(float x, float m) {
  return __builtin_amdgcn_exp2f((x - m) * 1.4426950408889634f);
}

// Both acceptance kernels; `mid` (optional) is recorded between them.
hipError_t launch_accept(const AccParams& p, hipStream_t s, hipEvent_t mid = nullptr);
// the two halves of launch_accept: row statistics, then decision and sample
hipError_t launch_rowstats(const AccParams& p, hipStream_t s);
hipError_t launch_decide(const AccParams& p, hipStream_t s);
// Debug check of the device-resident acceptance inputs: *flag (device) ends
// as the OR of 1 (draft token id outside [0, V)), 2 (uniform outside [0, 1))
// and 4 (draft probability at a draft token not > 0).
hipError_t launch_accept_validate(const AccParams& p, uint32_t* flag, hipStream_t s);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* out, int blocks, hipStream_t s);
// The acceptance floor probe's two kernels (stream, then the chain of
// dependent round trips) over num_rows (>= B) rows of v_bytes each.
hipError_t launch_accept_floor(const void* rows, int64_t row_bytes, int64_t v_bytes, int64_t chunk_bytes, int nch,
                               int num_rows, int B, uint32_t* sink, int32_t* tickets, uint64_t* sums, uint32_t* out,
                               hipStream_t s);

// The no-allocation entry point's device scratch (a static device array of
// kNoAllocScratchBytes) and its host staging (a static host array of
// kNoAllocStagingBytes).  noalloc_scratch returns the current device's
// address of the array, looked up once per device.
constexpr size_t kNoAllocScratchBytes = SPEC_NOALLOC_SCRATCH_BYTES;
constexpr size_t kNoAllocStagingBytes = SPEC_NOALLOC_STAGING_BYTES;
hipError_t noalloc_scratch(void** ptr);

}  // namespace sv
