// Internal layout shared by the host planner and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/specverify.h"

namespace sv {

constexpr int kMaxNodes = 32;          // verify positions per request (chain k+1 or tree)
constexpr int kAccChunk = 4096;        // vocabulary entries per acceptance work-group
constexpr int kAccThreads = 256;

// One request of the step, as the kernels see it.
struct ReqInfo {
  int32_t ctx;      // c_i
  int32_t nq;       // n_i verify positions
  int32_t q0;       // first query / target-logit / uniform row
  int32_t kv0;      // first KV row
  int32_t d0;       // first draft-probability row
  int32_t nseg;     // KV splits of this request (1 = direct output)
  int32_t part0;    // first partial row (nseg > 1)
  int32_t node0;    // first entry of the request's node table (per-request trees)
};

// One node of a per-request token tree (the staged node table, and the
// acceptance kernels' device copy of it).
struct NodeInfo {
  uint32_t anc;     // ancestors-or-self bit mask
  int8_t parent;    // -1 for the root
  int8_t qrank;     // the request's draft-probability row of this node (nodes with children), else -1
  int8_t depth;
  int8_t pqrank;    // qrank of the parent (-1 for the root)
};
static_assert(sizeof(NodeInfo) == 8, "8-byte node entries");

// One attention work item: a KV range of one (request, KV head, query-head group).
// The request's fields are repeated here so a work-group needs one scalar
// load of 64 bytes before it can issue its first transfer.
struct AttnItem {
  int32_t req;
  int32_t kvh;
  int32_t head_lo;  // first query head of the group
  int32_t nheads;   // query heads in the group (rows = nheads * n_i)
  int32_t kb, ke;   // KV positions [kb, ke) relative to the request's first KV row
  int32_t seg;      // split index (partial slot) or -1 for direct output
  int32_t ctx;      // the request's c_i, n_i, first query row, first KV row, first partial
  int32_t nq;
  int32_t q0;
  int32_t kv0;
  int32_t part0;
  int32_t node0;    // the request's first node-table entry (per-request trees)
  int32_t stream;   // split items: the (request, KV head, head group) stream's arrival counter
  int32_t nseg;     // the request's KV pieces
  int32_t pad;
};

static_assert(sizeof(ReqInfo) == 32, "ReqInfo is copied as two 16-byte units");
static_assert(sizeof(AttnItem) == 64, "one 64-byte scalar load per work item");

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

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  int64_t q_st, q_sh, kv_st, kv_sh;   // element strides
  float* out;
  float* part_o;      // [P, d] unnormalised partial outputs
  float2* part_ml;    // [P] (running max in log2 units, running sum)
  const AttnItem* items;    // read where the host staged them (see below)
  const ReqInfo* reqs;      // device copies read by the split combine
  const int32_t* row_req;   // query row -> request
  // The plan stays in the caller's pinned staging buffer, mapped into the
  // device address space: each work-group reads its own item from there, so
  // no upload pass precedes the kernel.  The combine reads the request table
  // and the row map many times, so the split kernel's last `mirror_wg`
  // work-groups copy them (mirror_n16 16-byte units, ahead of the items in
  // the staged block) into device memory first.  mirror_n16 = 0: no copy.
  const uint4* mirror_src;
  uint4* mirror_dst;
  int32_t mirror_n16;
  int32_t mirror_wg;
  int32_t n_parts;           // rows of the partial buffers
  float scale_log2;   // scale * log2(e)
  int32_t Hq, Hkv, G, D;
  int32_t n_items;
  int32_t Nq;
  // paged KV cache (bt != nullptr): page pools, the block table and its row
  // stride, tokens per page (a multiple of 32), pages in the pool, page bytes
  const int32_t* bt;
  int32_t bt_stride;
  int32_t page_tokens;
  int32_t num_pages;
  int64_t page_bytes;
  uint32_t anc[kMaxNodes];   // ancestors-or-self masks (kernel arguments: uniform loads)
  // per-request trees (per_req = 1): each request's masks in its node-table
  // entries, read where the host staged them
  const NodeInfo* nodes;
  int32_t per_req;
  // Split combine inside the split kernel (bf16 path): each split stream's
  // pieces check in on counters[stream] ((call tag << 32) | arrivals), and
  // the last one to arrive combines the stream's partials.  The tag is new
  // on every call, so a counter holding another call's value (or anything
  // else) starts over at its first arrival and never needs clearing.
  unsigned long long* counters;
  uint32_t call_tag;
  int32_t fused;
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

// Largest number of query rows (heads x verify positions) one work item holds.
int max_rows_per_item(int dtype_bf16, int D);

hipError_t launch_attention(const AttnParams& p, int dtype_bf16, int nr_max, hipStream_t s);
// LDS bytes of the bf16 split kernel's build for head dim D and nr row tiles
// (the fused combine stages its weights there).
int attn_lds_bytes(int D, int nr);
hipError_t launch_combine(const AttnParams& p, hipStream_t s);
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

// The no-allocation entry point's device scratch (a static device array of
// kNoAllocScratchBytes) and its host staging (a static host array of
// kNoAllocStagingBytes).  noalloc_scratch returns the current device's
// address of the array, looked up once per device.
constexpr size_t kNoAllocScratchBytes = SPEC_NOALLOC_SCRATCH_BYTES;
constexpr size_t kNoAllocStagingBytes = SPEC_NOALLOC_STAGING_BYTES;
hipError_t noalloc_scratch(void** ptr);

}  // namespace sv
