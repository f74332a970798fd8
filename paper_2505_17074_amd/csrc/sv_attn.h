// The verify attention kernels' work items, parameters and launchers.
#pragma once

#include "sv_common.h"

namespace sv {

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

static_assert(sizeof(AttnItem) == 64, "one 64-byte scalar load per work item");

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
  int64_t pool_bytes;        // num_pages * page_bytes
  int32_t pool32;            // pool_bytes < 2^32: the paged build with one descriptor per item
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
  // Work-groups of the bf16 split kernel (grid >= n_items).  Work-group b <
  // first_round takes item b; every later one claims the next item from
  // *claim ((call tag << 32) | next item; a word holding another tag starts
  // over at first_round) and leaves when none is left.  Later work-groups are
  // dispatched as earlier ones end, so the XCDs that drain their items sooner
  // take more of the rest.  first_round = grid = n_items: no claims.
  int32_t grid;
  int32_t first_round;
  unsigned long long* claim;
};

// Largest number of query rows (heads x verify positions) one work item holds.
int max_rows_per_item(int dtype_bf16, int D);

hipError_t launch_attention(const AttnParams& p, int dtype_bf16, int nr_max, hipStream_t s);
// Work-groups of the bf16 split kernel's build for head dim D, nr waves and
// the paged or packed layout that one compute unit holds at once, as the
// device reports it; 0 where it cannot be asked (no device).  paged: 0 the
// packed build, 1 the paged build with a descriptor per tile, 2 the paged
// build with one descriptor per item (pools whose byte offsets fit 32 bits).
int attn_resident_per_cu(int D, int nr, int paged);
// The paged build a launch with these pool sizes takes (1 or 2).
inline int paged_build(int64_t num_pages, int64_t page_bytes) {
  return num_pages * page_bytes <= (int64_t)0xFFFFFFFF ? 2 : 1;
}
// LDS bytes of the bf16 split kernel's build for head dim D and nr row tiles
// (the fused combine stages its weights there).
int attn_lds_bytes(int D, int nr);
hipError_t launch_combine(const AttnParams& p, hipStream_t s);

}  // namespace sv
