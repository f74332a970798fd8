// C ABI of the verify step: argument checks, the host plan, workspace
// layout and the launch sequence.  Every check runs before the first HIP call.
#include "../../include/specverify.h"

#include <hip/hip_runtime.h>

#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "sv_internal.h"

namespace {

using sv::AttnItem;
using sv::ReqInfo;
using sv::Topo;

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Plan {
  // request view
  int B = 0;
  bool tree = false;
  bool per_req = false;             // a token tree per request
  std::vector<sv::NodeInfo> nodes;  // per-request trees: every request's node table
  int64_t Nq = 0, Nkv = 0, Nd = 0;
  std::vector<ReqInfo> reqs;
  std::vector<int32_t> row_req;
  Topo topo{};
  // attention
  bool has_attn = false;
  std::vector<AttnItem> items;
  int64_t parts = 0;      // partial rows
  int nr_max = 1;
  int split = 0;
  int64_t split_streams = 0;   // (request, KV head, head group) streams cut into pieces
  bool fused = false;          // the split kernel combines its own partials
  int64_t grid = 0;            // work-groups of the split kernel
  int64_t first_round = 0;     // work-groups that take their own index's item
  bool claim_word = false;     // the workspace holds the claim word
  // acceptance
  bool has_acc = false;
  int nch = 0;
  // layout (bytes)
  size_t off_reqs = 0, off_rowreq = 0, off_items = 0, off_nodes = 0, plan_bytes = 0;
  size_t off_acc_reqs = 0, off_acc_nodes = 0, off_tickets = 0, off_seq = 0;
  size_t off_part_o = 0, off_part_ml = 0, off_rowstats = 0, off_masses = 0, off_flag = 0, off_counters = 0;
  size_t off_claim = 0;
  size_t device_bytes = 0;
};

// A BFS parent array: parent[0] = -1, 0 <= parent[n] < n.
bool valid_tree(const int32_t* parent, int nodes) {
  if (nodes < 1 || nodes > SPEC_MAX_TREE_NODES || !parent || parent[0] != -1) return false;
  for (int n = 1; n < nodes; ++n)
    if (parent[n] < 0 || parent[n] >= n) return false;
  return true;
}

spec_status_t check_requests(const spec_requests_t* r) {
  if (!r || r->num_requests < 1 || !r->ctx_len) return SPEC_ERR_INVALID_ARG;
  if (r->tree_nodes < 0 || r->tree_nodes > SPEC_MAX_TREE_NODES) return SPEC_ERR_INVALID_ARG;
  if (r->node_count) {
    // per-request trees: no shared tree besides them
    if (r->tree_nodes != 0 || !r->tree_parents) return SPEC_ERR_INVALID_ARG;
    int64_t o = 0;
    for (int i = 0; i < r->num_requests; ++i) {
      if (!valid_tree(r->tree_parents + o, r->node_count[i])) return SPEC_ERR_INVALID_ARG;
      o += r->node_count[i];
    }
  } else if (r->tree_nodes > 0) {
    if (!valid_tree(r->tree_parent, r->tree_nodes)) return SPEC_ERR_INVALID_ARG;
  } else if (!r->draft_len) {
    return SPEC_ERR_INVALID_ARG;
  }
  int64_t nq = 0, nkv = 0;
  for (int i = 0; i < r->num_requests; ++i) {
    if (r->ctx_len[i] < 0) return SPEC_ERR_INVALID_ARG;
    int n = r->node_count ? r->node_count[i] : r->tree_nodes;
    if (n == 0) {
      if (r->draft_len[i] < 0 || r->draft_len[i] > SPEC_MAX_DRAFT) return SPEC_ERR_INVALID_ARG;
      n = r->draft_len[i] + 1;
    }
    nq += n;
    nkv += (int64_t)r->ctx_len[i] + n;
  }
  if (nq >= INT32_MAX / 2 || nkv >= INT32_MAX / 2) return SPEC_ERR_INVALID_ARG;
  return SPEC_OK;
}

spec_status_t check_attn(const spec_attn_args_t* a) {
  if (!a) return SPEC_ERR_INVALID_ARG;
  if (a->num_q_heads < 1 || a->num_kv_heads < 1 || a->num_q_heads % a->num_kv_heads)
    return SPEC_ERR_INVALID_ARG;
  if (a->dtype != SPEC_F32 && a->dtype != SPEC_BF16) return SPEC_ERR_INVALID_ARG;
  if (a->head_dim != 64 && a->head_dim != 128) return SPEC_ERR_UNSUPPORTED;
  if (!a->q || !a->k || !a->v || !a->out) return SPEC_ERR_INVALID_ARG;
  if (!aligned16(a->q) || !aligned16(a->k) || !aligned16(a->v) || !aligned16(a->out))
    return SPEC_ERR_INVALID_ARG;
  const int64_t vec = a->dtype == SPEC_F32 ? 4 : 8;   // elements per 16 bytes
  if (a->q_stride_tok < 1 || a->q_stride_head < 1 || a->kv_stride_tok < 1 || a->kv_stride_head < 1)
    return SPEC_ERR_INVALID_ARG;
  if (a->q_stride_tok % vec || a->q_stride_head % vec || a->kv_stride_tok % vec || a->kv_stride_head % vec)
    return SPEC_ERR_INVALID_ARG;
  if (a->split_kv < 0 || (a->split_kv > 0 && a->split_kv % 32)) return SPEC_ERR_INVALID_ARG;
  if (a->block_table) {
    // paged pools [num_pages, page_tokens, Hkv, d]: a token row holds every head
    if (a->page_tokens < 32 || a->page_tokens % 32 || a->num_pages < 1 || a->block_stride < 1)
      return SPEC_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(a->block_table) % 4) return SPEC_ERR_INVALID_ARG;
    if (a->kv_stride_head * (a->num_kv_heads - 1) + a->head_dim > a->kv_stride_tok) return SPEC_ERR_INVALID_ARG;
    if (a->dtype != SPEC_BF16) return SPEC_ERR_UNSUPPORTED;
    // one page's rows of one head are addressed with 32-bit offsets
    if ((int64_t)a->page_tokens * a->kv_stride_tok * 2 >= INT32_MAX) return SPEC_ERR_UNSUPPORTED;
  }
  return SPEC_OK;
}

spec_status_t check_accept(const spec_accept_args_t* a, int64_t Nq, int B) {
  if (!a) return SPEC_ERR_INVALID_ARG;
  if (a->dtype != SPEC_F32 && a->dtype != SPEC_BF16) return SPEC_ERR_INVALID_ARG;
  if (a->vocab < 1 || (int64_t)a->vocab > (int64_t)sv::kAccMaxChunks * sv::kAccChunk) return SPEC_ERR_INVALID_ARG;
  if (!a->target_logits || !a->uniforms || !a->accepted_len || !a->next_token) return SPEC_ERR_INVALID_ARG;
  if (Nq > B && (!a->draft_probs || !a->draft_tokens)) return SPEC_ERR_INVALID_ARG;
  const int64_t vec = a->dtype == SPEC_F32 ? 4 : 8;
  if (a->logits_stride < a->vocab || a->logits_stride % vec || !aligned16(a->target_logits))
    return SPEC_ERR_INVALID_ARG;
  if (a->draft_probs && (a->probs_stride < a->vocab || a->probs_stride % vec || !aligned16(a->draft_probs)))
    return SPEC_ERR_INVALID_ARG;
  if (a->tree_rule != SPEC_TREE_INDEPENDENT && a->tree_rule != SPEC_TREE_SEQUENTIAL) return SPEC_ERR_INVALID_ARG;
  return SPEC_OK;
}

// SPEC_DEBUG_VALIDATE set to a non-empty value other than "0" (read per call).
bool debug_validate() {
  const char* e = std::getenv("SPEC_DEBUG_VALIDATE");
  return e && e[0] && !(e[0] == '0' && e[1] == 0);
}

// Compute units of the current device (cached; 256 when it cannot be asked,
// e.g. for a size query on a host without a GPU).
int device_cus() {
  static int cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      n = 256;
    }
    cus[dev] = n;
  }
  return cus[dev];
}

// Work-groups of the bf16 split kernel that run at once per compute unit.
// Measured, not taken from the occupancy calculator (which allows 3 for the
// 4- and 5-wave builds): with 64 equal streams cut into 8 pieces each (512
// items on 256 compute units) every width, at d = 64 and d = 128, runs 7-27%
// faster than with 9 pieces each (576 items), whose last 64 items form a
// second, nearly empty round.
#ifndef SV_GROUPS_W5
#define SV_GROUPS_W5 2
#endif
int groups_per_cu(int waves) { return waves == 5 ? SV_GROUPS_W5 : 2; }

// Piece length for a stream of L >= 1 keys and a split of s >= 1 keys: the
// stream cut into ceil(L / s) equal parts, rounded up to 32 keys (a short
// trailing piece would leave its work-group idle most of the kernel while its
// partial costs the same).  Every piece but the last has this length.
int piece_len(int L, int64_t s) {
  const int64_t n0 = (L + s - 1) / s;
  return (int)(((L + n0 - 1) / n0 + 31) / 32 * 32);
}

// Keys per split piece.  `slots` = work-groups the device runs at once;
// `len[i]` = keys of request i, each the length of `mult[i]` streams (one per
// KV head and head group).  Pieces stay >= 40 * rows keys, so the fp32
// partials (rows x d x 4 bytes, written once and read once by the combine)
// remain a few percent of the K/V bytes a piece streams (32 rows x d x 2 x 2
// per 32 keys), and >= 256 keys.
//  - At least as many streams as slots: pieces of at most kMaxPiece keys,
//    dispatched longest first, the items past the first round claimed at run
//    time.  A work-group streams about 30 keys per microsecond, so a
//    4096-key piece started first runs nearly as long as the whole kernel on
//    a 128-request ragged batch (3200 keys per slot on average).  Measured
//    there with claims, attention alone: 2048-key pieces 158 us, 2560 150,
//    3072 146, 3328-3840 142-143, 4096 155 (and 155 without claims).
//  - Fewer streams than slots: the smallest split whose items all fit one
//    round of slots, so every work-group takes exactly one item and none waits
//    for a second round (on 8 requests of 16K-32K keys x 8 KV heads, 504 items
//    of <= 3264 keys: about 7% faster than 408 items of <= 4096 keys, and 24%
//    faster than 528 items of <= 3072).
#ifndef SV_MAX_PIECE
#define SV_MAX_PIECE 3584
#endif
constexpr int64_t kMaxPiece = SV_MAX_PIECE;
// Largest partial block (rows x pieces x d x 4 bytes) of one split stream
// that the split kernel's last piece combines itself; above it the separate
// combine kernel spreads the work over the device.  The last piece reads the
// block alone, after every other piece of the stream has finished: on the
// ragged GQA batch (streams of <= 55 KB) fusing shortens the attention by
// 5 us and the step by 10 us, while on the long-context batch (295 KB per
// stream) it lengthens the attention by 7 us.  The environment variable
// SPEC_FUSED_COMBINE_MAX_BYTES overrides the limit (tests use it to reach
// the fused path with any stream).
constexpr int64_t kFuseMaxBytes = 64 << 10;
int64_t fuse_max_bytes() {
  const char* e = std::getenv("SPEC_FUSED_COMBINE_MAX_BYTES");
  if (!e || !*e) return kFuseMaxBytes;
  char* end = nullptr;
  const long long v = std::strtoll(e, &end, 10);
  return (end && *end == 0 && v >= 0) ? (int64_t)v : kFuseMaxBytes;
}
constexpr int64_t kMaxSplit = 1 << 20;
// Work-groups launched beyond the item count when items are claimed at run
// time.  Work-group b runs on XCD b % 8, and the XCDs stream at different
// rates (the slowest 5-10 % below the fastest on ragged batches, the same
// XCDs on every device measured), so an XCD that drains its items sooner
// can use more work-groups than an eighth of the items; the surplus finds
// nothing left and ends at once.  Measured on the 128-request ragged batch,
// 0 to 384 surplus work-groups are within 0.5 us of each other: the claims'
// gain is their order (the next item to whichever slot frees first, across
// the XCDs), not the surplus.  The environment variable SPEC_ATTN_EXTRA_WG
// overrides the count.
int64_t env_count(const char* name, int64_t dflt, int64_t lo) {
  const char* e = std::getenv(name);
  if (!e || !*e) return dflt;
  char* end = nullptr;
  const long long v = std::strtoll(e, &end, 10);
  return (end && *end == 0 && v >= lo && v <= (1 << 20)) ? (int64_t)v : dflt;
}
// Work-groups that take their own index's item: by default every
// work-group the device holds at once.  The environment variable
// SPEC_ATTN_FIRST_ROUND overrides it (tests use it to reach the claims with
// few items).
int64_t claim_first_round(int64_t slots) { return env_count("SPEC_ATTN_FIRST_ROUND", slots, 1); }
int64_t claim_extra(int64_t n_items) {
  return env_count("SPEC_ATTN_EXTRA_WG", (n_items / 6 + 7) / 8 * 8, 0);
}
// Keys per piece of each request's streams (every KV head and head group of
// a request has the same length).  `slots` = work-groups the device runs at
// once; `len[i]` = keys of request i, each the length of `mult[i]` streams.
// Pieces stay >= 40 * rows keys, so the fp32 partials (rows x d x 4 bytes,
// written once and read once by the combine) remain a few percent of the K/V
// bytes a piece streams (32 rows x d x 2 x 2 per 32 keys), and >= 256 keys.
//  - At least as many streams as slots: pieces of at most kMaxPiece keys
//    (above), dispatched longest first.
//  - Fewer streams than slots: every work-group takes exactly one item (a
//    second, nearly empty round of items ran 7-27% slower), and the pieces
//    are cut so that the longest is as short as the slots allow: one piece
//    per stream to start with, then repeatedly one more piece for the
//    request whose pieces are currently longest, while its streams' extra
//    items still fit the slots.  Every work-group streams at about the same
//    rate, so the longest piece sets the kernel's end.
#ifndef SV_MIN_PIECE_ROWS
#define SV_MIN_PIECE_ROWS 40
#endif
std::vector<int> piece_lengths(const std::vector<int>& len, const std::vector<int>& mult, int rows_max, int64_t slots) {
  slots = std::max<int64_t>(slots, 1);
  int64_t lo = std::max<int64_t>(SV_MIN_PIECE_ROWS * (int64_t)rows_max, 256);
  lo = std::min<int64_t>((lo + 31) / 32 * 32, kMaxSplit);
  const size_t B = len.size();
  std::vector<int> out(B);
  int64_t streams = 0;
  for (size_t i = 0; i < B; ++i) streams += mult[i];
  if (streams >= slots) {
    for (size_t i = 0; i < B; ++i) out[i] = piece_len(len[i], std::max(kMaxPiece, lo));
    return out;
  }
  // greedy: a max-heap of (current piece length, request)
  std::vector<int64_t> n(B, 1);
  auto cur = [&](size_t i) { return ((int64_t)len[i] + n[i] - 1) / n[i]; };
  std::vector<std::pair<int64_t, size_t>> heap;
  heap.reserve(B);
  for (size_t i = 0; i < B; ++i) heap.emplace_back(cur(i), i);
  std::make_heap(heap.begin(), heap.end());
  int64_t total = streams;
  while (!heap.empty()) {
    std::pop_heap(heap.begin(), heap.end());
    const size_t i = heap.back().second;
    heap.pop_back();
    // one more piece for request i: its pieces must stay >= lo keys, and its
    // streams' extra items must fit the remaining slots
    if (((int64_t)len[i] + n[i]) / (n[i] + 1) < lo || total + mult[i] > slots) break;
    ++n[i];
    total += mult[i];
    heap.emplace_back(cur(i), i);
    std::push_heap(heap.begin(), heap.end());
  }
  for (size_t i = 0; i < B; ++i) {
    const int64_t piece = (cur(i) + 31) / 32 * 32;            // equal 32-aligned pieces
    out[i] = (int)std::min<int64_t>(std::max<int64_t>(piece, 32), kMaxSplit);
  }
  return out;
}

spec_status_t build_plan(const spec_requests_t* r, const spec_attn_args_t* attn,
                         const spec_accept_args_t* acc, Plan& P) {
  spec_status_t st = check_requests(r);
  if (st != SPEC_OK) return st;
  P.B = r->num_requests;
  P.per_req = r->node_count != nullptr;
  P.tree = r->tree_nodes > 0 || P.per_req;
  if (attn) {
    st = check_attn(attn);
    if (st != SPEC_OK) return st;
  }

  // topology tables
  std::memset(&P.topo, 0, sizeof(P.topo));
  const int tn = r->tree_nodes;
  int n_int = 0;
  for (int n = 0; n < sv::kMaxNodes; ++n) {
    P.topo.parent[n] = n - 1;
    P.topo.qrank[n] = -1;
    P.topo.depth[n] = n;
    P.topo.anc[n] = (n >= 31) ? 0xffffffffu : ((2u << n) - 1u);   // chain: nodes 0..n
  }
  if (P.tree && !P.per_req) {
    std::vector<bool> has_child(tn, false);
    for (int n = 1; n < tn; ++n) has_child[r->tree_parent[n]] = true;
    for (int n = 0; n < tn; ++n) {
      P.topo.parent[n] = r->tree_parent[n];
      P.topo.depth[n] = n == 0 ? 0 : P.topo.depth[r->tree_parent[n]] + 1;
      P.topo.anc[n] = (1u << n) | (n == 0 ? 0u : P.topo.anc[r->tree_parent[n]]);
      P.topo.qrank[n] = has_child[n] ? n_int++ : -1;
      if (has_child[n]) P.topo.inner[P.topo.qrank[n]] = n;
    }
    P.topo.nodes = tn;
    P.topo.n_inner = n_int;
  }

  // requests (and, per-request trees, every request's node table)
  P.reqs.resize(P.B);
  int64_t q0 = 0, kv0 = 0, d0 = 0, o = 0;
  for (int i = 0; i < P.B; ++i) {
    ReqInfo& q = P.reqs[i];
    q.ctx = r->ctx_len[i];
    q.nq = P.per_req ? r->node_count[i] : (P.tree ? tn : r->draft_len[i] + 1);
    q.q0 = (int32_t)q0;
    q.kv0 = (int32_t)kv0;
    q.d0 = (int32_t)d0;
    q.nseg = 1;
    q.part0 = 0;
    q.node0 = (int32_t)o;
    int inner_i = P.tree ? n_int : q.nq - 1;
    if (P.per_req) {
      const int32_t* par = r->tree_parents + o;
      const int nn = q.nq;
      bool has_child[sv::kMaxNodes] = {};
      for (int n = 1; n < nn; ++n) has_child[par[n]] = true;
      inner_i = 0;
      const size_t base = P.nodes.size();
      P.nodes.resize(base + nn);
      for (int n = 0; n < nn; ++n) {
        sv::NodeInfo& e = P.nodes[base + n];
        e.parent = (int8_t)par[n];
        e.depth = (int8_t)(n == 0 ? 0 : P.nodes[base + par[n]].depth + 1);
        e.anc = (1u << n) | (n == 0 ? 0u : P.nodes[base + par[n]].anc);
        e.qrank = (int8_t)(has_child[n] ? inner_i++ : -1);
        e.pqrank = (int8_t)(n == 0 ? -1 : P.nodes[base + par[n]].qrank);
      }
      o += nn;
    }
    q0 += q.nq;
    kv0 += (int64_t)q.ctx + q.nq;
    d0 += inner_i;
  }
  P.Nq = q0;
  P.Nkv = kv0;
  P.Nd = d0;
  P.row_req.resize(P.Nq);
  for (int i = 0; i < P.B; ++i)
    for (int j = 0; j < P.reqs[i].nq; ++j) P.row_req[P.reqs[i].q0 + j] = i;

  if (acc) {
    st = check_accept(acc, P.Nq, P.B);
    if (st != SPEC_OK) return st;
    P.has_acc = true;
    P.nch = (acc->vocab + sv::kAccChunk - 1) / sv::kAccChunk;
  }

  if (attn) {
    const int64_t elem = attn->dtype == SPEC_F32 ? 4 : 2;
    for (int i = 0; i < P.B; ++i) {
      const int64_t L = (int64_t)P.reqs[i].ctx + P.reqs[i].nq;
      if (attn->block_table) {
        // every logical page of the request has a block table entry
        if ((L + attn->page_tokens - 1) / attn->page_tokens > attn->block_stride) return SPEC_ERR_INVALID_ARG;
      } else if (L * attn->kv_stride_tok * elem >= INT32_MAX) {
        // the packed path addresses one request's rows of one KV head with 32-bit offsets
        return SPEC_ERR_UNSUPPORTED;
      }
    }
    P.has_attn = true;
    const int bf = attn->dtype == SPEC_BF16;
    const int D = attn->head_dim;
    const int Hq = attn->num_q_heads, Hkv = attn->num_kv_heads, G = Hq / Hkv;
    const int rmax = sv::max_rows_per_item(bf, D);
    // query-head groups per request so that heads * n_i <= rmax
    std::vector<int> groups(P.B), hpg(P.B), len(P.B), mult(P.B);
    int rows_max = 1;
    for (int i = 0; i < P.B; ++i) {
      const int n = P.reqs[i].nq;
      const int hmax = std::max(1, rmax / n);          // heads that fit one item
      const int ng = (G + hmax - 1) / hmax;
      hpg[i] = (G + ng - 1) / ng;                      // balanced, still <= hmax
      groups[i] = (G + hpg[i] - 1) / hpg[i];
      len[i] = P.reqs[i].ctx + n;
      mult[i] = Hkv * groups[i];
      rows_max = std::max(rows_max, hpg[i] * n);
    }
    const int64_t slots = (int64_t)device_cus() * (bf ? groups_per_cu((rows_max + 15) / 16) : 2);
    std::vector<int> plen;
    if (attn->split_kv > 0) {
      plen.resize(P.B);
      for (int i = 0; i < P.B; ++i) plen[i] = piece_len(len[i], attn->split_kv);
    } else {
      plen = piece_lengths(len, mult, rows_max, slots);
    }
    P.split = 0;
    for (int i = 0; i < P.B; ++i) P.split = std::max(P.split, plen[i]);
    int64_t part = 0;
    int nr = 1;
    {
      int64_t n_items = 0;
      for (int i = 0; i < P.B; ++i) n_items += (int64_t)((len[i] + plen[i] - 1) / plen[i]) * mult[i];
      P.items.reserve((size_t)n_items);
    }
    for (int i = 0; i < P.B; ++i) {
      ReqInfo& q = P.reqs[i];
      const int L = len[i];
      const int piece = plen[i];
      q.nseg = (L + piece - 1) / piece;
      q.part0 = (int32_t)part;
      if (q.nseg > 1) part += (int64_t)q.nseg * q.nq * Hq;
      const int64_t stream0 = P.split_streams;
      if (q.nseg > 1) P.split_streams += (int64_t)Hkv * groups[i];
      for (int s = 0; s < q.nseg; ++s) {
        for (int g = 0; g < Hkv; ++g) {
          for (int gr = 0; gr < groups[i]; ++gr) {
            AttnItem it;
            it.req = i;
            it.kvh = g;
            it.head_lo = g * G + gr * hpg[i];
            it.nheads = std::min(hpg[i], G - gr * hpg[i]);
            it.kb = s * piece;
            it.ke = std::min(L, (s + 1) * piece);
            it.seg = q.nseg > 1 ? s : -1;
            it.ctx = q.ctx;
            it.nq = q.nq;
            it.q0 = q.q0;
            it.kv0 = q.kv0;
            it.part0 = q.part0;
            it.node0 = q.node0;
            it.stream = q.nseg > 1 ? (int32_t)(stream0 + (int64_t)g * groups[i] + gr) : -1;
            it.nseg = q.nseg;
            it.pad = 0;
            P.items.push_back(it);
            nr = std::max(nr, (it.nheads * q.nq + 15) / 16);
          }
        }
      }
    }
    // Longest items first: work-groups are dispatched in index order as slots
    // free up, so the last ones to start are the shortest and the kernel's
    // tail (slots idling while a few long items finish) stays short.  A
    // stable counting sort on the tile count (linear in the item count).
    {
      int max_t = 0;
      for (const AttnItem& it : P.items) max_t = std::max(max_t, (it.ke - it.kb + 31) / 32);
      std::vector<int> start(max_t + 2, 0);
      for (const AttnItem& it : P.items) ++start[max_t - (it.ke - it.kb + 31) / 32 + 1];
      for (int t = 1; t <= max_t + 1; ++t) start[t] += start[t - 1];
      std::vector<AttnItem> sorted(P.items.size());
      for (const AttnItem& it : P.items) sorted[start[max_t - (it.ke - it.kb + 31) / 32]++] = it;
      P.items.swap(sorted);
    }
    // Items past the first round go to whichever work-groups start next
    // (bf16 kernel; see claim_extra).  The first round is every work-group
    // the device holds at once (at least the plan's slots), so no claim
    // starts before a first-round work-group has ended.  The workspace keeps
    // the claim word whenever there are more items than slots, whatever the
    // device reports.
    const int64_t n_it = (int64_t)P.items.size();
    const int build = !attn->block_table ? 0
                      : sv::paged_build(attn->num_pages, (int64_t)attn->page_tokens * attn->kv_stride_tok * 2);
    const int64_t resident = (int64_t)device_cus() * sv::attn_resident_per_cu(D, nr, build);
    const int64_t first = claim_first_round(std::max(slots, resident));
    P.first_round = P.grid = n_it;
    P.claim_word = bf && n_it > std::min(first, slots);
    if (bf && n_it > first) {
      P.first_round = first;
      P.grid = n_it + claim_extra(n_it);
    }
    if (part >= INT32_MAX || P.grid >= INT32_MAX) return SPEC_ERR_INVALID_ARG;
    P.parts = part;
    P.nr_max = nr;
    // The bf16 kernel combines a split stream's partials itself (the last
    // piece to finish) when the stream's combine weights fit its LDS: rows x
    // (pieces + 1) floats.  Otherwise the split combine kernel runs after it.
    if (bf && part > 0) {
      int64_t lds = 0, blk = 0, stream_bytes = 0;
      for (int i = 0; i < P.B; ++i) {
        const ReqInfo& q = P.reqs[i];
        if (q.nseg <= 1) continue;
        const int64_t rows = (int64_t)hpg[i] * q.nq;
        lds = std::max<int64_t>(lds, rows * (2 * (int64_t)q.nseg + 1) * 4);
        blk = std::max<int64_t>(blk, (int64_t)q.nseg * q.nq * Hq * D * 4);
        stream_bytes = std::max<int64_t>(stream_bytes, rows * q.nseg * D * 4);
      }
      P.fused = lds <= sv::attn_lds_bytes(D, nr) && blk < ((int64_t)1 << 31) && stream_bytes <= fuse_max_bytes();
    }
  }

  // Staged block (the caller's pinned staging buffer; the kernels read it in
  // place): request table, row -> request map, attention items.  The device
  // workspace starts with room for the same block -- the split combine's
  // copies of the table and map, or all of it when the staging buffer is
  // not device-mapped and is copied -- followed by device-only scratch.
  size_t off = 0;
  P.off_reqs = off;
  off = align_up(off + sizeof(ReqInfo) * P.B);
  P.off_rowreq = off;
  off = align_up(off + sizeof(int32_t) * P.Nq);
  P.off_items = off;
  off = align_up(off + sizeof(AttnItem) * P.items.size());
  P.off_nodes = off;                   // per-request trees: the node table
  off = align_up(off + sizeof(sv::NodeInfo) * P.nodes.size());
  P.plan_bytes = off;
  P.off_acc_reqs = off;                // the acceptance kernels' copy of the table
  off = align_up(off + sizeof(ReqInfo) * (size_t)(P.has_acc ? P.B : 0));
  P.off_acc_nodes = off;               // and of the node table
  off = align_up(off + sizeof(sv::NodeInfo) * (P.has_acc ? P.nodes.size() : 0));
  P.off_tickets = off;                 // acceptance tickets, cleared on the device
  off = align_up(off + sizeof(int32_t) * (size_t)(P.has_acc ? P.B : 0));
  P.off_seq = off;                     // sequential sibling rule: exchange slots
  off = align_up(off + sizeof(sv::SeqSlot) * sv::kMaxNodes * sv::kSeqMaxGroups * (size_t)(P.has_acc && P.tree ? P.B : 0));
  const int D = attn ? attn->head_dim : 0;
  P.off_part_o = off;
  off = align_up(off + sizeof(float) * (size_t)P.parts * D);
  P.off_part_ml = off;
  off = align_up(off + sizeof(float) * 2 * (size_t)P.parts);
  P.off_counters = off;                // the fused combine's arrival counters
  off = align_up(off + sizeof(unsigned long long) * (size_t)(P.fused ? P.split_streams : 0));
  P.off_claim = off;                   // the split kernel's claim word
  off = align_up(off + (P.claim_word ? sizeof(unsigned long long) : 0));
  P.off_rowstats = off;
  off = align_up(off + sizeof(sv::ChunkStat) * (size_t)(P.has_acc ? P.Nq * P.nch : 0));
  P.off_masses = off;
  off = align_up(off + sizeof(double) * (size_t)(P.has_acc ? (int64_t)P.B * P.nch : 0));
  P.off_flag = off;                    // debug check result (SPEC_DEBUG_VALIDATE)
  off = align_up(off + (P.has_acc ? sizeof(uint32_t) : 0));
  P.device_bytes = off;
  return SPEC_OK;
}

// spec_verify runs the acceptance kernels (which read only logits, draft
// rows, tokens and uniforms) on a side stream forked from the caller's stream
// at the start of the call and joined back before returning, so they overlap
// the attention kernels.  One side stream and one fork/join event pair per
// device, created on first use at the default priority and kept for the life
// of the process; the mutex keeps concurrent callers' fork/join pairs apart.
struct SideStream {
  std::mutex mu;
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool ready = false;
};
constexpr int kMaxDevices = 64;
SideStream g_side[kMaxDevices];

SideStream* side_stream() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  SideStream& S = g_side[dev];
  std::lock_guard<std::mutex> lk(S.mu);
  if (!S.ready) {
    if (hipStreamCreateWithFlags(&S.s, hipStreamNonBlocking) != hipSuccess) return nullptr;
    // The pair only orders kernels of two streams on this device; every kernel
    // dispatch carries its own acquire and release fences, so the events skip
    // the system-scope fence (host visibility), which costs each step a
    // cache write-back (measured 1-3% of a step).
    constexpr unsigned kEv = hipEventDisableTiming | hipEventDisableSystemFence;
    if (hipEventCreateWithFlags(&S.fork, kEv) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&S.join, kEv) != hipSuccess) return nullptr;
    S.ready = true;
  }
  return &S;
}

// A fresh 32-bit tag per call for the fused combine's arrival counters, never
// 0 (fresh device memory is often zero).  The process's first tag is drawn
// from the clock and the process id, so memory left by an earlier process
// is as unlikely to match as anything else.
uint32_t next_call_tag() {
  static std::atomic<uint32_t> tag{
      (uint32_t)std::chrono::steady_clock::now().time_since_epoch().count() * 2654435761u ^ (uint32_t)getpid()};
  uint32_t t;
  do {
    t = tag.fetch_add(1, std::memory_order_relaxed);
  } while (t == 0);
  return t;
}

void write_staging(const Plan& P, void* host) {
  char* h = static_cast<char*>(host);
  // every section is written whole (alignment padding between sections is
  // copied along with the table and map but never read)
  std::memcpy(h + P.off_reqs, P.reqs.data(), sizeof(ReqInfo) * P.reqs.size());
  if (!P.items.empty()) std::memcpy(h + P.off_items, P.items.data(), sizeof(AttnItem) * P.items.size());
  std::memcpy(h + P.off_rowreq, P.row_req.data(), sizeof(int32_t) * P.row_req.size());
  if (!P.nodes.empty()) std::memcpy(h + P.off_nodes, P.nodes.data(), sizeof(sv::NodeInfo) * P.nodes.size());
}

// How run() places the work: the normal entry points overlap the two parts
// on a side stream and take the caller's staging; the no-allocation entry
// point keeps everything on the caller's stream and stages the plan in
// library-owned pageable memory, which is always copied.
struct RunMode {
  bool overlap = true;
  bool pageable = false;      // staging known not to be device-mapped
  std::mutex* staging_mu = nullptr;   // held while the staging is written and the copy enqueued
  const spec_lm_head_args_t* lm = nullptr;   // the LM head runs first, its statistics replace the row pass
  size_t off_tiles = 0;       // its tile statistics in the workspace
};

spec_status_t check_lm(const spec_lm_head_args_t* lm) {
  if (!lm || !lm->hidden || !lm->weight) return SPEC_ERR_INVALID_ARG;
  if (lm->hidden_dim < 32 || lm->hidden_dim % 32) return SPEC_ERR_INVALID_ARG;
  if (!aligned16(lm->hidden) || !aligned16(lm->weight)) return SPEC_ERR_INVALID_ARG;
  if (lm->hidden_stride < lm->hidden_dim || lm->hidden_stride % 8 || lm->weight_stride < lm->hidden_dim ||
      lm->weight_stride % 8)
    return SPEC_ERR_INVALID_ARG;
  // each work-group's rows are addressed with 32-bit offsets
  if ((int64_t)sv::kLmhNT * lm->weight_stride * 2 >= INT32_MAX ||
      (int64_t)sv::kLmhMaxTileRows * lm->hidden_stride * 2 >= INT32_MAX)
    return SPEC_ERR_UNSUPPORTED;
  return SPEC_OK;
}

// The LM-head call's plan: the acceptance plan plus the tile statistics
// [Nq, ceil(V / 256)] at the end of the workspace.
spec_status_t lm_plan(const spec_requests_t* req, const spec_lm_head_args_t* lm, const spec_accept_args_t* acc,
                      Plan& P, size_t& off_tiles, size_t& device_bytes) {
  if (!acc) return SPEC_ERR_INVALID_ARG;
  spec_status_t st = build_plan(req, nullptr, acc, P);
  if (st != SPEC_OK) return st;
  if ((st = check_lm(lm)) != SPEC_OK) return st;
  const int64_t ntiles = (acc->vocab + sv::kLmhNT - 1) / sv::kLmhNT;
  off_tiles = P.device_bytes;
  device_bytes = align_up(off_tiles + sizeof(sv::ChunkStat) * (size_t)(P.Nq * ntiles));
  return SPEC_OK;
}

spec_status_t run(const spec_requests_t* req, const spec_attn_args_t* attn, const spec_accept_args_t* acc,
                  void* ws, size_t ws_bytes, void* staging, size_t staging_bytes, void* stream,
                  const RunMode& mode = RunMode()) {
  Plan P;
  spec_status_t st = build_plan(req, attn, acc, P);
  if (st != SPEC_OK) return st;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) || ws_bytes < P.device_bytes) return SPEC_ERR_WORKSPACE;
  if (!staging || staging_bytes < P.plan_bytes) return SPEC_ERR_WORKSPACE;

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* d = static_cast<char*>(ws);
  // The kernels read the plan where it was staged when the staging buffer is
  // device-mapped pinned memory (no upload pass ahead of them); otherwise it
  // is copied into the workspace first.
  const char* pl = d;
  {
    std::unique_lock<std::mutex> lk;
    if (mode.staging_mu) lk = std::unique_lock<std::mutex>(*mode.staging_mu);
    write_staging(P, staging);
    void* mapped = nullptr;
    if (!mode.pageable && hipHostGetDevicePointer(&mapped, staging, 0) == hipSuccess && mapped &&
        aligned16(mapped)) {
      pl = static_cast<const char*>(mapped);
    } else {
      if (!mode.pageable) (void)hipGetLastError();   // clear the lookup's error state
      if (hipMemcpyAsync(d, staging, P.plan_bytes, hipMemcpyHostToDevice, s) != hipSuccess) return SPEC_ERR_HIP;
    }
  }

  sv::AttnParams a{};
  if (attn) {
    a.q = attn->q;
    a.k = attn->k;
    a.v = attn->v;
    a.q_st = attn->q_stride_tok;
    a.q_sh = attn->q_stride_head;
    a.kv_st = attn->kv_stride_tok;
    a.kv_sh = attn->kv_stride_head;
    a.out = attn->out;
    a.part_o = reinterpret_cast<float*>(d + P.off_part_o);
    a.part_ml = reinterpret_cast<float2*>(d + P.off_part_ml);
    a.items = reinterpret_cast<const AttnItem*>(pl + P.off_items);
    a.reqs = reinterpret_cast<const ReqInfo*>(d + P.off_reqs);
    a.row_req = reinterpret_cast<const int32_t*>(d + P.off_rowreq);
    a.grid = (int32_t)P.grid;
    a.first_round = (int32_t)P.first_round;
    if (P.fused || P.grid > P.first_round) a.call_tag = next_call_tag();
    if (P.grid > P.first_round) a.claim = reinterpret_cast<unsigned long long*>(d + P.off_claim);
    if (P.fused) {
      a.counters = reinterpret_cast<unsigned long long*>(d + P.off_counters);
      a.fused = 1;
    } else if (P.parts > 0 && pl != d) {      // the combine kernel runs: mirror its table and map
      const bool mfma = attn->dtype == SPEC_BF16;
      const int64_t threads = mfma ? 64 * (int64_t)P.nr_max : 256;
      const int64_t n16 = (int64_t)(P.off_items / 16);
      a.mirror_src = reinterpret_cast<const uint4*>(pl);
      a.mirror_dst = reinterpret_cast<uint4*>(d);
      a.mirror_n16 = (int32_t)n16;
      a.mirror_wg = (int32_t)std::min<int64_t>((int64_t)P.items.size(), (n16 + threads - 1) / threads);
    }
    a.n_parts = (int32_t)P.parts;
    const float scale = attn->scale > 0.f ? attn->scale : 1.f / std::sqrt((float)attn->head_dim);
    a.scale_log2 = scale * 1.4426950408889634f;
    a.Hq = attn->num_q_heads;
    a.Hkv = attn->num_kv_heads;
    a.G = a.Hq / a.Hkv;
    a.D = attn->head_dim;
    a.n_items = (int32_t)P.items.size();
    a.Nq = (int32_t)P.Nq;
    a.bt = attn->block_table;
    a.bt_stride = attn->block_stride;
    a.page_tokens = attn->page_tokens;
    a.num_pages = attn->num_pages;
    a.page_bytes = (int64_t)attn->page_tokens * attn->kv_stride_tok * 2;
    a.pool_bytes = (int64_t)attn->num_pages * a.page_bytes;
    a.pool32 = attn->block_table && sv::paged_build(attn->num_pages, a.page_bytes) == 2 ? 1 : 0;
    std::memcpy(a.anc, P.topo.anc, sizeof(a.anc));
    a.nodes = reinterpret_cast<const sv::NodeInfo*>(pl + P.off_nodes);
    a.per_req = P.per_req ? 1 : 0;
  }
  sv::AccParams c{};
  if (acc) {
    c.logits = acc->target_logits;
    c.probs = acc->draft_probs ? acc->draft_probs : acc->target_logits;
    c.l_st = acc->logits_stride;
    c.p_st = acc->draft_probs ? acc->probs_stride : acc->logits_stride;
    c.tokens = acc->draft_tokens;
    c.uniforms = acc->uniforms;
    c.acc_len = acc->accepted_len;
    c.next_tok = acc->next_token;
    c.acc_node = acc->accepted_node;
    c.reqs_src = reinterpret_cast<const ReqInfo*>(pl + P.off_reqs);
    c.reqs = reinterpret_cast<ReqInfo*>(d + P.off_acc_reqs);
    c.topo = P.topo;
    c.rowstats = reinterpret_cast<sv::ChunkStat*>(d + P.off_rowstats);
    c.tickets = reinterpret_cast<int32_t*>(d + P.off_tickets);
    c.masses = reinterpret_cast<double*>(d + P.off_masses);
    c.V = acc->vocab;
    c.nch = P.nch;
    c.B = P.B;
    c.Nq = (int32_t)P.Nq;
    c.tree = P.tree ? (acc->tree_rule == SPEC_TREE_SEQUENTIAL ? 2 : 1) : 0;   // 2: sequential siblings
    c.bf16 = acc->dtype == SPEC_BF16;
    c.nodes_src = reinterpret_cast<const sv::NodeInfo*>(pl + P.off_nodes);
    c.nodes = reinterpret_cast<sv::NodeInfo*>(d + P.off_acc_nodes);
    c.per_req = P.per_req ? 1 : 0;
    c.nodes_n16 = (int32_t)((sizeof(sv::NodeInfo) * P.nodes.size() + 15) / 16);
    c.all_stats = (P.per_req || mode.lm) ? 1 : 0;
    // sequential sibling rule: work-groups per request, enough to give every
    // compute unit one, at most kSeqMaxGroups and at most the 1024-thread
    // chunks of the vocabulary
    {
      const int64_t ch = 1024 * (acc->dtype == SPEC_BF16 ? 8 : 4);
      const int64_t nchunk = (acc->vocab + ch - 1) / ch;
      int64_t g = device_cus() / std::max(P.B, 1);
      // SPEC_SEQ_GROUPS (1..8) replaces the choice (the tests use it to run
      // every split of the vocabulary)
      if (const char* e = std::getenv("SPEC_SEQ_GROUPS")) {
        const long v = std::strtol(e, nullptr, 10);
        if (v >= 1 && v <= sv::kSeqMaxGroups) g = v;
      }
      g = std::min<int64_t>(std::min<int64_t>(g, sv::kSeqMaxGroups), nchunk);
      c.seq_groups = (int32_t)std::max<int64_t>(g, 1);
      c.seq_slots = reinterpret_cast<sv::SeqSlot*>(d + P.off_seq);
    }
  }

  // Optional device check of the acceptance inputs (the caller's contract),
  // before anything that writes an output is enqueued.
  if (acc && debug_validate()) {
    uint32_t* dflag = reinterpret_cast<uint32_t*>(d + P.off_flag);
    uint32_t hflag = 0;
    if (sv::launch_accept_validate(c, dflag, s) != hipSuccess) return SPEC_ERR_HIP;
    if (hipMemcpyAsync(&hflag, dflag, sizeof(hflag), hipMemcpyDeviceToHost, s) != hipSuccess) return SPEC_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return SPEC_ERR_HIP;
    if (hflag != 0) return SPEC_ERR_INVALID_ARG;
  }

  if (mode.lm) {
    // the LM head, then the decision and final sample (folding the head's
    // tile statistics), all on the caller's stream
    const spec_lm_head_args_t* lm = mode.lm;
    sv::LmhParams g{};
    g.hidden = static_cast<const uint16_t*>(lm->hidden);
    g.weight = static_cast<const uint16_t*>(lm->weight);
    g.h_st = lm->hidden_stride;
    g.w_st = lm->weight_stride;
    g.out = const_cast<void*>(acc->target_logits);
    g.o_st = acc->logits_stride;
    g.tiles = reinterpret_cast<sv::ChunkStat*>(d + mode.off_tiles);
    g.M = (int32_t)P.Nq;
    g.K = lm->hidden_dim;
    g.V = acc->vocab;
    g.ntiles = (acc->vocab + sv::kLmhNT - 1) / sv::kLmhNT;
    const sv::LmhGeometry geo = sv::lmh_geometry(g.M, g.ntiles, device_cus());
    g.rb = geo.rb;
    g.tile_rows = geo.tile_rows;
    g.m_tiles = geo.m_tiles;
    g.out_bf16 = acc->dtype == SPEC_BF16;
    // The decision kernel folds the tile statistics itself, and the GEMM does
    // the row-statistics kernel's other duties; the sequential sibling rule
    // reads chunk statistics, which the fold kernel writes.
    const bool fold = c.tree == 2;
    if (!fold) {
      c.tiles = g.tiles;
      c.ntiles = g.ntiles;
      g.reqs_src = c.reqs_src;
      g.reqs = c.reqs;
      g.tickets = c.tickets;
      g.nodes_src = c.nodes_src;
      g.nodes = c.nodes;
      g.nodes_n16 = c.per_req ? c.nodes_n16 : 0;
      g.B = c.B;
    }
    if (lm->event_begin && hipEventRecord(static_cast<hipEvent_t>(lm->event_begin), s) != hipSuccess) return SPEC_ERR_HIP;
    if (sv::launch_lmh(g, s) != hipSuccess) return SPEC_ERR_HIP;
    if (lm->event_end && hipEventRecord(static_cast<hipEvent_t>(lm->event_end), s) != hipSuccess) return SPEC_ERR_HIP;
    if (acc->event_begin && hipEventRecord(static_cast<hipEvent_t>(acc->event_begin), s) != hipSuccess) return SPEC_ERR_HIP;
    if (fold && sv::launch_foldstats(c, g.tiles, g.ntiles, s) != hipSuccess) return SPEC_ERR_HIP;
    if (acc->event_mid && hipEventRecord(static_cast<hipEvent_t>(acc->event_mid), s) != hipSuccess) return SPEC_ERR_HIP;
    if (sv::launch_decide(c, s) != hipSuccess) return SPEC_ERR_HIP;
    if (acc->event_end && hipEventRecord(static_cast<hipEvent_t>(acc->event_end), s) != hipSuccess) return SPEC_ERR_HIP;
    return SPEC_OK;
  }

  auto launch_acc = [&](hipStream_t st) -> bool {
    if (acc->event_begin && hipEventRecord(static_cast<hipEvent_t>(acc->event_begin), st) != hipSuccess) return false;
    if (sv::launch_accept(c, st, static_cast<hipEvent_t>(acc->event_mid)) != hipSuccess) return false;
    if (acc->event_end && hipEventRecord(static_cast<hipEvent_t>(acc->event_end), st) != hipSuccess) return false;
    return true;
  };
  auto launch_attn = [&](hipStream_t st) -> bool {
    if (attn->event_begin && hipEventRecord(static_cast<hipEvent_t>(attn->event_begin), st) != hipSuccess)
      return false;
    if (sv::launch_attention(a, attn->dtype == SPEC_BF16, P.nr_max, st) != hipSuccess) return false;
    if (P.parts > 0 && !P.fused && sv::launch_combine(a, st) != hipSuccess) return false;
    if (attn->event_end && hipEventRecord(static_cast<hipEvent_t>(attn->event_end), st) != hipSuccess) return false;
    return true;
  };

#ifndef SV_OVERLAP
#define SV_OVERLAP 1
#endif
  if (SV_OVERLAP && mode.overlap && attn && acc) {
    SideStream* S = side_stream();
    if (!S) return SPEC_ERR_HIP;
    std::lock_guard<std::mutex> lk(S->mu);
    if (hipEventRecord(S->fork, s) != hipSuccess || hipStreamWaitEvent(S->s, S->fork, 0) != hipSuccess)
      return SPEC_ERR_HIP;
    if (!launch_acc(S->s)) return SPEC_ERR_HIP;
    if (hipEventRecord(S->join, S->s) != hipSuccess) return SPEC_ERR_HIP;
    const bool ok = launch_attn(s);
    // join even after a failed launch, so the caller's stream never runs ahead
    if (hipStreamWaitEvent(s, S->join, 0) != hipSuccess || !ok) return SPEC_ERR_HIP;
    return SPEC_OK;
  }
  if (attn && !launch_attn(s)) return SPEC_ERR_HIP;
  if (acc && !launch_acc(s)) return SPEC_ERR_HIP;
  return SPEC_OK;
}

}  // namespace

extern "C" {

spec_status_t spec_workspace_bytes(const spec_requests_t* req, const spec_attn_args_t* attn,
                                   const spec_accept_args_t* acc, size_t* device_bytes, size_t* host_bytes) {
  if (!device_bytes || !host_bytes) return SPEC_ERR_INVALID_ARG;
  Plan P;
  const spec_status_t st = build_plan(req, attn, acc, P);
  if (st != SPEC_OK) return st;
  *device_bytes = P.device_bytes;
  *host_bytes = P.plan_bytes;
  return SPEC_OK;
}

spec_status_t spec_verify_attn(const spec_requests_t* req, const spec_attn_args_t* attn, void* workspace,
                               size_t workspace_bytes, void* host_staging, size_t host_staging_bytes,
                               void* stream) {
  if (!attn) return SPEC_ERR_INVALID_ARG;
  return run(req, attn, nullptr, workspace, workspace_bytes, host_staging, host_staging_bytes, stream);
}

spec_status_t spec_accept(const spec_requests_t* req, const spec_accept_args_t* acc, void* workspace,
                          size_t workspace_bytes, void* host_staging, size_t host_staging_bytes, void* stream) {
  if (!acc) return SPEC_ERR_INVALID_ARG;
  return run(req, nullptr, acc, workspace, workspace_bytes, host_staging, host_staging_bytes, stream);
}

spec_status_t spec_verify(const spec_requests_t* req, const spec_attn_args_t* attn, const spec_accept_args_t* acc,
                          void* workspace, size_t workspace_bytes, void* host_staging, size_t host_staging_bytes,
                          void* stream) {
  if (!attn || !acc) return SPEC_ERR_INVALID_ARG;
  return run(req, attn, acc, workspace, workspace_bytes, host_staging, host_staging_bytes, stream);
}

// The no-allocation variant of spec_verify: the library's static device
// scratch as the workspace, its static host array as the staging, and no
// side stream.  Pageable host memory: hipMemcpyAsync has read the plan out
// of the array before it returns, and the mutex keeps two host threads from
// writing the array at once.
spec_status_t spec_verify_noalloc(const spec_requests_t* req, const spec_attn_args_t* attn,
                                  const spec_accept_args_t* acc, void* stream) {
  static char host_staging[sv::kNoAllocStagingBytes];
  static std::mutex staging_mu;
  if (!attn || !acc) return SPEC_ERR_INVALID_ARG;
  Plan P;
  const spec_status_t st = build_plan(req, attn, acc, P);   // argument checks before any HIP call
  if (st != SPEC_OK) return st;
  if (P.device_bytes > sv::kNoAllocScratchBytes || P.plan_bytes > sv::kNoAllocStagingBytes) return SPEC_ERR_WORKSPACE;
  void* scratch = nullptr;
  if (sv::noalloc_scratch(&scratch) != hipSuccess) return SPEC_ERR_HIP;
  RunMode mode;
  mode.overlap = false;
  mode.pageable = true;
  mode.staging_mu = &staging_mu;
  return run(req, attn, acc, scratch, sv::kNoAllocScratchBytes, host_staging, sizeof(host_staging), stream, mode);
}

spec_status_t spec_lm_head_workspace_bytes(const spec_requests_t* req, const spec_lm_head_args_t* lm,
                                           const spec_accept_args_t* acc, size_t* device_bytes, size_t* host_bytes) {
  if (!device_bytes || !host_bytes) return SPEC_ERR_INVALID_ARG;
  Plan P;
  size_t off = 0, dev = 0;
  const spec_status_t st = lm_plan(req, lm, acc, P, off, dev);
  if (st != SPEC_OK) return st;
  *device_bytes = dev;
  *host_bytes = P.plan_bytes;
  return SPEC_OK;
}

spec_status_t spec_lm_head_accept(const spec_requests_t* req, const spec_lm_head_args_t* lm,
                                  const spec_accept_args_t* acc, void* workspace, size_t workspace_bytes,
                                  void* host_staging, size_t host_staging_bytes, void* stream) {
  Plan P;
  size_t off = 0, dev = 0;
  const spec_status_t st = lm_plan(req, lm, acc, P, off, dev);
  if (st != SPEC_OK) return st;
  if (workspace_bytes < dev) return SPEC_ERR_WORKSPACE;
  RunMode mode;
  mode.overlap = false;
  mode.lm = lm;
  mode.off_tiles = off;
  return run(req, nullptr, acc, workspace, workspace_bytes, host_staging, host_staging_bytes, stream, mode);
}

const char* spec_status_str(spec_status_t status) {
  switch (status) {
    case SPEC_OK: return "ok";
    case SPEC_ERR_INVALID_ARG: return "invalid argument";
    case SPEC_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case SPEC_ERR_WORKSPACE: return "workspace or staging buffer too small or misaligned";
    case SPEC_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int32_t spec_abi_version(void) { return SPEC_ABI_VERSION; }

spec_status_t spec_stream_read_probe(const void* src, size_t bytes, uint32_t* out, int32_t blocks, void* stream) {
  if (!src || !out || bytes == 0 || bytes % 16 || !aligned16(src) || blocks < 1 || blocks > 65536)
    return SPEC_ERR_INVALID_ARG;
  return sv::launch_stream_read(src, bytes, out, blocks, static_cast<hipStream_t>(stream)) == hipSuccess
             ? SPEC_OK
             : SPEC_ERR_HIP;
}

// The floor probe's workspace: the stream's words [num_rows, chunks], the
// tickets [B], the published values [B, chunks].
static size_t floor_layout(int32_t V, int32_t num_rows, int32_t B, size_t* off_tickets, size_t* off_sums) {
  const int64_t nch = ((int64_t)V + 4095) / 4096;
  size_t off = align_up(sizeof(uint32_t) * (size_t)((int64_t)num_rows * nch));
  *off_tickets = off;
  off = align_up(off + sizeof(int32_t) * (size_t)B);
  *off_sums = off;
  return align_up(off + sizeof(uint64_t) * (size_t)((int64_t)B * nch));
}

size_t spec_accept_floor_probe_bytes(int32_t V, int32_t num_rows, int32_t B) {
  if (V < 1 || B < 1 || num_rows < B) return 0;
  size_t a, b;
  return floor_layout(V, num_rows, B, &a, &b);
}

spec_status_t spec_accept_floor_probe(const void* rows, int64_t row_stride, int32_t elem_bytes, int32_t V,
                                      int32_t num_rows, int32_t B, void* ws, size_t ws_bytes, uint32_t* out,
                                      void* stream) {
  if (!rows || !ws || !out || !aligned16(rows) || !aligned16(ws) || (elem_bytes != 2 && elem_bytes != 4) || V < 1 ||
      B < 1 || num_rows < B || row_stride < V || (row_stride * elem_bytes) % 16 != 0)
    return SPEC_ERR_INVALID_ARG;
  const int64_t nch = ((int64_t)V + 4095) / 4096;
  if ((int64_t)num_rows * nch > INT32_MAX) return SPEC_ERR_INVALID_ARG;
  size_t ot, os;
  if (ws_bytes < floor_layout(V, num_rows, B, &ot, &os)) return SPEC_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  return sv::launch_accept_floor(rows, row_stride * elem_bytes, (int64_t)V * elem_bytes, 4096 * (int64_t)elem_bytes,
                                 (int)nch, num_rows, B, reinterpret_cast<uint32_t*>(w),
                                 reinterpret_cast<int32_t*>(w + ot), reinterpret_cast<uint64_t*>(w + os), out,
                                 static_cast<hipStream_t>(stream)) == hipSuccess
             ? SPEC_OK
             : SPEC_ERR_HIP;
}

}  // extern "C"
