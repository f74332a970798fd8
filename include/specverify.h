/*
 * specverify.h -- C ABI of the MI355X (gfx950) batched speculative-decoding
 * verify step.
 *
 * One verify step serves the requests a speculative-decoding scheduler has
 * picked for this round (the LAPS-SD setting of arXiv 2505.17074, Sec. 3:
 * requests with a context, a draft of candidate tokens and a target model
 * that verifies all of them in one parallel forward, Sec. 2.2).  For each
 * request i with c_i cached KV positions and a draft of k_i tokens:
 *
 *   1. verify attention: the k_i + 1 verify queries (the last accepted token
 *      plus the drafts) -- or the nodes of a token tree -- attend over the
 *      request's cached keys and, inside the verify block, over their own
 *      ancestors-or-self (causal for a chain, tree-ancestor for a tree);
 *   2. acceptance: target softmax of each verify position, the acceptance
 *      test of Eq. (1) (draft j is accepted iff u_j * q_j(x_j) < p_j(x_j),
 *      i.e. u_j < min(1, p/q), with p the TARGET and q the DRAFT
 *      distribution), the resample from the residual max(0, p - q) at the
 *      first rejection (Sec. 2.2), or the target's one additional token when
 *      every draft is accepted (Sec. 4.3, the "+1" of Eq. (6));
 *   3. outputs: each request's accepted count a_i -- what the scheduler's
 *      acceptance-rate estimate consumes (Sec. 4.3) -- and its next token.
 *
 * The KV cache is either packed per request or paged through block tables
 * (spec_attn_args_t); token trees are verified by independent per-node
 * tests or by sequential sibling verification (spec_accept_args_t).  The
 * scheduler that consumes a_i has its own ABI in specsched.h.
 *
 * Conventions for every entry point
 *   - Device pointers point to memory on the current HIP device; host
 *     pointers are read during the call only.  The library keeps no pointer
 *     after it returns and allocates no device memory: the caller passes a
 *     device workspace and a pinned host staging buffer sized by
 *     spec_workspace_bytes().
 *   - `stream` is a hipStream_t (NULL = the null stream).  All device work
 *     is enqueued on it in order; nothing synchronises the device.  Outputs
 *     are valid once the stream has passed the call.
 *   - The host staging buffer is written by the call and read on `stream`:
 *     when it is pinned (hipHostMalloc), the call's kernels read the plan
 *     through its device mapping, with no copy ahead of them; otherwise an
 *     asynchronous copy brings it into the workspace.  Either way it must
 *     stay untouched until the stream has passed the call.  Calls in flight
 *     at the same time need separate workspaces and staging buffers.
 *   - All argument checks run on the host before any HIP call; on an error
 *     nothing is enqueued and no output is touched.  Device-resident values
 *     (draft token ids in [0, V), uniforms in [0, 1), a positive draft
 *     probability at each draft token, finite logits) are the caller's
 *     contract.  They are not checked unless the environment variable
 *     SPEC_DEBUG_VALIDATE is set to a non-empty value other than "0": then
 *     spec_accept and spec_verify first check the first three on the device,
 *     wait for `stream`, and return SPEC_ERR_INVALID_ARG if any fails (the
 *     check is then the only work enqueued, and no output is touched).  Without the check an out-of-range token id is
 *     clamped into [0, V): its results are meaningless, but nothing outside
 *     the arguments is read.
 *   - The device workspace needs no initialisation and may hold anything
 *     between calls: every byte a call reads is written earlier in the same
 *     call, except the split-KV arrival counters and the attention's item
 *     claim word, which carry a tag that is new on every call and start over
 *     when it does not match.
 *   - When the bf16 verify attention has more work items than the device
 *     holds work-groups at once, the work-groups past that first round claim
 *     the next item at run time (the outputs do not depend on which
 *     work-group runs an item).  The environment variables
 *     SPEC_ATTN_FIRST_ROUND (a work-group count >= 1) and SPEC_ATTN_EXTRA_WG
 *     (surplus work-groups >= 0) override the first round and the surplus;
 *     they exist for tests.
 *   - When the verify attention cuts a request's KV range into pieces, the
 *     last piece of each (request, KV head, head group) to finish combines
 *     the pieces' partial outputs (bf16 inputs, partial blocks up to 64 KB
 *     per stream); otherwise a separate combine kernel follows.  The
 *     environment variable SPEC_FUSED_COMBINE_MAX_BYTES (a byte count)
 *     replaces the 64 KB limit; the outputs agree either way within the
 *     attention tolerance, and each choice is deterministic.
 *   - Results are deterministic: the same inputs give bit-identical outputs
 *     (fixed reduction orders, no floating-point atomics).
 *   - A call captured into a HIP graph may be replayed any number of times,
 *     also with other calls on the same workspace in between: the tagged
 *     words are left by each call ready for its own tag again.  A replay
 *     reads the plan staged at capture, so the staging buffer must keep it
 *     (for spec_verify_noalloc, whose staging is one static array, no other
 *     spec_verify_noalloc call with different requests may run between the
 *     capture and a replay).
 */
#ifndef SPECVERIFY_H
#define SPECVERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define SPEC_API __attribute__((visibility("default")))
#else
#define SPEC_API
#endif

#define SPEC_ABI_VERSION 5
#define SPEC_MAX_DRAFT 16        /* chain drafts per request */
#define SPEC_MAX_TREE_NODES 32   /* token-tree nodes per request, root included */

typedef enum spec_status {
  SPEC_OK = 0,
  SPEC_ERR_INVALID_ARG = 1,   /* a null pointer, size, stride or tree that breaks the contract */
  SPEC_ERR_UNSUPPORTED = 2,   /* valid but not built: head_dim not 64/128, a dtype/shape combination */
  SPEC_ERR_WORKSPACE = 3,     /* workspace or staging too small or misaligned */
  SPEC_ERR_HIP = 4            /* a HIP runtime call failed (launch, copy) */
} spec_status_t;

typedef enum spec_tree_rule {
  SPEC_TREE_INDEPENDENT = 0,
  SPEC_TREE_SEQUENTIAL = 1
} spec_tree_rule_t;

typedef enum spec_dtype {
  SPEC_F32 = 0,
  SPEC_BF16 = 1
} spec_dtype_t;

/*
 * The requests of one step (host memory).
 *   num_requests  B >= 1.
 *   ctx_len[B]    c_i >= 0: KV positions cached before the verify block.
 *   draft_len[B]  chain mode: k_i in [0, SPEC_MAX_DRAFT] drafts (k_i = 0 is
 *                 plain decoding: no test, one sample from the target).
 *                 Ignored (may be NULL) in tree mode.
 *   tree_nodes    0 = no shared tree.  Otherwise every request verifies the
 *                 same token-tree topology of tree_nodes nodes (1 ..
 *                 SPEC_MAX_TREE_NODES), node 0 being the last accepted token.
 *   tree_parent   [tree_nodes], BFS order: parent[0] = -1, 0 <= parent[n] < n.
 *   node_count    NULL, or per-request token trees (tree_nodes must then be
 *                 0; draft_len is ignored): request i verifies its own tree
 *                 of node_count[i] nodes (1 .. SPEC_MAX_TREE_NODES), the
 *                 SpecInfer setup of one speculated tree per request.
 *   tree_parents  [sum node_count] with node_count: request i's BFS parent
 *                 array at tree_parents[o_i .. o_i + node_count[i]), o_i the
 *                 running sum of node_count over requests < i; each array as
 *                 tree_parent above.
 *
 * Derived counts: n_i = k_i + 1 (chain), tree_nodes (shared tree) or
 * node_count[i] verify positions; Nq = sum n_i;  Nkv = sum (c_i + n_i);
 * Nd = sum of the number of nodes that have children (k_i for a chain).
 * Request i's rows of every packed array start at the running sum of the
 * matching count over requests < i.
 */
typedef struct spec_requests {
  int32_t num_requests;
  const int32_t* ctx_len;
  const int32_t* draft_len;
  int32_t tree_nodes;
  const int32_t* tree_parent;
  const int32_t* node_count;
  const int32_t* tree_parents;
} spec_requests_t;

/*
 * Verify attention (device memory).
 *   q     [Nq, Hq, d]  request i's verify positions (node order), strides
 *         q_stride_tok / q_stride_head in elements, last dim contiguous.
 *   k, v  [Nkv, Hkv, d] request i's c_i cached rows followed by its n_i
 *         verify rows (already appended by the caller); shared strides
 *         kv_stride_tok / kv_stride_head in elements, last dim contiguous.
 *   out   [Nq, Hq, d] float32, contiguous.
 *   Query head h reads KV head h / (Hq / Hkv).  scale <= 0 selects
 *   1/sqrt(d).  dtype SPEC_BF16 (MFMA path) or SPEC_F32; d in {64, 128}.
 *   split_kv 0 = automatic split of long contexts; otherwise the number of
 *   KV positions per split (a positive multiple of 32) -- results agree
 *   across splits within fp32 rounding.  Requests split more than once are
 *   merged by a second (combine) kernel.
 *
 * Paged KV cache (block_table != NULL; the PagedAttention layout the paper
 * cites as serving practice, Sec. 6.2): k and v are page pools
 * [num_pages, page_tokens, Hkv, d], kv_stride_tok / kv_stride_head their
 * strides inside a page (a page spans page_tokens * kv_stride_tok elements).
 * block_table (device, int32) holds request i's page ids at
 * block_table[i * block_stride + j] for its logical pages
 * j = 0 .. ceil((c_i + n_i) / page_tokens) - 1: logical KV row t of request
 * i is row t % page_tokens of page block_table[i * block_stride +
 * t / page_tokens], its verify rows last as in the packed layout.
 * page_tokens is a positive multiple of 32; block_stride must hold every
 * request's pages; bf16 only (SPEC_ERR_UNSUPPORTED for f32).  Page ids in
 * [0, num_pages) are the caller's contract: an id outside is clamped into
 * the pool, so nothing outside it is read, but its rows are meaningless.
 * With the same rows the paged and packed layouts give bit-identical
 * outputs.
 */
typedef struct spec_attn_args {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  spec_dtype_t dtype;
  float scale;
  const void* q;
  int64_t q_stride_tok;
  int64_t q_stride_head;
  const void* k;
  const void* v;
  int64_t kv_stride_tok;
  int64_t kv_stride_head;
  float* out;
  int32_t split_kv;
  /* Optional profiling: hipEvent_t handles recorded on `stream` right before
   * the split-KV attention kernel and right after the last attention kernel
   * (the split combine when some request is split, else the split-KV kernel
   * itself) (NULL = not recorded). */
  void* event_begin;
  void* event_end;
  /* Paged KV cache (above); block_table NULL = the packed layout. */
  const int32_t* block_table;
  int32_t block_stride;
  int32_t page_tokens;
  int32_t num_pages;
  int32_t pad0;
} spec_attn_args_t;

/*
 * Acceptance and final sample (device memory).
 *   target_logits [Nq, V]  row r = verify position r; row stride
 *                 logits_stride elements (>= V).
 *   draft_probs   [Nd, V]  the draft distribution of each node that has
 *                 children, used as stored (not renormalised); row stride
 *                 probs_stride.  Same dtype as target_logits.
 *   draft_tokens  [Nq - B] int32, one per non-root node: request i's are at
 *                 q0_i - i .. q0_i - i + n_i - 2 (node n at offset n - 1).
 *   uniforms      [Nq] float32 in [0, 1): request i's node n >= 1 is tested
 *                 with uniforms[q0_i + n - 1]; uniforms[q0_i + n_i - 1]
 *                 drives the final sample.
 *   accepted_len  [B] out: accepted drafts a_i (tree: depth of the deepest
 *                 accepted node).
 *   next_token    [B] out: the token sampled after the accepted prefix.
 *   accepted_node [B] out (may be NULL): the deepest accepted node (chain:
 *                 equals accepted_len).
 * Tree rules (tree_rule; ignored for chains):
 *   SPEC_TREE_INDEPENDENT (0): node n is accepted iff its parent is and its
 *     own test passes against the parent's target and draft rows; the
 *     deepest accepted node wins, the smallest BFS index on ties; the final
 *     token is drawn from that node's target row if it is a leaf, else from
 *     the residual.
 *   SPEC_TREE_SEQUENTIAL (1): SpecInfer's sequential sibling verification
 *     (multi-step speculative sampling; the token-tree system the paper's
 *     evaluation follows, Sec. 5.1), which emits tokens distributed exactly
 *     as the target when each node's children are drafted i.i.d. from its
 *     draft row.  From the root, the current node's children are tested in
 *     BFS order against a running distribution p' (first the node's target
 *     row): child c is accepted iff u_c * q(x_c) < p'(x_c); a rejection
 *     replaces p' by max(0, p' - q) normalised (unchanged if that has zero
 *     mass).  The first accepted child becomes the current node; when none
 *     is, or the node is a leaf, the final token is drawn from p'.
 *     accepted_node is the last current node, accepted_len its depth.
 *     Each request's walk runs on up to 8 work-groups that split the
 *     vocabulary (one per compute unit when there are few requests); the
 *     environment variable SPEC_SEQ_GROUPS (1..8) fixes that number.  Their
 *     waits on each other are bounded: a request whose wait gives up (not
 *     expected in any normal run) gets -1 in all three outputs.
 * Inverse-CDF convention: token ids ascending, the smallest id whose
 * cumulative weight exceeds u * (total weight); zero weights never chosen.
 */
typedef struct spec_accept_args {
  int32_t vocab;
  spec_dtype_t dtype;
  const void* target_logits;
  int64_t logits_stride;
  const void* draft_probs;
  int64_t probs_stride;
  const int32_t* draft_tokens;
  const float* uniforms;
  int32_t* accepted_len;
  int32_t* next_token;
  int32_t* accepted_node;
  /* Optional profiling: hipEvent_t handles recorded on the stream the
   * acceptance kernels run on, right before the first, right after the last,
   * and between the row-statistics kernel and the decision kernel
   * (NULL = none). */
  void* event_begin;
  void* event_end;
  void* event_mid;
  int32_t tree_rule;   /* SPEC_TREE_INDEPENDENT (0) or SPEC_TREE_SEQUENTIAL (1) */
  int32_t pad0;
} spec_accept_args_t;

/*
 * The target model's LM head (device memory): the verify positions' logits
 * logits = hidden . weight^T, the forward that produces the target
 * distributions the acceptance test of Eq. (1) compares with the draft's
 * (Sec. 2.2).
 *   hidden  [Nq, hidden_dim] bf16: the final hidden state of each verify
 *           position (row r = verify position r), row stride hidden_stride
 *           elements.
 *   weight  [vocab, hidden_dim] bf16: the LM head's weight, one row per
 *           vocabulary entry, row stride weight_stride elements.
 *   hidden_dim a positive multiple of 32; strides >= hidden_dim and
 *   multiples of 8; both pointers 16-byte aligned.  The products accumulate
 *   in fp32 (bf16 x bf16 products are exact in fp32).
 *   event_begin / event_end: optional hipEvent_t recorded on `stream` right
 *   before and right after the GEMM kernel (NULL = none).
 */
typedef struct spec_lm_head_args {
  int32_t hidden_dim;
  int32_t pad0;
  const void* hidden;
  int64_t hidden_stride;
  const void* weight;
  int64_t weight_stride;
  void* event_begin;
  void* event_end;
} spec_lm_head_args_t;

/* Workspace sizes for a call with these arguments (either args pointer may
 * be NULL when that part is not run).  The device workspace must be
 * 256-byte aligned; the host staging buffer should be pinned
 * (hipHostMalloc), so that the kernels read the plan where it was staged. */
SPEC_API spec_status_t spec_workspace_bytes(const spec_requests_t* req,
                                   const spec_attn_args_t* attn,
                                   const spec_accept_args_t* acc,
                                   size_t* device_bytes,
                                   size_t* host_bytes);

/* Step 1 alone: verify attention into attn->out. */
SPEC_API spec_status_t spec_verify_attn(const spec_requests_t* req,
                               const spec_attn_args_t* attn,
                               void* workspace, size_t workspace_bytes,
                               void* host_staging, size_t host_staging_bytes,
                               void* stream);

/* Steps 2-3 alone: acceptance and the final sample. */
SPEC_API spec_status_t spec_accept(const spec_requests_t* req,
                          const spec_accept_args_t* acc,
                          void* workspace, size_t workspace_bytes,
                          void* host_staging, size_t host_staging_bytes,
                          void* stream);

/* The whole verify step with one staged plan.  The logits are inputs, so the
 * two parts are independent: the acceptance kernels run on a library-owned
 * side stream (one per device, created on first use at the default priority)
 * that forks from `stream` at the start of the call and is joined back into `stream`
 * before the call returns, overlapping the attention kernels.  Completion is
 * still ordered by `stream` alone. */
SPEC_API spec_status_t spec_verify(const spec_requests_t* req,
                          const spec_attn_args_t* attn,
                          const spec_accept_args_t* acc,
                          void* workspace, size_t workspace_bytes,
                          void* host_staging, size_t host_staging_bytes,
                          void* stream);

/*
 * The whole verify step without any allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, outputs and kernels as
 * spec_verify, but no workspace or staging arguments: the library uses
 *   - a static device array of SPEC_NOALLOC_SCRATCH_BYTES in its own code
 *     object (each GPU it runs on holds one until the process ends) as the
 *     device workspace, and
 *   - a static host array of SPEC_NOALLOC_STAGING_BYTES for the plan, copied
 *     into that scratch with hipMemcpyAsync on `stream` (pageable memory:
 *     the copy has read the plan when the call returns),
 * and runs both parts on `stream` one after the other (no side stream).
 * The call makes no hipMalloc, hipFree, stream or event creation.
 * SPEC_ERR_WORKSPACE when the step needs more scratch or staging than that
 * (spec_workspace_bytes gives both sizes).  Every call on a GPU shares that
 * GPU's scratch, which keeps the last call's contents: calls that overlap on
 * one GPU (two streams, or two host threads without ordering between their
 * streams) race and must not be made; calls ordered on one stream are safe.
 */
#define SPEC_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
#define SPEC_NOALLOC_STAGING_BYTES ((size_t)1 << 20)
SPEC_API spec_status_t spec_verify_noalloc(const spec_requests_t* req,
                                           const spec_attn_args_t* attn,
                                           const spec_accept_args_t* acc,
                                           void* stream);

/* The LM head fused with acceptance and the final sample: the GEMM writes
 * the logits once into acc->target_logits (an OUTPUT here: [Nq, vocab] in
 * acc->dtype, fp32 or rounded to bf16, row stride acc->logits_stride) and,
 * in its epilogue, the maximum and the sum of exp(l - max) of every
 * (row, 256-entry tile) of the stored logits; the acceptance then folds those
 * into its normalisers instead of streaming the logits again, and reads the
 * logits only for its tests and the final sample.  Results equal spec_accept
 * on the same logits except where u * S lies within rounding of a boundary
 * (both are exact up to fp32 rounding of the normalisers).  Everything runs
 * on `stream`.  Workspace sizes from spec_lm_head_workspace_bytes. */
SPEC_API spec_status_t spec_lm_head_accept(const spec_requests_t* req,
                                           const spec_lm_head_args_t* lm,
                                           const spec_accept_args_t* acc,
                                           void* workspace, size_t workspace_bytes,
                                           void* host_staging, size_t host_staging_bytes,
                                           void* stream);

/* Workspace sizes for spec_lm_head_accept (as spec_workspace_bytes). */
SPEC_API spec_status_t spec_lm_head_workspace_bytes(const spec_requests_t* req,
                                                    const spec_lm_head_args_t* lm,
                                                    const spec_accept_args_t* acc,
                                                    size_t* device_bytes,
                                                    size_t* host_bytes);

/* Static text for a status code. */
SPEC_API const char* spec_status_str(spec_status_t status);

/* SPEC_ABI_VERSION of the built library. */
SPEC_API int32_t spec_abi_version(void);

/* Diagnostics: the device's plain streaming read rate, reported beside the
 * vendor HBM peak.  Reads `bytes` bytes at `src` (device memory, 16-byte
 * aligned, `bytes` a multiple of 16) once, with coalesced 16-byte loads from
 * `blocks` work-groups of 256 threads, and writes one word per work-group to
 * `out` [blocks] (device memory; the words only keep the loads live).
 * Enqueued on `stream`; the caller times it.  SPEC_ERR_INVALID_ARG for a
 * null pointer, a misaligned `src` or size, or blocks outside [1, 65536]. */
SPEC_API spec_status_t spec_stream_read_probe(const void* src, size_t bytes, uint32_t* out, int32_t blocks,
                                              void* stream);

/* Diagnostics: a floor for the acceptance kernels (spec_accept), reported
 * beside their time.  Two kernels with the acceptance's memory traffic and
 * its chain of dependent round trips (Eq. (1)'s tests need the rows'
 * normalisers, the residual or extra-token sample of Sec. 2.2 and Sec. 4.3
 * needs every chunk's mass, then the chosen chunk's entries) and none of its
 * arithmetic: the first reads every entry of `num_rows` rows of V entries
 * (elem_bytes 4 or 2, row stride `row_stride` elements) once in 4096-entry
 * chunks of whole 16-byte units (a row's last bytes past its last whole unit
 * are not read); the second, per request (B <= num_rows, request i owning rows
 * [i r, (i + 1) r), r = num_rows / B) and chunk, loads a word of the
 * first's output, a word chosen by it, a chunk of a row chosen by that,
 * publishes a value and takes a ticket, and the request's last work-group
 * loads the published values and a chunk chosen by them, and writes one
 * word to `out` [B] (device memory; the words only keep the loads live).
 * `rows` (device memory, 16-byte aligned, row stride a multiple of 16 bytes)
 * is only read; `ws` is device memory of spec_accept_floor_probe_bytes()
 * bytes, needing no initialisation.  Enqueued on `stream`; the caller times
 * it.
 * SPEC_ERR_INVALID_ARG for a null or misaligned pointer or a bad size,
 * SPEC_ERR_WORKSPACE for a short workspace. */
SPEC_API size_t spec_accept_floor_probe_bytes(int32_t V, int32_t num_rows, int32_t B);
SPEC_API spec_status_t spec_accept_floor_probe(const void* rows, int64_t row_stride, int32_t elem_bytes, int32_t V,
                                               int32_t num_rows, int32_t B, void* ws, size_t ws_bytes, uint32_t* out,
                                               void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SPECVERIFY_H */
