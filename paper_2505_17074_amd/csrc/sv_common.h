// Request and node tables shared by the host planner and every gfx950 kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sv {

constexpr int kMaxNodes = 32;          // verify positions per request (chain k+1 or tree)

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
static_assert(sizeof(ReqInfo) == 32, "ReqInfo is copied as two 16-byte units");

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

}  // namespace sv
