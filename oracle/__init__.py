"""CPU oracle of the batched speculative-decoding verify step (fp64, NumPy).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the CPU-baseline leg of the benchmark may import anything under ``oracle/``;
the product path (the C-ABI library and its Python binding) never does, and
the two share no code: no kernels, headers, helpers, tables or pre/post
processing.  The only thing both sides consume is the seeded input arrays
produced by ``paper_2505_17074_amd.workload``, which this package does not
import either: every function here takes plain arrays.

What it computes (each function cites the passage it follows):

* ``attention.verify_attention`` -- the k+1 (or tree-node) verify queries of
  each request attend over that request's cached keys plus the verify block
  under a causal or tree-ancestor mask (Sec. 2.1 KV cache; Sec. 2.2 parallel
  verification of all candidate tokens in one LLM forward).
* ``accept.accept_chain`` / ``accept.accept_tree`` / ``accept.verify_accept``
  -- the acceptance rule of Eq. (1), the resample from the residual
  distribution on rejection (Sec. 2.2), and the one extra LLM token when every
  candidate is accepted (Sec. 4.3, the "+1" of Eq. (6)).

* ``lm_head.lm_head_logits`` -- the target model's LM head over the verify
  positions' final hidden states (the forward of Sec. 2.2 whose output is
  the target distributions of Eq. (1)).

* ``scheduler.simulate`` -- the LAPS-SD request scheduler of Algorithm 1
  (Sec. 4: priority queues with exponential thresholds, demotion by attained
  service, the acceptance-rate stability test, the Eq. (6) estimate, and
  perceptible-SJF / non-perceptible-FCFS inside a queue) and the FCFS, LAS
  and predicted-length SJF baselines, round by round on integer microsecond
  times.

Everything is computed in float64 from the stored input values (bf16 and fp32
widen to fp64 exactly).  Both parts are exact results with a plain definition,
so the oracle is that definition written out, not an approximation.
"""
from .attention import verify_attention, ancestors_or_self, widen  # noqa: F401
from .lm_head import lm_head_logits  # noqa: F401
from .accept import (accept_chain, accept_tree, accept_tree_sequential, verify_accept, softmax64,  # noqa: F401
                     inverse_cdf, NEAR_TIE, NEAR_TIE_MASS)
