"""MI355X-native batched speculative-decoding verification.

The verify step that sits under a speculative-decoding request scheduler
(LAPS-SD, arXiv 2505.17074): verify attention of each request's k+1 (or
tree-node) queries over its ragged KV cache, then the fused target softmax,
acceptance test (Eq. (1)), residual / extra-token sample and per-request
accepted count.  Every step runs in the HIP kernels of ``libspecverify.so``;
this package only marshals arguments (``binding``), builds packed device
batches (``batch``) and draws seeded synthetic inputs (``workload``).
"""
__all__ = ["workload", "binding", "batch"]
