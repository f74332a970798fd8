"""fp64 oracle of the target model's LM head (test infrastructure; see the
package header).

The verify step's target distributions come from one forward of the target
model over every verify position (Sec. 2.2); the last layer of that forward
is the LM head, a linear map of each position's final hidden state to one
logit per vocabulary entry:

    logits[r, v] = sum_k hidden[r, k] * weight[v, k]

with `weight` in the linear layer's layout, one row per vocabulary entry.
The inputs are stored in bf16 (raw uint16 bit patterns), widened exactly to
fp64, and the sum is taken in fp64.  The acceptance oracle then takes these
(or the GPU's stored) logits as its target logits.
"""
from __future__ import annotations

import numpy as np

from .attention import widen


def lm_head_logits(hidden: np.ndarray, weight: np.ndarray, dtype: str = "bf16") -> np.ndarray:
    """fp64 [rows, vocab] = widen(hidden) @ widen(weight)^T."""
    H = widen(hidden, dtype)
    Wt = widen(weight, dtype)
    if H.shape[1] != Wt.shape[1]:
        raise ValueError("hidden and weight must share the hidden dimension")
    return H @ Wt.T
