"""Pins of the LM-head oracle: brute force, a library routine, closed forms."""
import math

import numpy as np
import torch

from oracle import lm_head_logits
from paper_2505_17074_amd import workload as W

RNG = np.random.default_rng(55)


def _bf16(shape, scale=1.0):
    return W.to_bf16_bits((RNG.standard_normal(shape) * scale).astype(np.float32))


def test_brute_force_loops():
    h, w = _bf16((3, 5)), _bf16((4, 5))
    hf, wf = W.bf16_bits_to_f32(h), W.bf16_bits_to_f32(w)
    ref = [[math.fsum(float(hf[r, k]) * float(wf[v, k]) for k in range(5)) for v in range(4)] for r in range(3)]
    np.testing.assert_allclose(lm_head_logits(h, w), np.array(ref), rtol=1e-15, atol=1e-15)


def test_matches_torch_fp64_matmul():
    h, w = _bf16((7, 64)), _bf16((33, 64), 0.25)
    ref = torch.from_numpy(W.bf16_bits_to_f32(h).astype(np.float64)) @ \
        torch.from_numpy(W.bf16_bits_to_f32(w).astype(np.float64)).T
    np.testing.assert_allclose(lm_head_logits(h, w), ref.numpy(), rtol=1e-14, atol=1e-14)


def test_one_hot_hidden_selects_a_weight_column():
    w = _bf16((10, 16))
    h = np.zeros((16, 16), np.float32)
    h[np.arange(16), np.arange(16)] = 1.0
    out = lm_head_logits(W.to_bf16_bits(h), w)
    np.testing.assert_array_equal(out, W.bf16_bits_to_f32(w).astype(np.float64).T)


def test_linear_in_hidden_and_weight():
    h1, h2, w = _bf16((4, 32)), _bf16((4, 32)), _bf16((9, 32))
    s = W.to_bf16_bits(W.bf16_bits_to_f32(h1) * 2)          # exact in bf16
    np.testing.assert_array_equal(lm_head_logits(s, w), 2 * lm_head_logits(h1, w))
    both = lm_head_logits(np.concatenate([h1, h2]), w)
    np.testing.assert_array_equal(both[:4], lm_head_logits(h1, w))
    np.testing.assert_array_equal(both[4:], lm_head_logits(h2, w))
