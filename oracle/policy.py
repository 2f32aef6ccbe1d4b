"""fp64 CPU oracle of the block-size policy (run once per prompt after prefill).

TEST INFRASTRUCTURE ONLY: the test suite is the only caller.

Sec. 2.3-2.4 and Eq. 9: the predictive distribution of the prompt's last token,
p = softmax(z), is the input of an MLP (two hidden layers of width 2048 by default,
Sec. 3.1) whose outputs score the candidates {B-k, ..., B+k}; the block size is the
argmax.  Readings: the hidden activation is ReLU (the paper does not name one); the
input is the plain softmax of the logits (the paper's "raw" distribution, with no
further normalisation); ties go to the smallest candidate.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def _f64(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu").to(torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float64)


@dataclass
class PolicyResult:
    scores: np.ndarray       # [P, 2k+1]
    block_size: np.ndarray   # [P]
    margin: np.ndarray       # [P] best score minus the runner-up


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """p_i = exp(z_i - max z) / sum_j exp(z_j - max z), per row."""
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def block_size_policy(logits, w1, b1, w2, b2, w3, b3, base_block, radius) -> PolicyResult:
    p = softmax_rows(_f64(logits))
    h1 = np.maximum(p @ _f64(w1).T + _f64(b1), 0.0)
    h2 = np.maximum(h1 @ _f64(w2).T + _f64(b2), 0.0)
    o = h2 @ _f64(w3).T + _f64(b3)
    best = np.argmax(o, axis=1)  # first maximum: the smallest candidate on ties
    srt = np.sort(o, axis=1)
    margin = srt[:, -1] - srt[:, -2] if o.shape[1] > 1 else np.full(o.shape[0], np.inf)
    return PolicyResult(o, (base_block - radius + best).astype(np.int32), margin)
