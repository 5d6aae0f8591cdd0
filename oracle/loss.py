"""Per-half losses L+ and L- (oracle side).

Algorithm 2 evaluates the model's loss under each perturbation.  The paper's tasks
use prompt-based losses on labelled data; with synthetic inputs the build's reading
is (a) next-token cross-entropy, the mean over the B (S - 1) shifted positions of
-log softmax(logits_p)[token_{p+1}], for the decoder models, and (b) for a single
adapted layer, the mean squared error against a fixed target.  Both are summed in
float64 here.

Pins (tests/test_oracle_core.py): uniform logits give exactly ln V; the loss of a
one-hot-dominant row tends to 0; L+(Z) = L-(-Z) through the linear layer; MSE of
the target itself is 0.
"""
from __future__ import annotations

import numpy as np


def next_token_ce(logits: np.ndarray, tokens: np.ndarray) -> float:
    """Mean next-token cross entropy.  logits [B][S][V] (position p predicts token p+1)."""
    lg = np.asarray(logits, dtype=np.float64)
    b, s, v = lg.shape
    pred = lg[:, :-1, :].reshape(-1, v)
    tgt = np.asarray(tokens, dtype=np.int64)[:, 1:].reshape(-1)
    mx = pred.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(pred - mx).sum(axis=1))
    return float(np.mean(lse - pred[np.arange(pred.shape[0]), tgt]))


def mse(y: np.ndarray, target: np.ndarray) -> float:
    """Mean of (y - target)^2 over all elements."""
    d = np.asarray(y, dtype=np.float64) - np.asarray(target, dtype=np.float64)
    return float(np.mean(d * d))
