"""Squared loss of the paper on the fp64 oracle -- test infrastructure only.

Section 3, "Training", Eq. (14): E = (y* - y)^2 with y* the target and y the
network's output.  Reading where the paper is brief: y is the per-voxel
softmax output of the final linear layer, y* the one-hot label, the squares
are summed over the classes and averaged over all voxels of the batch (as the
cross-entropy is).  Gradients by the chain rule, in plain numpy:
    d  = dE/dp = 2 (p - y*) / M
    dz = p * (d - sum_k p_k d_k)          (through the softmax)
    dW = dz^T x,  db = sum_v dz,  dx = dz W
"""
from __future__ import annotations

import numpy as np


def softmax_sq(x2, w, b, labels=None, grad=False):
    """Final linear layer + per-row softmax; mean (over rows) of the squared
    error against the one-hot labels when labels are given."""
    x2 = np.asarray(x2, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    M = x2.shape[0]
    K = w.shape[0]
    z = x2 @ w.T + b
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    p = e / e.sum(axis=1, keepdims=True)
    out = {"p": p, "loss": None}
    if labels is None:
        return out
    lab = np.asarray(labels).reshape(M)
    assert lab.min() >= 0 and lab.max() < K
    y = np.zeros((M, K))
    y[np.arange(M), lab] = 1.0
    out["loss"] = float(((p - y) ** 2).sum() / M)
    if grad:
        d = 2.0 * (p - y) / M
        dz = p * (d - (p * d).sum(axis=1, keepdims=True))
        out.update({"dx": dz @ w, "dw": dz.T @ x2, "db": dz.sum(axis=0)})
    return out
