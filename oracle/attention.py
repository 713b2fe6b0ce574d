"""Exact and candidate-restricted softmax attention in float64.

Paper: Sec. "Background and Problem Formulation", Eq. full_attention
(alpha_i = softmax_i <k_i, q>, o = sum_i alpha_i v_i) and Eqs. approx_weight /
approx_output (the same softmax restricted to a candidate set C(q)).  The
paper writes the raw score <k_i, q>; the optional ``scale`` multiplies every
score (1 reproduces the paper's formula, 1/sqrt(D) the usual model scaling).
Index -1 marks an empty slot and is ignored.
"""

import numpy as np


def _softmax_weighted_sum(scores, V):
    mx = np.max(scores)
    e = np.exp(scores - mx)
    return (e[:, None] * V).sum(axis=0) / e.sum()


def full_attention(q, K, V, scale=1.0):
    """Eq. full_attention over all n keys."""
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    s = scale * (K @ np.asarray(q, dtype=np.float64))
    return _softmax_weighted_sum(s, V)


def sparse_attention(q, K, V, idx, scale=1.0):
    """Eqs. approx_weight / approx_output over the keys listed in idx."""
    idx = np.asarray(idx, dtype=np.int64)
    idx = idx[idx >= 0]
    D = np.asarray(V).shape[1]
    if idx.shape[0] == 0:
        return np.zeros(D)
    K = np.asarray(K, dtype=np.float64)[idx]
    V = np.asarray(V, dtype=np.float64)[idx]
    s = scale * (K @ np.asarray(q, dtype=np.float64))
    return _softmax_weighted_sum(s, V)
