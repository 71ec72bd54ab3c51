"""Exact softmax attention (float64).

Every configuration in the paper's Section 2.1 ends its decode step in ordinary
attention over the keys and values its cache keeps: quantization changes the
values (KVQuant), eviction changes the set (H2O), sparse attention picks a
subset (RocketKV).  This module is that final step written out.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def softmax_attention(q, k, v):
    """Attention of query rows over keys/values, float64.

    q [G][d], k [n][d], v [n][d]  ->  (out [G][d], probs [G][n])

    probs[g, j] = exp(q_g . k_j / sqrt(d)) / sum_j' exp(q_g . k_j' / sqrt(d)),
    out[g] = sum_j probs[g, j] v_j.  The row maximum is subtracted before the
    exponential, which leaves the quotient unchanged.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    d = q.shape[-1]
    s = (q @ k.T) / np.sqrt(d)
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=-1, keepdims=True)
    return p @ v, p


def value_rms(v):
    """Root-mean-square of the effective value rows attended over (the error normaliser)."""
    v = np.asarray(v, np.float64)
    return float(np.sqrt(np.mean(v * v))) if v.size else 1.0
