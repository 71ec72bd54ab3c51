"""Hybrid sparse attention, the decode stage of RocketKV.

Section 2.1 (RocketKV paragraph): during each decode step, attention runs over
only a subset of the earlier tokens.  Readings used where the paper is silent:
  * per (sequence, kv head) and step, channel magnitudes a_c = sum_g |q_gc|
    over the kv head's query heads pick the n_c = 32 largest channels (lower
    channel index on equal magnitudes), taken in ascending channel order;
  * the approximate score of every retained token j is
    shat_j = sum_{c in C} qbar_c * k_jc with qbar_c = sum_g q_gc;
  * the top min(k, n) tokens by shat are selected (lower position on equal
    scores), with k = T / 2 by default, and exact attention runs over them.

The channel and score steps are written in float32 with a fixed order and no
fused multiply-add, so that the selected indices are reproducible bit for bit:
a_c and qbar_c add the query heads in ascending order; shat accumulates
acc = fl32(acc + fl32(qbar_c * k_jc)) over ascending c starting from 0.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def _head_sum(x):
    """fp32 sum over axis 0 in ascending order."""
    x = np.asarray(x, np.float32)
    acc = np.zeros(x.shape[1:], np.float32)
    for g in range(x.shape[0]):
        acc = (acc + x[g]).astype(np.float32)
    return acc


def select_channels(q, n_channels):
    """q [G][d] fp16 -> ascending channel indices of the n_channels largest sum_g |q_gc|."""
    a = _head_sum(np.abs(np.asarray(q).astype(np.float32)))
    c = np.arange(a.size)
    order = np.lexsort((c, -a))
    return np.sort(order[:min(int(n_channels), a.size)])


def approx_scores(q, k_rows, channels):
    """q [G][d] fp16, k_rows [n][d] fp16 -> shat [n] float32 (see the module docstring)."""
    qbar = _head_sum(np.asarray(q).astype(np.float32))
    k = np.asarray(k_rows).astype(np.float32)
    acc = np.zeros(k.shape[0], np.float32)
    for c in channels:
        prod = (qbar[c] * k[:, c]).astype(np.float32)
        acc = (acc + prod).astype(np.float32)
    return acc


def topk_indices(scores, k):
    """Ascending indices of the min(k, n) largest scores, lower index on equal scores."""
    s = np.asarray(scores)
    idx = np.arange(s.size)
    order = np.lexsort((idx, -s.astype(np.float64)))
    return np.sort(order[:min(int(k), s.size)])


def default_topk(keep_tokens, topk=0):
    return int(topk) if int(topk) > 0 else int(keep_tokens) // 2
