"""SnapKV prefill eviction, the first stage of RocketKV.

Section 2.1 (RocketKV paragraph): SnapKV scores prompt tokens by the attention
they receive from an observation window at the end of the prompt, aggregated,
and keeps the most relevant ones; a setting r x reduces the cache to about
1/r of its size after prefill.

Readings used where the paper is silent:
  * keep budget T tokens (T = n0 / r for the paper's ratio settings, an
    absolute token count otherwise); window w = min(32, n0); if T >= n0 nothing
    is evicted;
  * window row i sits at position n0 - w + i and attends causally to keys
    0 .. n0 - w + i (softmax over those keys, scale 1/sqrt(d));
  * vote v_j = sum over the kv head's query heads and the w window rows of the
    attention probability on key j, for j < n0 - w;
  * the votes are max-pooled with an odd kernel (7), stride 1, clipped at the
    ends of [0, n0 - w);
  * the T - w highest pooled votes are kept (lower position on equal votes),
    together with all w window tokens.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def window_votes(q_window, k_prompt):
    """Attention probability mass every prompt key receives from the window rows.

    q_window [w][G][d], k_prompt [n0][d]  ->  votes [n0] float64 (all keys, window included)"""
    q = np.asarray(q_window, np.float64)
    k = np.asarray(k_prompt, np.float64)
    w, g, d = q.shape
    n0 = k.shape[0]
    votes = np.zeros(n0)
    for i in range(w):
        row = n0 - w + i
        s = (q[i] @ k[:row + 1].T) / np.sqrt(d)       # [G][row + 1]
        s = s - s.max(axis=1, keepdims=True)
        e = np.exp(s)
        votes[:row + 1] += (e / e.sum(axis=1, keepdims=True)).sum(axis=0)
    return votes


def max_pool(v, kernel):
    """Stride-1 max pool with an odd kernel, the window clipped at both ends."""
    v = np.asarray(v, np.float64)
    h = int(kernel) // 2
    n = len(v)
    return np.array([v[max(0, j - h):min(n, j + h + 1)].max() for j in range(n)]) if n else v


def keep_budget(cfg, n0):
    """Tokens SnapKV keeps for a configuration row: `keep_tokens`, or for the paper's r-times
    settings (`keep_ratio` = r > 0) floor(n0 / r), but never fewer than the window rows, which
    are always kept (reading of Section 2.1, RocketKV paragraph: the ratio compresses the
    prompt's cache)."""
    r = int(cfg.get("keep_ratio", 0))
    if r > 0:
        return max(int(n0) // r, int(cfg.get("window", 32)))
    return int(cfg["keep_tokens"])


def snap_keep(q_window, k_prompt, keep_tokens, window=32, pool=7):
    """Positions kept by SnapKV (ascending) for one (sequence, kv head)."""
    n0 = np.asarray(k_prompt).shape[0]
    T = int(keep_tokens)
    if T >= n0:
        return np.arange(n0)
    w = min(int(window), n0)
    votes = window_votes(np.asarray(q_window)[-w:], k_prompt)[:n0 - w]
    u = max_pool(votes, pool)
    cand = np.arange(n0 - w)
    order = np.lexsort((cand, -u))                    # pooled vote desc, then position asc
    return np.sort(np.concatenate([cand[order[:T - w]], np.arange(n0 - w, n0)]))


def pooled_votes(q_window, k_prompt, window=32, pool=7):
    """The pooled votes snap_keep ranks, exposed for tie-band checks."""
    n0 = np.asarray(k_prompt).shape[0]
    w = min(int(window), n0)
    return max_pool(window_votes(np.asarray(q_window)[-w:], k_prompt)[:n0 - w], pool)
