"""H2O heavy-hitter eviction.

Section 2.1 (H2O paragraph): each token carries an accumulated attention score,
the attention it receives from later tokens; when the cache exceeds its budget,
older tokens with the lowest accumulated scores are evicted; a setting p % is a
budget relative to the prompt length.

Readings used where the paper is silent:
  * budget B = floor(p * n0 / 100), fixed at prefill; it is split into R =
    floor(B / 2) most-recent tokens and H = B - R heavy hitters;
  * under grouped-query attention one score per (sequence, kv head) is kept,
    the sum over the kv head's query heads;
  * prefill score of prompt token j: S_j = sum_g sum_{i >= j} softmax_i[j], the
    causal attention it receives from every prompt row i (its own included);
    the cache keeps the R most recent prompt tokens plus the H highest S_j
    among the rest, preferring the newer token on equal scores;
  * decode step at position p: append the new token with score 0, attend over
    the retained set (new token included), add each query head's attention
    probability to the scores, then, if more than B tokens are held, evict the
    token with the lowest score among positions < p - R + 1, the older one on
    equal scores.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np

from .attention import softmax_attention


def budget(budget_pct, n0):
    """(B, R): total budget and recent-window size for a p % setting at prompt length n0."""
    b = (int(budget_pct) * int(n0)) // 100
    return b, b // 2


def prefill_scores(q_prompt, k_prompt, row_chunk=512):
    """Accumulated prefill attention per prompt token of one (sequence, kv head).

    q_prompt [n0][G][d] (the kv head's query heads), k_prompt [n0][d]  ->  S [n0] float64"""
    q = np.asarray(q_prompt, np.float64)
    k = np.asarray(k_prompt, np.float64)
    n0, g, d = q.shape
    S = np.zeros(n0)
    for a in range(0, n0, row_chunk):
        b = min(n0, a + row_chunk)
        rows = np.arange(a, b)
        for gi in range(g):
            s = (q[a:b, gi] @ k[:b].T) / np.sqrt(d)          # rows [a, b) x keys [0, b)
            s[np.arange(b)[None, :] > rows[:, None]] = -np.inf  # causal: key j <= row i
            s = s - s.max(axis=1, keepdims=True)
            e = np.exp(s)
            p = e / e.sum(axis=1, keepdims=True)
            S[:b] += p.sum(axis=0)
    return S


def prefill_keep(S, B, R):
    """Positions kept after prefill (ascending): the last R plus the top B - R of the rest.

    Among the candidates [0, n0 - R), higher score wins and the newer token wins a tie."""
    n0 = len(S)
    if B >= n0:
        return np.arange(n0)
    cand = np.arange(n0 - R)
    order = np.lexsort((-cand, -np.asarray(S)[cand]))   # score desc, then position desc
    keep = np.sort(np.concatenate([cand[order[:B - R]], np.arange(n0 - R, n0)]))
    return keep


class H2OHead:
    """Retained set of one (sequence, kv head): positions, effective K/V rows, float64 scores."""

    def __init__(self, positions, k_rows, v_rows, scores, B, R):
        self.pos = np.asarray(positions, np.int64)
        self.k = np.asarray(k_rows, np.float64)
        self.v = np.asarray(v_rows, np.float64)
        self.score = np.asarray(scores, np.float64)
        self.B, self.R = int(B), int(R)

    def attend(self, k_new, v_new, q, p):
        """Append token p, attend, accumulate.  q [G][d] -> out [G][d] float64."""
        self.pos = np.append(self.pos, p)
        self.k = np.vstack([self.k, np.asarray(k_new, np.float64)[None]])
        self.v = np.vstack([self.v, np.asarray(v_new, np.float64)[None]])
        self.score = np.append(self.score, 0.0)
        out, probs = softmax_attention(q, self.k, self.v)
        self.score = self.score + probs.sum(axis=0)
        return out

    def eviction_candidates(self, p):
        """Indices (into the retained arrays) that may be evicted after the step at position p."""
        return np.nonzero(self.pos < p - self.R + 1)[0]

    def choose_eviction(self, p):
        """Position the method evicts after the step at p, or None when within budget."""
        if len(self.pos) <= self.B:
            return None
        c = self.eviction_candidates(p)
        order = np.lexsort((self.pos[c], self.score[c]))     # score asc, then position asc
        return int(self.pos[c[order[0]]])

    def evict(self, position):
        i = int(np.nonzero(self.pos == position)[0][0])
        keep = np.arange(len(self.pos)) != i
        self.pos, self.k, self.v, self.score = (self.pos[keep], self.k[keep], self.v[keep],
                                                self.score[keep])
