"""Pins of the oracle's H2O, SnapKV and RocketKV selection steps.

Each is pinned to something other than itself: pure-Python brute force with
math.exp on tiny inputs, rank counting instead of sorting, probability-mass
conservation, a library max filter, an independent float32 emulation through
struct, and the reductions to dense attention the methods have when nothing is
evicted or every token is selected.
"""
import math
import struct

import numpy as np
import pytest

from oracle import h2o, rocketkv, snapkv
from oracle.attention import softmax_attention
from oracle.sequence import Sequence
from workloads import make_workload, prompt_kv, prompt_q, step_inputs


def _brute_column_sums(q, k):
    """S_j = sum_g sum_{i >= j} causal softmax, by explicit loops."""
    n0, G, d = q.shape
    S = [0.0] * n0
    for g in range(G):
        for i in range(n0):
            logits = [sum(float(q[i, g, c]) * float(k[j, c]) for c in range(d)) / math.sqrt(d)
                      for j in range(i + 1)]
            m = max(logits)
            e = [math.exp(x - m) for x in logits]
            tot = sum(e)
            for j in range(i + 1):
                S[j] += e[j] / tot
    return S


def _rank_keep(scores, positions, h, prefer_newer):
    """Keep j iff fewer than h candidates beat it (higher score, or equal score and the tie rule)."""
    kept = []
    for a, sa in zip(positions, scores):
        beats = 0
        for b, sb in zip(positions, scores):
            if b == a:
                continue
            if sb > sa or (sb == sa and ((b > a) if prefer_newer else (b < a))):
                beats += 1
        if beats < h:
            kept.append(a)
    return sorted(kept)


def test_h2o_prefill_scores_brute_force():
    r = np.random.default_rng(20)
    q = r.standard_normal((12, 3, 4))
    k = r.standard_normal((12, 4))
    np.testing.assert_allclose(h2o.prefill_scores(q, k, row_chunk=5), _brute_column_sums(q, k),
                               rtol=0, atol=1e-13)


def test_h2o_prefill_keep_rank_counting_with_ties():
    r = np.random.default_rng(21)
    for trial in range(50):
        n0 = int(r.integers(4, 16))
        S = r.integers(0, 4, n0).astype(float)          # many exact ties
        B = int(r.integers(1, n0 + 2))
        R = int(r.integers(0, B + 1))
        keep = h2o.prefill_keep(S, B, R)
        if B >= n0:
            assert list(keep) == list(range(n0))
            continue
        cand = list(range(n0 - R))
        brute = sorted(_rank_keep([S[j] for j in cand], cand, B - R, prefer_newer=True)
                       + list(range(n0 - R, n0)))
        assert list(keep) == brute


def test_h2o_prefill_mass_conservation():
    r = np.random.default_rng(22)
    q, k = r.standard_normal((300, 4, 32)), r.standard_normal((300, 32)) * 2
    S = h2o.prefill_scores(q, k, row_chunk=77)
    assert abs(S.sum() - 4 * 300) < 1e-9
    assert np.all(S > 0)


def _h2o_case(pct, n0=64, steps=24, G=2, hkv=2, d=16, seed=23):
    wl = make_workload("custom", seed=seed, n_seqs=1, n_q_heads=G * hkv, n_kv_heads=hkv,
                       head_dim=d, prompt_lens=[n0], steps=steps,
                       config_ids=[0], boost_frac=0.05, boost=3.0)
    kp, vp = prompt_kv(wl, 0)
    qp = prompt_q(wl, 0)
    return wl, kp, vp, qp


def test_h2o_large_budget_equals_dense():
    wl, kp, vp, qp = _h2o_case(0)
    dense = Sequence({"method": "fp16"}, kp, vp, wl.n_q_heads)
    h = Sequence({"method": "h2o", "budget_pct": 1000}, kp, vp, wl.n_q_heads, q_prompt=qp)
    for t in range(wl.steps):
        kn, vn, q = step_inputs(wl, t)
        a, _ = dense.step(kn[0], vn[0], q[0])
        b, info = h.step(kn[0], vn[0], q[0])
        assert all(e is None for e in info["evict"])
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_h2o_mass_conservation_and_brute_force_decode():
    """Scores kept + scores evicted == G * (prompt rows + decode steps); and a list-based
    brute-force simulation with math.exp reproduces the retained sets and outputs."""
    wl, kp, vp, qp = _h2o_case(0, n0=14, steps=10, G=2, hkv=1, d=4, seed=24)
    seq = Sequence({"method": "h2o", "budget_pct": 50}, kp, vp, wl.n_q_heads, q_prompt=qp)
    B, R = h2o.budget(50, 14)
    # brute force state
    S = _brute_column_sums(qp[:, 0:2].astype(np.float64), kp[:, 0].astype(np.float64))
    cand = list(range(14 - R))
    keep = sorted(_rank_keep([S[j] for j in cand], cand, B - R, True) + list(range(14 - R, 14)))
    assert list(seq.heads[0].pos) == keep
    state = {j: S[j] for j in keep}
    rows = {j: (kp[j, 0].astype(float), vp[j, 0].astype(float)) for j in range(14)}
    evicted_mass = sum(S[j] for j in range(14) if j not in keep)
    for t in range(wl.steps):
        kn, vn, q = step_inputs(wl, t)
        p = 14 + t
        out, info = seq.step(kn[0], vn[0], q[0])
        rows[p] = (kn[0, 0].astype(float), vn[0, 0].astype(float))
        state[p] = 0.0
        pos = sorted(state)
        for g in range(2):
            logits = [sum(float(q[0, g, c]) * rows[j][0][c] for c in range(4)) / 2.0 for j in pos]
            m = max(logits)
            e = [math.exp(x - m) for x in logits]
            tot = sum(e)
            o = [sum(e[i] / tot * rows[j][1][c] for i, j in enumerate(pos)) for c in range(4)]
            np.testing.assert_allclose(out[g], o, atol=1e-12)
            for i, j in enumerate(pos):
                state[j] += e[i] / tot
        if len(state) > B:
            cands = [j for j in pos if j < p - R + 1]
            victim = min(cands, key=lambda j: (state[j], j))
            assert info["evict"][0] == victim
            evicted_mass += state.pop(victim)
        seq.apply_evictions(info["evict"])
        assert list(seq.heads[0].pos) == sorted(state)
        np.testing.assert_allclose(seq.heads[0].score, [state[j] for j in sorted(state)], atol=1e-12)
        total = sum(state.values()) + evicted_mass
        assert abs(total - 2 * (14 + t + 1)) < 1e-9


def test_h2o_all_recent_is_a_sliding_window():
    r = np.random.default_rng(25)
    S = r.random(40)
    assert list(h2o.prefill_keep(S, 10, 10)) == list(range(30, 40))
    hd = h2o.H2OHead(np.arange(30, 40), r.standard_normal((10, 8)), r.standard_normal((10, 8)),
                     r.random(10), B=10, R=10)
    for p in range(40, 50):
        hd.attend(r.standard_normal(8), r.standard_normal(8), r.standard_normal((1, 8)), p)
        hd.evict(hd.choose_eviction(p))
        assert list(hd.pos) == list(range(p - 9, p + 1))


def test_snapkv_keeps_everything_when_budget_covers_prompt():
    r = np.random.default_rng(26)
    k, qw = r.standard_normal((100, 16)), r.standard_normal((32, 2, 16))
    assert list(snapkv.snap_keep(qw, k, 100)) == list(range(100))
    assert list(snapkv.snap_keep(qw, k, 500)) == list(range(100))


def test_snapkv_votes_mass_and_brute_force():
    r = np.random.default_rng(27)
    n0, w, G, d = 20, 5, 2, 4
    k, qw = r.standard_normal((n0, d)), r.standard_normal((w, G, d))
    votes = snapkv.window_votes(qw, k)
    assert abs(votes.sum() - G * w) < 1e-12
    brute = [0.0] * n0
    for i in range(w):
        row = n0 - w + i
        for g in range(G):
            lg = [sum(qw[i, g, c] * k[j, c] for c in range(d)) / 2.0 for j in range(row + 1)]
            m = max(lg)
            e = [math.exp(x - m) for x in lg]
            for j in range(row + 1):
                brute[j] += e[j] / sum(e)
    np.testing.assert_allclose(votes, brute, atol=1e-13)


def test_snapkv_pool_matches_library_max_filter_and_keep_brute_force():
    ndimage = pytest.importorskip("scipy.ndimage")
    r = np.random.default_rng(28)
    for n in (1, 2, 7, 50):
        v = r.random(n)
        for ker in (1, 3, 7):
            np.testing.assert_array_equal(snapkv.max_pool(v, ker),
                                          ndimage.maximum_filter1d(v, ker, mode="nearest"))
    for trial in range(30):
        n0, w, T = int(r.integers(10, 40)), 4, int(r.integers(5, 12))
        k, qw = r.standard_normal((n0, 4)), r.standard_normal((w, 1, 4))
        k[r.integers(0, n0, 3)] = k[0]                 # duplicate keys -> exact vote ties
        keep = snapkv.snap_keep(qw, k, T, window=w, pool=3)
        u = snapkv.pooled_votes(qw, k, window=w, pool=3)
        cand = list(range(n0 - w))
        brute = sorted(_rank_keep([u[j] for j in cand], cand, T - w, prefer_newer=False)
                       + list(range(n0 - w, n0)))
        assert list(keep) == brute
    # pool 1 is a plain top-(T - w) of the raw votes
    k, qw = r.standard_normal((60, 8)), r.standard_normal((8, 2, 8))
    votes = snapkv.window_votes(qw, k)[:52]
    top = np.argsort(-votes, kind="stable")[:12]
    assert list(snapkv.snap_keep(qw, k, 20, window=8, pool=1)) == sorted(list(top) + list(range(52, 60)))


def _fl32(x):
    return struct.unpack("f", struct.pack("f", x))[0]


def test_rocket_approx_scores_match_struct_float32_emulation():
    r = np.random.default_rng(29)
    q = r.standard_normal((4, 32)).astype(np.float16)
    k = (r.standard_normal((40, 32)) * 3).astype(np.float16)
    ch = rocketkv.select_channels(q, 8)
    s = rocketkv.approx_scores(q, k, ch)
    qbar = []
    for c in range(32):
        acc = 0.0
        for g in range(4):
            acc = _fl32(acc + float(q[g, c]))
        qbar.append(acc)
    for j in range(40):
        acc = 0.0
        for c in ch:
            acc = _fl32(acc + _fl32(qbar[c] * float(k[j, c])))
        assert np.float32(acc) == s[j]


def test_rocket_channel_and_token_selection_rank_counting():
    r = np.random.default_rng(30)
    for trial in range(40):
        q = r.integers(-3, 4, (2, 16)).astype(np.float16)           # many equal magnitudes
        ch = rocketkv.select_channels(q, 5)
        a = [_fl32(abs(float(q[0, c])) + abs(float(q[1, c]))) for c in range(16)]
        assert list(ch) == _rank_keep(a, list(range(16)), 5, prefer_newer=False)
        sc = r.integers(0, 5, 25).astype(np.float32)
        kk = int(r.integers(1, 30))
        assert list(rocketkv.topk_indices(sc, kk)) == _rank_keep(list(sc), list(range(25)), kk, False)


def test_rocket_full_channels_rank_like_exact_logits():
    r = np.random.default_rng(31)
    q = r.standard_normal((1, 64)).astype(np.float16)
    k = r.standard_normal((300, 64)).astype(np.float16)
    s = rocketkv.approx_scores(q, k, np.arange(64))
    exact = k.astype(np.float64) @ q[0].astype(np.float64)
    np.testing.assert_allclose(s, exact, atol=1e-4)
    order = np.argsort(-exact)
    gaps = -np.diff(exact[order])
    clear = np.nonzero(gaps > 1e-3)[0]
    for i in clear[:50]:
        top = set(rocketkv.topk_indices(s, i + 1))
        assert top == set(order[:i + 1])


def test_rocket_dense_when_budget_covers_everything():
    wl = make_workload("custom", n_seqs=1, n_q_heads=4, n_kv_heads=2, head_dim=32,
                       prompt_lens=[80], steps=6, config_ids=[0])
    kp, vp = prompt_kv(wl, 0)
    qp = prompt_q(wl, 0)
    dense = Sequence({"method": "fp16"}, kp, vp, 4)
    rk = Sequence({"method": "rocket", "keep_tokens": 100, "window": 32, "pool": 7,
                   "topk": 1000, "n_channels": 32}, kp, vp, 4, q_prompt=qp)
    for t in range(6):
        kn, vn, q = step_inputs(wl, t)
        a, _ = dense.step(kn[0], vn[0], q[0])
        b, info = rk.step(kn[0], vn[0], q[0])
        assert all(len(s["slots"]) == 80 + t + 1 for s in info["selected"])
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_dense_sequence_is_exact_attention_over_the_stream():
    torch = pytest.importorskip("torch")
    wl = make_workload("tiny")
    kp, vp = prompt_kv(wl, 0)
    seq = Sequence({"method": "fp16"}, kp, vp, 4)
    kn, vn, q = step_inputs(wl, 0)
    out, _ = seq.step(kn[0], vn[0], q[0])
    for h in range(4):
        K = np.vstack([kp[:, h], kn[0, h][None]]).astype(np.float64)
        V = np.vstack([vp[:, h], vn[0, h][None]]).astype(np.float64)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[0, h:h + 1].astype(np.float64))[None], torch.from_numpy(K)[None],
            torch.from_numpy(V)[None])[0].numpy()
        np.testing.assert_allclose(out[h:h + 1], ref, atol=1e-12)


def test_uq_sixteen_bits_tracks_dense():
    wl = make_workload("tiny")
    kp, vp = prompt_kv(wl, 0)
    dense = Sequence({"method": "fp16"}, kp, vp, 4)
    uq = Sequence({"method": "uq", "bits": 16, "group": 64}, kp, vp, 4)
    for t in range(3):
        kn, vn, q = step_inputs(wl, t)
        a, _ = dense.step(kn[0], vn[0], q[0])
        b, _ = uq.step(kn[0], vn[0], q[0])
        np.testing.assert_allclose(a, b, atol=2e-3)


def test_rocket_ratio_budget_is_prompt_over_r():
    """The paper's r-times RocketKV settings keep floor(prompt_len / r) tokens (never fewer than
    the window): at a 32768-token prompt, 8x, 16x and 32x are the 4096-, 2048- and 1024-token
    budgets, and the keep-set equals the absolute-budget keep-set."""
    from workloads import config
    for r, T in ((8, 4096), (16, 2048), (32, 1024)):
        assert snapkv.keep_budget(config(f"Rocket-{r}x"), 32768) == T
        assert snapkv.keep_budget(config(f"Rocket-{T}"), 32768) == T
    assert snapkv.keep_budget(config("Rocket-32x"), 500) == 32      # 15 < window
    rng = np.random.default_rng(3)
    n0, G, d = 700, 2, 16
    q = rng.standard_normal((32, G, d)).astype(np.float16)
    k = rng.standard_normal((n0, d)).astype(np.float16)
    a = snapkv.snap_keep(q, k, snapkv.keep_budget(config("Rocket-8x"), n0), 32, 7)
    b = snapkv.snap_keep(q, k, n0 // 8, 32, 7)
    assert np.array_equal(a, b) and len(a) == n0 // 8
