"""Pins of the oracle's quantizers and codebook fit.

KVQuant-style codes are pinned to brute-force nearest-entry search in exact
rational arithmetic, the outlier rule to exact order-statistic counts, the
uniform quantizer to its half-step round-trip bound at 16 bits and to exact
grids, and the Lloyd fit to the published Lloyd-Max Gaussian levels.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import codebook, kvquant, uniform


def _brute_nearest(xhat, cb):
    """Nearest entry by exact distance, lower index on an exact tie."""
    x = Fraction(float(xhat))
    best, bd = 0, None
    for i, c in enumerate(cb):
        dist = abs(x - Fraction(float(c)))
        if bd is None or dist < bd:
            best, bd = i, dist
    return best


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_codes_are_brute_force_nearest(bits):
    r = np.random.default_rng(bits)
    cb = np.sort(r.uniform(-1, 1, 1 << bits).astype(np.float32))
    mids = kvquant.midpoints(cb)
    xs = np.concatenate([r.uniform(-1.5, 1.5, 3000), cb, -cb]).astype(np.float32)
    codes = kvquant.codes_of(xs, cb)
    for x, c in zip(xs, codes):
        # exclude values whose float32 midpoint differs from the exact one only by rounding
        near = np.any(np.abs(np.float64(x) - (cb[:-1].astype(np.float64) + cb[1:]) / 2) < 1e-6)
        if not near:
            assert c == _brute_nearest(x, cb), (x, c)
    assert np.all(np.diff(codes[np.argsort(xs, kind="stable")].astype(int)) >= 0)  # monotone
    assert codes.min() >= 0 and codes.max() <= (1 << bits) - 1
    # exactly representable midpoints go to the lower code
    assert mids.dtype == np.float32


def test_exact_midpoint_goes_to_lower_code():
    cb = np.array([-1.0, -0.25, 0.25, 1.0], np.float32)        # midpoints -0.625, 0, 0.625 exact
    xs = np.array([-0.625, 0.0, 0.625, -0.6249999, 0.6250001], np.float32)
    assert list(kvquant.codes_of(xs, cb)) == [0, 1, 2, 1, 3]
    for x in xs[:3]:
        assert kvquant.codes_of(np.array([x], np.float32), cb)[0] == _brute_nearest(x, cb)


def test_key_outlier_counts_follow_the_order_statistic():
    r = np.random.default_rng(7)
    n0, d = 4096, 64
    k = (r.standard_normal((n0, d)) * r.lognormal(0, .5, d)).astype(np.float16)
    for bp in (100, 250):
        no = kvquant.outlier_count(n0, bp)
        tau, inv = kvquant.calibrate_keys(k, bp)
        _, out = kvquant.quantize_keys(k, tau, inv, np.array([-1, 1], np.float32), bp)
        counts = out.sum(0)
        assert np.all(counts <= no)
        # each channel: out count + number of entries tied with tau above index no == no
        a = np.abs(k.astype(np.float32))
        for c in range(d):
            assert counts[c] == int((a[:, c] > tau[c]).sum())
            assert int((a[:, c] >= tau[c]).sum()) >= no + 1
        assert no == (n0 * bp + 5000) // 10000
    assert kvquant.outlier_count(4096, 100) == 41
    assert kvquant.outlier_count(128, 100) == 1


def test_no_outliers_at_zero_fraction():
    r = np.random.default_rng(8)
    k = (r.standard_normal((300, 32)) * 5).astype(np.float16)
    tau, inv = kvquant.calibrate_keys(k, 0)
    assert np.array_equal(tau, np.abs(k.astype(np.float32)).max(0))
    _, out = kvquant.quantize_keys(k, tau, inv, np.array([-1, 0, 1], np.float32), 0)
    assert not out.any()
    _, s, outv = kvquant.quantize_values(k, np.array([-1, 1], np.float32), 0)
    assert not outv.any() and np.array_equal(s, np.abs(k.astype(np.float32)).max(1))


def test_value_scale_is_second_largest_at_one_percent():
    r = np.random.default_rng(9)
    v = r.standard_normal((50, 128)).astype(np.float16)
    _, s, out = kvquant.quantize_values(v, np.array([-1, 1], np.float32), 100)
    a = np.sort(np.abs(v.astype(np.float32)), 1)
    assert np.array_equal(s, a[:, -2])
    # one outlier per token unless the two largest magnitudes tie in fp16
    assert np.array_equal(out.sum(1), (a[:, -1] > a[:, -2]).astype(int))


def test_codebook_points_round_trip():
    """Keys and values placed on codebook points (times a power-of-two threshold) dequantize exactly."""
    cb = np.array([-1.0, -0.375, 0.375, 1.0], np.float32)
    # prompt whose per-channel 41st-largest |k| is exactly 2 (threshold), no value above except 41
    n0 = 4096
    base = np.tile(np.array([-2.0, -0.75, 0.75, 2.0], np.float32), n0 // 4)
    k = np.stack([base, -base], 1).astype(np.float16)
    k[:41, :] = np.float16(8.0)                               # 41 outliers per channel
    tau, inv = kvquant.calibrate_keys(k, 100)
    assert np.all(tau == 2.0) and np.all(inv == 0.5)
    codes, out = kvquant.quantize_keys(k, tau, inv, cb, 100)
    eff = kvquant.dequantize_keys(k, codes, out, tau, cb)
    assert np.array_equal(eff, k.astype(np.float64))
    assert out.sum() == 82


def test_uniform_sixteen_bit_round_trip():
    """At 16 bits every value comes back within half a quantization step (plus float32 slack)."""
    r = np.random.default_rng(10)
    x = (r.standard_normal((500, 64)) * 3).astype(np.float16)
    codes, mn, rr = uniform.quantize_groups(x, 16)
    back = uniform.dequantize_groups(codes, mn, rr, 16)
    step = rr.astype(np.float64)[:, None] / 65535.0
    err = np.abs(back - x.astype(np.float64))
    assert np.all(err <= step * 0.5 * 1.05 + 1e-12)
    assert np.all(codes.min(1) == 0) and np.all(codes.max(1) == 65535)


def test_uniform_grid_values_are_exact():
    x = np.array([[0, 1, 2, 3, 15, 7, 9, 14] * 8], np.float16)      # min 0, max 15 -> step 1 at 4 bits
    codes, mn, rr = uniform.quantize_groups(x, 4)
    assert np.array_equal(codes, x.astype(np.int64))
    assert np.array_equal(uniform.dequantize_groups(codes, mn, rr, 4), x.astype(np.float64))


def test_uniform_codes_are_nearest_grid_point():
    r = np.random.default_rng(11)
    x = r.standard_normal((200, 64)).astype(np.float16)
    codes, mn, rr = uniform.quantize_groups(x, 4)
    for i in range(200):
        lo, span = Fraction(float(mn[i])), Fraction(float(rr[i]))
        for j in range(64):
            t = (Fraction(float(x[i, j])) - lo) * 15 / span
            frac = t - int(t)
            if abs(frac - Fraction(1, 2)) > Fraction(1, 10**4):
                assert codes[i, j] == round(t), (i, j)


def test_uniform_key_tail_stays_fp16():
    r = np.random.default_rng(12)
    k = r.standard_normal((64 * 3 + 17, 64)).astype(np.float16)
    eff = uniform.effective_keys(k, 4)
    assert np.array_equal(eff[192:], k[192:].astype(np.float64))
    assert not np.array_equal(eff[:192], k[:192].astype(np.float64))
    # per (block, channel) the min and max survive exactly
    blk = k[:64].astype(np.float64)
    assert np.array_equal(eff[:64].min(0), blk.min(0))
    np.testing.assert_allclose(eff[:64].max(0), blk.max(0), rtol=1e-6)


def test_lloyd_matches_published_gaussian_levels(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "lloyd_max_gaussian.json")))
    x = np.random.default_rng(13).standard_normal(400_000)
    for bits, half in g["levels"].items():
        cb = codebook.lloyd_codebook(x, int(bits), max_iter=300)
        expect = np.concatenate([-np.array(half[::-1]), np.array(half)])
        np.testing.assert_allclose(cb, expect, atol=0.02)


def test_lloyd_fixed_point_and_separated_clusters():
    r = np.random.default_rng(14)
    centers = np.array([-3.0, -1.0, 0.5, 4.0])
    x = np.concatenate([c + 0.01 * r.standard_normal(1000) for c in centers])
    cb = np.sort(codebook.lloyd_centroids(x, 2))
    np.testing.assert_allclose(cb, [x[i * 1000:(i + 1) * 1000].mean() for i in range(4)], atol=1e-6)
    # at convergence every centroid is the mean of the samples nearest to it
    y = r.standard_normal(20000)
    cb = codebook.lloyd_centroids(y, 3, max_iter=1000)
    a = np.argmin(np.abs(y[:, None] - cb[None]), 1)
    for i in range(8):
        assert abs(y[a == i].mean() - cb[i]) < 1e-6


def test_stored_codebook_is_the_fp16_rounding_of_the_centroids():
    y = np.random.default_rng(15).standard_normal(20000) * 0.37
    for bits in (2, 3, 4):
        c = np.sort(codebook.lloyd_centroids(y, bits))
        cb = codebook.lloyd_codebook(y, bits)
        assert cb.dtype == np.float32 and np.all(np.diff(cb) >= 0)
        # every entry is an fp16 value, within half an fp16 ulp of its centroid
        assert np.array_equal(cb.astype(np.float16).astype(np.float32), cb)
        ulp = np.spacing(np.abs(c).astype(np.float16)).astype(np.float64)
        assert np.all(np.abs(cb.astype(np.float64) - c) <= ulp / 2)


def test_kvq_sequence_dequant_error_is_bounded_by_the_codebook_gap():
    """With a 16-entry uniform codebook on [-1, 1], every non-outlier effective key lies within
    half a gap (1/15) times its channel threshold of the fp16 key, and outliers are exact."""
    from oracle.sequence import Sequence
    from workloads import make_workload, prompt_kv, step_inputs
    wl = make_workload("custom", n_seqs=1, n_q_heads=4, n_kv_heads=2, head_dim=64,
                       prompt_lens=[300], steps=2, config_ids=[0])
    kp, vp = prompt_kv(wl, 0)
    cb = np.linspace(-1, 1, 16).astype(np.float32)
    seq = Sequence({"method": "kvq", "bits": 4, "outlier_bp": 100}, kp, vp, 4,
                   codebooks={4: (cb, cb)})
    kn, vn, q = step_inputs(wl, 0)
    seq.step(kn[0], vn[0], q[0])
    for h in range(2):
        kq = seq.kq[h]
        raw = kq["raw"].astype(np.float64)
        err = np.abs(kq["eff"] - raw)
        tau = seq.tau[h].astype(np.float64)
        inl = ~kq["outlier"]
        assert np.all(err[inl] <= (tau[None, :] / 15 + 1e-6 * tau[None, :]).repeat(301, 0)[inl])
        assert np.all(err[kq["outlier"]] == 0)
        vq = seq.vq[h]
        verr = np.abs(vq["eff"] - vq["raw"].astype(np.float64))
        assert np.all(verr[~vq["outlier"]] <= (vq["scale"][:, None] / 15 * (1 + 1e-6)).repeat(64, 1)[~vq["outlier"]])


def test_uniform_value_groups_are_consecutive_channels():
    """Values are grouped per token over 64 consecutive channels: the exact minimum of every
    (token, channel 64g .. 64g + 63) group comes back exactly, its maximum to float32 rounding,
    and every code equals a brute-force quantizer of that slice in exact rationals (a grouping
    over any other channel sets moves some group's extremes and codes)."""
    r = np.random.default_rng(16)
    n, d = 40, 256
    v = (r.standard_normal((n, d)) * r.lognormal(0, 0.7, d)).astype(np.float16)
    eff = uniform.effective_values(v, 4)
    codes, mn, rr = uniform.quantize_value_rows(v, 4)
    assert codes.shape == (n, d) and mn.shape == (n, d // 64)
    for t in range(n):
        for g in range(d // 64):
            sl = slice(64 * g, 64 * g + 64)
            x = [Fraction(float(a)) for a in v[t, sl]]
            lo, hi = min(x), max(x)
            assert Fraction(float(eff[t, sl].min())) == lo
            assert abs(float(eff[t, sl].max()) - float(hi)) <= 1e-6 * max(abs(float(hi)), 1e-3)
            assert Fraction(float(mn[t, g])) == lo
            for j, xj in enumerate(x):
                u = (xj - lo) * 15 / (hi - lo)
                if abs(u - int(u) - Fraction(1, 2)) > Fraction(1, 10**4):
                    assert codes[t, 64 * g + j] == round(u), (t, g, j)


def _brute_threshold(col, n_o):
    """n_o-th largest magnitude (0-based), found by counting rather than sorting: the value a
    with at most n_o magnitudes strictly above it and at least n_o + 1 at or above it."""
    mags = [abs(Fraction(float(x))) for x in col]
    for a in mags:
        above = sum(1 for m in mags if m > a)
        atleast = sum(1 for m in mags if m >= a)
        if above <= n_o < atleast:
            return a
    raise AssertionError("no order statistic")


@pytest.mark.parametrize("bp", [100, 400])
def test_normalised_inliers_brute_force(bp):
    """The codebook-fitting samples: per channel (keys) or per token (values), every entry at or
    below its threshold, scaled by the float32 reciprocal of the threshold; the threshold is
    found by counting magnitudes in exact rationals."""
    r = np.random.default_rng(17 + bp)
    k = (r.standard_normal((150, 8)) * r.lognormal(0, 1.0, 8)).astype(np.float16)
    v = r.standard_normal((30, 64)).astype(np.float16)
    want_k = []
    for c in range(k.shape[1]):
        tau = _brute_threshold(k[:, c], kvquant.outlier_count(k.shape[0], bp))
        inv = np.float32(1.0) / np.float32(float(tau))
        want_k += [float(np.float32(np.float32(float(x)) * inv)) for x in k[:, c]
                   if abs(Fraction(float(x))) <= tau]
    got_k = kvquant.normalised_inliers_keys(k, bp)
    assert sorted(got_k.tolist()) == sorted(want_k)
    want_v = []
    for t in range(v.shape[0]):
        s = _brute_threshold(v[t], kvquant.outlier_count(v.shape[1], bp))
        inv = np.float32(1.0) / np.float32(float(s))
        want_v += [float(np.float32(np.float32(float(x)) * inv)) for x in v[t] if abs(Fraction(float(x))) <= s]
    got_v = kvquant.normalised_inliers_values(v, bp)
    assert sorted(got_v.tolist()) == sorted(want_v)
    assert np.all(np.abs(got_k) <= 1.0 + 2 ** -23) and np.all(np.abs(got_v) <= 1.0 + 2 ** -23)
