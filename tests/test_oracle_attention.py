"""Pins of the oracle's exact attention: closed forms, a library routine, a split form."""
import json
import math
import os

import numpy as np
import pytest

from oracle.attention import softmax_attention


def test_closed_form_fixture(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "attention_closed_form.json")))
    out, p = softmax_attention(np.array(g["q"]), np.array(g["k"]), np.array(g["v"]))
    np.testing.assert_allclose(p, g["probs"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(out, g["out"], rtol=0, atol=1e-14)


def test_single_key_returns_its_value():
    r = np.random.default_rng(1)
    v = r.standard_normal((1, 16))
    out, p = softmax_attention(r.standard_normal((3, 16)), r.standard_normal((1, 16)), v)
    assert np.array_equal(p, np.ones((3, 1)))
    assert np.array_equal(out, np.repeat(v, 3, axis=0))


@pytest.mark.parametrize("case", ["zero_query", "identical_keys"])
def test_uniform_weights_give_the_mean(case):
    r = np.random.default_rng(2)
    n, d = 37, 32
    v = r.standard_normal((n, d))
    if case == "zero_query":
        q, k = np.zeros((2, d)), r.standard_normal((n, d))
    else:
        q, k = r.standard_normal((2, d)), np.repeat(r.standard_normal((1, d)), n, axis=0)
    out, _ = softmax_attention(q, k, v)
    np.testing.assert_allclose(out, np.repeat(v.mean(0, keepdims=True), 2, 0), atol=1e-14)


def test_dominant_key_selects_its_value():
    r = np.random.default_rng(3)
    d = 64
    k = r.standard_normal((50, d)) * 0.01
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    k[17, 0] = 100.0 * math.sqrt(d)         # logit 100 above the others
    v = r.standard_normal((50, d))
    out, _ = softmax_attention(q, k, v)
    np.testing.assert_allclose(out[0], v[17], atol=1e-30 + 1e-40, rtol=1e-12)


def test_matches_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(4)
    for n, d, g in [(1, 64, 4), (129, 128, 4), (1000, 64, 1), (513, 128, 8)]:
        q, k, v = r.standard_normal((g, d)), r.standard_normal((n, d)) * 2, r.standard_normal((n, d))
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None])[0].numpy()
        out, _ = softmax_attention(q, k, v)
        np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_split_lse_merge_reaches_the_same_value():
    """A streaming split over token chunks with log-sum-exp merging gives the same output."""
    r = np.random.default_rng(5)
    n, d = 1000, 128
    q, k, v = r.standard_normal((4, d)), r.standard_normal((n, d)) * 3, r.standard_normal((n, d))
    parts = []
    for a in range(0, n, 96):
        s = q @ k[a:a + 96].T / math.sqrt(d)
        m = s.max(1)
        e = np.exp(s - m[:, None])
        parts.append((m, e.sum(1), e @ v[a:a + 96]))
    M = np.max([p[0] for p in parts], axis=0)
    L = sum(p[1] * np.exp(p[0] - M) for p in parts)
    O = sum(p[2] * np.exp(p[0] - M)[:, None] for p in parts) / L[:, None]
    out, _ = softmax_attention(q, k, v)
    np.testing.assert_allclose(O, out, rtol=0, atol=1e-12)


def test_permutation_invariance():
    r = np.random.default_rng(6)
    q, k, v = r.standard_normal((4, 64)), r.standard_normal((200, 64)), r.standard_normal((200, 64))
    perm = r.permutation(200)
    a, _ = softmax_attention(q, k, v)
    b, _ = softmax_attention(q, k[perm], v[perm])
    np.testing.assert_allclose(a, b, atol=1e-14)
