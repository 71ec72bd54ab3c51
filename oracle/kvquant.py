"""KVQuant-style non-uniform b-bit quantization with fp16 outliers.

Follows Section 2.1 (KVQuant paragraph): keys are quantized per channel,
because outliers sit in consistent channels; outlier values are stored in
uncompressed fp16; a setting is named by its bit width b in {2, 3, 4}.

The paper fixes nothing further, so these readings are used:
  * Keys: per (sequence, kv head, channel) a threshold tau_c is calibrated once
    on the prompt as the n_o-th largest |k| (0-based, descending), with
    n_o = floor((n0 * bp + 5000) / 10000) and bp the outlier fraction in basis
    points (100 = 1 %).  tau_c stays frozen for decode tokens.
  * Values: per token, s_t is the n_ov-th largest |v| over the d channels,
    n_ov = floor((d * bp + 5000) / 10000).
  * A value is an outlier iff |x| > threshold (strict).  bp = 0 disables
    outliers: the threshold is then the maximum and nothing is extracted.
  * Normalisation is symmetric: xhat = fl32(x * fl32(1 / threshold)), or 0 when
    the threshold is 0.
  * Code = number of codebook midpoints m_i = fl32((cb_i + cb_{i+1}) * 0.5)
    strictly below xhat, i.e. the nearest codebook entry with exact midpoints
    going to the lower code.  Outliers still receive (clamped) codes.
  * Effective (dequantized) value: cb[code] * threshold, except outliers,
    whose effective value is the fp16 value itself (replace, not add).

The normalise-and-compare steps are written in float32 so that codes are
reproducible bit for bit; dequantization is float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def outlier_count(n, outlier_bp):
    """Number of elements above the threshold order statistic for n elements at bp basis points."""
    return (int(n) * int(outlier_bp) + 5000) // 10000


def _order_stat_desc(a, idx, axis):
    """idx-th largest (0-based) of |a| along `axis`; 0 where idx is out of range."""
    srt = -np.sort(-np.abs(a), axis=axis)
    n = a.shape[axis]
    if idx >= n:
        shp = list(a.shape)
        del shp[axis]
        return np.zeros(shp, a.dtype)
    return np.take(srt, idx, axis=axis)


def _reciprocal(t):
    """fl32(1 / t) for t > 0, else 0 (float32 in, float32 out)."""
    t = np.asarray(t, np.float32)
    out = np.zeros_like(t)
    np.divide(np.float32(1.0), t, out=out, where=t > 0)
    return out


def midpoints(cb):
    """Decision thresholds between consecutive ascending codebook entries, float32."""
    cb = np.asarray(cb, np.float32)
    return ((cb[:-1] + cb[1:]) * np.float32(0.5)).astype(np.float32)


def codes_of(xhat, cb):
    """Nearest-codebook-entry code of each normalised value: count of midpoints strictly below."""
    m = midpoints(cb)
    xhat = np.asarray(xhat, np.float32)
    return (xhat[..., None] > m).sum(axis=-1).astype(np.uint8)


def calibrate_keys(k_prompt, outlier_bp):
    """Per-channel key thresholds of one (sequence, kv head).

    k_prompt [n0][d] fp16  ->  (tau [d] float32, inv [d] float32)"""
    x = np.asarray(k_prompt).astype(np.float32)
    if outlier_bp == 0:
        tau = np.abs(x).max(axis=0)
    else:
        tau = _order_stat_desc(x, outlier_count(x.shape[0], outlier_bp), axis=0)
    tau = np.asarray(tau, np.float32)
    return tau, _reciprocal(tau)


def quantize_keys(k, tau, inv, cb, outlier_bp):
    """Codes and outlier mask of key rows k [n][d] under frozen per-channel thresholds."""
    x = np.asarray(k).astype(np.float32)
    xhat = (x * np.asarray(inv, np.float32)[None, :]).astype(np.float32)
    codes = codes_of(xhat, cb)
    if outlier_bp > 0:
        outlier = np.abs(x) > np.asarray(tau, np.float32)[None, :]
    else:
        outlier = np.zeros(x.shape, bool)
    return codes, outlier


def dequantize_keys(k, codes, outlier, tau, cb):
    """Effective keys (float64): cb[code] * tau_c, or the fp16 value at outliers."""
    deq = np.asarray(cb, np.float64)[codes] * np.asarray(tau, np.float64)[None, :]
    return np.where(outlier, np.asarray(k).astype(np.float64), deq)


def quantize_values(v, cb, outlier_bp):
    """Per-token scales, codes and outlier mask of value rows v [n][d].

    -> (codes [n][d] uint8, scale [n] float32, outlier [n][d] bool)"""
    x = np.asarray(v).astype(np.float32)
    if outlier_bp == 0:
        s = np.abs(x).max(axis=1)
    else:
        s = _order_stat_desc(x, outlier_count(x.shape[1], outlier_bp), axis=1)
    s = np.asarray(s, np.float32)
    xhat = (x * _reciprocal(s)[:, None]).astype(np.float32)
    codes = codes_of(xhat, cb)
    outlier = (np.abs(x) > s[:, None]) if outlier_bp > 0 else np.zeros(x.shape, bool)
    return codes, s, outlier


def dequantize_values(v, codes, outlier, scale, cb):
    """Effective values (float64): cb[code] * s_t, or the fp16 value at outliers."""
    deq = np.asarray(cb, np.float64)[codes] * np.asarray(scale, np.float64)[:, None]
    return np.where(outlier, np.asarray(v).astype(np.float64), deq)


def normalised_inliers_keys(k, outlier_bp):
    """Normalised non-outlier key values of one (sequence, kv head) [n][d], for codebook fitting."""
    tau, inv = calibrate_keys(k, outlier_bp)
    x = np.asarray(k).astype(np.float32)
    xhat = (x * inv[None, :]).astype(np.float32)
    keep = np.abs(x) <= tau[None, :]
    return xhat[keep].astype(np.float64)


def normalised_inliers_values(v, outlier_bp):
    """Normalised non-outlier value entries of rows v [n][d], for codebook fitting."""
    x = np.asarray(v).astype(np.float32)
    _, s, _ = quantize_values(v, np.zeros(2, np.float32), outlier_bp)
    xhat = (x * _reciprocal(s)[:, None]).astype(np.float32)
    keep = np.abs(x) <= s[:, None]
    return xhat[keep].astype(np.float64)
