"""Uniform (asymmetric min/max) b-bit group quantization.

This is the per-channel-key / per-token-value uniform quantizer with group 64
used as the eleventh configuration: the paper itself only evaluates KVQuant's
non-uniform variant, so this is a reading of "b-bit KV quantization with keys
per channel" (Section 2.1, KVQuant paragraph) in its simplest uniform form.

For one group of values x (fp16):
  mn, mx = min, max (exact in float32);  r = fl32(mx - mn)
  inv = fl32((2^b - 1) / r) if r > 0 else 0
  code = clamp(rint_half_even(fl32(fl32(x - mn) * inv)), 0, 2^b - 1)
  effective value = mn + code * r / (2^b - 1)        (float64)

Keys: groups are one channel over a 64-token block; tokens of an incomplete
final block stay in fp16 until the block fills.  Values: groups are 64
consecutive channels of one token.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def quantize_groups(x, bits):
    """Quantize along the last axis.  x [..., g] fp16 -> (codes int64, mn f32, r f32)."""
    xf = np.asarray(x).astype(np.float32)
    mn = xf.min(axis=-1)
    mx = xf.max(axis=-1)
    r = (mx - mn).astype(np.float32)
    levels = np.float32((1 << int(bits)) - 1)
    inv = np.zeros_like(r)
    np.divide(levels, r, out=inv, where=r > 0)
    y = ((xf - mn[..., None]).astype(np.float32) * inv[..., None]).astype(np.float32)
    codes = np.clip(np.rint(y), 0, levels).astype(np.int64)
    return codes, mn, r


def dequantize_groups(codes, mn, r, bits):
    levels = float((1 << int(bits)) - 1)
    return (np.asarray(mn, np.float64)[..., None]
            + np.asarray(codes, np.float64) * (np.asarray(r, np.float64)[..., None] / levels))


def quantize_key_blocks(k, bits, group=64):
    """Keys [n][d] -> codes [nb*group][d], mn [nb][d], r [nb][d] over the nb full blocks."""
    k = np.asarray(k)
    nb = k.shape[0] // group
    blocks = k[:nb * group].reshape(nb, group, k.shape[1]).transpose(0, 2, 1)  # [nb][d][g]
    codes, mn, r = quantize_groups(blocks, bits)
    return codes.transpose(0, 2, 1).reshape(nb * group, k.shape[1]), mn, r


def effective_keys(k, bits, group=64):
    """Effective keys of a token stream: full blocks dequantized, the tail block left in fp16."""
    k = np.asarray(k)
    nb = k.shape[0] // group
    out = k.astype(np.float64)
    if nb:
        codes, mn, r = quantize_key_blocks(k, bits, group)
        c = codes.reshape(nb, group, k.shape[1]).transpose(0, 2, 1)
        deq = dequantize_groups(c, mn, r, bits).transpose(0, 2, 1).reshape(nb * group, k.shape[1])
        out[:nb * group] = deq
    return out


def quantize_value_rows(v, bits, group=64):
    """Values [n][d] -> codes [n][d], mn [n][d/group], r [n][d/group]."""
    v = np.asarray(v)
    n, d = v.shape
    codes, mn, r = quantize_groups(v.reshape(n, d // group, group), bits)
    return codes.reshape(n, d), mn, r


def effective_values(v, bits, group=64):
    v = np.asarray(v)
    n, d = v.shape
    codes, mn, r = quantize_value_rows(v, bits, group)
    return dequantize_groups(codes.reshape(n, d // group, group), mn, r, bits).reshape(n, d)
