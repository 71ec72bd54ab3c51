"""Seeded synthetic decode workloads.

Both the GPU path and the CPU oracle consume these arrays; nothing in this
module computes any part of a compression method.  Every draw comes from its
own ``numpy.random.Generator(PCG64(SeedSequence([seed, workload, kind, index])))``
stream, so a sequence's tensors do not depend on how many other sequences or
steps are drawn.  All values are drawn in float32 and rounded to IEEE binary16
with round-to-nearest-even.

Distributions (shaped like a Llama-3-8B attention layer, the model of the
paper's Section 3.1):
  * queries and values ~ N(0, 1);
  * keys = N(0, 1) * sigma_c with sigma_c ~ lognormal(0, 0.5) per
    (sequence, kv head, channel) and two channels per kv head scaled by 8
    (the per-channel outlier structure KVQuant's key quantization targets);
  * the ``h2o`` workload additionally scales 5 % of key rows by 3
    (Bernoulli per row, prompt and decode alike) to create heavy hitters.
"""
from dataclasses import dataclass, field

import numpy as np

from .configs import config

# stream kinds
_SIGMA, _OUTCH, _KP, _VP, _QP, _STEP, _LENS, _CFG, _BOOST, _CALIB = range(1, 11)

WORKLOAD_IDS = {"custom": 0, "tiny": 1, "llama_layer": 2, "h2o": 3, "rocket": 4, "mixed": 5}


@dataclass
class Workload:
    name: str
    n_seqs: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prompt_lens: list
    config_ids: list
    steps: int
    seed: int = 0
    boost_frac: float = 0.0
    boost: float = 1.0
    wid: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    def cfg(self, s):
        return config(int(self.config_ids[s]))


def _rng(seed, wid, kind, index=0):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wid, kind, index])))


def _h(x):
    return np.asarray(x, np.float32).astype(np.float16)


def make_workload(name, seed=0, config_ids=None, **kw):
    """Build one of the named workloads; keyword arguments override fields.

    tiny        1 seq, 4q/4kv x 64, prompt 512, 16 steps
    llama_layer 8 seqs, 32q/8kv x 128, prompt 4096, 128 steps
    h2o         8 seqs, 32q/8kv x 128, prompt 8192, 256 steps, boosted key rows
    rocket      4 seqs, 32q/8kv x 128, prompt 32768, 256 steps
    mixed       64 seqs, 32q/8kv x 128, prompts log-uniform in [1024, 32768],
                config drawn uniformly from the 11 rows, 128 steps
    custom      give every field explicitly
    """
    wid = WORKLOAD_IDS[name]
    if name == "tiny":
        base = dict(n_seqs=1, n_q_heads=4, n_kv_heads=4, head_dim=64, prompt_lens=[512], steps=16)
    elif name == "llama_layer":
        base = dict(n_seqs=8, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_lens=[4096] * 8,
                    steps=128)
    elif name == "h2o":
        base = dict(n_seqs=8, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_lens=[8192] * 8,
                    steps=256, boost_frac=0.05, boost=3.0)
    elif name == "rocket":
        base = dict(n_seqs=4, n_q_heads=32, n_kv_heads=8, head_dim=128, prompt_lens=[32768] * 4,
                    steps=256)
    elif name == "mixed":
        n = kw.pop("n_seqs", 64)
        r = _rng(seed, wid, _LENS)
        lens = np.rint(np.exp(r.uniform(np.log(1024.0), np.log(32768.0), size=n))).astype(int)
        cfgs = _rng(seed, wid, _CFG).integers(0, 11, size=n)
        base = dict(n_seqs=n, n_q_heads=32, n_kv_heads=8, head_dim=128,
                    prompt_lens=[int(x) for x in lens], steps=128)
        if config_ids is None:
            config_ids = [int(c) for c in cfgs]
    elif name == "custom":
        base = {}
    else:
        raise KeyError(name)
    base.update(kw)
    if config_ids is None:
        config_ids = [0] * base["n_seqs"]
    if isinstance(config_ids, (int, str)):
        config_ids = [config_ids] * base["n_seqs"]
    ids = [config(c)["id"] if isinstance(c, str) else int(c) for c in config_ids]
    return Workload(name=name, seed=seed, wid=wid, config_ids=ids, **base)


def key_sigma(wl, s):
    """Per-(kv head, channel) key scale of sequence s: lognormal(0, 0.5), 2 channels x 8."""
    sig = _rng(wl.seed, wl.wid, _SIGMA, s).lognormal(0.0, 0.5, size=(wl.n_kv_heads, wl.head_dim))
    r = _rng(wl.seed, wl.wid, _OUTCH, s)
    for h in range(wl.n_kv_heads):
        ch = r.choice(wl.head_dim, size=min(2, wl.head_dim), replace=False)
        sig[h, ch] *= 8.0
    return sig.astype(np.float32)


def _boost_rows(wl, kind, s, n):
    if wl.boost_frac <= 0.0:
        return None
    r = _rng(wl.seed, wl.wid, _BOOST, kind * 1_000_003 + s)
    return np.where(r.random(size=(n, wl.n_kv_heads)) < wl.boost_frac, wl.boost, 1.0).astype(np.float32)


def prompt_kv(wl, s):
    """Prompt keys and values of sequence s: two fp16 arrays [n0][Hkv][d]."""
    n0 = int(wl.prompt_lens[s])
    shape = (n0, wl.n_kv_heads, wl.head_dim)
    k = _rng(wl.seed, wl.wid, _KP, s).standard_normal(size=shape, dtype=np.float32)
    k *= key_sigma(wl, s)[None]
    b = _boost_rows(wl, 0, s, n0)
    if b is not None:
        k *= b[:, :, None]
    v = _rng(wl.seed, wl.wid, _VP, s).standard_normal(size=shape, dtype=np.float32)
    return _h(k), _h(v)


def prompt_q(wl, s, last=None):
    """Prompt queries of sequence s, fp16 [rows][Hq][d]: all n0 rows, or only the last `last`.

    Rows are drawn in fixed 256-row blocks, so row i has the same value whichever
    slice is asked for and a short tail is cheap to draw."""
    n0 = int(wl.prompt_lens[s])
    last = n0 if last is None else min(int(last), n0)
    row = wl.n_q_heads * wl.head_dim
    first = n0 - last
    blk0 = first // 256
    out = []
    for b in range(blk0, (n0 + 255) // 256):
        rb = _rng(wl.seed, wl.wid, _QP, (s << 20) + b)
        out.append(rb.standard_normal(size=(min(256, n0 - b * 256), row), dtype=np.float32))
    q = np.concatenate(out)[first - blk0 * 256:] if out else np.zeros((0, row), np.float32)
    return _h(q).reshape(last, wl.n_q_heads, wl.head_dim)


def step_inputs(wl, t):
    """Decode step t: (k_new [S][Hkv][d], v_new [S][Hkv][d], q [S][Hq][d]), fp16."""
    S, hk, hq, d = wl.n_seqs, wl.n_kv_heads, wl.n_q_heads, wl.head_dim
    r = _rng(wl.seed, wl.wid, _STEP, t)
    k = r.standard_normal(size=(S, hk, d), dtype=np.float32)
    v = r.standard_normal(size=(S, hk, d), dtype=np.float32)
    q = r.standard_normal(size=(S, hq, d), dtype=np.float32)
    for s in range(S):
        k[s] *= key_sigma(wl, s)
        b = _boost_rows(wl, 1 + t, s, 1)
        if b is not None:
            k[s] *= b[0][:, None]
    return _h(k), _h(v), _h(q)


def calib_kv(wl, tokens=1024):
    """Separate calibration draw (seed + 1000) for fitting KVQuant codebooks: fp16 [tokens][Hkv][d]."""
    cw = Workload(name=wl.name, n_seqs=1, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads,
                  head_dim=wl.head_dim, prompt_lens=[tokens], config_ids=[0], steps=0,
                  seed=wl.seed + 1000, wid=wl.wid)
    return prompt_kv(cw, 0)
