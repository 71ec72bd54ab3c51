"""Multi-step decode of one sequence under one compression configuration.

A decode step appends the new token's key and value to the cache, picks the
tokens to attend to, runs exact attention over their effective values, and
updates any eviction state (Section 2.1 describes each method; Table 1 lists
the configurations).  Query heads h*G .. h*G + G - 1 share kv head h.

``Sequence.step`` returns the float64 output [Hq][d] together with the
per-kv-head effective value rows attended over (for the RMS error normaliser).
The H2O and SnapKV decisions can be overridden from outside (``adopt_*``):
softmax-derived scores are not reproducible bit for bit across precisions, so a
harness may adopt another implementation's choice inside a declared tie band
and continue in lock step.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np

from . import h2o, kvquant, rocketkv, snapkv, uniform
from .attention import softmax_attention


class Sequence:
    def __init__(self, cfg, k_prompt, v_prompt, n_q_heads, q_prompt=None, codebooks=None, keep=None):
        """cfg: a configuration row (dict); k_prompt, v_prompt [n0][Hkv][d] fp16;
        q_prompt: [n0][Hq][d] (H2O) or at least the last `window` rows (RocketKV);
        codebooks: {bits: (cb_k, cb_v)} float32 ascending (KVQuant);
        keep: optional per-kv-head prefill keep-sets for H2O / RocketKV, adopted instead of
        scoring the prompt (H2O scores then start at 0) — for callers that time decode only."""
        self.cfg = dict(cfg)
        self.method = cfg["method"]
        self.kp = np.asarray(k_prompt)
        self.vp = np.asarray(v_prompt)
        self.n0, self.hkv, self.d = self.kp.shape
        self.hq = int(n_q_heads)
        self.G = self.hq // self.hkv
        self.p = self.n0                      # position of the next token
        m = self.method
        if m in ("fp16", "uq"):
            self.k = [self.kp[:, h].copy() for h in range(self.hkv)]   # fp16 token streams
            self.v = [self.vp[:, h].copy() for h in range(self.hkv)]
        elif m == "kvq":
            self._init_kvq(codebooks)
        elif m == "h2o":
            self.B, self.R = h2o.budget(cfg["budget_pct"], self.n0)
            self.heads = None
            if keep is not None:
                self.S = [np.zeros(self.n0) for _ in range(self.hkv)]
                self.adopt_h2o_prefill(keep)
            else:
                self.qp = np.asarray(q_prompt)
                self.S = [h2o.prefill_scores(self.qp[:, h * self.G:(h + 1) * self.G], self.kp[:, h])
                          for h in range(self.hkv)]
                self.adopt_h2o_prefill([h2o.prefill_keep(self.S[h], self.B, self.R)
                                        for h in range(self.hkv)])
        elif m == "rocket":
            self.T = snapkv.keep_budget(cfg, self.n0)
            self.w = int(cfg.get("window", 32))
            self.pool = int(cfg.get("pool", 7))
            self.nc = int(cfg.get("n_channels", 32))
            self.topk = rocketkv.default_topk(self.T, cfg.get("topk", 0))
            if keep is not None:
                self.adopt_snap_keep(keep)
            else:
                qw = np.asarray(q_prompt)[-min(self.w, self.n0):]
                self.qw = qw
                self.adopt_snap_keep([snapkv.snap_keep(qw[:, h * self.G:(h + 1) * self.G],
                                                       self.kp[:, h], self.T, self.w, self.pool)
                                      for h in range(self.hkv)])
        elif m != "fp16":
            raise ValueError(m)

    # ---- KVQuant ---------------------------------------------------------------------------
    def _init_kvq(self, codebooks):
        b = int(self.cfg["bits"])
        self.bp = int(self.cfg.get("outlier_bp", 100))
        self.cbk, self.cbv = (np.asarray(c, np.float32) for c in codebooks[b])
        self.tau, self.inv = [], []
        self.kq, self.vq = [], []         # per head dict of arrays over all tokens so far
        for h in range(self.hkv):
            tau, inv = kvquant.calibrate_keys(self.kp[:, h], self.bp)
            self.tau.append(tau)
            self.inv.append(inv)
            self.kq.append(self._kvq_k(self.kp[:, h], h))
            self.vq.append(self._kvq_v(self.vp[:, h]))

    def _kvq_k(self, rows, h):
        codes, out = kvquant.quantize_keys(rows, self.tau[h], self.inv[h], self.cbk, self.bp)
        eff = kvquant.dequantize_keys(rows, codes, out, self.tau[h], self.cbk)
        return {"codes": codes, "outlier": out, "eff": eff, "raw": np.asarray(rows)}

    def _kvq_v(self, rows):
        codes, s, out = kvquant.quantize_values(rows, self.cbv, self.bp)
        eff = kvquant.dequantize_values(rows, codes, out, s, self.cbv)
        return {"codes": codes, "outlier": out, "eff": eff, "scale": s, "raw": np.asarray(rows)}

    @staticmethod
    def _cat(a, b):
        return {key: np.concatenate([a[key], b[key]]) for key in a}

    # ---- eviction state adoption -------------------------------------------------------------
    def adopt_h2o_prefill(self, keeps):
        """Set the retained prompt positions of every kv head (ascending arrays)."""
        self.heads = []
        for h, keep in enumerate(keeps):
            keep = np.asarray(keep, np.int64)
            self.heads.append(h2o.H2OHead(keep, self.kp[keep, h], self.vp[keep, h],
                                          self.S[h][keep], self.B, self.R))

    def adopt_snap_keep(self, keeps):
        """Set the SnapKV-retained prompt positions of every kv head (ascending arrays)."""
        self.keep = [np.asarray(k, np.int64) for k in keeps]
        self.rk = [self.kp[k, h].copy() for h, k in enumerate(self.keep)]
        self.rv = [self.vp[k, h].copy() for h, k in enumerate(self.keep)]
        self.rpos = [k.copy() for k in self.keep]

    # ---- one decode step -------------------------------------------------------------------
    def step(self, k_new, v_new, q):
        """k_new, v_new [Hkv][d] fp16, q [Hq][d] fp16 -> (out [Hq][d] float64, info)."""
        G, d = self.G, self.d
        out = np.zeros((self.hq, d))
        info = {"v_eff": [], "selected": [], "evict": []}
        p = self.p
        for h in range(self.hkv):
            qh = np.asarray(q[h * G:(h + 1) * G])
            m = self.method
            if m == "fp16":
                self.k[h] = np.vstack([self.k[h], k_new[h][None]])
                self.v[h] = np.vstack([self.v[h], v_new[h][None]])
                kk, vv = self.k[h].astype(np.float64), self.v[h].astype(np.float64)
            elif m == "uq":
                self.k[h] = np.vstack([self.k[h], k_new[h][None]])
                self.v[h] = np.vstack([self.v[h], v_new[h][None]])
                b, g = int(self.cfg.get("bits", 4)), int(self.cfg.get("group", 64))
                kk = uniform.effective_keys(self.k[h], b, g)
                vv = uniform.effective_values(self.v[h], b, g)
            elif m == "kvq":
                self.kq[h] = self._cat(self.kq[h], self._kvq_k(k_new[h][None], h))
                self.vq[h] = self._cat(self.vq[h], self._kvq_v(v_new[h][None]))
                kk, vv = self.kq[h]["eff"], self.vq[h]["eff"]
            elif m == "h2o":
                hd = self.heads[h]
                out[h * G:(h + 1) * G] = hd.attend(k_new[h], v_new[h], qh, p)
                info["v_eff"].append(hd.v.copy())
                info["evict"].append(hd.choose_eviction(p))
                continue
            elif m == "rocket":
                self.rk[h] = np.vstack([self.rk[h], k_new[h][None]])
                self.rv[h] = np.vstack([self.rv[h], v_new[h][None]])
                self.rpos[h] = np.append(self.rpos[h], p)
                ch = rocketkv.select_channels(qh, self.nc)
                sh = rocketkv.approx_scores(qh, self.rk[h], ch)
                sel = rocketkv.topk_indices(sh, self.topk)
                info["selected"].append({"channels": ch, "slots": sel, "positions": self.rpos[h][sel],
                                         "scores": sh})
                kk = self.rk[h][sel].astype(np.float64)
                vv = self.rv[h][sel].astype(np.float64)
            o, _ = softmax_attention(qh.astype(np.float64), kk, vv)
            out[h * G:(h + 1) * G] = o
            info["v_eff"].append(vv)
        self.p += 1
        return out, info

    def apply_evictions(self, positions):
        """H2O: evict the given position per kv head (None = nothing)."""
        for h, pos in enumerate(positions):
            if pos is not None:
                self.heads[h].evict(pos)
