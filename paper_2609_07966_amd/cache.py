"""Torch-facing convenience over the C ABI: owns the arena tensor and marshals tensors to pointers.

PyTorch only provides device memory and the stream here; every step of the decode path runs in
libmkv's HIP kernels.
"""
import struct

from . import _lib as L


def _ptr(t):
    return 0 if t is None else int(t.data_ptr())


class KVCache:
    """One mixed-configuration KV cache (one attention layer's worth).

    shape: (n_seqs, n_q_heads, n_kv_heads, head_dim, max_new_tokens)
    cfgs:  per-sequence configuration dicts (workloads.configs rows)
    codebooks: flat 56 float32 values (b = 2, 3, 4: key then value codebook), or None
    """

    def __init__(self, shape, cfgs, prompt_lens, codebooks=None, device="cuda", stream=None):
        import torch
        self.torch = torch
        self.shape = tuple(int(x) for x in shape)
        self.S, self.Hq, self.Hkv, self.D, self.max_new = self.shape
        self.cfgs = [dict(c) for c in cfgs]
        self.prompt_lens = [int(x) for x in prompt_lens]
        self.nbytes = L.mkv_cache_bytes(self.shape, self.cfgs, self.prompt_lens)
        self.arena = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        base = self.arena.data_ptr()
        self.arena_ptr = (base + 255) & ~255
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.arena.device)
        self.h = L.mkv_cache_create(self.shape, self.cfgs, self.prompt_lens, codebooks, self.arena_ptr,
                                    self.nbytes, self.stream.cuda_stream)

    def close(self):
        if getattr(self, "h", None):
            L.mkv_cache_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def s(self):
        return self.stream.cuda_stream

    # ---- prefill -----------------------------------------------------------------------------
    def append_prompt(self, k, v):
        """k, v: device fp16 [sum prompt_len][Hkv][D] (sequences in order)."""
        cu = [0]
        for n in self.prompt_lens:
            cu.append(cu[-1] + n)
        L.mkv_append_quantize(self.h, _ptr(k), _ptr(v), cu, self.s)

    def h2o_prefill(self, q_prompt):
        L.mkv_h2o_update_evict(self.h, _ptr(q_prompt), self.s)

    def snap_prefill(self, q_window):
        L.mkv_snap_prefill_evict(self.h, _ptr(q_window), self.s)

    # ---- decode ------------------------------------------------------------------------------
    def append(self, k, v):
        L.mkv_append_quantize(self.h, _ptr(k), _ptr(v), list(range(self.S + 1)), self.s)

    def topk(self, q, pos_out=None):
        L.mkv_topk_select(self.h, _ptr(q), _ptr(pos_out), self.s)

    def attention(self, q, out):
        L.mkv_decode_attention(self.h, _ptr(q), _ptr(out), self.s)

    def evict(self):
        L.mkv_h2o_update_evict(self.h, 0, self.s)

    def step(self, k, v, q, out):
        L.mkv_decode_step(self.h, _ptr(k), _ptr(v), _ptr(q), _ptr(out), self.s)

    # ---- inspection --------------------------------------------------------------------------
    def export(self, seq, kv_head, what, dtype=None):
        import numpy as np
        raw = L.mkv_export(self.h, seq, kv_head, what)
        if dtype is None:
            dtype = {"codes_k": np.uint8, "codes_v": np.uint8, "scales_k": np.float32, "scales_v": np.float32,
                     "scores": np.float32}.get(what, np.int32)
        return np.frombuffer(raw, dtype=dtype).copy()

    def counts(self, seq, kv_head):
        return struct.unpack("4i", L.mkv_export(self.h, seq, kv_head, "counts"))

    def n_tiles(self):
        """-> (all attention tiles, tiles of uniform 4-bit sequences, tiles of RocketKV sequences)."""
        return L.mkv_attention_tiles(self.h)
