"""ctypes binding of libmkv (include/mkv.h): the same entry points, argument marshalling only.

Device memory and streams are passed as integers (raw pointers / hipStream_t).  Every compute
step runs in the library's HIP kernels; if the library is missing this module raises at import
of ``lib()`` rather than falling back to anything else.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("MKV_LIB", os.path.join(_HERE, "libmkv.so"))

METHODS = {"fp16": 0, "uq": 1, "kvq": 2, "h2o": 3, "rocket": 4}

EXPORT = {
    "counts": 0, "positions": 1, "codes_k": 2, "codes_v": 3, "outliers_k": 4, "outliers_v": 5,
    "scales_k": 6, "scales_v": 7, "scores": 8, "topk": 9, "channels": 10,
}

PROFILE_KINDS = {"partial": 0, "combine": 1, "append": 2, "topk": 3, "append_score": 4}


class mkv_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("method", "bits", "group", "outlier_bp", "budget_pct",
                                              "keep_tokens", "window", "pool", "topk", "n_channels",
                                              "keep_ratio")]


class mkv_candidate(ctypes.Structure):
    _fields_ = [("method", ctypes.c_int32), ("level", ctypes.c_int32), ("latency", ctypes.c_double),
                ("memory", ctypes.c_double), ("p_correct", ctypes.c_double)]


class mkv_shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_seqs", "n_q_heads", "n_kv_heads", "head_dim",
                                              "max_new_tokens")]


class MkvError(RuntimeError):
    def __init__(self, status, text):
        super().__init__(f"mkv status {status}: {text}")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int32
_SIGS = {
    "mkv_status_str": (ctypes.c_char_p, [_I]),
    "mkv_last_error": (ctypes.c_char_p, []),
    "mkv_cache_bytes": (_I, [ctypes.POINTER(mkv_shape), ctypes.POINTER(mkv_config), ctypes.POINTER(_I),
                             ctypes.POINTER(ctypes.c_size_t)]),
    "mkv_cache_create": (_I, [ctypes.POINTER(mkv_shape), ctypes.POINTER(mkv_config), ctypes.POINTER(_I),
                              ctypes.POINTER(ctypes.c_float), _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)]),
    "mkv_cache_destroy": (_I, [_P]),
    "mkv_append_quantize": (_I, [_P, _P, _P, ctypes.POINTER(_I), _P]),
    "mkv_h2o_update_evict": (_I, [_P, _P, _P]),
    "mkv_snap_prefill_evict": (_I, [_P, _P, _P]),
    "mkv_topk_select": (_I, [_P, _P, _P, _P]),
    "mkv_decode_attention": (_I, [_P, _P, _P, _P]),
    "mkv_decode_attention_noalloc": (_I, [_P, _P, _P, _P]),
    "mkv_decode_step": (_I, [_P, _P, _P, _P, _P, _P]),
    "mkv_export": (_I, [_P, _I, _I, _I, _P, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]),
    "mkv_fit_codebooks": (_I, [_P, _P, _I, _I, _I, _I, _I, ctypes.POINTER(ctypes.c_float),
                               ctypes.POINTER(ctypes.c_float)]),
    "mkv_profile_enable": (_I, [_P, _I, _I]),
    "mkv_profile_read": (_I, [_P, _I, ctypes.POINTER(_I), ctypes.POINTER(ctypes.c_double)]),
    "mkv_attention_tiles": (_I, [_P, ctypes.POINTER(_I), ctypes.POINTER(_I), ctypes.POINTER(_I)]),
    "mkv_select_config": (_I, [ctypes.POINTER(mkv_candidate), _I, ctypes.c_double, ctypes.c_double,
                               ctypes.POINTER(_I), ctypes.POINTER(_I)]),
    "mkv_kv_memory": (_I, [ctypes.POINTER(mkv_shape), ctypes.POINTER(mkv_config), _I, _I,
                           ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]),
    "mkv_probe_read_bandwidth": (_I, [_P, ctypes.c_size_t, _P, _I, ctypes.POINTER(ctypes.c_double), _P]),
}
SYMBOLS = tuple(_SIGS)


def lib():
    """Load libmkv.so (built by ``paper_2609_07966_amd.build``); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libmkv.so not found at {LIB_PATH}; run paper_2609_07966_amd.build.build()")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def _check(status):
    if status != 0:
        L = lib()
        raise MkvError(status, f"{L.mkv_status_str(status).decode()}: {L.mkv_last_error().decode()}")


def make_config(row):
    """A configuration dict (see workloads.configs) -> mkv_config."""
    c = mkv_config()
    c.method = METHODS[row["method"]]
    c.bits = int(row.get("bits", 0))
    c.group = int(row.get("group", 0))
    c.outlier_bp = int(row.get("outlier_bp", 0))
    c.budget_pct = int(row.get("budget_pct", 0))
    c.keep_tokens = int(row.get("keep_tokens", 0))
    c.window = int(row.get("window", 0))
    c.pool = int(row.get("pool", 0))
    c.topk = int(row.get("topk", 0))
    c.n_channels = int(row.get("n_channels", 0))
    c.keep_ratio = int(row.get("keep_ratio", 0))
    return c


def _arrays(shape, cfgs, prompt_lens):
    sh = mkv_shape(*[int(x) for x in shape])
    n = sh.n_seqs
    ca = (mkv_config * n)(*[make_config(r) if isinstance(r, dict) else r for r in cfgs])
    pl = (_I * n)(*[int(x) for x in prompt_lens])
    return sh, ca, pl


def mkv_cache_bytes(shape, cfgs, prompt_lens):
    """shape = (n_seqs, n_q_heads, n_kv_heads, head_dim, max_new_tokens)."""
    sh, ca, pl = _arrays(shape, cfgs, prompt_lens)
    out = ctypes.c_size_t()
    _check(lib().mkv_cache_bytes(ctypes.byref(sh), ca, pl, ctypes.byref(out)))
    return out.value


def mkv_cache_create(shape, cfgs, prompt_lens, codebooks, arena_ptr, arena_bytes, stream):
    sh, ca, pl = _arrays(shape, cfgs, prompt_lens)
    cb = None
    if codebooks is not None:
        flat = [float(x) for x in codebooks]
        cb = (ctypes.c_float * len(flat))(*flat)
    h = _P()
    _check(lib().mkv_cache_create(ctypes.byref(sh), ca, pl, cb, _P(arena_ptr), arena_bytes, _P(stream),
                                  ctypes.byref(h)))
    return h


def mkv_cache_destroy(h):
    _check(lib().mkv_cache_destroy(h))


def mkv_append_quantize(h, k_ptr, v_ptr, cu_new, stream):
    cu = (_I * len(cu_new))(*[int(x) for x in cu_new])
    _check(lib().mkv_append_quantize(h, _P(k_ptr), _P(v_ptr), cu, _P(stream)))


def mkv_h2o_update_evict(h, q_prompt_ptr, stream):
    _check(lib().mkv_h2o_update_evict(h, _P(q_prompt_ptr) if q_prompt_ptr else None, _P(stream)))


def mkv_snap_prefill_evict(h, q_window_ptr, stream):
    _check(lib().mkv_snap_prefill_evict(h, _P(q_window_ptr) if q_window_ptr else None, _P(stream)))


def mkv_topk_select(h, q_ptr, pos_out_ptr, stream):
    _check(lib().mkv_topk_select(h, _P(q_ptr), _P(pos_out_ptr) if pos_out_ptr else None, _P(stream)))


def mkv_decode_attention(h, q_ptr, out_ptr, stream):
    _check(lib().mkv_decode_attention(h, _P(q_ptr), _P(out_ptr), _P(stream)))


def mkv_decode_attention_noalloc(h, q_ptr, out_ptr, stream):
    _check(lib().mkv_decode_attention_noalloc(h, _P(q_ptr), _P(out_ptr), _P(stream)))


def mkv_decode_step(h, k_ptr, v_ptr, q_ptr, out_ptr, stream):
    _check(lib().mkv_decode_step(h, _P(k_ptr), _P(v_ptr), _P(q_ptr), _P(out_ptr), _P(stream)))


def mkv_export(h, seq, kv_head, what, cap=1 << 26):
    """Returns the exported bytes."""
    buf = ctypes.create_string_buffer(cap)
    n = ctypes.c_size_t()
    _check(lib().mkv_export(h, int(seq), int(kv_head), EXPORT.get(what, what), buf, cap, ctypes.byref(n)))
    return buf.raw[:n.value]


def mkv_fit_codebooks(k_bytes, v_bytes, n_tokens, n_kv_heads, head_dim, bits, outlier_bp):
    """k_bytes, v_bytes: host fp16 buffers [n_tokens][n_kv_heads][head_dim] (bytes-like)."""
    nc = 1 << int(bits)
    a, b = (ctypes.c_float * nc)(), (ctypes.c_float * nc)()
    kb = ctypes.create_string_buffer(bytes(k_bytes), len(k_bytes))
    vb = ctypes.create_string_buffer(bytes(v_bytes), len(v_bytes))
    _check(lib().mkv_fit_codebooks(kb, vb, int(n_tokens), int(n_kv_heads), int(head_dim), int(bits),
                                   int(outlier_bp), a, b))
    return list(a), list(b)


def mkv_profile_enable(h, enable, max_launches):
    """enable: mask of PROFILE_KINDS values to time (bit k = kind k), 0 = off."""
    _check(lib().mkv_profile_enable(h, int(enable), int(max_launches)))


def mkv_profile_read(h, kind):
    n, ms = _I(), ctypes.c_double()
    _check(lib().mkv_profile_read(h, PROFILE_KINDS.get(kind, kind), ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


def mkv_probe_read_bandwidth(buf_ptr, nbytes, sink_ptr, reps, stream=0):
    """Best single-pass read rate (GB/s) of a plain streaming kernel over a device buffer."""
    g = ctypes.c_double()
    _check(lib().mkv_probe_read_bandwidth(buf_ptr, nbytes, sink_ptr, reps, ctypes.byref(g), stream))
    return g.value


def mkv_kv_memory(shape, cfg, prompt_len, n_generated):
    """-> (resident, peak) KV-cache bytes of one sequence (host only)."""
    sh = mkv_shape(*[int(x) for x in shape])
    c = make_config(cfg)
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().mkv_kv_memory(ctypes.byref(sh), ctypes.byref(c), int(prompt_len), int(n_generated),
                               ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def mkv_select_config(cands, l_max, m_max):
    """cands: sequence of (method name, level, latency, memory, p_correct).
    -> (chosen index, violated flag)."""
    arr = (mkv_candidate * len(cands))(*[mkv_candidate(METHODS[m], int(lv), float(l), float(mem), float(p))
                                         for m, lv, l, mem, p in cands])
    ch, vi = _I(), _I()
    _check(lib().mkv_select_config(arr, len(cands), float(l_max), float(m_max), ctypes.byref(ch), ctypes.byref(vi)))
    return ch.value, bool(vi.value)


def mkv_attention_tiles(h):
    """-> (all partial tiles, tiles of uniform 4-bit sequences, tiles of RocketKV sequences)."""
    n, n_uq, n_rk = _I(), _I(), _I()
    _check(lib().mkv_attention_tiles(h, ctypes.byref(n), ctypes.byref(n_uq), ctypes.byref(n_rk)))
    return n.value, n_uq.value, n_rk.value
