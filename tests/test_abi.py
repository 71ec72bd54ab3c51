"""Host-side checks of the C ABI that need no GPU: the library loads, exports every declared
symbol, validates shapes and configurations, sizes arenas, and fits codebooks on the host
exactly as the oracle does."""
import os
import re

import numpy as np
import pytest

from workloads import CONFIGS, calib_kv, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2609_07966_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_07966_amd import build
        build.build()
    _lib.lib()
    return _lib


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "mkv.h")).read()
    return sorted(set(re.findall(r"^\s*(?:mkv_status|const char \*)\s*(mkv_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(L):
    import ctypes
    h = ctypes.CDLL(L.LIB_PATH)
    syms = declared_symbols()
    assert len(syms) >= 15
    for s in syms:
        assert hasattr(h, s), s
    assert set(syms) == set(L.SYMBOLS)


def _shape(S=2, Hq=8, Hkv=2, D=128, mn=16):
    return (S, Hq, Hkv, D, mn)


def test_cache_bytes_for_every_config(L):
    sizes = {}
    for row in CONFIGS:
        sizes[row["name"]] = L.mkv_cache_bytes(_shape(S=1), [row], [4096])
        assert sizes[row["name"]] > 0
    # compressed caches are smaller than the fp16 one, in bit order
    assert sizes["KVQ2"] < sizes["KVQ3"] < sizes["KVQ4"] < sizes["FP16"]
    assert sizes["UQ4-g64"] < sizes["FP16"]
    # the mixed batch of the paper-shaped workload fits easily in one GPU's memory
    wl = make_workload("mixed")
    total = L.mkv_cache_bytes((wl.n_seqs, 32, 8, 128, 128), [wl.cfg(s) for s in range(wl.n_seqs)], wl.prompt_lens)
    assert total < 40 << 30


@pytest.mark.parametrize("shape,cfg,plen,status", [
    ((1, 6, 4, 128, 8), {"method": "fp16"}, 10, 1),        # Hq % Hkv != 0
    ((1, 48, 4, 128, 8), {"method": "fp16"}, 10, 5),       # G = 12 unsupported
    ((1, 8, 2, 96, 8), {"method": "fp16"}, 10, 5),         # head_dim 96 unsupported
    ((1, 8, 2, 128, 8), {"method": "fp16"}, 0, 1),         # empty prompt
    ((1, 8, 2, 128, 8), {"method": "kvq", "bits": 5, "outlier_bp": 100}, 10, 1),
    ((1, 8, 2, 128, 8), {"method": "kvq", "bits": 4, "outlier_bp": 9000}, 10, 1),
    ((1, 8, 2, 128, 8), {"method": "uq", "bits": 2, "group": 64}, 10, 5),
    ((1, 8, 2, 128, 8), {"method": "h2o", "budget_pct": 10}, 5, 1),   # budget rounds to 0 tokens
    ((1, 8, 2, 128, 8), {"method": "rocket", "keep_tokens": 16, "window": 32, "pool": 7,
                         "n_channels": 32}, 100, 1),                  # keep < window
    ((1, 8, 2, 128, 8), {"method": "rocket", "keep_tokens": 64, "window": 32, "pool": 6,
                         "n_channels": 32}, 100, 1),                  # even pool
    ((1, 8, 2, 64, 8), {"method": "rocket", "keep_tokens": 64, "window": 32, "pool": 7,
                        "n_channels": 65}, 100, 1),                   # more channels than head_dim
])
def test_validation_errors(L, shape, cfg, plen, status):
    with pytest.raises(L.MkvError) as e:
        L.mkv_cache_bytes(shape, [cfg], [plen])
    assert e.value.status == status
    assert L.lib().mkv_last_error().decode() != ""


def test_arena_grows_with_context_and_steps(L):
    a = L.mkv_cache_bytes(_shape(S=1, mn=16), [CONFIGS[0]], [1000])
    b = L.mkv_cache_bytes(_shape(S=1, mn=16), [CONFIGS[0]], [2000])
    c = L.mkv_cache_bytes(_shape(S=1, mn=64), [CONFIGS[0]], [1000])
    assert a < b and a < c
    # the H2O decode region is the budget, but the prompt is staged for prefill scoring
    h = L.mkv_cache_bytes(_shape(S=1), [CONFIGS[6]], [8192])
    f = L.mkv_cache_bytes(_shape(S=1), [CONFIGS[0]], [8192])
    assert h > 0 and f > 0


@pytest.mark.parametrize("buf,nbytes,sink,reps", [
    (0, 1 << 18, 4096, 1),          # NULL buffer
    (4096, 1 << 18, 0, 1),          # NULL sink
    (4096, (1 << 18) + 16, 4096, 1),  # not a multiple of 256 KiB
    (4096, 0, 4096, 1),             # empty
    (4096, 1 << 18, 4096, 0),       # no timed pass
])
def test_read_probe_validation(L, buf, nbytes, sink, reps):
    # rejected on the host before any device work (the pointers are never dereferenced)
    with pytest.raises(L.MkvError) as e:
        L.mkv_probe_read_bandwidth(buf, nbytes, sink, reps)
    assert e.value.status == 1


def test_status_strings(L):
    for s in range(7):
        assert L.lib().mkv_status_str(s)
    assert L.lib().mkv_status_str(99) == b"unknown status"


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_host_codebook_fit_equals_oracle(L, bits):
    """The library's host codebook fit reproduces the oracle's Lloyd fit on the same draw."""
    from oracle import codebook, kvquant
    wl = make_workload("custom", n_seqs=1, n_q_heads=8, n_kv_heads=2, head_dim=64, prompt_lens=[1],
                       steps=0, config_ids=[0])
    k, v = calib_kv(wl, tokens=256)
    ks = np.concatenate([kvquant.normalised_inliers_keys(k[:, h], 100) for h in range(2)])
    vs = np.concatenate([kvquant.normalised_inliers_values(v[:, h], 100) for h in range(2)])
    ref_k = codebook.lloyd_codebook(ks, bits)
    ref_v = codebook.lloyd_codebook(vs, bits)
    got_k, got_v = L.mkv_fit_codebooks(k.tobytes(), v.tobytes(), 256, 2, 64, bits, 100)
    np.testing.assert_array_equal(np.array(got_k, np.float32), ref_k)
    np.testing.assert_array_equal(np.array(got_v, np.float32), ref_v)


def test_create_rejects_short_arena_and_bad_codebooks_on_the_host(L):
    """mkv_cache_create checks the arena and the codebooks before any device work, so these
    rejections need no GPU (the fake arena address is never dereferenced)."""
    cfgs = [CONFIGS[0], CONFIGS[3]]
    shape = _shape(S=2, mn=4)
    need = L.mkv_cache_bytes(shape, cfgs, [300, 400])
    cb = []
    for b in (2, 3, 4):
        grid = np.linspace(-1, 1, 1 << b).astype(np.float16).astype(np.float32).tolist()
        cb += grid + grid
    fake = 1 << 40

    def status(codebooks, nbytes=need, ptr=fake):
        with pytest.raises(L.MkvError) as e:
            L.mkv_cache_create(shape, cfgs, [300, 400], codebooks, ptr, nbytes, 0)
        return e.value.status

    assert status(cb, need - 1) == 2
    assert status(cb, need, fake + 64) == 1
    assert status(None) == 1
    bad = list(cb)
    bad[5] += 1e-4
    assert status(bad) == 1
    desc = list(cb)
    desc[8], desc[9] = desc[9], desc[8]
    assert status(desc) == 1


def test_fit_codebooks_reports_its_errors(L):
    with pytest.raises(L.MkvError) as e:
        L.mkv_fit_codebooks(b"\0" * 256, b"\0" * 256, 2, 1, 64, 9, 100)
    assert e.value.status == 1 and "bits" in L.lib().mkv_last_error().decode()
