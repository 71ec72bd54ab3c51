"""GPU parity: every configuration through the C ABI against the CPU oracle, in lock step.

Sizes are chosen so the oracle finishes in seconds while the GPU path spans several attention
tiles and ragged tails (prompt lengths that are not multiples of 64 or of the tile size)."""
import numpy as np
import pytest

from workloads import make_workload

pytestmark = pytest.mark.gpu


def _run(wl, steps, check_codes=True, fused=False):
    """fused: drive the cache by mkv_decode_step (append and top-k in one launch) instead of the
    separate calls."""
    from gpu_harness import Run, log
    log(f"[parity] {wl.name} S={wl.n_seqs} Hq={wl.n_q_heads} Hkv={wl.n_kv_heads} d={wl.head_dim} "
        f"prompts={wl.prompt_lens} cfgs={wl.config_ids} steps={steps} fused={fused}")
    r = Run(wl, steps, fused=fused).run(check_codes=check_codes)
    log(f"[parity]   max normalised error {r.max_err:.2e}, near-ties adopted {r.near_ties}")
    return r


@pytest.fixture(autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import sys, os
    sys.path.insert(0, os.path.dirname(__file__))
    from paper_2609_07966_amd import _lib
    _lib.lib()


@pytest.mark.parametrize("cfg", ["FP16", "UQ4-g64"])
def test_tiny_decode(cfg):
    _run(make_workload("tiny", config_ids=cfg), 16)


def test_llama_shaped_fp16_and_kvquant():
    wl = make_workload("custom", seed=3, n_seqs=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[1000, 777, 1500, 64], steps=8,
                       config_ids=["FP16", "KVQ4", "KVQ3", "KVQ2"])
    _run(wl, 8)


def test_kvquant_all_bits_ragged():
    wl = make_workload("custom", seed=4, n_seqs=3, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[2500, 333, 1029], steps=70, config_ids=["KVQ2", "KVQ3", "KVQ4"])
    _run(wl, 70)


def test_uniform_block_boundaries():
    # prompts end just before, at and after a 64-token block boundary; 70 steps cross more
    wl = make_workload("custom", seed=5, n_seqs=3, n_q_heads=16, n_kv_heads=4, head_dim=128,
                       prompt_lens=[63, 128, 1001], steps=70, config_ids=["UQ4-g64"] * 3)
    _run(wl, 70)


def test_h2o_evictions():
    wl = make_workload("custom", seed=6, n_seqs=3, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[600, 901, 1200], steps=40, config_ids=["H2O-20", "H2O-50", "H2O-10"],
                       boost_frac=0.05, boost=3.0)
    _run(wl, 40)


@pytest.mark.parametrize("fused", [False, True])
def test_rocket_prefill_and_topk(fused):
    wl = make_workload("custom", seed=7, n_seqs=2, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[3000, 2100], steps=10, config_ids=["Rocket-1024", "Rocket-2048"])
    _run(wl, 10, fused=fused)


def test_rocket_large_retained_sets():
    # retained sets past 4 x 1024 tokens (a lane scores 8 tokens) and past the 10240 score keys
    # the top-k holds in LDS (keys in the global scratch), through the fused append and top-k
    wl = make_workload("custom", seed=18, n_seqs=2, n_q_heads=4, n_kv_heads=1, head_dim=64,
                       prompt_lens=[12000, 6000], steps=4, config_ids=[0, 0])
    wl.config_ids = [8, 8]
    cfgs = [{"id": 8, "name": "Rocket-11000", "method": "rocket", "keep_tokens": 11000, "window": 32, "pool": 7,
             "topk": 0, "n_channels": 16},
            {"id": 8, "name": "Rocket-5000", "method": "rocket", "keep_tokens": 5000, "window": 32, "pool": 7,
             "topk": 0, "n_channels": 32}]
    wl.cfg = lambda s: dict(cfgs[s])
    _run(wl, 4, fused=True)


def test_mixed_batch_every_config():
    r = np.random.default_rng(8)
    lens = [int(x) for x in np.rint(np.exp(r.uniform(np.log(200), np.log(3000), 11)))]
    wl = make_workload("custom", seed=8, n_seqs=11, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=lens, steps=6, config_ids=list(range(11)))
    _run(wl, 6, fused=True)


@pytest.mark.parametrize("hq,hkv,d", [(32, 4, 64), (8, 8, 128), (16, 8, 64)])
def test_mixed_other_head_shapes(hq, hkv, d):
    wl = make_workload("custom", seed=9, n_seqs=6, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                       prompt_lens=[700, 1300, 257, 900, 2050, 600], steps=5,
                       config_ids=["FP16", "KVQ3", "UQ4-g64", "H2O-20", "Rocket-1024", "KVQ2"])
    _run(wl, 5, fused=True)


def test_edge_cases():
    # one-token prompt (fp16); prompt shorter than the window and than the keep budget (RocketKV
    # keeps everything, top-k covers everything -> dense); H2O budget above prompt + steps (dense)
    wl = make_workload("custom", seed=10, n_seqs=4, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[1, 20, 500, 300], steps=12, config_ids=[0, 0, 0, 0])
    wl.config_ids = [0, 8, 8, 5]
    cfgs = [{"id": 0, "name": "FP16", "method": "fp16"},
            {"id": 8, "name": "Rocket", "method": "rocket", "keep_tokens": 1024, "window": 32, "pool": 7,
             "topk": 0, "n_channels": 32},
            {"id": 8, "name": "Rocket-dense", "method": "rocket", "keep_tokens": 256, "window": 32, "pool": 7,
             "topk": 4096, "n_channels": 32},
            {"id": 5, "name": "H2O-dense", "method": "h2o", "budget_pct": 1000}]
    wl.cfg = lambda s: dict(cfgs[s])
    _run(wl, 12, fused=True)


def test_kvquant_without_outliers():
    # outlier_bp = 0: no outliers anywhere, every value from its code (and no key-outlier pool to
    # fill); ragged prompts so that the decode tokens cross 4-token value blocks
    wl = make_workload("custom", seed=12, n_seqs=3, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[300, 517, 129], steps=10, config_ids=[0, 0, 0])
    wl.config_ids = [2, 3, 4]
    cfgs = [{"id": 2, "name": "KVQ4-no-outliers", "method": "kvq", "bits": 4, "outlier_bp": 0},
            {"id": 3, "name": "KVQ3-no-outliers", "method": "kvq", "bits": 3, "outlier_bp": 0},
            {"id": 4, "name": "KVQ2", "method": "kvq", "bits": 2, "outlier_bp": 100}]
    wl.cfg = lambda s: dict(cfgs[s])
    _run(wl, 10)


def test_kvquant_large_outlier_budgets():
    # several value outliers per token (outlier_bp 500 at d = 128: 6 per token) and about 3-6 key
    # outliers per token: the multi-entry paths of the append and the attention
    wl = make_workload("custom", seed=13, n_seqs=3, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[400, 233, 650], steps=10, config_ids=[0, 0, 0])
    wl.config_ids = [2, 3, 4]
    cfgs = [{"id": 2, "name": "KVQ4-5%", "method": "kvq", "bits": 4, "outlier_bp": 500},
            {"id": 3, "name": "KVQ3-3%", "method": "kvq", "bits": 3, "outlier_bp": 300},
            {"id": 4, "name": "KVQ2-2.5%", "method": "kvq", "bits": 2, "outlier_bp": 250}]
    wl.cfg = lambda s: dict(cfgs[s])
    _run(wl, 10)


def test_small_budgets_and_selections():
    # H2O budgets of a few tokens (B = 3 and 1: eviction from the first decode step on; with
    # B = 1 the recent part R = floor(B / 2) is empty); RocketKV with a top-k of 8
    wl = make_workload("custom", seed=14, n_seqs=3, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[300, 150, 700], steps=12, config_ids=[0, 0, 0])
    wl.config_ids = [5, 5, 8]
    cfgs = [{"id": 5, "name": "H2O-1%", "method": "h2o", "budget_pct": 1},
            {"id": 5, "name": "H2O-B1", "method": "h2o", "budget_pct": 1},
            {"id": 8, "name": "Rocket-top8", "method": "rocket", "keep_tokens": 64, "window": 32, "pool": 7,
             "topk": 8, "n_channels": 32}]
    wl.cfg = lambda s: dict(cfgs[s])
    _run(wl, 12, fused=True)


def test_tiny_prompts_quantized():
    # prompts of 1, 2 and 5 tokens under the quantizers (KVQuant calibrates its key thresholds on
    # a handful of rows; uniform 4-bit starts with every key in the fp16 residual) and H2O
    # (B = 1 at 5 prompt tokens); 9 steps complete the first 4-token value blocks
    wl = make_workload("custom", seed=15, n_seqs=4, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       prompt_lens=[1, 2, 5, 5], steps=9, config_ids=["KVQ4", "UQ4-g64", "KVQ2", "H2O-20"])
    _run(wl, 9)


def test_paper_grid_settings():
    # the paper's own settings (Table 1) beyond the benchmark grid: H2O at 40 % and 60 % of the
    # prompt, and RocketKV at 8x, 16x and 32x compression of each prompt (keep prompt_len / r
    # tokens, at least the window); lock step against the oracle
    wl = make_workload("custom", seed=17, n_seqs=5, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[900, 1300, 3000, 2500, 4100], steps=6,
                       config_ids=["H2O-40", "H2O-60", "Rocket-8x", "Rocket-16x", "Rocket-32x"],
                       boost_frac=0.05, boost=3.0)
    _run(wl, 6, fused=True)


@pytest.mark.parametrize("hq,n0", [(4, 13001), (8, 7001)])
def test_h2o_large_retained_sets(hq, n0):
    # H2O-50 with one kv head of d = 64: B = 6500 (G = 4) and 3500 (G = 8) retained slots, more
    # than the combine pass scores in one round of its workgroup (6144 and 3072 slots), so the
    # score accumulation and the victim search also run their later rounds
    wl = make_workload("custom", seed=16, n_seqs=1, n_q_heads=hq, n_kv_heads=1, head_dim=64,
                       prompt_lens=[n0], steps=4, config_ids=["H2O-50"], boost_frac=0.05, boost=3.0)
    _run(wl, 4)


def test_batch_invariance():
    """Every sequence of a mixed batch gets exactly (bit for bit) the outputs, codes, selections
    and evictions of its solo run: the ragged launch shares no arithmetic between sequences."""
    import torch
    from gpu_harness import log, oracle_codebooks
    from paper_2609_07966_amd.cache import KVCache
    from workloads import prompt_kv, prompt_q, step_inputs
    wl = make_workload("custom", seed=11, n_seqs=6, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[1500, 700, 2100, 1300, 1800, 900], steps=6,
                       config_ids=["FP16", "UQ4-g64", "KVQ3", "H2O-20", "Rocket-1024", "KVQ2"])
    steps, S, Hkv = 6, wl.n_seqs, wl.n_kv_heads
    _, flat = oracle_codebooks(wl)
    cfgs = [wl.cfg(s) for s in range(S)]
    prompts = [prompt_kv(wl, s) for s in range(S)]
    ins = [step_inputs(wl, t) for t in range(steps)]

    def h(x):
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()

    def run(seqs):
        log(f"[parity] batch invariance: sequences {seqs}")
        c = KVCache((len(seqs), wl.n_q_heads, Hkv, wl.head_dim, steps), [cfgs[s] for s in seqs],
                    [wl.prompt_lens[s] for s in seqs], codebooks=list(flat))
        c.append_prompt(h(np.concatenate([prompts[s][0] for s in seqs])),
                        h(np.concatenate([prompts[s][1] for s in seqs])))
        hq = [prompt_q(wl, s) for s in seqs if cfgs[s]["method"] == "h2o"]
        if hq:
            c.h2o_prefill(h(np.concatenate(hq)))
        rq = [prompt_q(wl, s, last=32) for s in seqs if cfgs[s]["method"] == "rocket"]
        if rq:
            c.snap_prefill(h(np.concatenate(rq)))
        out = torch.empty((len(seqs), wl.n_q_heads, wl.head_dim), dtype=torch.float32, device="cuda")
        res = {s: {"out": []} for s in seqs}
        for t in range(steps):
            kn, vn, q = ins[t]
            c.append(h(kn[seqs]), h(vn[seqs]))
            c.topk(h(q[seqs]))
            c.attention(h(q[seqs]), out)
            o = out.cpu().numpy()
            for i, s in enumerate(seqs):
                res[s]["out"].append(o[i].copy())
                if cfgs[s]["method"] == "rocket":
                    res[s][("topk", t)] = [c.export(i, hh, "topk") for hh in range(Hkv)]
            c.evict()
        for i, s in enumerate(seqs):
            for what in ("positions", "codes_k", "codes_v", "scores"):
                if what == "scores" and cfgs[s]["method"] != "h2o":
                    continue
                if what.startswith("codes") and cfgs[s]["method"] not in ("kvq", "uq"):
                    continue
                res[s][what] = [c.export(i, hh, what) for hh in range(Hkv)]
        c.close()
        return res

    batch = run(list(range(S)))
    for s in range(S):
        solo = run([s])[s]
        for key, val in solo.items():
            for a, b in zip(batch[s][key], val):
                np.testing.assert_array_equal(a, b, err_msg=f"sequence {s} ({cfgs[s]['name']}): {key}")
