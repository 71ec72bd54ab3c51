"""GPU parity: every configuration through the C ABI against the CPU oracle, in lock step.

Sizes are chosen so the oracle finishes in seconds while the GPU path spans several attention
tiles and ragged tails (prompt lengths that are not multiples of 64 or of the tile size)."""
import numpy as np
import pytest

from workloads import make_workload

pytestmark = pytest.mark.gpu


def _run(wl, steps, check_codes=True):
    from gpu_harness import Run, log
    log(f"[parity] {wl.name} S={wl.n_seqs} Hq={wl.n_q_heads} Hkv={wl.n_kv_heads} d={wl.head_dim} "
        f"prompts={wl.prompt_lens} cfgs={wl.config_ids} steps={steps}")
    r = Run(wl, steps).run(check_codes=check_codes)
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


def test_rocket_prefill_and_topk():
    wl = make_workload("custom", seed=7, n_seqs=2, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[3000, 2100], steps=10, config_ids=["Rocket-1024", "Rocket-2048"])
    _run(wl, 10)


def test_mixed_batch_every_config():
    r = np.random.default_rng(8)
    lens = [int(x) for x in np.rint(np.exp(r.uniform(np.log(200), np.log(3000), 11)))]
    wl = make_workload("custom", seed=8, n_seqs=11, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=lens, steps=6, config_ids=list(range(11)))
    _run(wl, 6)


@pytest.mark.parametrize("hq,hkv,d", [(32, 4, 64), (8, 8, 128), (16, 8, 64)])
def test_mixed_other_head_shapes(hq, hkv, d):
    wl = make_workload("custom", seed=9, n_seqs=6, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                       prompt_lens=[700, 1300, 257, 900, 2050, 600], steps=5,
                       config_ids=["FP16", "KVQ3", "UQ4-g64", "H2O-20", "Rocket-1024", "KVQ2"])
    _run(wl, 5)


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
    _run(wl, 12)
