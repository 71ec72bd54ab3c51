"""One captured decode step, replayed: the same results as the eager calls, and a device-side
capacity check once a replayed step runs past max_new_tokens.

Every decode quantity that changes from step to step (counts, positions, the H2O victim, the
KVQuant outlier fill) lives in device state, so a step captured once can be replayed with new
inputs written into the captured buffers.  Replays alternate with eager work (input copies,
synchronizations, exports) and every replay is checked."""
import numpy as np
import pytest

from workloads import make_workload


def _setup(wl, max_new, stream=None):
    import torch
    from gpu_harness import oracle_codebooks
    from paper_2609_07966_amd.cache import KVCache
    from workloads import prompt_kv, prompt_q
    S = wl.n_seqs
    cfgs = [wl.cfg(s) for s in range(S)]
    _, flat = oracle_codebooks(wl)

    def h(x):
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()

    c = KVCache((S, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, max_new), cfgs, wl.prompt_lens,
                codebooks=list(flat), stream=stream)
    prompts = [prompt_kv(wl, s) for s in range(S)]
    c.append_prompt(h(np.concatenate([p[0] for p in prompts])), h(np.concatenate([p[1] for p in prompts])))
    hq = [prompt_q(wl, s) for s in range(S) if cfgs[s]["method"] == "h2o"]
    if hq:
        c.h2o_prefill(h(np.concatenate(hq)))
    rq = [prompt_q(wl, s, last=32) for s in range(S) if cfgs[s]["method"] == "rocket"]
    if rq:
        c.snap_prefill(h(np.concatenate(rq)))
    torch.cuda.synchronize()
    return c, cfgs


def _state(c, cfgs, Hkv):
    res = {}
    for i, cf in enumerate(cfgs):
        for hh in range(Hkv):
            res[(i, hh, "counts")] = np.array(c.counts(i, hh))
            res[(i, hh, "positions")] = c.export(i, hh, "positions")
            if cf["method"] == "h2o":
                res[(i, hh, "scores")] = c.export(i, hh, "scores")
            if cf["method"] in ("kvq", "uq"):
                res[(i, hh, "codes_k")] = c.export(i, hh, "codes_k")
                res[(i, hh, "codes_v")] = c.export(i, hh, "codes_v")
            if cf["method"] == "rocket":
                res[(i, hh, "topk")] = c.export(i, hh, "topk")
    return res


@pytest.mark.gpu
def test_graph_replay_matches_eager():
    import torch
    from gpu_harness import log
    from workloads import step_inputs
    wl = make_workload("custom", seed=21, n_seqs=7, n_q_heads=32, n_kv_heads=8, head_dim=128,
                       prompt_lens=[900, 1300, 700, 1700, 2300, 1100, 600], steps=8,
                       config_ids=["FP16", "UQ4-g64", "KVQ4", "KVQ2", "H2O-10", "Rocket-1024", "H2O-50"])
    steps, S, Hkv, Hq, D = 8, wl.n_seqs, wl.n_kv_heads, wl.n_q_heads, wl.head_dim
    log("[graph] eager and captured caches: 7 sequences, 8 decode steps")
    eager, cfgs = _setup(wl, steps)
    side = torch.cuda.Stream()
    graphed, _ = _setup(wl, steps, stream=side)
    kb = torch.zeros((S, Hkv, D), dtype=torch.float16, device="cuda")
    vb = torch.zeros_like(kb)
    qb = torch.zeros((S, Hq, D), dtype=torch.float16, device="cuda")
    out_e = torch.empty((S, Hq, D), dtype=torch.float32, device="cuda")
    out_g = torch.full_like(out_e, float("nan"))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        graphed.step(kb, vb, qb, out_g)
    torch.cuda.synchronize()
    for t in range(steps):
        kn, vn, q = (torch.from_numpy(x).cuda() for x in step_inputs(wl, t))
        eager.step(kn, vn, q, out_e)
        kb.copy_(kn)
        vb.copy_(vn)
        qb.copy_(q)
        out_g.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"[graph] replay {t}")
        np.testing.assert_array_equal(out_g.cpu().numpy(), out_e.cpu().numpy(), err_msg=f"step {t}")
        if t in (0, steps - 1):
            a, b = _state(eager, cfgs, Hkv), _state(graphed, cfgs, Hkv)
            assert a.keys() == b.keys()
            for key in a:
                np.testing.assert_array_equal(b[key], a[key], err_msg=f"step {t}: {key}")
    eager.close()
    graphed.close()


@pytest.mark.gpu
def test_graph_replay_past_capacity_drops_tokens():
    """Replays beyond max_new_tokens leave the full regions unchanged (no write past them); H2O
    keeps evicting and appending within its budget."""
    import torch
    from gpu_harness import log
    from workloads import step_inputs
    max_new, replays = 3, 7
    wl = make_workload("custom", seed=22, n_seqs=6, n_q_heads=8, n_kv_heads=4, head_dim=64,
                       prompt_lens=[300, 257, 400, 350, 500, 280], steps=replays,
                       config_ids=["FP16", "UQ4-g64", "KVQ3", "H2O-20", "Rocket-1024", "KVQ4"])
    S, Hkv, Hq, D = wl.n_seqs, wl.n_kv_heads, wl.n_q_heads, wl.head_dim
    side = torch.cuda.Stream()
    c, cfgs = _setup(wl, max_new, stream=side)
    kept0 = [c.counts(i, 0)[0] for i in range(S)]
    kb = torch.zeros((S, Hkv, D), dtype=torch.float16, device="cuda")
    vb = torch.zeros_like(kb)
    qb = torch.zeros((S, Hq, D), dtype=torch.float16, device="cuda")
    out = torch.empty((S, Hq, D), dtype=torch.float32, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        c.step(kb, vb, qb, out)
    torch.cuda.synchronize()
    for t in range(replays):
        kn, vn, q = (torch.from_numpy(x).cuda() for x in step_inputs(wl, t))
        kb.copy_(kn)
        vb.copy_(vn)
        qb.copy_(q)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"[graph] capacity replay {t}")
        assert np.isfinite(out.cpu().numpy()).all(), f"replay {t}"
    for i, cf in enumerate(cfgs):
        for hh in range(Hkv):
            held, next_pos = c.counts(i, hh)[:2]
            m = cf["method"]
            if m in ("fp16", "rocket"):
                assert held == kept0[i] + max_new, (cf["name"], hh, held)
            elif m in ("uq", "kvq"):
                # regions are rounded up to 4-token blocks
                assert kept0[i] + max_new <= held <= kept0[i] + max_new + 3, (cf["name"], hh, held)
            else:  # H2O: at most budget + 1 held, and every replay appended a token
                assert held <= kept0[i] + replays and next_pos == wl.prompt_lens[i] + replays, (cf["name"], hh)
    c.close()
