"""KV-cache memory of one sequence under one configuration (the peak KV memory of the paper's
Table 1; Section 2.2 compares the methods by it).

The count is of the state each method keeps, in the storage format of the GPU cache: what a
token, channel or slot costs is fixed by the format (fp16 K and V rows; b-bit codes; float32
thresholds, scales and group (min, step) pairs; 32-bit outlier entries and CSR row pointers;
per-slot positions, scores and saved logits; RocketKV's channel-major key copy).  ``resident``
counts the tokens kept after the step, ``peak`` the largest state from prefill on: H2O and
RocketKV hold the whole fp16 prompt (and H2O its prefill scores) beside the kept slots before
their prefill eviction.  KVQuant key outliers: n_o per channel over the prompt (the order
statistic's bound) and outlier_bp / 10000 of each decode token's channels (their expected
number).

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from .h2o import budget as h2o_budget
from .kvquant import outlier_count
from .snapkv import keep_budget


def kv_memory(cfg, n0, n_gen, n_kv_heads, head_dim, group):
    """-> (resident, peak) bytes of one sequence: cfg a configuration row, n0 prompt tokens,
    n_gen decode steps, group = query heads per kv head."""
    d, m = int(head_dim), cfg["method"]
    n = n0 + n_gen
    fp16_row = 2 * 2 * d                                   # one token's key and value in fp16
    if m == "fp16":
        resident = peak = n * fp16_row
    elif m == "uq":
        blocks = n // 64                                   # complete 64-token key blocks
        keys = blocks * 64 * d * 4 // 8 + blocks * d * 2 * 4 + (n - 64 * blocks) * d * 2
        values = n * d * 4 // 8 + n * (d // 64) * 2 * 4
        resident = peak = keys + values
    elif m == "kvq":
        b, bp = int(cfg["bits"]), int(cfg.get("outlier_bp", 100))
        codes = 2 * n * d * b // 8
        thresholds = d * 2 * 4                              # tau and 1/tau per channel
        scales = n * 4                                      # one per token (values)
        csr = (n + 1) * 4
        key_out = min(outlier_count(n0, bp), n0) * d + (n_gen * d * bp + 5000) // 10000
        v_slots = max(1, outlier_count(d, bp)) if bp > 0 else 1
        value_out = n * v_slots * (4 + 4)                   # the entry and the attention's difference
        resident = peak = codes + thresholds + scales + csr + key_out * 4 + value_out
    elif m == "h2o":
        B, _ = h2o_budget(cfg["budget_pct"], n0)
        kept = min(B, n0)
        slot = fp16_row + 4 + 4 + 4 * int(group)            # rows, position, score, saved logits
        resident = min(B, kept + n_gen) * slot
        prefill = n0 * fp16_row + n0 * 4 + kept * slot      # the prompt and its scores beside the slots
        decode = (min(B + 1, kept + n_gen) if n_gen else kept) * slot
        peak = max(prefill, decode)
    elif m == "rocket":
        T = keep_budget(cfg, n0)
        kept = min(T, n0)
        k = int(cfg.get("topk", 0)) or T // 2
        slot = fp16_row + d * 2 + 4 + 4                     # rows, channel-major key copy, position, score key
        resident = (kept + n_gen) * slot + k * 4
        peak = max(n0 * fp16_row + kept * slot, resident)
    else:
        raise ValueError(m)
    return resident * int(n_kv_heads), peak * int(n_kv_heads)
