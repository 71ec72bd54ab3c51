"""The eleven KV-cache compression configurations, as plain data.

Each row names a method and its parameters; no arithmetic of the method lives
here.  IDs follow one fixed order:

  0      FP16            uncompressed cache (Table 1, "Uncompressed")
  1      UQ4-g64         uniform 4-bit, keys per channel over 64-token blocks,
                         values per token over 64-channel groups
  2,3,4  KVQ4/3/2        KVQuant-style non-uniform b-bit with fp16 outliers
                         (Section 2.1, KVQuant paragraph)
  5,6,7  H2O-10/20/50    heavy-hitter eviction with a budget of p% of the
                         prompt (Section 2.1, H2O paragraph)
  8,9,10 Rocket-1024/2048/4096
                         SnapKV prefill eviction to T tokens, then top-(T/2)
                         sparse decode attention (Section 2.1, RocketKV
                         paragraph)

The paper's own settings (Section 2.1, Table 1) add:

  11,12  H2O-40/60       heavy-hitter eviction at 40 % and 60 % of the prompt
  13,14,15 Rocket-8x/16x/32x
                         SnapKV keeping prompt_len / r tokens (r = 8, 16, 32),
                         then top-(T/2) sparse decode attention

PAPER_GRID lists the paper's ten configurations (Table 1) by name.
"""

CONFIGS = [
    {"id": 0, "name": "FP16", "method": "fp16"},
    {"id": 1, "name": "UQ4-g64", "method": "uq", "bits": 4, "group": 64},
    {"id": 2, "name": "KVQ4", "method": "kvq", "bits": 4, "outlier_bp": 100},
    {"id": 3, "name": "KVQ3", "method": "kvq", "bits": 3, "outlier_bp": 100},
    {"id": 4, "name": "KVQ2", "method": "kvq", "bits": 2, "outlier_bp": 100},
    {"id": 5, "name": "H2O-10", "method": "h2o", "budget_pct": 10},
    {"id": 6, "name": "H2O-20", "method": "h2o", "budget_pct": 20},
    {"id": 7, "name": "H2O-50", "method": "h2o", "budget_pct": 50},
    {"id": 8, "name": "Rocket-1024", "method": "rocket", "keep_tokens": 1024,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
    {"id": 9, "name": "Rocket-2048", "method": "rocket", "keep_tokens": 2048,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
    {"id": 10, "name": "Rocket-4096", "method": "rocket", "keep_tokens": 4096,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
    {"id": 11, "name": "H2O-40", "method": "h2o", "budget_pct": 40},
    {"id": 12, "name": "H2O-60", "method": "h2o", "budget_pct": 60},
    {"id": 13, "name": "Rocket-8x", "method": "rocket", "keep_ratio": 8, "keep_tokens": 0,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
    {"id": 14, "name": "Rocket-16x", "method": "rocket", "keep_ratio": 16, "keep_tokens": 0,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
    {"id": 15, "name": "Rocket-32x", "method": "rocket", "keep_ratio": 32, "keep_tokens": 0,
     "window": 32, "pool": 7, "topk": 0, "n_channels": 32},
]

PAPER_GRID = ["FP16", "KVQ4", "KVQ3", "KVQ2", "H2O-60", "H2O-40", "H2O-20", "Rocket-8x",
              "Rocket-16x", "Rocket-32x"]

BY_NAME = {c["name"]: c for c in CONFIGS}


def config(ident):
    """Return a copy of a config row by ID or name."""
    row = CONFIGS[ident] if isinstance(ident, int) else BY_NAME[ident]
    return dict(row)

