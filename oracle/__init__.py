"""CPU oracle for KV-compressed decode attention (MetaKV, arXiv 2609.07966).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or run
this package; only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` use it.  It shares no code with the HIP path.

It is a plain, slow and obviously correct statement of what one decode step
computes under each of the paper's KV-cache compression configurations
(Section 2.1; Table 1):

  attention.py  exact softmax attention in float64 — the quantity every
                configuration ends in ("attention over what the cache keeps")
  kvquant.py    KVQuant-style b-bit keys per channel / values per token with
                fp16 outliers (Section 2.1, KVQuant paragraph)
  uniform.py    uniform b-bit group quantizer (per-channel keys over 64-token
                blocks, per-token values over 64-channel groups)
  codebook.py   1-D Lloyd k-means for the non-uniform codebooks
  h2o.py        H2O accumulated-attention scoring and eviction (Section 2.1,
                H2O paragraph)
  snapkv.py     SnapKV observation-window prefill eviction (Section 2.1,
                RocketKV paragraph, first stage)
  rocketkv.py   Hybrid sparse attention top-k selection (Section 2.1,
                RocketKV paragraph, second stage)
  sequence.py   per-configuration multi-step decode of one sequence

Readings the paper leaves open (budget split, tie rules, outlier fraction,
codebook fitting, ...) are stated in each function's docstring.  Floating
point is float64 except where a step is specified in float32 so that integer
decisions (quantization codes, top-k indices) are reproducible bit for bit;
those steps say so.
"""
