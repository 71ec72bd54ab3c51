"""Host-side checks of the benchmark: the one-GPU contract, the algorithmic byte model behind the
roofline figure, and the gating of the recorded HBM traffic on the kernel sources."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


# Bytes per (kv head, token) at head_dim 128, G = 4, outlier budget 1 %: rows are 2 x 128 fp16;
# H2O also writes G float32 logits; RocketKV reads a 4-byte slot index; KVQuant-b reads b-bit key
# and value codes, a value scale, a CSR word, one value-outlier slot and 1.28 key outliers
# (4 bytes each); uniform 4-bit reads 4-bit codes plus a (min, step) pair per 64 keys of a channel
# and per 64 channels of a value.
@pytest.mark.parametrize("cfg, per_token", [
    ({"method": "fp16"}, 512.0),
    ({"method": "h2o", "budget_pct": 10 ** 6}, 512.0 + 16),
    ({"method": "rocket", "keep_tokens": 10 ** 6, "topk": 10 ** 6}, 516.0),
    ({"method": "kvq", "bits": 4, "outlier_bp": 100}, 128 + 4 + 4 + 4 + 4 * 1.28),
    ({"method": "kvq", "bits": 3, "outlier_bp": 100}, 96 + 4 + 4 + 4 + 4 * 1.28),
    ({"method": "kvq", "bits": 2, "outlier_bp": 100}, 64 + 4 + 4 + 4 + 4 * 1.28),
])
def test_bytes_per_token(cfg, per_token):
    n0 = 4095  # with the step's appended token: 4096 tokens
    assert bench.active_tokens(cfg, n0, 0) == 4096
    assert bench.token_bytes(cfg, n0, 0, 128, 4) == pytest.approx(4096 * per_token)


def test_uniform_bytes_full_blocks_and_fp16_tail():
    cfg = {"method": "uq"}
    # 4096 tokens: 64 full key blocks, 160 B per token
    assert bench.token_bytes(cfg, 4095, 0, 128, 4) == pytest.approx(4096 * 160.0)
    # 4100 tokens: the 4 tokens of the incomplete key block are read as fp16 (256 B) instead
    assert bench.token_bytes(cfg, 4099, 0, 128, 4) == pytest.approx(4096 * 160.0 + 4 * (256 + 80))


def test_active_tokens_follow_each_method():
    assert bench.active_tokens({"method": "kvq", "bits": 4}, 1000, 9) == 1010
    # H2O: the budget plus the step's token, never more
    h = {"method": "h2o", "budget_pct": 20}
    assert bench.active_tokens(h, 1000, 0) == 201
    assert bench.active_tokens(h, 1000, 50) == 201
    # RocketKV: the top-k of what SnapKV kept plus the decode tokens; all of it while that is smaller
    r = {"method": "rocket", "keep_tokens": 1024, "topk": 0}
    assert bench.active_tokens(r, 5000, 3) == 512
    assert bench.active_tokens(r, 300, 3) == 304


def test_traffic_record_is_gated_on_the_kernel_sources(tmp_path, monkeypatch):
    rec = tmp_path / "rec.md"
    good = bench.kernel_source_hash()

    def write(h):
        rec.write_text("# record\n\n- fetch_bytes_per_launch: `1000`\n- write_bytes_per_launch: `24`\n"
                       f"- source_sha256: `{h}`\n")

    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "TRAFFIC_RECORD", "rec.md")
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: good)
    write(good)
    assert bench.recorded_traffic() == 1024.0
    write("0" * 64)
    assert bench.recorded_traffic() is None
    rec.unlink()
    assert bench.recorded_traffic() is None
