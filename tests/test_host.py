"""Host-side checks that need no GPU: the benchmark's contract and byte counts, the guard
that keeps a stale traffic profile out of the report, and the input recipe of the
synthetic workloads (the stand-ins for the paper's models and datasets)."""
import hashlib
import json
import math
import os
import subprocess
import sys

import pytest
import torch

from paper_2606_01563_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "single" in r.stderr and "--gpus 1" in r.stderr
    assert r.stdout == ""


def test_decode_bytes_match_the_per_head_formula():
    """512 len + 68612 bytes per KV head and step at d = 128, G = 4 (K/V rows, the d x d
    summary, its vectors and count, queries in and outputs out), plus the appended row
    read and written and lens read and written."""
    for n in (1, 128, 2049):
        assert bench.decode_bytes(1, 4, 128, n) == 512 * n + 68612 + 2 * 512 + 8
    assert bench.decode_bytes(288, 4, 128, 100) == 288 * bench.decode_bytes(1, 4, 128, 100)
    # the eviction step also writes the summary back and moves one row
    assert (bench.evict_bytes(1, 4, 128, 128) - bench.decode_bytes(1, 4, 128, 129)
            == 4 * 128 * 128 + 8 * 128 + 4 + 2 * 2 * 128 * 2)


def test_compress_bytes_read_k_and_v_once():
    n, d, L = 32768, 128, 512
    assert bench.compress_bytes(8, n, d, L) >= 2 * 8 * n * d * 2


def test_traffic_profile_is_ignored_once_the_sources_change(tmp_path, monkeypatch):
    """bench.measured_traffic reports HBM traffic only while the sha256 of the sources the
    counters were taken with still matches."""
    src = tmp_path / "src.txt"
    src.write_text("kernel v1")
    prof = tmp_path / "profiles"
    prof.mkdir()
    data = {"decode_sources_sha256": hashlib.sha256(b"kernel v1").hexdigest(),
            "sources": ["src.txt"], "traffic_over_algorithmic": {"128": 1.5, "256": 1.25}}
    (prof / "traffic_decode_w.md").write_text("x\n```json\n" + json.dumps(data) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w", {128: 100.0, 256: 200.0}) == pytest.approx((150 + 250) / 2)
    assert bench.measured_traffic("w", {128: 100.0, 512: 1.0}) is None   # budget not profiled
    src.write_text("kernel v2")
    assert bench.measured_traffic("w", {128: 100.0}) is None
    assert bench.measured_traffic("missing", {128: 100.0}) is None


def test_workloads_have_the_paper_shapes():
    """GQA 32/8 heads, head dim 128 and bf16 for the two models; the budgets, window and
    32K / 128K contexts of the runs; the tiny fp32 case."""
    q = synth.WORKLOADS["qwen3_4b_stack_n32768"]
    assert (q.n_q_heads, q.n_kv_heads, q.head_dim, q.ctx_len, q.window, q.layers) == \
        (32, 8, 128, 32768, 32, 36)
    assert q.budgets == (128, 256, 512, 1024, 2048) and q.dtype == torch.bfloat16
    r = synth.WORKLOADS["ruler_n131072"]
    assert (r.ctx_len, r.window, r.queries) == (131072, 64, "needle")
    t = synth.WORKLOADS["tiny_fp32_n2048"]
    assert (t.dtype, t.head_dim, t.n_kv_heads, t.ctx_len) == (torch.float32, 64, 1, 2048)


def test_synthetic_keys_and_values_share_a_rank_four_component():
    """The planted law: the value-key cross-covariance of a head has four singular values
    near 9 (3 U_v c against 3 U_k c) and the rest near sampling noise."""
    wl = synth.shrink(synth.WORKLOADS["llama31_8b_layer_n8192"], ctx_len=4096, n_kv_heads=1,
                      n_q_heads=4, rope_base=None)
    x = synth.make_layer(wl, 0, decode_steps=1)
    k = x["k"][0, 0].float()
    v = x["v"][0, 0].float()
    kc, vc = k - k.mean(0), v - v.mean(0)
    sv = torch.linalg.svdvals(vc.T @ kc / k.shape[0])
    assert torch.all((sv[:4] > 7.0) & (sv[:4] < 11.0)), sv[:6]
    assert sv[4] < 0.5, sv[:6]


def test_synthetic_inputs_are_seeded_and_rope_preserves_norms():
    wl = synth.shrink(synth.WORKLOADS["llama31_8b_layer_n8192"], ctx_len=512, batch=1)
    a = synth.make_layer(wl, 3, decode_steps=2)
    b = synth.make_layer(wl, 3, decode_steps=2)
    for name in a:
        assert torch.equal(a[name], b[name]), name
    c = synth.make_layer(wl, 4, decode_steps=2)
    assert not torch.equal(a["k"], c["k"])
    x = torch.randn(7, 128)
    y = synth.rope(x, torch.arange(7) * 1000, 5e5)
    torch.testing.assert_close(y.norm(dim=-1), x.norm(dim=-1), rtol=1e-5, atol=1e-5)


def test_needle_queries_concentrate_attention():
    """Needle queries sit on a planted needle key: its logit is far above the background
    (the concentrated-attention regime of the long-context retrieval runs)."""
    wl = synth.shrink(synth.WORKLOADS["ruler_n131072"], ctx_len=4096, n_q_heads=4,
                      n_kv_heads=1, dtype=torch.float32)
    x = synth.make_layer(wl, 0, decode_steps=8)
    k = x["k"][0, 0]
    q = x["q_dec"][:, 0].reshape(-1, wl.head_dim)               # [T * Hq, d]
    s = q @ k.T / math.sqrt(wl.head_dim)
    top = s.max(dim=1).values
    bg_std = s.std(dim=1)
    needles = set(int(p) for p in x["needles"][0, 0])
    assert all(int(i) in needles for i in s.argmax(dim=1))
    assert float((top / bg_std).min()) > 5.0
