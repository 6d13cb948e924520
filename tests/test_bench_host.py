"""Host-side checks of bench.py: the algorithmic work per unit behind its
roofline figures (the hot-path survey's derivation at DeepSeek-V3 shapes and
at the tiny shape), the digest that keeps stale traffic counters out of the
JSON line, and the one-GPU refusal.  CPU only."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_flops_per_pair_matches_derivation():
    # 2*H*2I (gate and up) + 2*I*H (down) per routed pair
    assert bench.flops_per_pair(W.CONFIGS["decode"]) == 88_080_384
    assert bench.flops_per_pair(W.CONFIGS["tiny"]) == 786_432


@pytest.mark.parametrize("P,touched", [(17, 11), (5119, 29), (65536, 13), (0, 0)])
def test_layer_bytes_matches_derivation(P, touched):
    # per touched expert: 3*H*I weight bytes + 10,752 scale bytes; per token:
    # hidden row, its scales, the fp32 logits and the bf16 output row
    for name in ("decode", "prefill", "skewed"):
        cfg = W.CONFIGS[name]
        want = 44_050_944 * touched + 22_752 * cfg.T + 4 * 256
        assert bench.layer_bytes(cfg, P, touched) == want


def test_gemm1_bytes_paths():
    dec, pre = W.CONFIGS["decode"], W.CONFIGS["prefill"]
    # weights and scales of W13 per touched expert, then rows in and out
    w13 = 2 * 2048 * 7168 + 4 * 32 * 56
    assert bench.gemm1_bytes(dec, 0, 1) == w13
    assert bench.small_tile_path(dec) and not bench.small_tile_path(pre)
    # the column-split path writes fp32 SwiGLU rows, the tile path FP8 codes and scales
    assert bench.gemm1_bytes(dec, 1, 0) == 7168 + 4 * 56 + 4 * 2048
    assert bench.gemm1_bytes(pre, 1, 0) == 7168 + 4 * 56 + 2048 + 4 * 16


def test_code_only_ignores_comments_and_spacing():
    a = "int f(int x) {  // doubles\n  return 2 * x; /* twice */\n}\n"
    b = "int f(int x) {\n\n    return 2 * x;\n}"
    c = "int f(int x) {\n  return 3 * x;\n}"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)


def test_read_traffic_needs_current_digest(tmp_path, monkeypatch):
    path = tmp_path / "gemm1_traffic_{cfg}.txt"
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(path))
    assert bench.read_traffic("x") is None  # no file
    f = tmp_path / "gemm1_traffic_x.txt"
    f.write_text("# note\nsource_digest=0000000000000000\n"
                 "fetch_bytes_per_launch=100\nwrite_bytes_per_launch=20\n")
    assert bench.read_traffic("x") is None  # stale digest
    f.write_text(f"source_digest={bench.source_digest()}\n"
                 "fetch_bytes_per_launch=100\nwrite_bytes_per_launch=20\n")
    assert bench.read_traffic("x") == 120


def test_committed_traffic_files_parse():
    for name in ("decode", "prefill", "skewed"):
        p = os.path.join(ROOT, "profiles", f"gemm1_traffic_{name}.txt")
        assert os.path.exists(p), p
        kv = dict(line.strip().split("=", 1) for line in open(p)
                  if "=" in line and not line.startswith("#"))
        assert len(kv["source_digest"]) == 16
        assert float(kv["fetch_bytes_per_launch"]) > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
