"""Host-side logic of bench.py and the binding (CPU): the one-GPU contract,
the algorithmic flop count behind the step TFLOP/s, the source-hash gate on
the committed HBM traffic records, and the position-table size check."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4"])
def test_algorithmic_flops_sum_of_the_products(key):
    """2 M N K for each of the four projections of every block (M rows of
    image plus text tokens) plus QK^T and PV (2 Tj^2 dh each, per head)."""
    c = synth.CONFIGS[key]
    M = c.batch * (c.tokens + c.text_tokens)
    D, F, Tj = c.hidden, c.mlp_hidden, c.tokens + c.text_tokens
    gemms = [(M, 3 * D, D), (M, D, D), (M, F, D), (M, D, F)]
    per_block = sum(2.0 * m * n * k for m, n, k in gemms) + c.batch * c.heads * 2 * (2.0 * Tj * Tj * c.head_dim)
    assert bench.algorithmic_flops(c) == pytest.approx(c.n_blocks * per_block, rel=1e-12)


def test_algorithmic_flops_other_mlp_width():
    c = synth.CONFIGS["c1"].with_(mlp_hidden=1000, n_blocks=2)
    M, D = c.batch * c.tokens, c.hidden
    expect = 2 * (2.0 * M * D * (3 * D + D) + 2.0 * M * D * 1000 * 2 + 4.0 * c.batch * c.tokens ** 2 * D)
    assert bench.algorithmic_flops(c) == pytest.approx(expect, rel=1e-12)


def test_traffic_record_only_for_the_current_source(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    rec = {"kernel_class": "attention", "workload": "w", "hbm_bytes_per_launch": 123.0,
           "source_hash": bench.source_hash(bench.CLASSES["attention"][1])}
    (tmp_path / "attention_w_traffic.json").write_text(json.dumps(rec))
    assert bench.traffic_from_profile("attention", "w") == 123.0
    rec["source_hash"] = "0" * 16  # taken on another version of the kernel
    (tmp_path / "attention_w_traffic.json").write_text(json.dumps(rec))
    assert bench.traffic_from_profile("attention", "w") is None
    assert bench.traffic_from_profile("attention", "absent") is None


def test_position_table_must_cover_the_tokens():
    """A position table shorter than the token count would be read past its
    end by the patch embedding on the device; the binding and the bench
    refuse it on the host."""
    import torch
    import synth
    import paper_2605_25550_amd as dm
    cfg = synth.CONFIGS["c2"]
    shape = dm.shape_of(cfg)
    dm._check_pos(shape, None)
    dm._check_pos(shape, torch.zeros(cfg.tokens, cfg.hidden))
    for bad in (torch.zeros(cfg.tokens - 1, cfg.hidden), torch.zeros(cfg.tokens, cfg.hidden + 1),
                torch.zeros(cfg.tokens * cfg.hidden)):
        with pytest.raises(ValueError):
            dm._check_pos(shape, bad)
    with pytest.raises(ValueError):
        bench.Workload(cfg.with_(tokens=2 * cfg.tokens), torch, dm)
