"""Host logic of bench.py: the algorithmic work behind the roofline figures, the
latency-vs-p_t figure, and the refusal of more than one GPU (no device needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_attention_work_hand_values():
    # Hq 16, Hkv 8: 4096 bytes of keys and values per token (8 heads x 128 x 2 B x 2),
    # a query or output row of 16 x 128 bf16 = 4096 bytes.
    # Decoder with 10 keys: 10 x 4096 + 4096 + 4096 bytes, 4 x 128 x 16 x 10 flops.
    # Prompt chunk of 4 tokens over a 2-token prefix (6 keys): pairs 4 x 2 + 4 x 5 / 2 = 18.
    dec_b, pre_b, dec_f, pre_f = bench.attn_work(16, 8, [1, 4], [10, 6])
    assert dec_b == 10 * 4096 + 2 * 4096
    assert dec_f == 4 * 128 * 16 * 10
    assert pre_b == 6 * 4096 + 4 * 2 * 4096
    assert pre_f == 4 * 128 * 16 * 18
    # a chunk with no prefix is plain causal: p (p + 1) / 2 pairs
    _, _, _, f = bench.attn_work(64, 8, [8], [8])
    assert f == 4 * 128 * 64 * 36


def test_append_work_reads_and_writes_each_new_row_once():
    # 3 tokens x 8 KV heads x (key + value) x 128 x 2 B, read once and written once
    assert bench.append_work(8, 3) == 3 * 8 * 2 * 128 * 2 * 2


def _line():
    lat = {str(p): {"iter_ms_mean": 1.0 + p / 1e4, "iter_ms_first_mid_last": [0.9, 1.0, 1.2],
                    "t_lb_us": 800.0} for p in (512, 1024)}
    other = {str(p): {"iter_ms_mean": 0.9, "iter_ms_first_mid_last": [0.8, 0.9, 1.1],
                      "t_lb_us": 20.0} for p in (64, 128)}
    return {"value": 5.0e5, "latency_vs_pt": lat, "controller": {"decode_only_iter_ms": 0.95},
            "other_shapes": {"qwen3-0.6b": {"latency_vs_pt": other, "decode_only_iter_ms": 25.0,
                                            "layers_per_iteration_timed": 28}}}


def test_latency_figure_is_written(tmp_path):
    pytest.importorskip("matplotlib")
    path = tmp_path / "lat.png"
    bench.plot_latency(_line(), str(path))
    with open(path, "rb") as f:
        assert f.read(8) == b"\x89PNG\r\n\x1a\n"


def test_more_than_one_gpu_is_refused_before_any_device_call():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_source_hash_covers_the_kernel_and_its_policy():
    names = {os.path.basename(f) for f in bench.KERNEL_SOURCES}
    assert {"attention_mixed.hip", "dlfp_host.cpp", "dlfp.h"} <= names
    assert len(bench.source_hash()) == 64
