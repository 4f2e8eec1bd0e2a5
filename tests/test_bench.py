"""CPU checks of bench.py's contract: one GPU only, and the CPU baseline's fields."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_fields():
    import oracle
    if not os.path.exists(oracle._LIB):
        pytest.skip("oracle library not built")
    import bench
    import synth
    layer = synth.make_layer(synth.CONFIGS["tiny"], 1)
    rec = bench.cpu_baseline(layer, seconds=0.2)
    assert rec["kind"] == "oracle" and rec["unit"] == "ct-terms/s"
    assert rec["value"] > 0 and 1 <= rec["cores"] <= 16
    assert "positions" in rec["sample"]


def test_algorithmic_bytes_match_the_roofline_formula():
    import synth
    for name in ("vgg11", "vit768", "bert_ffn"):
        layer = synth.make_layer(synth.CONFIGS[name], 1)
        assert synth.algorithmic_bytes(layer) == 8 * layer.L * layer.N * (2 * layer.n_in + layer.n_pm + 2 * layer.n_out)
