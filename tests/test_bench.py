"""Checks of bench.py: one GPU only, the CPU baseline's fields, the roofline bytes
(CPU), and the layer-step timing path (GPU)."""
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


@pytest.mark.gpu
def test_layer_step_timing_runs():
    """bench.time_pipeline on the Tiny layer (63 rotations at N = 2^12, the
    weighted sum, the rescale): the eager and the HIP-graph timings exist and
    the stages add up to the step."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import bench
    import synth
    import paper_2609_35352_amd as fiona
    fiona.lib()
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=dev)
    rec = bench.time_pipeline(synth.make_layer(synth.CONFIGS["tiny"], 1), dev, 3, 1, stream)
    assert rec["rotations"] == 63
    for k in ("rotate_ms", "weighted_sum_ms", "rescale_ms", "step_ms", "graph_step_ms"):
        assert rec[k] > 0, k
    parts = rec["rotate_ms"] + rec["weighted_sum_ms"] + rec["rescale_ms"]
    assert abs(parts - rec["step_ms"]) <= 0.25 * rec["step_ms"] + 0.05
