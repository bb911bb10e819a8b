"""Host-side checks of the benchmark's bookkeeping (no GPU).

The roofline fractions bench.py reports divide algorithmic bytes by measured time.  These tests pin
those byte counts against an independent enumeration: every tensor of the model's own tensor list
that a block forward reads (by shape and storage type; the embedding only at the block's rows), the
K/V cache read and written, and the float logits; the gate/up launch's two weight matrices, its input
rows and its SwiGLU output.  They also check that a committed counter summary stops supplying
`traffic` as soon as a kernel source it was taken from changes, and that a multi-GPU request is
refused before anything touches a device.
"""
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

import bench
from paper_2403_18647_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _weights_read(sh):
    total = 0
    for n in synth.tensor_names(sh):
        if n == "embed":
            continue   # only the block's rows of the embedding are read
        count = int(np.prod(synth.tensor_shape(sh, n)))
        total += count * (4 if synth.is_gain(n) else 2)   # float32 gains, bf16 matrices
    return total


@pytest.mark.parametrize("shape", [synth.LLAMA7B, synth.LLAMA13B])
@pytest.mark.parametrize("B,q,ctx", [(1, 6, 639), (4, 6, 1100), (1, 11, 2100), (8, 11, 16384)])
def test_block_bytes_counts_every_tensor_the_forward_reads(shape, B, q, ctx):
    d, L, V = shape.d_model, shape.n_layers, shape.vocab
    kv_read = L * 2 * B * ctx * d * 2          # K and V of every layer, bf16
    kv_write = L * 2 * B * q * d * 2
    expect = _weights_read(shape) + B * q * d * 2 + kv_read + kv_write + B * q * V * 4
    assert bench.block_bytes(shape, B, q, ctx) == expect


def test_block_bytes_of_the_headline_workload():
    """7B, one sequence, k = 5 (6 rows) at the mean decode context of a 512-token prompt and 256
    new tokens (639 keys): 32 layers x (4 d^2 + 3 d F) x 2 B = 12,952,010,752; LM head 32016 x 4096 x 2
    = 262,275,072; 65 gains x 4096 x 4 = 1,064,960; K/V read 2 x 32 x 4096 x 639 x 2 = 335,020,032 and
    written 2 x 32 x 4096 x 6 x 2 = 3,145,728; embedding rows 49,152; logits 6 x 32016 x 4 = 768,384."""
    assert bench.block_bytes(synth.LLAMA7B, 1, 6, 639) == 13_554_334_080


def test_gateup_bytes():
    sh = synth.LLAMA7B
    d, F = sh.d_model, sh.d_ffn
    w = sum(int(np.prod(synth.tensor_shape(sh, n))) for n in ("l0.w_gate", "l0.w_up")) * 2
    # several rows: bf16 normalised rows in, bf16 SwiGLU product out
    assert bench.gateup_bytes(sh, 6) == w + 6 * d * 2 + 6 * F * 2 == 180_536_320
    # one row: the float row x o g and its per-16-column sums of squares
    assert bench.gateup_bytes(sh, 1) == w + d * 4 + (d // 16) * 4 + F * 2


def test_metric_names_follow_the_workload():
    assert bench.metric_for(synth.workload("7b")) == bench.METRIC_7B
    assert "@bs1 (13B shape, k=10, greedy)" in bench.metric_for(synth.workload("13b"))
    assert "@bs4 (7B shape, k=5, nucleus)" in bench.metric_for(synth.workload("7b_bs4_nucleus"))


def _copy_tree(tmp_path):
    os.makedirs(tmp_path / "profiles")
    os.makedirs(tmp_path / "paper_2403_18647_amd" / "csrc")
    for f in ("block_forward_7b_decode.md", "gateup_gemm_7b_decode.md"):
        shutil.copy(os.path.join(ROOT, "profiles", f), tmp_path / "profiles" / f)
    src = os.path.join(ROOT, "paper_2403_18647_amd", "csrc")
    for f in os.listdir(src):
        if f.endswith(".hip"):
            shutil.copy(os.path.join(src, f), tmp_path / "paper_2403_18647_amd" / "csrc" / f)


def _recorded(path, key):
    for line in open(path).read().splitlines():
        if line.startswith(key + ": "):
            return int(line.split(": ", 1)[1])
    raise AssertionError(f"{key} not in {path}")


@pytest.mark.parametrize("source", ["gemm.hip", "attention.hip", "prefill.hip", "misc.hip"])
def test_counter_traffic_is_null_once_a_source_changed(tmp_path, monkeypatch, source):
    _copy_tree(tmp_path)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    block = bench.profiled_block_traffic("7b")
    gateup = bench.profiled_traffic("7b")
    # the committed summaries may predate the current sources; then both already read None
    if block is not None:
        assert block == _recorded(tmp_path / "profiles" / "block_forward_7b_decode.md", "traffic_bytes_per_block")
    if gateup is not None:
        assert gateup == _recorded(tmp_path / "profiles" / "gateup_gemm_7b_decode.md", "traffic_bytes_per_launch")
    with open(tmp_path / "paper_2403_18647_amd" / "csrc" / source, "a") as f:
        f.write("\n// edited\n")
    assert bench.profiled_block_traffic("7b") is None
    if source == "gemm.hip":
        assert bench.profiled_traffic("7b") is None
    assert bench.profiled_block_traffic("13b") is None   # no summary for this workload


def test_multi_gpu_request_is_refused_before_any_device_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and r.stdout == ""
    assert "one GPU" in r.stderr
