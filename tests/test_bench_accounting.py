"""The benchmark's algorithmic byte and flop counts against the per-coordinate accounting of the
step: logits, first and second moments read and written (24 bytes per logit under Adam, 16
under Lion), W read once, R written by the backward and read by the contraction, G written by
the contraction and read by the backward, 2 O I^2 flops for the contraction (Eq. 1 for a linear
layer)."""
import importlib.util
import os

import pytest

from paper_2604_18556_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(inputs.WORKLOADS))
def test_step_bytes_per_coordinate(name):
    b = _bench()
    w = inputs.WORKLOADS[name]
    K = {"shift": 5, "ternary": 2}.get(w.relaxation, len(w.levels))
    gs = 16 if w.layout == "superblock" else w.group_size
    n = w.batch * w.out_features * w.in_features
    wb = 2 if w.precision == "bf16" else 4
    base = 1 if w.relaxation == "shift" else 0
    work = b.algorithmic_work(w, fused=True, want_loss=True, lr_scales=w.lr_scales)
    scale = (24.0 if w.lr_scales > 0 else 4.0) / gs
    # backward: state, G, W (loss and next sample), next R, scales
    assert work["backward"][1] == pytest.approx(n * (24 * K + base + 4 + wb + wb + scale))
    # contraction: R read, G written, H read
    assert work["contract"][2] == n * (wb + 4) + w.batch * w.in_features ** 2 * wb
    assert work["contract"][1] == 2.0 * w.batch * w.out_features * w.in_features ** 2
    # whole fused step with frozen-size H left out: 24K + 14 bytes per coordinate in bf16
    if wb == 2 and base == 0:
        total = work["backward"][1] + work["contract"][2] - w.batch * w.in_features ** 2 * wb
        assert total == pytest.approx(n * (24 * K + 14 + scale))


def test_lion_and_samples():
    b = _bench()
    w = inputs.WORKLOADS["attn-4096x4096-k3"]
    n = w.out_features * w.in_features
    adam = b.algorithmic_work(w, True, True, w.lr_scales)["backward"][1]
    lion = b.algorithmic_work(w, True, True, w.lr_scales, lion=True)["backward"][1]
    two = b.algorithmic_work(w, True, True, w.lr_scales, samples=2)["backward"][1]
    # Lion keeps one moment: 8 bytes per logit less (logits and m read and written)
    assert adam - lion == pytest.approx(n * 8 * 3 + n * 8.0 / w.group_size)
    # every further sample adds its G read
    assert two - adam == pytest.approx(n * 4)


def test_harden_bytes():
    b = _bench()
    w = inputs.WORKLOADS["attn-4096x4096-k3"]
    n = w.out_features * w.in_features
    assert b.harden_bytes(w, hard_loss=False) == n * (12 + 1) + n // 128 * 8
    assert b.harden_bytes(w, hard_loss=True) == n * (12 + 1 + 4) + n // 128 * 8


def test_recorded_backward_traffic_matches_the_algorithmic_bytes():
    """The HBM bytes measured for the backward (FETCH_SIZE + WRITE_SIZE, copy-calibrated) stay
    within a few percent of what the step must move: the kernel re-reads nothing."""
    import json
    b = _bench()
    path = os.path.join(ROOT, "profiles", "traffic.json")
    rec = json.load(open(path))
    checked = 0
    for key, r in rec.items():
        kernel, name = key.split(":", 1)
        if kernel != "backward" or name not in inputs.WORKLOADS:
            continue
        w = inputs.WORKLOADS[name]
        alg = b.algorithmic_work(w, fused=True, want_loss=True, lr_scales=w.lr_scales)["backward"][1]
        assert 0.98 <= r["bytes_per_launch"] / alg <= 1.05, (name, r["bytes_per_launch"], alg)
        checked += 1
    assert checked >= 2


def test_bench_refuses_more_than_one_gpu():
    """The library has no multi-GPU path: --gpus above 1 exits with a message, before any GPU
    work."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
