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


def test_recorded_mfma_flops_are_the_algorithmic_flops():
    """The bf16 flops the matrix-core counters record for one step contraction
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512, in profiles/mfma_contract_*.txt) are exactly the
    2 O I^2 of P = R H: the kernel does no redundant products."""
    import glob
    b = _bench()
    files = glob.glob(os.path.join(ROOT, "profiles", "mfma_contract_*.txt"))
    assert files
    for path in files:
        name = os.path.basename(path)[len("mfma_contract_"):-len(".txt")]
        w = inputs.WORKLOADS[name]
        alg = b.algorithmic_work(w, fused=True, want_loss=True, lr_scales=w.lr_scales)["contract"][1]
        rows = [ln.split() for ln in open(path) if ln.startswith("contract ")]
        step = [r for r in rows if r[1] == "step"]
        assert len(step) == 1, path
        gflop = float(step[0][6])
        assert abs(gflop * 1e9 - alg) <= 0.05e9, (name, gflop, alg / 1e9)


def test_mfma_summary_arithmetic(tmp_path, capsys):
    """The MFMA summary on two hand-made dispatches: clock = GRBM_GUI_ACTIVE per XCC over the
    dispatch time, busy share = busy cycles over (active cycles x SIMDs), flops = 512 per MOPS
    unit; a contraction after the first harden kernel is listed as a hard-loss one."""
    from paper_2604_18556_amd import rocprof_summary as rs
    agent = tmp_path / "agent.csv"
    agent.write_text("Agent_Type,Num_Xcc,Simd_Count\nCPU,1,0\nGPU,8,1024\n")
    cc = tmp_path / "cc.csv"
    lines = ["Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp"]
    t = 0

    def dispatch(d, kernel, dur_ns, counters):
        nonlocal t
        for c, v in counters.items():
            lines.append(f'{d},"{kernel}",{c},{v},{t},{t + dur_ns}')
        t += dur_ns + 1000

    # 100 us at 2.0 GHz on each of 8 XCCs: 200000 cycles per XCC; half of 1024 SIMDs' cycles busy
    dispatch(1, "gsq::k_contract_bf16(x)", 100_000,
             {"GRBM_GUI_ACTIVE": 8 * 200_000, "SQ_VALU_MFMA_BUSY_CYCLES": 0.5 * 200_000 * 1024,
              "SQ_INSTS_VALU_MFMA_MOPS_BF16": 2 ** 20, "SQ_LDS_BANK_CONFLICT": 0})
    dispatch(2, "gsq::k_harden<3>(x)", 10_000, {"GRBM_GUI_ACTIVE": 8 * 20_000})
    dispatch(3, "gsq::k_contract_bf16(x)", 200_000,
             {"GRBM_GUI_ACTIVE": 8 * 400_000, "SQ_VALU_MFMA_BUSY_CYCLES": 0.25 * 400_000 * 1024,
              "SQ_INSTS_VALU_MFMA_MOPS_BF16": 2 ** 20, "SQ_LDS_BANK_CONFLICT": 7})
    cc.write_text("\n".join(lines) + "\n")
    rs.main(["mfma", str(cc), "--agent", str(agent)])
    out = {tuple(ln.split()[:2]): ln.split() for ln in capsys.readouterr().out.splitlines()
           if ln.startswith("contract ")}
    step, hard = out[("contract", "step")], out[("contract", "hard")]
    assert step[2] == "1" and float(step[3]) == pytest.approx(100.0)
    assert float(step[4]) == pytest.approx(2.0) and float(step[5]) == pytest.approx(0.5)
    gflop = 2 ** 20 * 512 / 1e9
    assert float(step[6]) == pytest.approx(gflop, abs=0.05)
    assert float(step[7]) == pytest.approx(gflop / 100e-6 / 1e3, abs=1)      # TFLOP/s
    # hard-loss row: "contract hard loss n us ..." has one more token before the numbers
    assert float(hard[6]) == pytest.approx(0.25) and float(hard[5]) == pytest.approx(2.0)


def test_measured_traffic_only_for_the_profiled_configuration():
    """The roofline's traffic comes from PMC passes of the Adam, one-draw, fused, loss-every-step
    run; any other configuration (Lion, several draws) reports it as null."""
    b = _bench()
    w = inputs.WORKLOADS["moe-64x2048x7168-superblock"]
    per_kernel = {"backward": {"bound": "hbm", "achieved": 6000.0, "peak": 8000.0, "unit": "GB/s",
                               "frac": 0.75, "avg_ms": 30.0, "ms_per_step": 30.0},
                  "contract": {"bound": "mfma", "achieved": 1200.0, "peak": 2500.0, "unit": "TFLOP/s",
                               "frac": 0.48, "avg_ms": 11.0, "ms_per_step": 11.0}}
    r = b.dominant_roofline(per_kernel, w, profiled=False)
    assert r["kernel"] == "backward" and r["traffic"] is None
    r = b.dominant_roofline(per_kernel, w, profiled=True)
    assert r["traffic"] == b.measured_traffic("backward", w.name)
