#!/usr/bin/env python3
"""GSQ layer-step benchmark on one MI355X.

A step is one full pass of the hot path over one layer (here: a batch of layers): Philox
Gumbel noise, the tempered softmax sample and residual (Alg. 1), the contraction P = R H with
the loss (Eq. 1), the gradient of logits and scales, and the Adam update.  The default
workload is the largest one that fits one GPU: 64 routed MoE experts of 2048 x 7168, each with
its own H (7168 x 7168, from Zipf(1.2)-skewed routed token counts), 8 levels
{+-0.5 .. +-3.5} in 256-weight super-blocks of 16 x 16 with frozen 6-bit sub-block scales
(the K-quant-style layout of §4.4 and App. E; experts solved independently as in App. G.1),
stepped with the linear temperature schedule 1.0 -> 0.05 over 200 steps.  Inputs are seeded
and synthetic and resident in HBM before timing starts.

Prints one JSON line: steps/s, the roofline of the dominant kernel (its duration measured
with HIP events on the library's stream during the timed steps), the CPU oracle timed on a
bounded sample of the same workload, (key "target_layer") the kernel rooflines of a short
run on the 4096 x 14336 MLP down projection, whose contraction is the matrix-core target,
(key "local_shift_variant") a short run of the same experts under the local-shift relaxation,
and (keys "lion_variant", "multi_sample_variant") short runs of the default workload under Lion
and with two noise draws per step.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
    python bench.py --copy-calibration   # plain device copy of known size, for PMC scaling
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GSQ steps/sec per layer (fwd+bwd+update) + % HBM / MFMA peak, 1 MI355X"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_FP64_TFLOPS = 78.6        # fp64 vector (the FP32 precision accumulates in fp64)
DEFAULT_WORKLOAD = "moe-64x2048x7168-superblock"
TARGET_LAYER = "mlp-down-4096x14336-k8"   # the layer the matrix-core target names
VARIANT_OF = {"moe-64x2048x7168-superblock": "moe-64x2048x7168-superblock-shift8"}
ONCE_REPS = 5                  # timed calls of gsq_harden / gsq_pack


def algorithmic_work(w, fused, want_loss, lr_scales, lion=False, samples=1):
    """Per-launch algorithmic bytes / flops of each step kernel.

    Per coordinate, bf16 W and R, fp32 logits / moments / gradient, K levels, groups of gs:
      forward   4K (logits) + 2 (W) + 2 (R)                      + 4/gs (scale)
      backward  12K read + 12K write (logits, m, v; Lion: no v) + 4 M (G of each of the
                M samples) + scale state + [fused or loss] 2 (W) + [fused] 2 (next R)
    K is the number of logits per coordinate (the grid size, 5 for the local shift, 2 for
    the ternary mask and sign); the local shift also reads one byte of base index.
      contract  2 O I^2 flops per layer
    """
    B, O, I, gs = w.batch, w.out_features, w.in_features, w.group_size
    K = {"shift": 5, "ternary": 2}.get(w.relaxation, len(w.levels))   # logits per coordinate
    base = 1 if w.relaxation == "shift" else 0                        # u8 initial grid index
    if w.layout == "superblock":
        gs = 16
    n = B * O * I
    wb = 2 if w.precision == "bf16" else 4
    state = 16 if lion else 24                  # bytes per logit: logits, m (, v), read + write
    scale_b = (state if lr_scales > 0 else 4.0) / gs
    fwd = n * (4 * K + base + 2 * wb + 4.0 / gs)
    w_read = wb if (fused or want_loss) else 0    # W, for the next sample and / or the loss
    bwd = n * (state * K + base + 4 * samples + scale_b + w_read + (wb if fused else 0))
    flops = 2.0 * B * O * I * I
    contract_bytes = n * (wb + 4) + B * I * I * wb
    return {"forward": ("hbm", fwd), "backward": ("hbm", bwd), "contract": ("flops", flops, contract_bytes)}


def harden_bytes(w, hard_loss):
    """Algorithmic bytes of gsq_harden: the K logit planes, the shift's base index, one code byte,
    and with a hard loss W and the hard residual; plus the scales read and the fp16 scales
    written (4 + 4 bytes per group)."""
    K = {"shift": 5, "ternary": 2}.get(w.relaxation, len(w.levels))
    gs = 16 if w.layout == "superblock" else w.group_size
    n = w.batch * w.out_features * w.in_features
    wb = 2 if w.precision == "bf16" else 4
    per = 4 * K + (1 if w.relaxation == "shift" else 0) + 1 + (2 * wb if hard_loss else 0)
    return n * per + n // gs * 8


def source_sha(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed PMC summary, if it matches the current source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(f"{kernel}:{workload}")
    except (ValueError, OSError):
        return None
    if not rec:
        return None
    src = os.path.join(ROOT, "paper_2604_18556_amd", "csrc", rec["source"])
    if not os.path.exists(src) or source_sha(src) != rec["source_sha256"]:
        return None
    return rec["bytes_per_launch"]


# Oracle sample size, in coordinates x K^2 per step (its backward forms K x K level differences
# per coordinate): about 2 s of host work per step on 16 cores.
CPU_WORK_PER_STEP = 38_000_000


def cpu_sample(w, rows=None, experts=None):
    """(experts, rows per expert) of the oracle's bounded sample of workload ``w``.

    Rows and experts are independent problems given their H, so a sample of them, scaled by
    the fraction of coordinates it covers, extrapolates to the whole step.  By default the
    sample holds about CPU_WORK_PER_STEP coordinates x K^2: two experts of a batched workload."""
    K = {"shift": 5, "ternary": 2}.get(w.relaxation, len(w.levels))
    n_exp = min(w.batch, 2) if experts is None else max(1, min(experts, w.batch))
    if rows is None:
        rows = int(round(CPU_WORK_PER_STEP / (n_exp * w.in_features * K * K)))
    rows = max(1, min(rows, w.out_features))
    return n_exp, rows


def cpu_baseline(w, W, Hd, rows, experts, steps, lr_scales, opt_kw):
    """The oracle, untuned, on ``rows`` rows of ``experts`` layers for ``steps`` steps (host
    cores); only those layers' H leave the GPU."""
    import numpy as np
    from oracle import gsq as ref
    blas = []
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        threads = max([p.get("num_threads", 1) for p in info] or [1])
        blas = [f"{p.get('internal_api')} {p.get('version')} ({p.get('num_threads')} threads)"
                for p in info if p.get("user_api") == "blas"]
    except Exception:
        threads = os.cpu_count()
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    # the first `experts` layers as a batch of their own: noise indices ((b O) + o) I + i do not
    # depend on the batch size, so this is the same computation as on the whole batch
    rcfg = ref.Config(w.out_features, w.in_features, w.levels, w.group_size, batch=experts,
                      layout=w.layout, precision=w.precision, seed=0, relaxation=w.relaxation,
                      alpha=3.0 if w.relaxation == "ternary" else 6.0)
    sel = np.arange(rows)
    Ws = W[:experts]
    Hs = ref.symmetrize(Hd[:experts].cpu().numpy())
    Hc = ref.to_contraction_precision(rcfg, Hs)
    st = ref.init_layer(rcfg, Ws, rows=sel)
    t0 = time.perf_counter()
    for t in range(steps):
        prm = ref.StepParams(tau=ref.tau_schedule(t, w.steps), lr_scales=lr_scales, **opt_kw)
        st, _ = ref.step(rcfg, Ws, Hs, st, prm, rows=sel, Hc=Hc)
    sec = (time.perf_counter() - t0) / steps
    frac = (experts * rows) / (w.batch * w.out_features)
    what = f"{rows} of {w.out_features} rows" + (f" of {experts} of {w.batch} experts" if w.batch > 1 else "")
    return {"value": frac / sec, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{what} x {steps} steps ({sec:.2f} s/step); extrapolated to the whole "
                      f"{'batch' if w.batch > 1 else 'layer'} by the coordinate fraction "
                      f"{frac:.4g} (rows and experts are independent given their H)",
            "cpu_count": os.cpu_count(), "cpu_model": cpu_model, "numpy": np.__version__,
            "blas": blas}


def library_gemm(w, dev, reps=20):
    """The same contraction through the vendor BLAS (torch.mm: bf16 operands, fp32 output, as G
    needs), for one layer of the workload, as a reference beside the library's own kernel."""
    import torch
    O, I = w.out_features, w.in_features
    gen = torch.Generator(device=dev).manual_seed(0)
    a = torch.randn(O, I, device=dev, dtype=torch.bfloat16, generator=gen)
    b = torch.randn(I, I, device=dev, dtype=torch.bfloat16, generator=gen)

    def f():
        return torch.mm(a, b.t(), out_dtype=torch.float32)
    for _ in range(3):
        f()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        f()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a, b
    return {"ms_per_layer": ms, "ms_per_step": ms * w.batch,
            "TFLOP/s": 2.0 * O * I * I / (ms * 1e-3) / 1e12,
            "note": "torch.mm of a bf16 O x I by a bf16 I x I matrix with fp32 output "
                    "(hipBLASLt), not part of the step"}


def copy_calibration(dev, gib=1):
    import torch
    n = gib * (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(5):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / 5
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 6,
                      "ms_per_copy": ms, "copy_GBs": 2 * n * 4 / (ms * 1e-3) / 1e9}))


def kernel_table(kern, work, w, steps):
    """Per-kernel averages of a timed pass (gsq_timing_read over ``steps`` steps) against their
    rooflines: algorithmic bytes over the HBM peak, or flops over the matrix-core peak."""
    per_kernel = {}
    for name, (ms, cnt) in kern.items():
        if cnt == 0:
            continue
        avg = ms / cnt
        entry = {"launches": cnt, "avg_ms": avg, "ms_per_step": ms / steps}
        if name in ("forward", "backward"):
            gbs = work[name][1] / (avg * 1e-3) / 1e9
            entry.update(bound="hbm", achieved=gbs, peak=PEAK_HBM_GBS, unit="GB/s",
                         frac=gbs / PEAK_HBM_GBS, bytes_per_launch=work[name][1])
        elif name == "contract":
            tf = work[name][1] / (avg * 1e-3) / 1e12
            peak = PEAK_BF16_TFLOPS if w.precision == "bf16" else PEAK_FP64_TFLOPS
            entry.update(bound="mfma" if w.precision == "bf16" else "alu", achieved=tf, peak=peak,
                         unit="TFLOP/s", frac=tf / peak, flops_per_launch=work[name][1])
        per_kernel[name] = entry
    return per_kernel


KERNEL_SOURCE = {"forward": "gsq_elem.hip", "backward": "gsq_elem.hip", "contract": "gsq_contract.hip"}


def dominant_roofline(per_kernel, w, profiled=True):
    """The roofline object of the kernel with the largest time per step.  ``profiled``: the run
    has the launch configuration of the committed PMC passes (Adam, one sample, the loss every
    step, the next sample fused), so their measured traffic applies; otherwise it is null."""
    dom = max((k for k in per_kernel if "bound" in per_kernel[k]),
              key=lambda k: per_kernel[k]["ms_per_step"])
    d = per_kernel[dom]
    return {"bound": d["bound"], "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"],
            "frac": d["frac"], "traffic": measured_traffic(dom, w.name) if profiled else None,
            "kernel": dom,
            "avg_ms": d["avg_ms"], "source": KERNEL_SOURCE[dom]}


def make_config(B, w):
    return B.LayerConfig(w.out_features, w.in_features, w.levels, w.group_size, w.batch,
                         {"superblock": B.LAYOUT_SUPERBLOCK, "base3": B.LAYOUT_BASE3}.get(w.layout, B.LAYOUT_GROUP),
                         B.PREC_BF16 if w.precision == "bf16" else B.PREC_FP32, seed=0,
                         alpha=3.0 if w.relaxation == "ternary" else 6.0,
                         relaxation={"shift": B.RELAX_SHIFT, "ternary": B.RELAX_TERNARY}.get(
                             w.relaxation, B.RELAX_GRID))


def tau_at(t, T):
    """Linear anneal 1.0 -> 0.05 over T steps, the last step at 0.05 (repeats after T)."""
    t %= T
    return 1.0 + (0.05 - 1.0) * t / (T - 1)


def short_run(name, dev, steps=10, warmup=3, opt=None, samples=1):
    """A short run of a workload (same schedule, fused next sample, loss every step; Adam unless
    ``opt`` gives other step parameters, ``samples`` draws per step): steps/s over ``steps``
    timed steps after ``warmup``, then the kernel rooflines of the next ``steps`` steps, each
    launch between the library's HIP events on its stream.  The measured traffic of the
    committed PMC passes is attached only to runs in their configuration (Adam, one sample)."""
    import torch
    from paper_2604_18556_amd import binding as B
    from paper_2604_18556_amd import inputs
    w = inputs.WORKLOADS[name]
    W, Hd = inputs.make_layer(w, device=dev)
    Wd = torch.from_numpy(W).to(dev).to(torch.bfloat16)
    layer = B.Layer(make_config(B, w), Wd, Hd)
    del W, Wd, Hd
    loss = torch.zeros(w.batch, device=dev)

    opt = opt or {}

    def run(t0, n):
        for t in range(t0, t0 + n):
            layer.step(B.StepParams(tau=tau_at(t, w.steps), lr_scales=w.lr_scales,
                                    tau_next=tau_at(t + 1, w.steps), samples=samples, **opt),
                       loss_out=loss)
    run(0, warmup)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    run(warmup, steps)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / steps
    layer.timing(True)
    layer.timing_read(reset=True)
    run(warmup + steps, steps)
    kern = layer.timing_read(reset=True)
    layer.check()
    layer.destroy()
    lion = opt.get("optimizer") == B.OPT_LION
    per_kernel = kernel_table(kern, algorithmic_work(w, True, True, w.lr_scales, lion, samples), w, steps)
    out = {"workload": name, "value": 1e3 / ms_step, "unit": "steps/s", "ms_per_step": ms_step,
           "steps": steps, "warmup": warmup, "optimizer": "lion" if lion else "adam",
           "samples_per_step": samples}
    profiled = not lion and samples == 1
    for k in ("forward", "contract", "backward"):
        if k not in per_kernel:
            continue
        e = per_kernel[k]
        out[k] = {key: e[key] for key in ("avg_ms", "ms_per_step", "bound", "achieved", "peak", "unit",
                                          "frac")}
        out[k]["traffic"] = measured_traffic(k, name) if profiled else None
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--loss-every", type=int, default=1, help="request the loss every n steps")
    ap.add_argument("--no-library-gemm", action="store_true",
                    help="skip timing the same contraction through the vendor BLAS")
    ap.add_argument("--no-fuse", action="store_true", help="do not draw the next sample in the backward pass")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=None,
                    help="rows per sampled layer of the oracle baseline (default: about "
                         f"{CPU_WORK_PER_STEP:,} coordinates x K^2 per step)")
    ap.add_argument("--cpu-experts", type=int, default=None,
                    help="layers of a batched workload in the oracle sample (default 2)")
    ap.add_argument("--cpu-steps", type=int, default=6)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--target-layer", default=TARGET_LAYER,
                    help="workload of the short extra run reported under target_layer ('' skips it)")
    ap.add_argument("--variant", default=None,
                    help="workload of a second short run reported under local_shift_variant "
                         "(default: the local-shift form of the default MoE workload; '' skips it)")
    ap.add_argument("--no-side-runs", action="store_true",
                    help="skip the short Lion and two-sample runs of the default workload "
                         "(lion_variant, multi_sample_variant)")
    ap.add_argument("--optimizer", choices=("adam", "lion"), default="adam",
                    help="adam (default) or lion (the paper's optimiser; lr 1e-4, weight decay 1.0)")
    ap.add_argument("--samples", type=int, default=1,
                    help="independent Gumbel draws averaged per step (gradient accumulation)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the GSQ layer step is measured per GPU and the library "
              f"has no multi-GPU path (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2604_18556_amd import binding as B
    from paper_2604_18556_amd import inputs

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        copy_calibration(dev)
        return

    w = inputs.WORKLOADS[args.workload]
    if args.variant is None:
        args.variant = VARIANT_OF.get(w.name, "")
    W, Hd = inputs.make_layer(w, device=dev)
    Wd = torch.from_numpy(W).to(dev)
    if w.precision == "bf16":
        Wd = Wd.to(torch.bfloat16)
    cfg = make_config(B, w)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    layer = B.Layer(cfg, Wd, Hd)
    torch.cuda.synchronize()
    init_ms = (time.perf_counter() - t0) * 1e3

    T = w.steps
    fused = not args.no_fuse
    lion = args.optimizer == "lion"
    lion_kw = dict(optimizer=B.OPT_LION, lr_logits=1e-4, weight_decay=1.0)   # Tab. 7's Lion
    opt_kw = lion_kw if lion else {}
    loss = torch.zeros(w.batch, device=dev)

    def run(t0, n):
        for i in range(n):
            t = t0 + i
            p = B.StepParams(tau=tau_at(t, T), lr_scales=w.lr_scales,
                             tau_next=tau_at(t + 1, T) if fused else 0.0, samples=args.samples,
                             **opt_kw)
            layer.step(p, loss_out=loss if (t % args.loss_every == 0) else None)

    run(0, args.warmup)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # throughput: K steps with nothing else on the stream
    start.record()
    run(args.warmup, args.steps)
    end.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(end)
    # kernel durations: the next K steps of the same schedule, every launch between HIP events
    # recorded by the library on its stream (the events themselves add gaps between launches,
    # which is why they stay out of the throughput pass)
    layer.timing(True)
    layer.timing_read(reset=True)
    t_start = time.perf_counter()
    run(args.warmup + args.steps, args.steps)
    kern = layer.timing_read(reset=True)
    ms_timed_pass = (time.perf_counter() - t_start) * 1e3
    layer.timing(False)
    layer.check()
    ms_step = ms_total / args.steps

    # once per layer: harden (+ hard loss) and pack
    codes = torch.empty(w.batch, w.out_features, w.in_features, dtype=torch.uint8, device=dev)
    hl = torch.empty(w.batch, device=dev)
    packed = torch.empty(B.packed_size(cfg), dtype=torch.uint8, device=dev)
    # one untimed call of each (first launches), then the average of ONCE_REPS timed calls
    layer.harden(codes=codes, hard_loss=hl)
    layer.pack(packed)
    layer.timing(True)
    layer.timing_read(reset=True)
    for _ in range(ONCE_REPS):
        layer.harden(codes=codes, hard_loss=hl)
    once = {k: (ms / ONCE_REPS, n) for k, (ms, n) in layer.timing_read(reset=True).items()}
    for _ in range(ONCE_REPS):
        layer.pack(packed)
    once_pack = {k: (ms / ONCE_REPS, n) for k, (ms, n) in layer.timing_read(reset=True).items()}
    layer.timing(False)

    work = algorithmic_work(w, fused, args.loss_every == 1, w.lr_scales, lion, args.samples)
    per_kernel = kernel_table(kern, work, w, args.steps)
    roofline = dominant_roofline(per_kernel, w, profiled=not lion and args.samples == 1 and fused
                                 and args.loss_every == 1)

    # the step's ideal time: each kernel's algorithmic bytes at the HBM peak, or flops at the
    # matrix-core peak, added (the kernels run one after another)
    ideal_ms = 0.0
    for name, entry in per_kernel.items():
        if entry.get("unit") == "GB/s":
            ideal_ms += entry["ms_per_step"] / entry["avg_ms"] * entry["bytes_per_launch"] / (PEAK_HBM_GBS * 1e9) * 1e3
        elif entry.get("unit") == "TFLOP/s":
            ideal_ms += entry["ms_per_step"] / entry["avg_ms"] * entry["flops_per_launch"] / (entry["peak"] * 1e12) * 1e3
    h_ms = once["harden"][0]
    h_bytes = harden_bytes(w, hard_loss=True)
    p_ms = once_pack["pack"][0]

    lib_gemm = None
    if w.precision == "bf16" and not args.no_library_gemm:
        try:
            lib_gemm = library_gemm(w, dev)
        except (RuntimeError, TypeError) as ex:   # an older torch without out_dtype
            lib_gemm = {"error": str(ex)[:200]}

    layer.destroy()
    del Wd
    target = variant = None
    if args.target_layer and args.target_layer != w.name:
        target = short_run(args.target_layer, dev)
        target["note"] = ("the layer the matrix-core target names: its contraction's fraction of "
                          "the bf16 peak (2.5 PFLOP/s) and the backward's of the HBM peak")
    if args.variant and args.variant != w.name:
        variant = short_run(args.variant, dev)
        variant["note"] = ("the same experts with the local-shift relaxation (5 logits over "
                           "shifts of the round-to-nearest index), App. E's procedure for "
                           "K-quant sets of more than four values")
    lion_run = multi = None
    if w.name == DEFAULT_WORKLOAD and not args.no_side_runs and not lion and args.samples == 1:
        lion_run = short_run(w.name, dev, opt=lion_kw)
        lion_run["note"] = ("the same workload under Lion, the paper's optimiser (Tab. 7: lr 1e-4, "
                            "weight decay 1.0): one moment, 16 instead of 24 state bytes per logit")
        multi = short_run(w.name, dev, samples=2)
        multi["note"] = ("the same workload with two independent noise draws per step, gradients "
                         "and loss averaged (gradient accumulation over resampled noise, §3.3): a "
                         "second sample pass and contraction, and the backward reads both G")

    cpu = None
    if not args.no_cpu_baseline:
        ref_opt = dict(samples=args.samples)
        if lion:
            ref_opt.update(optimizer="lion", lr_logits=1e-4, weight_decay=1.0)
        n_exp, rows = cpu_sample(w, args.cpu_rows, args.cpu_experts)
        cpu = cpu_baseline(w, W, Hd, rows, n_exp, args.cpu_steps, w.lr_scales, ref_opt)

    out = {
        "metric": METRIC,
        "value": 1e3 / ms_step,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.precision == "bf16" else "fp32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "out_features": w.out_features,
                   "in_features": w.in_features, "levels": len(w.levels), "group_size": w.group_size,
                   "layout": w.layout, "precision": w.precision, "relaxation": w.relaxation,
                   "calibration_tokens": w.tokens,
                   "tau_schedule": f"linear 1.0 -> 0.05 over {T} steps", "optimizer": args.optimizer,
                   "next_sample_fused": fused, "loss_every": args.loss_every,
                   "samples_per_step": args.samples, "parallelism": "none"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": per_kernel,
        "kernel_timing_pass": {"steps": args.steps, "wall_ms": ms_timed_pass,
                               "note": "per-kernel HIP events; throughput is timed without them"},
        "step_roofline": {"ideal_ms": ideal_ms, "frac": ideal_ms / ms_step,
                          "note": "sum over the step's kernels of algorithmic bytes / 8 TB/s and "
                                  "flops / matrix-core peak, over the measured step time"},
        "once_per_layer": {"init_ms": init_ms,
                           "harden_ms": h_ms, "harden_bytes": h_bytes,
                           "harden_GBps": h_bytes / (h_ms * 1e-3) / 1e9 if h_ms > 0 else None,
                           "pack_ms": p_ms, "pack_harden_ms": once_pack["harden"][0],
                           "hard_loss_contract_ms": once["contract"][0],
                           "note": f"mean of {ONCE_REPS} calls after one untimed call; harden: codes, hard residual and fp16 scales (gsq_harden with "
                                   "a hard loss); pack: the bit-packing kernels of gsq_pack, which "
                                   "first re-derives the codes (pack_harden_ms)"},
        "library_gemm": lib_gemm,
        "target_layer": target,
        "local_shift_variant": variant,
        "lion_variant": lion_run,
        "multi_sample_variant": multi,
        "gpu_vs_cpu": None if cpu is None else (1e3 / ms_step) / cpu["value"],
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
