"""Parity over a whole optimisation run at full size (the trajectory contract for the bf16
workloads): the library runs every step of a workload's schedule on the full layer, in the
benchmark's launch configuration (next sample drawn by the backward pass), while the oracle runs
the same steps on sampled rows of sampled experts (rows are independent given H, and the noise
indices stay the global ones).  Both start from the oracle's initial state of those rows, uploaded
into the layer, so the two runs differ only by rounding inside the steps.

Along the run, at five checkpoints, the gradient G = dL/dW_hat of the sampled rows and their
loss terms sum_i R_oi P_oi (each side from its own R and G) are compared with the oracle's: at
the first step from identical states to the single-step bar (1e-3); later, the states having
drifted apart by rounding, G within CKPT_TOL_G (measured at most 1.4e-3 under Adam, 8e-3 under
Lion, whose steps keep their size whatever the gradient's) and the row losses within 1e-3
(measured at most 2.5e-4).

After the last step the hardened codes of the sampled rows must agree, except where the oracle's
own decision is a near tie (top-2 logit gap, or for the ternary pair the deciding logit, below
GAP_TOL of the largest logit).  The group scales must stay within the single-step bf16 tolerance.
The logits get RUN_TOL: Adam's update is normalised, so a rounding-level change in a gradient
that is close to zero can move that coordinate's logit by up to a step size at one step, and
such changes add up over the run (measured: 3e-5 to 2.6e-3 over 200-500 steps).  Lion runs are
bounded in units of the step size instead (see the test).
"""
import numpy as np
import pytest

from oracle import gsq as ref
from paper_2604_18556_amd import binding as B
from paper_2604_18556_amd import inputs

from gpu_common import oracle_params, rel_err

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RUNS = ["attn-4096x4096-k3", "attn-4096x4096-ternary", "mlp-up-14336x4096-k8",
        "mlp-down-4096x14336-k8", "mlp-down-4096x14336-shift8", "down-8192x28672-k4",
        "moe-64x2048x7168-superblock", "moe-64x2048x7168-superblock-shift8"]
GAP_TOL = 1e-4
RUN_TOL = 5e-3
CKPT_TOL_G = {"adam": 5e-3, "lion": 2e-2}
CKPT_TOL_LOSS = 1e-3


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    return torch.device("cuda:0")


def near_ties(rcfg, logits):
    """Coordinates whose hard decision the oracle takes within GAP_TOL of its largest logit."""
    lg = np.asarray(logits, np.float64)
    tol = GAP_TOL * np.abs(lg).max()
    if rcfg.relaxation == "ternary":
        return (np.abs(lg[..., 0]) < tol) | ((lg[..., 0] >= 0) & (np.abs(lg[..., 1]) < tol))
    srt = np.sort(lg, -1)
    return srt[..., -1] - srt[..., -2] < tol


# Lion (the paper's optimiser, Tab. 7's lr 1e-4 and weight decay 1.0) over whole runs too
LION = dict(optimizer=B.OPT_LION, lr_logits=1e-4, weight_decay=1.0)
CASES = [(n, {}) for n in RUNS] + [("attn-4096x4096-k3", LION),
                                   ("mlp-down-4096x14336-shift8", LION),
                                   ("moe-64x2048x7168-superblock", LION)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,opt", CASES,
                         ids=[n + ("-lion" if o else "") for n, o in CASES])
def test_full_run_on_sampled_rows(dev, name, opt):
    w = inputs.WORKLOADS[name]
    W, Hd = inputs.make_layer(w, device=dev)
    experts = [0] if w.batch == 1 else [0, w.batch - 1]
    Bn, O, I = w.batch, w.out_features, w.in_features
    rows = np.array([0, 1, O // 2, O - 1])
    alpha = 3.0 if w.relaxation == "ternary" else 6.0
    rcfg = ref.Config(O, I, w.levels, w.group_size, batch=Bn, precision="bf16", seed=0,
                      layout=w.layout, relaxation=w.relaxation, alpha=alpha)
    bcfg = B.LayerConfig(O, I, w.levels, w.group_size, Bn,
                         {"base3": B.LAYOUT_BASE3, "superblock": B.LAYOUT_SUPERBLOCK}.get(
                             w.layout, B.LAYOUT_GROUP), B.PREC_BF16, seed=0, alpha=alpha,
                         relaxation={"shift": B.RELAX_SHIFT, "ternary": B.RELAX_TERNARY}.get(
                             w.relaxation, B.RELAX_GRID))
    layer = B.Layer(bcfg, torch.from_numpy(W).to(dev).to(torch.bfloat16), Hd)
    Hs = ref.symmetrize(Hd[experts].cpu().numpy())
    del Hd
    torch.cuda.empty_cache()
    Hc = ref.to_contraction_precision(rcfg, Hs)   # rounded once for the whole run
    W64 = W.astype(np.float64)                     # converted once (the oracle takes float64 as is)
    K, gs = bcfg.K, bcfg.gs
    rows_t = torch.from_numpy(rows).to(dev)

    # the oracle's initial logits of the sampled rows replace the library's (init noise is
    # matched to a tolerance only); every other initial value is bit-identical
    st = ref.init_layer(rcfg, W, rows=rows, batches=experts)
    buf = torch.empty(Bn, O, I, K, device=dev)
    layer.get_state(logits=buf)
    for i, e in enumerate(experts):
        buf[e].index_copy_(0, rows_t, torch.from_numpy(st.logits[i].astype(np.float32)).to(dev))
    layer.set_state(0, logits=buf)

    T = w.steps
    ckpts = {0, T // 4, T // 2, 3 * T // 4, T - 1}
    worst = {"G": 0.0, "loss": 0.0}
    for t in range(T):
        tau = ref.tau_schedule(t, T)
        nxt = ref.tau_schedule(t + 1, T) if t + 1 < T else 0.0
        prm = B.StepParams(tau=tau, tau_next=nxt, lr_scales=w.lr_scales, **opt)
        layer.step(prm)
        if t not in ckpts:
            st, _ = ref.step(rcfg, W64, Hs, st, oracle_params(prm), rows=rows, batches=experts,
                             Hc=Hc)
            continue
        st, _, inter = ref.step(rcfg, W64, Hs, st, oracle_params(prm), rows=rows,
                                batches=experts, Hc=Hc, want=True)
        R = torch.empty(Bn, O, I, dtype=torch.bfloat16, device=dev)
        G = torch.empty(Bn, O, I, device=dev)
        layer.intermediates(residual=R, grad=G)
        Rg = np.stack([R[e].index_select(0, rows_t).float().cpu().numpy() for e in experts])
        Gg = np.stack([G[e].index_select(0, rows_t).cpu().numpy() for e in experts])
        del R, G
        eg = rel_err(Gg, inter["G"])
        lg_gpu = (Rg.astype(np.float64) * Gg * -0.5).sum(-1)           # per sampled row
        lg_ref = (inter["R"] * inter["G"] * -0.5).sum(-1)
        el = rel_err(lg_gpu, lg_ref)
        tol_g = 1e-3 if t == 0 else CKPT_TOL_G["lion" if opt else "adam"]
        print(f"  step {t}: G rel err {eg:.2e}, row losses rel err {el:.2e}")
        assert eg <= tol_g and el <= CKPT_TOL_LOSS, (t, eg, el)
        if t > 0:
            worst["G"], worst["loss"] = max(worst["G"], eg), max(worst["loss"], el)

    layer.get_state(logits=buf)
    lg = np.stack([buf[e].index_select(0, rows_t).cpu().numpy() for e in experts])
    del buf
    sbuf = torch.empty(Bn, O, I // gs, device=dev)
    layer.get_state(scales=sbuf)
    sc = np.stack([sbuf[e].index_select(0, rows_t).cpu().numpy() for e in experts])
    codes = torch.empty(Bn, O, I, dtype=torch.uint8, device=dev)
    layer.harden(codes=codes)
    c_gpu = np.stack([codes[e].index_select(0, rows_t).cpu().numpy() for e in experts])
    layer.destroy()

    c_ref = ref.hard_codes(rcfg, st)
    diff = c_gpu != c_ref
    ties = near_ties(rcfg, st.logits)
    print(f"{name}: {T} steps, {diff.sum()} of {diff.size} codes differ ({(diff & ties).sum()} "
          f"at near ties), logits rel err {rel_err(lg, st.logits):.2e}, scales rel err "
          f"{rel_err(sc, st.scales):.2e}; checkpoints after the first: G {worst['G']:.2e}, "
          f"row losses {worst['loss']:.2e}")
    if not opt:
        assert not np.any(diff & ~ties), np.argwhere(diff & ~ties)[:10]
        assert rel_err(sc, st.scales) <= 1e-3
        assert rel_err(lg, st.logits) <= RUN_TOL
        return
    # Lion steps every logit by lr (the sign of its momentum) whatever the gradient's size, so a
    # momentum within rounding of zero can send the runs 2 lr apart at that step. That happens
    # wherever a logit's gradient vanishes: far below the top, and also at the top once the
    # sample sits on its level (c_k - v -> 0), or for the shifts that a clipped window maps to
    # one level. Such drift leaves the codes alone: every differing code must be explained by
    # the drift of its own logits (the oracle's top-2 gap below their summed differences),
    # differing codes and drifting logits must stay rare, and no logit can drift more than
    # 2 lr per step.
    # Logits far below their coordinate's top (kappa times the gap over the run's largest tau
    # beyond -ln(FLT_MIN) = 87.3, e.g. the far levels of an 8-level grid under App. A's prior)
    # have a softmax weight below fp32's normal range at every step: the kernel's fp32 gradient
    # there is 0 or a denormal of a few bits, so Lion moves them by weight decay alone or by
    # steps of an unreliable sign, while the oracle's float64 weight is tiny but exact and
    # Lion's sign makes a full step of it every step. Those are counted apart; the bound on
    # drifting logits applies to all others.
    lr = opt["lr_logits"]
    d = np.abs(lg.astype(np.float64) - st.logits)
    L64 = np.asarray(st.logits, np.float64)
    underflow = (L64.max(-1, keepdims=True) - L64) * 1.0 / ref.tau_schedule(0, T) > 87.3  # kappa 1
    far = np.mean((d > 4 * lr) & ~underflow)
    far_u = np.mean((d > 4 * lr) & underflow)
    srt = np.sort(L64, -1)
    gap = srt[..., -1] - srt[..., -2]
    ds = np.abs(sc.astype(np.float64) - st.scales)
    far_s = np.mean(ds > 4 * w.lr_scales)
    print(f"  Lion: {far:.2e} of logits beyond 4 lr ({far_u:.2e} more where the fp32 weight "
          f"underflows, {underflow.mean():.2e} of all), max drift {d.max():.2e}; "
          f"{far_s:.2e} of scales beyond 4 lr_scales, max drift {ds.max():.2e}")
    assert far < 1e-2 and diff.mean() < 1e-3 and d.max() <= 2 * lr * T
    # the scales take the same sign steps (lr_scales); there are few of them per sampled row
    assert ds.max() <= 2 * w.lr_scales * T and far_s <= 2e-2
    for idx in map(tuple, np.argwhere(diff)):
        assert gap[idx] <= d[idx].sum(), (idx, gap[idx], d[idx])
