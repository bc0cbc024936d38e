"""GPU parity of the local-shift (§3.2, Eq. 6) and ternary mask x sign (§3.1, Alg. 2)
relaxations and of the base-3 layout: the HIP path through the C ABI against the CPU oracle.

Same bars as the full-grid tests: 1e-5 (FP32 precision) / 1e-3 (BF16 precision), max-normalised;
codes, base indices and packed bytes bit-exact.
"""
import numpy as np
import pytest

from oracle import gsq as ref
from oracle import pack as refpack
from oracle import philox
from paper_2604_18556_amd import binding as B
from paper_2604_18556_amd import inputs

from gpu_common import Pair, assert_state_close, layer_inputs, oracle_params, rel_err, warm_state

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 1e-3}
L3, L4, L8 = inputs.L3, inputs.L4, inputs.L8
L16 = tuple(x + 0.5 for x in range(-8, 8))


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    return torch.device("cuda:0")


def _rcfg(relax, O, I, levels, gs, prec, **kw):
    alpha = 3.0 if relax == "ternary" else 6.0       # Tab. 7: 3 for ternary, 6 for 2/3-bit
    return ref.Config(O, I, levels, gs, precision=prec, relaxation=relax, alpha=alpha, **kw)


# ------------------------------------------------------------------ noise
@pytest.mark.parametrize("relax,levels,Z", [("shift", L8, 5), ("ternary", L3, 2)])
def test_noise_of_the_relaxations_is_bit_exact(dev, relax, levels, Z):
    """FP32 precision: Gumbel values of the shift's five logits, logistic values of the ternary
    relaxation's two pairs, both evaluated in fp64 and rounded once, as the oracle does."""
    cfg = B.LayerConfig(4, 256, levels, 128, precision=B.PREC_FP32, seed=77,
                        relaxation={"shift": B.RELAX_SHIFT, "ternary": B.RELAX_TERNARY}[relax])
    n = 100_000
    out = torch.empty(n, Z, device=dev)
    B.gumbel(cfg, 3 * 2**32 - 17, n, 5, out)
    draw = philox.logistic if relax == "ternary" else philox.gumbel
    want = draw(77, np.arange(3 * 2**32 - 17, 3 * 2**32 - 17 + n), 5, Z)
    assert np.count_nonzero(out.cpu().numpy().astype(np.float64) != want) <= 2


def test_ternary_noise_bf16_path_is_close(dev):
    """BF16 precision: ln2 (log2 u - log2(1 - u)) with the hardware logarithm against the fp64
    value; the error is a few ulps of the larger logarithm."""
    cfg = B.LayerConfig(4, 256, L3, 128, precision=B.PREC_BF16, seed=5, relaxation=B.RELAX_TERNARY)
    n = 400_000
    out = torch.empty(n, 2, device=dev)
    B.gumbel(cfg, 0, n, 3, out)
    want = philox.logistic(5, np.arange(n), 3, 2)
    err = np.abs(out.cpu().numpy() - want)
    print(f"bf16-path logistic noise: max abs error {err.max():.3e}, mean {err.mean():.3e}")
    assert err.max() < 2e-5, err.max()


# ------------------------------------------------------------------ initialisation
@pytest.mark.parametrize("relax,prec,O,I,levels,gs,layout", [
    ("shift", "fp32", 256, 256, L8, 128, "group"),
    ("shift", "bf16", 70, 384, L16, 64, "group"),
    ("shift", "bf16", 40, 512, L8, 16, "superblock"),
    ("ternary", "fp32", 96, 256, L3, 128, "group"),
    ("ternary", "bf16", 130, 272, L3, 16, "base3"),
])
def test_init_matches_oracle(dev, relax, prec, O, I, levels, gs, layout):
    W, H = layer_inputs(O, I, bf16=prec == "bf16", seed=len(levels) + O)
    rcfg = _rcfg(relax, O, I, levels, gs, prec, layout=layout, seed=31, sigma_init=0.8)
    pair = Pair(rcfg, W, H, dev)
    st = ref.init_layer(rcfg, W)
    got = pair.get()
    np.testing.assert_array_equal(got.scales, st.scales)
    assert rel_err(got.logits, st.logits) <= 1e-6
    if relax == "shift":
        np.testing.assert_array_equal(got.base, st.base)
        assert st.base.min() == 0 and st.base.max() == len(levels) - 1   # both ends of the grid occur
    # noise-free warm start: hardening returns the round-to-nearest code
    rcfg0 = _rcfg(relax, O, I, levels, gs, prec, layout=layout, init_noise=False)
    pair0 = Pair(rcfg0, W, H, dev)
    codes = torch.empty(1, O, I, dtype=torch.uint8, device=dev)
    pair0.layer.harden(codes=codes)
    np.testing.assert_array_equal(codes.cpu().numpy(), ref.init_layer(rcfg0, W).extra["q0"])


# ------------------------------------------------------------------ one step from a shared state
CASES = [
    # relax, precision, O, I, levels, gs, tau, kappa
    ("shift", "fp32", 256, 256, L8, 128, 0.05, 1.0),
    ("shift", "fp32", 70, 384, L16, 64, 0.5, 2.0),
    ("shift", "bf16", 200, 384, L8, 128, 0.3, 1.0),
    ("shift", "bf16", 96, 272, L16, 16, 1.0, 1.0),
    ("ternary", "fp32", 256, 256, L3, 128, 0.05, 1.0),
    ("ternary", "fp32", 70, 384, L3, 64, 0.5, 2.0),
    ("ternary", "bf16", 200, 384, L3, 128, 0.3, 1.0),
    ("ternary", "bf16", 130, 512, L3, 128, 1.0, 1.0),
]


@pytest.mark.parametrize("relax,prec,O,I,levels,gs,tau,kappa", CASES)
@pytest.mark.parametrize("warm", [False, True])
def test_single_step_matches_oracle(dev, relax, prec, O, I, levels, gs, tau, kappa, warm):
    W, H = layer_inputs(O, I, bf16=prec == "bf16", seed=O + 2 * I)
    rcfg = _rcfg(relax, O, I, levels, gs, prec, seed=4)
    pair = Pair(rcfg, W, H, dev)
    st = ref.init_layer(rcfg, W)
    rng = np.random.default_rng(O)
    if warm:
        st = warm_state(st, rng)
        if relax == "shift":       # any base index, the clipped ends included
            st.base = rng.integers(0, len(levels), st.base.shape).astype(np.uint8)
    pair.put(st)
    prm = B.StepParams(tau=tau, kappa=kappa, lr_scales=5e-5)
    loss = pair.step(prm)
    R, G = pair.intermediates()
    new, L, inter = ref.step(rcfg, W, pair.Hs, st, oracle_params(prm), want=True)
    tol = TOL[prec]
    assert np.all(np.abs(loss - L) <= tol * np.abs(L)), (loss, L)
    assert rel_err(G, inter["G"]) <= tol, rel_err(G, inter["G"])
    assert rel_err(R, inter["R"]) <= (tol if prec == "fp32" else 2.0**-7)
    got = pair.get()
    assert_state_close(got, new, inter["G"], tol, st.t + 1, label=f"{relax} {prec} {O}x{I}",
                       dlogits=inter["dlogits"])
    if not warm:
        assert rel_err(got.m / (1 - np.float32(0.9)), inter["dlogits"]) <= tol
        assert rel_err(got.m_s / (1 - np.float32(0.9)), inter["dscales"]) <= tol
    if relax == "shift":
        np.testing.assert_array_equal(got.base, st.base)   # the base never moves


@pytest.mark.parametrize("prec,batch,O,I,gs,layout", [("bf16", 2, 48, 512, 16, "superblock"),
                                                       ("fp32", 1, 70, 384, 64, "group"),
                                                       ("bf16", 1, 130, 272, 16, "group")])
@pytest.mark.parametrize("opt", ["adam", "lion"])
def test_shift_step_with_frozen_scales(dev, prec, batch, O, I, gs, layout, opt):
    """The local shift with frozen scales (lr_scales = 0, as for the super-block experts), whose
    backward keeps every moment in flight (a code path of its own), from warm moments and any
    base indices, under Adam and Lion."""
    W, H = layer_inputs(O, I, batch=batch, bf16=prec == "bf16", seed=O + I)
    rcfg = ref.Config(O, I, L8, gs, batch=batch, layout=layout, precision=prec, seed=8,
                      relaxation="shift")
    pair = Pair(rcfg, W, H, dev)
    rng = np.random.default_rng(I)
    st = warm_state(ref.init_layer(rcfg, W), rng)
    st.base = rng.integers(0, 8, st.base.shape).astype(np.uint8)
    pair.put(st)
    kw = dict(optimizer=B.OPT_LION, lr_logits=1e-3, weight_decay=1.0) if opt == "lion" else {}
    prm = B.StepParams(tau=0.3, lr_scales=0.0, **kw)
    loss = pair.step(prm)
    R, G = pair.intermediates()
    new, L, inter = ref.step(rcfg, W, pair.Hs, st, oracle_params(prm), want=True)
    tol = TOL[prec]
    assert np.all(np.abs(loss - L) <= tol * np.abs(L)), (loss, L)
    assert rel_err(G, inter["G"]) <= tol
    got = pair.get()
    assert_state_close(got, new, inter["G"], tol, st.t + 1, label=f"frozen shift {prec} {O}x{I}",
                       dlogits=inter["dlogits"])
    np.testing.assert_array_equal(got.scales, st.scales)


@pytest.mark.parametrize("relax,prec", [("shift", "fp32"), ("ternary", "bf16")])
def test_lion_and_samples_step(dev, relax, prec):
    """The paper's optimiser (Lion, weight decay) and three averaged draws on the relaxations."""
    levels = L8 if relax == "shift" else L3
    W, H = layer_inputs(130, 384, bf16=prec == "bf16", seed=3)
    rcfg = _rcfg(relax, 130, 384, levels, 128, prec, seed=9)
    pair = Pair(rcfg, W, H, dev)
    st = warm_state(ref.init_layer(rcfg, W), np.random.default_rng(1))
    pair.put(st)
    prm = B.StepParams(tau=0.4, lr_logits=1e-3, lr_scales=5e-5, optimizer=B.OPT_LION,
                       weight_decay=1.0, samples=3)
    loss = pair.step(prm)
    _, G = pair.intermediates()
    new, L, inter = ref.step(rcfg, W, pair.Hs, st, oracle_params(prm), want=True)
    tol = TOL[prec]
    assert np.all(np.abs(loss - L) <= tol * np.abs(L))
    assert rel_err(G, inter["G"]) <= tol
    assert_state_close(pair.get(), new, inter["G"], tol, st.t + 1, label=f"lion {relax}",
                       dlogits=inter["dlogits"])


# ------------------------------------------------------------------ harden / pack
@pytest.mark.parametrize("relax,levels,gs,layout", [
    ("shift", L8, 128, "group"), ("shift", L16, 64, "group"), ("shift", L8, 16, "superblock"),
    ("ternary", L3, 128, "group"), ("ternary", L3, 64, "base3"), ("grid", L3, 16, "base3"),
])
def test_harden_and_pack_are_bit_exact(dev, relax, levels, gs, layout):
    O, I, batch = 37, 512, 2
    W, H = layer_inputs(O, I, batch=batch, seed=len(levels))
    rcfg = _rcfg(relax, O, I, levels, gs, "bf16", batch=batch, layout=layout, seed=2)
    pair = Pair(rcfg, W, H, dev)
    st = ref.init_layer(rcfg, W)
    rng = np.random.default_rng(len(levels) + gs)
    st.logits = rng.integers(-2, 3, st.logits.shape).astype(np.float32)   # exact ties and zeros
    if relax == "shift":
        st.base = rng.integers(0, len(levels), st.base.shape).astype(np.uint8)
    if layout != "superblock":
        st.scales = (st.scales * rng.uniform(0.5, 2, st.scales.shape)).astype(np.float32)
    pair.put(st)
    codes = torch.empty(batch, O, I, dtype=torch.uint8, device=dev)
    scales = torch.empty(st.scales.shape, device=dev)
    hl = torch.empty(batch, device=dev)
    pair.layer.harden(codes=codes, scales=scales, hard_loss=hl)
    c_ref, s_ref, hl_ref = ref.harden_layer(rcfg, W, pair.Hs, st)
    np.testing.assert_array_equal(codes.cpu().numpy(), c_ref)
    np.testing.assert_array_equal(scales.cpu().numpy(), s_ref)
    assert np.all(np.abs(hl.cpu().numpy() - hl_ref) <= 1e-3 * np.abs(hl_ref))
    packed = torch.empty(B.packed_size(pair.bcfg), dtype=torch.uint8, device=dev)
    pair.layer.pack(packed)
    if layout == "group":
        expect = refpack.pack_plain(c_ref, ref.scales_fp16(st.scales), len(levels), gs)
    elif layout == "base3":
        expect = refpack.pack_base3(c_ref, ref.scales_fp16(st.scales))
    else:
        sd, ssc, _ = ref.superblock_scales(W.astype(np.float64), rcfg)
        expect = refpack.pack_superblock(c_ref, sd, ssc)
    np.testing.assert_array_equal(packed.cpu().numpy(), expect)


# ------------------------------------------------------------------ trajectories (tiny fp32 layer)
@pytest.mark.parametrize("relax", ["shift", "ternary"])
def test_tiny_layer_trajectory(dev, relax):
    """40 fused steps, tau 1.0 -> 0.05: shift with Adam on the 3-bit grid, ternary with Lion
    (lr 1e-3, weight decay 1.0, Tab. 7's ternary setting); losses every step, final codes."""
    w = inputs.WORKLOADS["tiny-256x256-k4"]
    W, H = inputs.make_layer(w)
    levels = L8 if relax == "shift" else L3
    rcfg = _rcfg(relax, 256, 256, levels, 128, "fp32", seed=5)
    pair = Pair(rcfg, W, H, dev)
    st = ref.init_layer(rcfg, W)
    T = 40
    opt = dict(optimizer=B.OPT_LION, lr_logits=1e-3, weight_decay=1.0) if relax == "ternary" else {}
    for t in range(T):
        prm = B.StepParams(tau=ref.tau_schedule(t, T), lr_scales=5e-5,
                           tau_next=ref.tau_schedule(t + 1, T) if t + 1 < T else 0.0, **opt)
        lg = pair.step(prm)[0]
        st, L = ref.step(rcfg, W, pair.Hs, st, oracle_params(prm))
        assert abs(lg - L[0]) <= 1e-5 * abs(L[0]), (t, lg, L[0])
    got = pair.get()
    assert rel_err(got.logits, st.logits) <= 1e-5
    c_gpu, c_ref = ref.hard_codes(rcfg, got), ref.hard_codes(rcfg, st)
    assert np.count_nonzero(c_gpu != c_ref) == 0
