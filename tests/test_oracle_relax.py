"""Pins of the oracle's local-shift (§3.2, Eq. 6) and ternary mask x sign (§3.1, Eq. 2, Alg. 2)
relaxations, and of the base-3 packing of 3-level codes."""
import math
import os

import numpy as np
import pytest
from scipy import stats
from scipy.special import expit

from oracle import gsq, pack, philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
L8 = (-3.5, -2.5, -1.5, -0.5, 0.5, 1.5, 2.5, 3.5)
L5 = (-2.0, -1.0, 0.0, 1.0, 2.0)
L3 = (-1.0, 0.0, 1.0)


def _spd(rng, n):
    X = rng.standard_normal((2 * n, n)) * rng.lognormal(0, 0.5, n)
    return X.T @ X


def _loss(cfg, W, H, lg, sc, g, tau, kappa, base=None):
    s_coord = gsq.expand_scales(sc, cfg.gs)
    if cfg.relaxation == "ternary":
        _, _, R = gsq.ternary_forward(cfg, W, lg, s_coord, g, tau, kappa)
    else:
        _, _, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa, gsq.candidates(cfg, base))
    return gsq.contract(cfg, R, H)[1]


# ------------------------------------------------------------------ local shift
def test_shift_window_worked_example_on_an_8_level_grid():
    """Eq. 6 on the 3-bit grid: interior indices see the five neighbouring levels; at the ends
    the clip repeats the end level (written out by hand for this grid)."""
    cfg = gsq.Config(1, 16, L8, 16, relaxation="shift")
    c = gsq.candidates(cfg, np.arange(8))
    assert tuple(c[0]) == (-3.5, -3.5, -3.5, -2.5, -1.5)
    assert tuple(c[1]) == (-3.5, -3.5, -2.5, -1.5, -0.5)
    assert tuple(c[4]) == (-1.5, -0.5, 0.5, 1.5, 2.5)
    assert tuple(c[6]) == (0.5, 1.5, 2.5, 3.5, 3.5)
    assert tuple(c[7]) == (1.5, 2.5, 3.5, 3.5, 3.5)
    # the paper's 1-based form clip(j + delta, 1, 2^b) with j = j0 + 1 names the same levels
    for j0 in range(8):
        one_based = [min(max(j0 + 1 + d, 1), 8) for d in (-2, -1, 0, 1, 2)]
        assert tuple(c[j0]) == tuple(L8[j - 1] for j in one_based)


def test_shift_on_a_five_level_grid_centred_is_the_full_categorical():
    """With 5 levels and every j0 at the centre the window is the whole grid: a shift step is
    exactly a full-grid step (same noise, same state, same arithmetic)."""
    rng = np.random.default_rng(3)
    O, I = 4, 64
    W = rng.normal(0, 0.02, (1, O, I)).astype(np.float32)
    H = gsq.symmetrize(_spd(rng, I).astype(np.float32))
    cg = gsq.Config(O, I, L5, 32, precision="fp32", seed=5)
    cs = gsq.Config(O, I, L5, 32, precision="fp32", seed=5, relaxation="shift")
    st = gsq.init_layer(cg, W)
    st.m[:] = rng.standard_normal(st.m.shape).astype(np.float32) * 1e-3
    st.v[:] = rng.uniform(0.5, 2, st.v.shape).astype(np.float32) * 1e-6
    ss = st.copy()
    ss.base = np.full((1, O, I), 2, np.uint8)
    prm = gsq.StepParams(tau=0.4, kappa=1.5, samples=2)
    ng, lg_ = gsq.step(cg, W, H, st, prm)
    ns, ls_ = gsq.step(cs, W, H, ss, prm)
    np.testing.assert_array_equal(lg_, ls_)
    for k in ("logits", "m", "v", "scales"):
        np.testing.assert_array_equal(getattr(ng, k), getattr(ns, k))


def test_shift_low_temperature_limit_and_hardening():
    """tau -> 0 without noise: the soft weight is s c[clip(j0 + delta*)] with delta* the argmax
    shift, and hardening returns that code, for every j0 and every winning shift."""
    cfg = gsq.Config(1, 40, L8, 8, precision="fp64", relaxation="shift")
    j0 = np.repeat(np.arange(8), 5)[None]                   # 8 bases x 5 winners
    win = np.tile(np.arange(5), 8)[None]
    lg = np.where(np.arange(5) == win[..., None], 2.0, -1.0)
    s = np.full((1, 40), 0.03)
    _, v, _ = gsq.forward(cfg, np.zeros((1, 40)), lg, s, np.zeros((1, 40, 5)), 1e-6, 1.0,
                          gsq.candidates(cfg, j0))
    code = np.clip(j0 + win - 2, 0, 7)
    np.testing.assert_allclose(v, np.asarray(L8)[code], atol=1e-9)
    st = gsq.State(lg[None].astype(np.float32), None, None, None, None, None, base=j0[None].astype(np.uint8))
    np.testing.assert_array_equal(gsq.hard_codes(cfg, st)[0], code)


@pytest.mark.parametrize("tau,kappa", [(1.0, 1.0), (0.3, 2.0)])
def test_shift_backward_matches_finite_differences(tau, kappa):
    rng = np.random.default_rng(30)
    O, I, gs = 2, 32, 16
    cfg = gsq.Config(O, I, L8, gs, precision="fp64", relaxation="shift")
    H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, 5))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    base = rng.integers(0, 8, (O, I))
    base[0, :4] = [0, 1, 6, 7]                               # clipped windows included
    g = philox.gumbel(2, np.arange(O * I), 1, 5).reshape(O, I, 5)
    s_coord = gsq.expand_scales(sc, gs)
    cand = gsq.candidates(cfg, base)
    p, v, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa, cand)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.backward(cfg, (-2 * P)[None], s_coord[None], p[None], v[None], tau, kappa, cand[None])
    dl, ds = dl[0], ds[0]
    for idx in [(0, 0, 0), (0, 0, 4), (0, 3, 3), (1, 5, 2), (1, 31, 1)]:
        h = 1e-6 * max(1.0, abs(lg[idx]))
        a, b = lg.copy(), lg.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss(cfg, W, H, a, sc, g, tau, kappa, base) - _loss(cfg, W, H, b, sc, g, tau, kappa, base)) / (2 * h)
        assert abs(fd - dl[idx]) <= 1e-6 * max(abs(fd), np.abs(dl).max() * 1e-3), (idx, fd, dl[idx])
    for idx in [(0, 0), (1, 1)]:
        h = 1e-6 * sc[idx]
        a, b = sc.copy(), sc.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss(cfg, W, H, lg, a, g, tau, kappa, base) - _loss(cfg, W, H, lg, b, g, tau, kappa, base)) / (2 * h)
        assert abs(fd - ds[idx]) <= 1e-6 * abs(fd)


def test_shift_backward_matches_torch_autograd_of_the_gathered_grid():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(31)
    O, I, gs = 3, 64, 32
    cfg = gsq.Config(O, I, L8, gs, precision="fp64", relaxation="shift")
    H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, 5))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    base = rng.integers(0, 8, (O, I))
    g = philox.gumbel(1, np.arange(O * I), 0, 5).reshape(O, I, 5)
    tau, kappa = 0.4, 1.5
    s_coord = gsq.expand_scales(sc, gs)
    cand = gsq.candidates(cfg, base)
    p, v, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa, cand)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.backward(cfg, (-2 * P)[None], s_coord[None], p[None], v[None], tau, kappa, cand[None])
    # torch: the level of shift delta is the grid gathered at clamp(j0 + delta, 0, 7)
    idx = torch.clamp(torch.tensor(base)[..., None] + torch.arange(-2, 3), 0, 7)
    levels = torch.tensor(L8, dtype=torch.float64)[idx]
    tl = torch.tensor(lg, requires_grad=True)
    ts = torch.tensor(sc, requires_grad=True)
    pt = torch.softmax((kappa * tl + torch.tensor(g)) / tau, dim=-1)
    Rt = torch.tensor(W) - ts.repeat_interleave(gs, dim=-1) * (pt * levels).sum(-1)
    (Rt @ torch.tensor(H) * Rt).sum().backward()
    np.testing.assert_allclose(dl[0], tl.grad.numpy(), rtol=1e-9, atol=1e-12 * np.abs(dl).max())
    np.testing.assert_allclose(ds[0], ts.grad.numpy(), rtol=1e-9)


def test_shift_init_is_the_centred_prior_around_the_rtn_code():
    """App. A for b > 2: candidates are the shifts, centred at 0, mean-subtracted:
    -delta^2/2 + 1 = (-1, 1/2, 1, 1/2, -1), times alpha sigma_init; j0 is the RTN code and
    hardening the initial state returns it."""
    rng = np.random.default_rng(32)
    W = rng.normal(0, 0.02, (1, 6, 128)).astype(np.float32)
    cfg = gsq.Config(6, 128, L8, 64, init_noise=False, relaxation="shift", alpha=6.0, sigma_init=0.5)
    st = gsq.init_layer(cfg, W)
    np.testing.assert_array_equal(st.logits, np.broadcast_to(np.float32(3.0) * np.array(
        [-1, 0.5, 1, 0.5, -1], np.float32), st.logits.shape))
    q0 = gsq.rtn_codes(W, gsq.expand_scales(st.scales, 64), gsq.Config(6, 128, L8, 64))
    np.testing.assert_array_equal(st.base, q0)
    np.testing.assert_array_equal(gsq.hard_codes(cfg, st), q0)


# ------------------------------------------------------------------ ternary mask x sign
def test_ternary_pairs_are_sigmoids_of_twice_the_logit():
    """§3: a two-element GS with logits {-l, l} is a sigmoid of the noisy logit 2l, so the mask
    is sigmoid((2 kappa l_m + d_m) / tau) and the sign 2 sigmoid(...) - 1, d the pair's
    logistic noise (the difference of its two Gumbel values)."""
    rng = np.random.default_rng(40)
    n = 2000
    lg = rng.standard_normal((1, n, 2)) * 2
    d = philox.logistic(3, np.arange(n), 4, 2).reshape(1, n, 2)
    cfg = gsq.Config(1, n, L3, 16 if n % 16 == 0 else 1, precision="fp64", relaxation="ternary")
    for tau, kappa in ((1.0, 1.0), (0.2, 3.0)):
        p, v, _ = gsq.ternary_forward(cfg, np.zeros((1, n)), lg, np.ones((1, n)), d, tau, kappa)
        m = expit((2 * kappa * lg[..., 0] + d[..., 0]) / tau)
        b = 2 * expit((2 * kappa * lg[..., 1] + d[..., 1]) / tau) - 1
        np.testing.assert_allclose(p[..., 0, 1], m, rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(v, m * b, rtol=1e-10, atol=1e-15)


def test_ternary_pair_with_two_gumbels_equals_the_pair_with_their_difference():
    """Alg. 1 on {-l, l} with Gumbel values (g0, g1) gives the same probabilities as the pair
    driven by the single value d = g1 - g0 (the softmax sees only the difference)."""
    rng = np.random.default_rng(46)
    n = 3000
    l = rng.standard_normal(n) * 2
    g = philox.gumbel(8, np.arange(n), 2, 2)
    for tau, kappa in ((1.0, 1.0), (0.1, 2.5)):
        full = gsq.soft_sample(np.stack([-l, l], -1), g, tau, kappa)
        p0, p1 = gsq.binary_sample(l, g[:, 1] - g[:, 0], tau, kappa)
        np.testing.assert_allclose(p1, full[:, 1], rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(p0, full[:, 0], rtol=1e-12, atol=1e-300)


def test_ternary_mask_frequency_is_the_logistic_of_twice_the_logit():
    """The mask's noise is logistic, so at tau -> 0 the mask is 1 with probability
    sigmoid(2 kappa l) (checked with the generator's own noise), for the mask and the sign."""
    n = 200_000
    d = philox.logistic(9, np.arange(n), 7, 2)
    for l, kappa in ((0.3, 1.0), (-0.8, 0.5)):
        p = expit(2 * kappa * l)
        for j in (0, 1):
            frac = np.mean(2 * kappa * l + d[:, j] > 0)
            assert abs(frac - p) < 5 * math.sqrt(p * (1 - p) / n)


def test_ternary_low_temperature_limit():
    """tau -> 0: W_hat = s * [noisy mask logit > 0] * sign(noisy sign logit) (Alg. 2)."""
    rng = np.random.default_rng(41)
    n = 512
    cfg = gsq.Config(1, n, L3, 16, precision="fp64", relaxation="ternary")
    lg = rng.standard_normal((1, n, 2))
    d = philox.logistic(5, np.arange(n), 3, 2).reshape(1, n, 2)
    _, v, _ = gsq.ternary_forward(cfg, np.zeros((1, n)), lg, np.ones((1, n)), d, 1e-7, 1.0)
    hard = (2 * lg[..., 0] + d[..., 0] > 0) * np.sign(2 * lg[..., 1] + d[..., 1])
    np.testing.assert_allclose(v, hard, atol=1e-9)


@pytest.mark.parametrize("tau,kappa", [(1.0, 1.0), (0.3, 2.0)])
def test_ternary_backward_matches_finite_differences(tau, kappa):
    rng = np.random.default_rng(42)
    O, I, gs = 2, 32, 16
    cfg = gsq.Config(O, I, L3, gs, precision="fp64", relaxation="ternary")
    H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, 2))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    g = philox.logistic(2, np.arange(O * I), 1, 2).reshape(O, I, 2)
    s_coord = gsq.expand_scales(sc, gs)
    p, v, R = gsq.ternary_forward(cfg, W, lg, s_coord, g, tau, kappa)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.ternary_backward(cfg, (-2 * P)[None], s_coord[None], p[None], tau, kappa)
    dl, ds = dl[0], ds[0]
    for idx in [(0, 0, 0), (0, 0, 1), (1, 5, 0), (1, 31, 1), (0, 17, 1)]:
        h = 1e-6 * max(1.0, abs(lg[idx]))
        a, b = lg.copy(), lg.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss(cfg, W, H, a, sc, g, tau, kappa) - _loss(cfg, W, H, b, sc, g, tau, kappa)) / (2 * h)
        assert abs(fd - dl[idx]) <= 1e-6 * max(abs(fd), np.abs(dl).max() * 1e-3), (idx, fd, dl[idx])
    for idx in [(0, 0), (1, 1)]:
        h = 1e-6 * sc[idx]
        a, b = sc.copy(), sc.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss(cfg, W, H, lg, a, g, tau, kappa) - _loss(cfg, W, H, lg, b, g, tau, kappa)) / (2 * h)
        assert abs(fd - ds[idx]) <= 1e-6 * abs(fd)


def test_ternary_backward_matches_torch_autograd_of_alg2():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(43)
    O, I, gs = 3, 64, 32
    cfg = gsq.Config(O, I, L3, gs, precision="fp64", relaxation="ternary")
    H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, 2))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    g = philox.gumbel(1, np.arange(O * I), 0, 4).reshape(O, I, 4)
    d = np.stack([g[..., 1] - g[..., 0], g[..., 3] - g[..., 2]], -1)
    tau, kappa = 0.4, 1.5
    s_coord = gsq.expand_scales(sc, gs)
    p, v, R = gsq.ternary_forward(cfg, W, lg, s_coord, d, tau, kappa)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.ternary_backward(cfg, (-2 * P)[None], s_coord[None], p[None], tau, kappa)
    tl = torch.tensor(lg, requires_grad=True)
    ts = torch.tensor(sc, requires_grad=True)
    gt = torch.tensor(g)

    def gs_pair(l, gg, vals):
        pr = torch.softmax((kappa * torch.stack([-l, l], -1) + gg) / tau, dim=-1)
        return (pr * torch.tensor(vals, dtype=torch.float64)).sum(-1)

    m = gs_pair(tl[..., 0], gt[..., 0:2], (0.0, 1.0))
    b = gs_pair(tl[..., 1], gt[..., 2:4], (-1.0, 1.0))
    Rt = torch.tensor(W) - ts.repeat_interleave(gs, dim=-1) * m * b
    (Rt @ torch.tensor(H) * Rt).sum().backward()
    np.testing.assert_allclose(dl[0], tl.grad.numpy(), rtol=1e-9, atol=1e-12 * np.abs(dl).max())
    np.testing.assert_allclose(ds[0], ts.grad.numpy(), rtol=1e-9)


def test_ternary_init_is_eq3_scaled_by_eq4():
    """Eq. 3 for RTN ternary codes -1 / 0 / +1: (l_m, l_b) = (1, -1) / (-1, 0) / (1, 1), then
    Eq. 4 without noise multiplies by alpha sigma_init; hardening returns the RTN codes."""
    rng = np.random.default_rng(44)
    W = rng.normal(0, 0.02, (1, 4, 256)).astype(np.float32)
    cfg = gsq.Config(4, 256, L3, 128, init_noise=False, relaxation="ternary", alpha=3.0, sigma_init=1.0)
    st = gsq.init_layer(cfg, W)
    q0 = st.extra["q0"]
    assert set(np.unique(q0)) == {0, 1, 2}
    table = {0: (3.0, -3.0), 1: (-3.0, 0.0), 2: (3.0, 3.0)}
    for code, (lm, lb) in table.items():
        sel = q0 == code
        assert np.all(st.logits[sel][:, 0] == lm) and np.all(st.logits[sel][:, 1] == lb)
    np.testing.assert_array_equal(gsq.hard_codes(cfg, st), q0)


def test_ternary_hardening_thresholds_and_ties():
    """Alg. 2's final step: active iff l_m >= 0, positive iff l_b >= 0 (zero goes to active and
    positive); the code indexes (-1, 0, 1)."""
    cfg = gsq.Config(1, 16, L3, 16, relaxation="ternary")
    cases = [((0.0, 0.0), 2), ((0.0, -1e-30), 0), ((-1e-30, 5.0), 1), ((2.0, -3.0), 0),
             ((2.0, 0.0), 2), ((-2.0, -3.0), 1), ((1.0, 1.0), 2)]
    lg = np.array([c for c, _ in cases], np.float32)[None, None]
    st = gsq.State(lg, None, None, None, None, None)
    np.testing.assert_array_equal(gsq.hard_codes(cfg, st)[0, 0], [code for _, code in cases])


def test_ternary_init_noise_is_two_standard_normals_per_coordinate():
    W = np.random.default_rng(45).normal(0, 0.02, (1, 64, 256)).astype(np.float32)
    cfg = gsq.Config(64, 256, L3, 128, relaxation="ternary", alpha=3.0, sigma_init=1.0)
    noisy = gsq.init_layer(cfg, W).logits.astype(np.float64)
    clean = gsq.init_layer(gsq.Config(64, 256, L3, 128, relaxation="ternary", alpha=3.0,
                                      init_noise=False), W).logits
    eps = (noisy - clean).reshape(-1)
    assert abs(eps.mean()) < 5 / math.sqrt(eps.size) and abs(eps.var() - 1) < 0.05
    assert stats.kstest(eps, "norm").pvalue > 1e-4


# ------------------------------------------------------------------ base-3 packing
def test_base3_pack_matches_integer_arithmetic_and_round_trips():
    rng = np.random.default_rng(46)
    B, O, I, gs = 2, 3, 128, 64
    codes = rng.integers(0, 3, (B, O, I)).astype(np.uint8)
    codes.reshape(-1)[:8] = [2, 2, 2, 2, 2, 0, 1, 2]
    sc16 = rng.uniform(0.001, 0.1, (B, O, I // gs)).astype(np.float16)
    data = pack.pack_base3(codes, sc16)
    n = B * O * I
    assert data.size == pack.packed_size_base3(B, O, I, gs) == -(-n // 5) + 2 * B * O * I // gs
    assert data[0] == 242                       # 2 + 2*3 + 2*9 + 2*27 + 2*81
    flat = [int(c) for c in codes.reshape(-1)] + [0] * (-n % 5)
    for j in range(0, len(flat), 5):
        x = 0
        for t in reversed(flat[j:j + 5]):       # Horner: t0 + 3 (t1 + 3 (t2 + ...))
            x = 3 * x + t
        assert data[j // 5] == x
    c2, s2 = pack.unpack_base3(data, B, O, I, gs)
    np.testing.assert_array_equal(c2, codes)
    np.testing.assert_array_equal(s2.view(np.uint16), sc16.view(np.uint16))


def test_ternary_bits_per_parameter_of_table_1():
    """Tab. 1 books ternary GSQ at 1.71 bpp = log2(3) + 16/128 (entropy of a trit plus one fp16
    scale per 128); the byte-aligned base-3 format stores 8/5 + 16/128 = 1.725."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "bpp_table1_ternary.txt"))
            if l.strip() and l[0] != "#"]
    for K, gs, bpp in rows:
        K, gs = int(K), int(gs)
        assert f"{math.log2(K) + 16 / gs:.2f}" == bpp
        size = pack.packed_size_base3(1, 4096, 4096, gs)
        assert size * 8 / 4096 ** 2 == pytest.approx(1.6 + 16 / gs)
        assert size * 8 / 4096 ** 2 - float(bpp) < 0.02
