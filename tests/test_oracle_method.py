"""Pins of the oracle's method: each check is a fact fixed by the paper or by mathematics."""
import itertools

import numpy as np
import pytest

from oracle import gsq, philox

L4 = (-1.5, -0.5, 0.5, 1.5)
L3 = (-1.0, 0.0, 1.0)


def _spd(rng, n, tokens=None):
    X = rng.standard_normal((tokens or 2 * n, n)) * rng.lognormal(0, 0.5, n)
    return X, X.T @ X


def _state(cfg, rng, B=1, spread=2.0):
    O, I, K = cfg.out_features, cfg.in_features, cfg.K
    lg = (rng.standard_normal((B, O, I, K)) * spread).astype(np.float32)
    sc = rng.uniform(0.01, 0.03, (B, O, I // cfg.gs)).astype(np.float32)
    z = np.zeros_like(lg)
    zs = np.zeros_like(sc)
    return gsq.State(lg, z, z.copy(), sc, zs, zs.copy(), 0)


# ------------------------------------------------------------------ Alg. 1 limits and special cases
def test_low_temperature_limit_is_the_hard_gumbel_max_sample():
    """As tau -> 0 the soft sample collapses onto c[argmax(kappa l + g)] (§3, Alg. 1)."""
    rng = np.random.default_rng(0)
    cfg = gsq.Config(4, 256, L4, 128, precision="fp64")
    l = rng.standard_normal((4, 256, 4))
    g = philox.gumbel(0, np.arange(4 * 256), 5, 4).reshape(4, 256, 4)
    s = np.full((4, 256), 0.02)
    for kappa in (1.0, 3.0):
        p, v, _ = gsq.forward(cfg, np.zeros((4, 256)), l, s, g, 1e-6, kappa)
        hard = np.asarray(L4)[np.argmax(kappa * l + g, axis=-1)]
        np.testing.assert_allclose(s * v, s * hard, atol=1e-6 * 0.02 * 1.5, rtol=0)


def test_binary_case_is_a_sigmoid_of_twice_the_logit():
    """K = 2 with logits {-l, +l}: the softmax is a sigmoid of the noisy logit 2l (§3)."""
    rng = np.random.default_rng(1)
    l = rng.standard_normal(1000) * 2
    g = philox.gumbel(4, np.arange(1000), 0, 2)
    for tau, kappa in ((1.0, 1.0), (0.3, 2.0)):
        p = gsq.soft_sample(np.stack([-l, l], -1), g, tau, kappa)
        sig = 1 / (1 + np.exp(-(2 * kappa * l + g[:, 1] - g[:, 0]) / tau))
        np.testing.assert_allclose(p[:, 1], sig, rtol=1e-12, atol=1e-15)
    p = gsq.soft_sample(np.stack([-l, l], -1), np.zeros((1000, 2)), 1.0, 1.0)
    np.testing.assert_allclose(p[:, 1], 1 / (1 + np.exp(-2 * l)), rtol=1e-12)


def test_soft_sample_is_the_formula_of_alg1_without_max_shift():
    rng = np.random.default_rng(2)
    l = rng.standard_normal((50, 5))
    g = rng.gumbel(size=(50, 5))
    tau, kappa = 0.7, 1.3
    num = np.exp((kappa * l + g) / tau)
    np.testing.assert_allclose(gsq.soft_sample(l, g, tau, kappa), num / num.sum(1, keepdims=True),
                               rtol=1e-12)


# ------------------------------------------------------------------ Eq. 1 objective
def test_loss_through_H_equals_output_error_from_X():
    """tr(R H R^T) with H = X^T X equals ||X W_hat^T - X W^T||_F^2 of Eq. 1 (linear layer)."""
    rng = np.random.default_rng(3)
    O, I = 6, 256
    X, H = _spd(rng, I, 300)
    cfg = gsq.Config(O, I, L4, 128, precision="fp64")
    W = rng.normal(0, 0.02, (1, O, I))
    st = _state(cfg, rng)
    g = philox.gumbel(0, gsq.coord_index(cfg, 0, np.arange(O)), 0, 4).reshape(O, I, 4)
    s_coord = gsq.expand_scales(st.scales[0], 128)
    _, v, R = gsq.forward(cfg, W[0], st.logits[0], s_coord, g, 0.5, 1.0)
    _, L = gsq.contract(cfg, R, H)
    W_hat = s_coord * v
    direct = np.sum((X @ W_hat.T - X @ W[0].T) ** 2)
    assert abs(L - direct) <= 1e-12 * direct


def test_step_with_the_contraction_operand_rounded_beforehand_is_identical():
    """Long runs pass H already rounded to the contraction's precision: same values, same step."""
    rng = np.random.default_rng(4)
    cfg = gsq.Config(8, 256, L4, 128, batch=2, precision="bf16", seed=3)
    W = rng.normal(0, 0.02, (2, 8, 256))
    Hs = gsq.symmetrize(np.stack([_spd(rng, 256)[1] for _ in range(2)]))
    rows, batches = np.array([1, 6]), np.array([1])
    st = gsq.init_layer(cfg, W, rows=rows, batches=batches)
    prm = gsq.StepParams(tau=0.4, kappa=1.0, lr_logits=1e-2, lr_scales=5e-5)
    a, la = gsq.step(cfg, W, Hs[batches], st, prm, rows=rows, batches=batches)
    b, lb = gsq.step(cfg, W, Hs[batches], st, prm, rows=rows, batches=batches,
                     Hc=gsq.to_contraction_precision(cfg, Hs[batches]))
    np.testing.assert_array_equal(la, lb)
    for k in ("logits", "m", "v", "scales", "m_s", "v_s"):
        np.testing.assert_array_equal(getattr(a, k), getattr(b, k))


def test_zero_loss_when_weights_lie_on_the_grid():
    """W = s c[q*] with each group reaching the outer level: init recovers s and q*, hard loss 0,
    and the noise-free optimisation keeps q* (it is the global optimum, loss 0)."""
    rng = np.random.default_rng(4)
    O, I, gs = 8, 256, 128
    c = np.asarray(L4)
    s_true = (2.0 ** -6 * (1 + rng.integers(0, 8, (1, O, I // gs)) / 8)).astype(np.float32)
    q = rng.integers(0, 4, (1, O, I))
    q[..., ::gs] = 3                              # every group reaches +1.5
    W = (gsq.expand_scales(s_true, gs) * c[q]).astype(np.float32)
    X, H = _spd(rng, I)
    cfg = gsq.Config(O, I, L4, gs, precision="fp32", init_noise=False)
    st = gsq.init_layer(cfg, W)
    np.testing.assert_array_equal(st.scales, s_true)
    np.testing.assert_array_equal(st.extra["q0"], q)
    codes, eff, hl = gsq.harden_layer(cfg, W, gsq.symmetrize(H), st)
    np.testing.assert_array_equal(codes, q)
    assert hl[0] == 0.0
    prm = gsq.StepParams(tau=1.0, lr_scales=0.0)
    for t in range(20):
        prm.tau = gsq.tau_schedule(t, 20)
        st, _ = gsq.step(cfg, W, gsq.symmetrize(H), st, prm)
    np.testing.assert_array_equal(gsq.harden(st.logits), q)


@pytest.mark.parametrize("K,levels", [(3, L3), (4, L4)])
def test_bruteforce_hard_losses_and_diagonal_H_optimum(K, levels):
    """Enumerate all K^8 assignments of a 1 x 8 layer: the oracle's hard loss equals the direct
    output error from X for every one; with diagonal H the optimum is per-coordinate RTN."""
    rng = np.random.default_rng(10 + K)
    I, gs = 8, 8
    X, H = _spd(rng, I, 40)
    W = rng.normal(0, 0.02, (1, 1, I)).astype(np.float32)
    cfg = gsq.Config(1, I, levels, gs, precision="fp64")
    st = gsq.init_layer(gsq.Config(1, I, levels, gs, precision="fp64", init_noise=False), W)
    s = st.scales
    allq = np.array(list(itertools.product(range(K), repeat=I)), dtype=np.uint8)
    c = np.asarray(levels)
    Wq_all = s[0, 0, 0].astype(np.float64) * c[allq]
    direct = np.sum((X @ (Wq_all - W[0, 0].astype(np.float64)).T) ** 2, axis=0)
    for n in rng.choice(len(allq), 50, replace=False):
        hl = gsq.hard_loss(cfg, W, H, allq[n].reshape(1, 1, I), s)[0]
        assert abs(hl - direct[n]) <= 1e-9 * direct[n]
    direct_diag = np.einsum("ni,i,ni->n", Wq_all - W[0, 0], np.diag(H), Wq_all - W[0, 0])
    best = allq[np.argmin(direct_diag)]
    np.testing.assert_array_equal(best, st.extra["q0"][0, 0])
    # noise-free soft loss at tau -> 0 equals the hard loss of argmax(l)
    q = allq[int(np.argmin(direct))]
    lg = np.where(np.arange(K) == q[:, None], 3.0, 0.0)[None, None]
    p, v, R = gsq.forward(cfg, W[0], lg[0], gsq.expand_scales(s, gs)[0], np.zeros((1, I, K)), 1e-4, 1.0)
    assert abs(gsq.contract(cfg, R, H)[1] - direct.min()) <= 1e-9 * direct.min()


# ------------------------------------------------------------------ gradients
def _loss_fn(cfg, W, H, lg, sc, g, tau, kappa):
    s_coord = gsq.expand_scales(sc, cfg.gs)
    _, _, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa)
    return gsq.contract(cfg, R, H)[1]


@pytest.mark.parametrize("tau,kappa", [(1.0, 1.0), (0.3, 2.0)])
def test_backward_matches_central_finite_differences(tau, kappa):
    rng = np.random.default_rng(20)
    O, I, gs, K = 2, 32, 16, 4
    cfg = gsq.Config(O, I, L4, gs, precision="fp64")
    _, H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, K))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    g = philox.gumbel(1, np.arange(O * I), 2, K).reshape(O, I, K)
    s_coord = gsq.expand_scales(sc, gs)
    p, v, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.backward(cfg, (-2 * P)[None], s_coord[None], p[None], v[None], tau, kappa)
    dl, ds = dl[0], ds[0]
    for idx in [(0, 0, 0), (1, 5, 2), (0, 31, 3), (1, 17, 1)]:
        h = 1e-6 * max(1.0, abs(lg[idx]))
        a, b = lg.copy(), lg.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss_fn(cfg, W, H, a, sc, g, tau, kappa) - _loss_fn(cfg, W, H, b, sc, g, tau, kappa)) / (2 * h)
        assert abs(fd - dl[idx]) <= 1e-6 * max(abs(fd), np.abs(dl).max() * 1e-3)
    for idx in [(0, 0), (1, 1)]:
        h = 1e-6 * sc[idx]
        a, b = sc.copy(), sc.copy()
        a[idx] += h
        b[idx] -= h
        fd = (_loss_fn(cfg, W, H, lg, a, g, tau, kappa) - _loss_fn(cfg, W, H, lg, b, g, tau, kappa)) / (2 * h)
        assert abs(fd - ds[idx]) <= 1e-6 * abs(fd)


def test_backward_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(21)
    O, I, gs, K = 3, 64, 32, 3
    cfg = gsq.Config(O, I, L3, gs, precision="fp64")
    _, H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    lg = rng.standard_normal((O, I, K))
    sc = rng.uniform(0.01, 0.03, (O, I // gs))
    g = philox.gumbel(1, np.arange(O * I), 0, K).reshape(O, I, K)
    tau, kappa = 0.4, 1.5
    s_coord = gsq.expand_scales(sc, gs)
    p, v, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa)
    P, _ = gsq.contract(cfg, R, H)
    dl, ds = gsq.backward(cfg, (-2 * P)[None], s_coord[None], p[None], v[None], tau, kappa)
    tl = torch.tensor(lg, requires_grad=True)
    ts = torch.tensor(sc, requires_grad=True)
    pt = torch.softmax((kappa * tl + torch.tensor(g)) / tau, dim=-1)
    vt = (pt * torch.tensor(L3, dtype=torch.float64)).sum(-1)
    Rt = torch.tensor(W) - ts.repeat_interleave(gs, dim=-1) * vt
    (Rt @ torch.tensor(H) * Rt).sum().backward()
    np.testing.assert_allclose(dl[0], tl.grad.numpy(), rtol=1e-9, atol=1e-12 * np.abs(dl).max())
    np.testing.assert_allclose(ds[0], ts.grad.numpy(), rtol=1e-9)


def test_logit_gradient_obeys_lemma_b1():
    """App. B, Lemma B.1: |dL/da_i| <= (G/tau)(1 - y_max) with G = ||dL/dy||_1; dl = kappa dL/da."""
    rng = np.random.default_rng(22)
    O, I, K = 4, 128, 4
    cfg = gsq.Config(O, I, L4, 128, precision="fp64")
    _, H = _spd(rng, I)
    W = rng.normal(0, 0.02, (O, I))
    for tau in (1.0, 0.2, 0.05):
        lg = rng.standard_normal((O, I, K)) * 3
        sc = np.full((O, 1), 0.02)
        g = philox.gumbel(0, np.arange(O * I), 0, K).reshape(O, I, K)
        kappa = 1.7
        s_coord = gsq.expand_scales(sc, 128)
        p, v, R = gsq.forward(cfg, W, lg, s_coord, g, tau, kappa)
        G = -2 * gsq.contract(cfg, R, H)[0]
        dl = gsq.backward(cfg, G[None], s_coord[None], p[None], v[None], tau, kappa)[0][0]
        Gy = np.abs(G * s_coord)[..., None] * np.abs(np.asarray(L4)).sum()
        # 1 - y_max written as the mass of the other levels (no cancellation when y_max -> 1)
        top = np.argmax(p, -1)[..., None]
        tail = np.where(np.arange(K) == top, 0.0, p).sum(-1, keepdims=True)
        bound = kappa * Gy / tau * tail
        assert np.all(np.abs(dl) <= bound * (1 + 1e-9) + 1e-300)
        # second inequality of the lemma: 1 - y_max <= (K - 1) exp(-Delta / tau)
        a = kappa * lg + g
        srt = np.sort(a, -1)
        assert np.all(tail[..., 0] <= (K - 1) * np.exp(-(srt[..., -1] - srt[..., -2]) / tau) * (1 + 1e-9))


def test_adam_matches_torch_optim_adam():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(23)
    th = rng.standard_normal(1000).astype(np.float32)
    m = np.zeros_like(th)
    v = np.zeros_like(th)
    p = torch.tensor(th.astype(np.float64), requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-2, betas=(0.9, 0.95), eps=1e-8)
    cur = th
    for n in range(1, 8):
        gr = rng.standard_normal(1000) * 10.0 ** rng.integers(-6, 1, 1000)
        cur, m, v = gsq.adam(cur, m, v, gr, 1e-2, 0.9, 0.95, 1e-8, n)
        p.grad = torch.tensor(gr)
        opt.step()
        # torch keeps float64 state; the oracle stores float32 each step
        np.testing.assert_allclose(cur, p.detach().numpy(), rtol=0, atol=2e-6)


def test_adamw_matches_torch_optim_adamw():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(24)
    th = rng.standard_normal(500).astype(np.float32)
    m = np.zeros_like(th)
    v = np.zeros_like(th)
    p = torch.tensor(th.astype(np.float64), requires_grad=True)
    opt = torch.optim.AdamW([p], lr=1e-2, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.5)
    cur = th
    for n in range(1, 6):
        gr = rng.standard_normal(500) * 10.0 ** rng.integers(-4, 1, 500)
        cur, m, v = gsq.adam(cur, m, v, gr, 1e-2, 0.9, 0.95, 1e-8, n, wd=0.5)
        p.grad = torch.tensor(gr)
        opt.step()
        np.testing.assert_allclose(cur, p.detach().numpy(), rtol=0, atol=2e-6)


def test_lion_properties():
    """Lion's defining properties (Chen et al., 2023): without momentum it is signSGD; every
    step has size exactly lr; weight decay alone scales by (1 - lr wd); the sign follows the
    beta1 interpolation, not the stored moment; the moment then moves with beta2."""
    rng = np.random.default_rng(25)
    th = rng.standard_normal(1000)
    g = rng.standard_normal(1000)
    t1, m1 = gsq.lion(th, np.zeros(1000), g, 0.01, 0.0, 0.0)
    np.testing.assert_allclose(t1, th - 0.01 * np.sign(g), atol=1e-6)
    np.testing.assert_allclose(m1, g, rtol=1e-6)
    m = rng.standard_normal(1000)
    t2, _ = gsq.lion(th, m, g, 0.01, 0.9, 0.99)
    np.testing.assert_allclose(np.abs(t2 - th), 0.01, rtol=1e-4)
    t3, _ = gsq.lion(th, np.zeros(1000), np.zeros(1000), 0.01, 0.9, 0.99, wd=2.0)
    np.testing.assert_allclose(t3, th * (1 - 0.02), rtol=1e-6)
    # moment and gradient of opposite signs: the step follows 0.9 m + 0.1 g
    m4 = np.array([1.0, -1.0, 0.05, -0.05])
    g4 = np.array([-5.0, 5.0, -5.0, 5.0])
    t4, m4b = gsq.lion(np.zeros(4), m4, g4, 1.0, 0.9, 0.99)
    np.testing.assert_array_equal(t4, -np.sign(0.9 * m4 + 0.1 * g4).astype(np.float32))
    np.testing.assert_allclose(m4b, 0.99 * m4 + 0.01 * g4, rtol=1e-6)


# ------------------------------------------------------------------ initialisation (Eq. 4, App. A)
def test_init_logits_prior_and_noise():
    rng = np.random.default_rng(30)
    W = rng.normal(0, 0.02, (1, 8, 256)).astype(np.float32)
    base = gsq.Config(8, 256, L4, 128, init_noise=False, alpha=6.0, sigma_init=1.0)
    st = gsq.init_layer(base, W)
    q0 = st.extra["q0"]
    # the prior favours the RTN level, is mean-free over the levels, and is the Gaussian bump
    np.testing.assert_array_equal(np.argmax(st.logits, -1), q0)
    np.testing.assert_allclose(st.logits.astype(np.float64).sum(-1), 0, atol=1e-5)
    c = np.asarray(L4)
    bump = -0.5 * (c - c[q0][..., None]) ** 2
    np.testing.assert_allclose(st.logits, 6 * (bump - bump.mean(-1, keepdims=True)), rtol=1e-6)
    noisy = gsq.init_layer(gsq.Config(8, 256, L4, 128, init_noise=True, sigma_init=0.5), W)
    eps = philox.init_normals(0, np.arange(8 * 256), 4).reshape(1, 8, 256, 4)
    np.testing.assert_allclose(noisy.logits, 0.5 * (eps + st.logits), rtol=1e-6, atol=1e-6)


def test_rtn_codes_and_absmax_scales_by_enumeration():
    rng = np.random.default_rng(31)
    W = rng.normal(0, 0.02, (1, 4, 256)).astype(np.float32)
    W[0, 0, :128] = 0.0                                   # an all-zero group
    cfg = gsq.Config(4, 256, L4, 128, init_noise=False)
    st = gsq.init_layer(cfg, W)
    for o in range(4):
        for g in range(2):
            grp = W[0, o, 128 * g:128 * (g + 1)]
            s = np.float32(np.abs(grp).max()) / np.float32(1.5) if np.abs(grp).max() > 0 else 1.0
            assert st.scales[0, o, g] == np.float32(s)
            for i in range(0, 128, 7):
                u = float(np.float32(grp[i]) / np.float32(s))
                best = min(range(4), key=lambda k: (abs(u - L4[k]), k))
                assert st.extra["q0"][0, o, 128 * g + i] == best


def test_superblock_scales_reconstruct_exactly():
    rng = np.random.default_rng(32)
    W = rng.normal(0, 0.02, (2, 4, 512)).astype(np.float32)
    W[0, 0, :16] = 0
    cfg = gsq.Config(4, 512, tuple(np.arange(-3.5, 4, 1.0)), layout="superblock", batch=2)
    d, sc, eff = gsq.superblock_scales(W, cfg)
    assert d.dtype == np.float16 and sc.max() <= 63
    d32 = np.repeat(d.astype(np.float32), 16, axis=-1)
    assert np.all(eff == d32 * sc.astype(np.float32))    # exact float32 product
    raw = np.abs(W.reshape(2, 4, 32, 16)).max(-1) / np.float32(3.5)
    assert np.all(np.abs(eff - raw) <= 0.5 * d32 * (1 + 1e-6) + 1e-12)
    assert eff[0, 0, 0] == 0


# ------------------------------------------------------------------ a planted mistake is caught
def test_a_planted_sign_error_in_the_backward_is_caught(monkeypatch):
    """Plant a plausible mistake in the oracle's backward (c_k + v instead of c_k - v) and check
    that the finite-difference pin rejects it."""
    orig = gsq.backward

    def wrong(cfg, G, s_coord, p, v, tau, kappa):
        c = cfg.levels64()
        dlog = (G * s_coord * (kappa / tau))[..., None] * p * (c + v[..., None])
        return dlog, orig(cfg, G, s_coord, p, v, tau, kappa)[1]

    monkeypatch.setattr(gsq, "backward", wrong)
    with pytest.raises(AssertionError):
        test_backward_matches_central_finite_differences(1.0, 1.0)


# ------------------------------------------------------------------ multi-sample averaging (§3.3)
def _tiny_problem(seed=40):
    rng = np.random.default_rng(seed)
    O, I, K = 2, 16, 3
    _, H = _spd(rng, I)
    W = rng.normal(0, 0.02, (1, O, I))
    cfg = gsq.Config(O, I, L3, 16, precision="fp64", seed=3)
    st = _state(cfg, rng, spread=0.5)
    return cfg, W, H, st


def test_many_sample_gradient_matches_an_independent_monte_carlo_estimate():
    """With M draws the averaged gradient estimates E_g[dL/dl]; numpy's own Gumbel generator
    (an independent source) estimates the same expectation."""
    cfg, W, H, st = _tiny_problem()
    tau, M = 0.5, 3000
    prm = gsq.StepParams(tau=tau, lr_scales=1e-5, samples=M)
    _, _, inter = gsq.step(cfg, W, H, st, prm, want=True)
    ours = inter["dlogits"][0]
    rng = np.random.default_rng(77)
    s_coord = gsq.expand_scales(st.scales[0], 16)
    acc = []
    for _ in range(M):
        g = rng.gumbel(size=(2, 16, 3))
        p, v, R = gsq.forward(cfg, W[0], st.logits[0], s_coord, g, tau, 1.0)
        G = -2 * gsq.contract(cfg, R, H)[0]
        acc.append(gsq.backward(cfg, G[None], s_coord[None], p[None], v[None], tau, 1.0)[0][0])
    acc = np.stack(acc)
    ref_mean, sem = acc.mean(0), acc.std(0) / np.sqrt(M)
    # difference of two independent means: standard error sqrt(2) * sem
    assert np.all(np.abs(ours - ref_mean) <= 6 * np.sqrt(2) * sem + 1e-12)


def test_sample_averaging_divides_the_gradient_variance():
    """Var of the M-sample gradient across steps (independent noise per step) ~ Var / M."""
    cfg, W, H, st = _tiny_problem(41)
    var = {}
    for M in (1, 4):
        grads = []
        for t in range(150):
            s = st.copy()
            s.t = t
            prm = gsq.StepParams(tau=0.5, samples=M)
            grads.append(gsq.step(cfg, W, H, s, prm, want=True)[2]["dlogits"][0])
        var[M] = np.stack(grads).var(0).sum()
    assert 2.5 < var[1] / var[4] < 6.0, var[1] / var[4]
