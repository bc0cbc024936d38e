"""Helpers shared by the GPU parity tests: running the C ABI and the oracle on the same state."""
import numpy as np

from oracle import gsq as ref
from paper_2604_18556_amd import binding as B

PREC = {"fp32": B.PREC_FP32, "bf16": B.PREC_BF16}
LAYOUT = {"group": B.LAYOUT_GROUP, "superblock": B.LAYOUT_SUPERBLOCK, "base3": B.LAYOUT_BASE3}
RELAX = {"grid": B.RELAX_GRID, "shift": B.RELAX_SHIFT, "ternary": B.RELAX_TERNARY}


def rel_err(a, b):
    """max |a - b| / max |b| over the tensor (the parity metric); 0 when both are zero."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.abs(b).max() if b.size else 0.0
    num = np.abs(a - b).max() if b.size else 0.0
    return 0.0 if num == 0 else num / den


def layer_inputs(O, I, batch=1, bf16=True, seed=0, tokens=None):
    """A small seeded layer shaped like the workloads: N(0, 0.02^2) weights with 0.1 % x10
    outliers (bf16-representable if asked), H from Student-t(4) tokens with LogNormal channel
    scales."""
    from paper_2604_18556_amd import inputs
    rng = np.random.default_rng(100 + seed)
    W = rng.normal(0, 0.02, (batch, O, I)).astype(np.float32)
    W.reshape(-1)[rng.choice(W.size, max(1, W.size // 1000), replace=False)] *= 10
    if bf16:
        W = inputs.to_bf16_values(W)
    Hs = []
    for b in range(batch):
        X = rng.standard_t(4, (tokens or 2 * I, I)) * rng.lognormal(0, 0.5, I)
        Hs.append((X.T @ X).astype(np.float32))
    return W, np.stack(Hs)


def warm_state(st, rng):
    """A state with non-zero optimiser moments (as after some steps)."""
    st = st.copy()
    st.m = (rng.standard_normal(st.m.shape) * 1e-3).astype(np.float32)
    st.v = (rng.uniform(0.5, 2, st.v.shape) * 1e-6).astype(np.float32)
    st.m_s = (rng.standard_normal(st.m_s.shape) * 1e-4).astype(np.float32)
    st.v_s = (rng.uniform(0.5, 2, st.v_s.shape) * 1e-8).astype(np.float32)
    st.t = 7
    return st


def configs(rcfg):
    """(binding config, oracle config) for one oracle Config."""
    return B.LayerConfig(rcfg.out_features, rcfg.in_features, tuple(rcfg.levels), rcfg.group_size,
                         rcfg.batch, LAYOUT[rcfg.layout], PREC[rcfg.precision], rcfg.seed,
                         rcfg.alpha, rcfg.sigma_init, rcfg.init_noise,
                         RELAX[rcfg.relaxation]), rcfg


class Pair:
    """A GPU layer and the oracle state it mirrors."""

    def __init__(self, rcfg, W, H, dev, scales_init=None):
        import torch
        self.torch = torch
        self.dev = dev
        self.bcfg, self.rcfg = configs(rcfg)
        self.W = np.asarray(W, np.float32)
        self.H = np.asarray(H, np.float32)
        wt = torch.from_numpy(self.W).to(dev)
        if rcfg.precision == "bf16":
            wt = wt.to(torch.bfloat16)
        s0 = None
        if scales_init is not None:
            s0 = torch.from_numpy(np.ascontiguousarray(scales_init, np.float32)).to(dev)
        self.layer = B.Layer(self.bcfg, wt, torch.from_numpy(self.H).to(dev), scales_init=s0)
        self.Hs = ref.symmetrize(self.H)

    # -- state transfer
    def shapes(self):
        c = self.rcfg
        return (c.batch, c.out_features, c.in_features, c.K), (c.batch, c.out_features,
                                                              c.in_features // c.gs)

    def get(self):
        t = self.torch
        ls, ss = self.shapes()
        out = {k: t.empty(ls, device=self.dev) for k in ("logits", "m", "v")}
        out.update({k: t.empty(ss, device=self.dev) for k in ("scales", "m_s", "v_s")})
        if self.rcfg.relaxation == "shift":
            out["base"] = t.empty(ls[:3], dtype=t.uint8, device=self.dev)
        step = self.layer.get_state(**out)
        st = ref.State(*(out[k].cpu().numpy() for k in ("logits", "m", "v", "scales", "m_s", "v_s")),
                       step)
        if "base" in out:
            st.base = out["base"].cpu().numpy()
        return st

    def put(self, st):
        t = self.torch
        kw = {k: t.from_numpy(np.ascontiguousarray(getattr(st, k), np.float32)).to(self.dev)
              for k in ("logits", "m", "v", "m_s", "v_s")}
        if self.rcfg.layout != "superblock":
            kw["scales"] = t.from_numpy(np.ascontiguousarray(st.scales, np.float32)).to(self.dev)
        if st.base is not None:
            kw["base"] = t.from_numpy(np.ascontiguousarray(st.base, np.uint8)).to(self.dev)
        self.layer.set_state(st.t, **kw)

    def intermediates(self):
        t = self.torch
        c = self.rcfg
        shape = (c.batch, c.out_features, c.in_features)
        R = t.empty(shape, device=self.dev, dtype=t.bfloat16 if c.precision == "bf16" else t.float32)
        G = t.empty(shape, device=self.dev)
        self.layer.intermediates(R, G)
        return R.float().cpu().numpy(), G.cpu().numpy()

    def step(self, prm, want_loss=True):
        t = self.torch
        loss = t.zeros(self.rcfg.batch, device=self.dev) if want_loss else None
        self.layer.step(prm, loss_out=loss)
        return None if loss is None else loss.cpu().numpy().astype(np.float64)


def oracle_params(p):
    return ref.StepParams(p.tau, p.kappa, p.lr_logits, p.lr_scales, p.beta1, p.beta2, p.eps,
                          p.gumbel_noise, "lion" if p.optimizer == B.OPT_LION else "adam",
                          p.weight_decay, p.samples)


def assert_state_close(gpu, orc, G_oracle, tol, n, label="", gate=None, dlogits=None):
    """Updated logits / moments / scales agree to ``tol`` (max-normalised).

    Adam's first-moment ratio m / sqrt(v) from zero moments (and Lion's sign) jumps with
    the sign of a gradient, so a logit may differ by up to 2 lr where the oracle's gradient
    is within the contraction's error of zero: |dL/dl| <= gate * max|dL/dl| when
    ``dlogits`` is given, else |G| <= gate * max|G| with G = dL/dW_hat.  Those coordinates
    are counted and must be rare; m and v, which are continuous in the gradient, have no
    exception.
    """
    gate = tol if gate is None else gate
    assert rel_err(gpu.m, orc.m) <= tol, f"{label} m {rel_err(gpu.m, orc.m):.2e}"
    assert rel_err(gpu.v, orc.v) <= tol, f"{label} v {rel_err(gpu.v, orc.v):.2e}"
    dl = np.abs(gpu.logits.astype(np.float64) - orc.logits)
    scale = np.abs(orc.logits).max()
    badc = dl > tol * scale
    if badc.any():
        if dlogits is not None:
            near0 = np.abs(dlogits) <= gate * np.abs(dlogits).max()
        else:
            near0 = (np.abs(G_oracle) <= gate * np.abs(G_oracle).max())[..., None]
        unexplained = badc & ~np.broadcast_to(near0, badc.shape)
        assert not unexplained.any(), (
            f"{label} logits differ at {int(unexplained.sum())} coordinates away from G = 0 "
            f"(max {dl[unexplained].max():.3e})")
        assert badc.sum() <= max(2, 1e-3 * badc.size), f"{label} {int(badc.sum())} sign flips"
    assert rel_err(gpu.scales, orc.scales) <= tol, f"{label} scales {rel_err(gpu.scales, orc.scales):.2e}"
    assert gpu.t == orc.t == n
