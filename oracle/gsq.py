"""Plain CPU oracle of one GSQ layer: init, relaxed step, hardening.  Test infrastructure only.

Written from the paper (Gumbel-Softmax Quantization, arXiv 2604.18556), in
float64 unless a storage precision is part of the path:

* the optimiser state (logits, moments, scales) is stored in float32;
* the noise g is float32 (the generator's output, see ``oracle.philox``);
* in the "bf16" precision the residual R and H enter the contraction rounded to
  bfloat16 (round-to-nearest-even), as the kernel's inputs are; the
  contraction itself is accumulated in float64 here;
* in the "fp32" precision R and H enter the contraction as float32 values.

Notation (the paper's where it has one): W is O x I, groups of ``gs``
consecutive inputs along a row share one scale s (§4.1 "Quantization
configuration"); every coordinate carries K logits over grid levels
c_0 < ... < c_{K-1} (§3.2, Eq. 5); H = X^T X is the layer's calibration Gram
matrix, so the reconstruction error of Eq. 1 for a linear layer is
tr((W - W_hat) H (W - W_hat)^T).

Three relaxations of a coordinate's choice (``Config.relaxation``):
* "grid": one categorical over all K grid levels (§3.2, Eq. 5);
* "shift": for wider grids, a categorical over the five index shifts
  delta in {-2..2} around a fixed initial grid index j0, the level being
  c[clip(j0 + delta)] (§3.2 "Higher bit-widths", Eq. 6);
* "ternary": the mask x sign form of §3.1 (Eq. 2, Alg. 2), two binary
  relaxations per coordinate with logits {-l, l} each.

Where the paper is silent, the reading taken is stated at the function that
takes it.
"""
from dataclasses import dataclass, field

import numpy as np

from . import philox

F32 = np.float32

RELAXATIONS = ("grid", "shift", "ternary")
SHIFTS = np.array([-2, -1, 0, 1, 2])          # the local-shift window of §3.2 (Eq. 6)
TERNARY_LEVELS = (-1.0, 0.0, 1.0)


# ----------------------------------------------------------------------------- rounding helpers
def round_f32(x):
    """Round float64 values to float32 and back (exact representable values)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_bf16(x):
    """Round to bfloat16 with round-to-nearest-even, returned as float64.

    bfloat16 keeps the top 16 bits of an IEEE float32: the value is first
    rounded to float32, then the low 16 bits are rounded away (ties to even).
    NaN/Inf are not expected here.
    """
    b = np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    b = (b + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def to_contraction_precision(cfg, x):
    """Round an operand of the contraction to the path's storage type.

    "bf16": bfloat16 (RNE); "fp32": float32; "fp64": unrounded (used only by the
    mathematical pins, e.g. finite differences).
    """
    if cfg.precision == "bf16":
        return round_bf16(x)
    if cfg.precision == "fp32":
        return round_f32(x)
    return np.asarray(x, np.float64)


# ----------------------------------------------------------------------------- configuration
@dataclass
class Config:
    """One layer (or a batch of independent layers, e.g. MoE experts)."""
    out_features: int
    in_features: int
    levels: tuple                      # the grid c_0 < ... < c_{n-1}
    group_size: int = 128              # gs, along the input dimension (§4.1)
    batch: int = 1
    layout: str = "group"              # "group" | "superblock" | "base3" (3-level grids)
    precision: str = "fp32"            # "fp32" | "bf16" | "fp64": dtype of R and H in the contraction
    seed: int = 0
    alpha: float = 6.0                 # warm-start strength of Eq. 4 (Tab. 7: 6 for 2/3-bit)
    sigma_init: float = 1.0            # overall logit scale of Eq. 4
    init_noise: bool = True
    relaxation: str = "grid"           # "grid" | "shift" | "ternary"

    def __post_init__(self):
        assert self.relaxation in RELAXATIONS, self.relaxation
        if self.relaxation == "ternary":
            assert tuple(float(c) for c in self.levels) == TERNARY_LEVELS
        if self.layout == "base3":
            assert len(self.levels) == 3

    @property
    def K(self):
        """Logits per coordinate."""
        return {"grid": len(self.levels), "shift": len(SHIFTS), "ternary": 2}[self.relaxation]

    @property
    def n_grid(self):
        """Grid cardinality (the number of code values)."""
        return len(self.levels)

    @property
    def n_noise(self):
        """Noise values per coordinate and draw: one Gumbel value per logit of a categorical,
        or one logistic value per binary pair (ternary: the mask's, then the sign's)."""
        return 2 if self.relaxation == "ternary" else self.K

    @property
    def gs(self):
        return 16 if self.layout == "superblock" else self.group_size

    def levels64(self):
        return np.asarray(self.levels, dtype=np.float32).astype(np.float64)


@dataclass
class StepParams:
    tau: float
    kappa: float = 1.0
    lr_logits: float = 1e-2
    lr_scales: float = 5e-5
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    gumbel_noise: bool = True
    optimizer: str = "adam"            # "adam" (AdamW when weight_decay > 0) | "lion"
    weight_decay: float = 0.0          # decoupled, on logits and scales
    samples: int = 1                   # independent Gumbel draws averaged per step (§3.3)


def as_f32_params(prm):
    """The step's scalars as the float32 values the library receives."""
    f = lambda x: float(np.float32(x))
    return StepParams(f(prm.tau), f(prm.kappa), f(prm.lr_logits), f(prm.lr_scales),
                      f(prm.beta1), f(prm.beta2), f(prm.eps), bool(prm.gumbel_noise),
                      prm.optimizer, f(prm.weight_decay), max(1, int(prm.samples)))


@dataclass
class State:
    """Optimiser state of one layer, float32 storage (logits in O x I x K order)."""
    logits: np.ndarray                 # (B, O, I, K) float32
    m: np.ndarray
    v: np.ndarray
    scales: np.ndarray                 # (B, O, I // gs) float32
    m_s: np.ndarray
    v_s: np.ndarray
    t: int = 0
    sb_d: np.ndarray = None            # super-block fp16 d, (B, O, I // 256)
    sb_sc: np.ndarray = None           # super-block 6-bit sub-scales, (B, O, I // 16)
    extra: dict = field(default_factory=dict)
    base: np.ndarray = None            # local shift: initial grid index j0, (B, O, I) uint8

    def copy(self):
        c = State(self.logits.copy(), self.m.copy(), self.v.copy(), self.scales.copy(),
                  self.m_s.copy(), self.v_s.copy(), self.t,
                  None if self.sb_d is None else self.sb_d.copy(),
                  None if self.sb_sc is None else self.sb_sc.copy(),
                  base=None if self.base is None else self.base.copy())
        return c


# ----------------------------------------------------------------------------- initialisation
def symmetrize(H):
    """(H + H^T) / 2, rounded to float32.

    The objective only sees the symmetric part of H (tr(R H R^T) = tr(R H^T R^T)),
    so symmetrising changes nothing mathematically and makes the gradient
    -2 R H exact (reading: the library symmetrises its copy of H).
    """
    H = np.asarray(H, dtype=np.float64)
    return round_f32((H + np.swapaxes(H, -1, -2)) * 0.5)


def group_absmax_scales(W, cfg):
    """Initial group scales: s = max|W_group| / max_k |c_k| (float32 division).

    The paper takes the initial scale from its warm start (GPTQ, Eq. 4's
    paragraph); the warm start here is round-to-nearest, whose symmetric scale
    maps the group's largest magnitude onto the outermost grid level.  An
    all-zero group gets s = 1 (reading).
    """
    B, O, I = W.shape
    gs = cfg.group_size
    absmax = np.abs(W.reshape(B, O, I // gs, gs)).max(axis=-1).astype(np.float32)
    cmax = np.float32(np.abs(cfg.levels64()).max())
    s = absmax / cmax                                   # IEEE float32 division
    s[s == 0] = 1.0
    return s.astype(np.float32)


def superblock_scales(W, cfg):
    """K-quant-style scales: 256-weight super-blocks of 16 sub-blocks of 16.

    Each sub-block j has a raw absmax scale s_j = max|W_j| / max|c|; the
    super-block stores d = fp16(max_j s_j / 63) and 6-bit integers
    sc_j = clamp(rint(s_j / d), 0, 63), and the effective scale is d * sc_j
    (§4.4 and App. E keep the optimised weights in the deployment format; the
    byte layout is ours).  Returns (d fp16 (B,O,I/256), sc uint8 (B,O,I/16),
    effective float32 scales (B,O,I/16)).
    """
    B, O, I = W.shape
    cmax = np.float32(np.abs(cfg.levels64()).max())
    absmax = np.abs(W.reshape(B, O, I // 16, 16)).max(axis=-1).astype(np.float32)
    raw = (absmax / cmax).astype(np.float32)
    per_sb = raw.reshape(B, O, I // 256, 16)
    d = (per_sb.max(axis=-1) / np.float32(63.0)).astype(np.float32).astype(np.float16)
    d32 = d.astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(d32[..., None] > 0, per_sb / d32[..., None], np.float32(0)).astype(np.float32)
    sc = np.clip(np.rint(q), 0, 63).astype(np.uint8)
    eff = (d32[..., None] * sc.astype(np.float32)).astype(np.float32)
    return d, sc.reshape(B, O, I // 16), eff.reshape(B, O, I // 16)


def expand_scales(scales, gs):
    """Per-coordinate view of group scales: (B, O, I/gs) -> (B, O, I)."""
    return np.repeat(scales, gs, axis=-1)


def rtn_codes(W, s_coord, cfg):
    """Round-to-nearest level index q0 = argmin_k |fl32(W / s) - c_k|, ties to the lower k.

    The ratio is taken in float32 (IEEE division); distances to the levels are
    exact.  A zero scale (an all-zero super-block sub-block) uses ratio 0.
    """
    c = cfg.levels64()
    W32 = np.asarray(W, dtype=np.float32)
    s32 = np.asarray(s_coord, dtype=np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        u = np.where(s32 != 0, W32 / s32, np.float32(0)).astype(np.float64)
    dist = np.abs(u[..., None] - c)                     # exact in float64
    return np.argmin(dist, axis=-1)                      # first minimum = lower index


def prior_logits(q0, cfg):
    """Gaussian-prior warm-start logits (App. A), mean-subtracted per coordinate.

    l_k = -(x_k - mu)^2 / 2 over the coordinate's candidates x_k, then the mean
    over k is removed.  Full grid: x_k = c_k, mu = c_{q0}.  Local shift: the
    candidates are the shifts themselves, x_k = delta_k, and mu = 0, since the
    warm-start code is already the window's centre j0 (App. A).
    """
    if cfg.relaxation == "shift":
        x = SHIFTS.astype(np.float64)
        l = np.broadcast_to(-0.5 * x ** 2, np.shape(q0) + (len(x),))
    else:
        c = cfg.levels64()
        mu = c[q0][..., None]
        l = -0.5 * (c - mu) ** 2
    return l - l.mean(axis=-1, keepdims=True)


def ternary_warm_logits(q0):
    """Eq. 3: mask logit +1 where the warm-start code is non-zero, -1 where it is zero; sign
    logit +1 / -1 for a +1 / -1 code and 0 for a zero code.  q0 indexes (-1, 0, 1).
    Returns (..., 2) as (mask, sign)."""
    val = np.asarray(q0).astype(np.int64) - 1
    lm = np.where(val != 0, 1.0, -1.0)
    lb = val.astype(np.float64)
    return np.stack([lm, lb], axis=-1)


def init_logits(q0, cfg, eps=None):
    """Eq. 4: l = sigma_init * (eps + alpha * l_warm); eps ~ N(0, I) or zero.  The warm
    logits are App. A's prior (grid, shift) or Eq. 3's signs (ternary, not mean-subtracted)."""
    lp = ternary_warm_logits(q0) if cfg.relaxation == "ternary" else prior_logits(q0, cfg)
    noise = 0.0 if eps is None else eps
    sigma, alpha = float(np.float32(cfg.sigma_init)), float(np.float32(cfg.alpha))
    return round_f32(sigma * (noise + alpha * lp)).astype(np.float32)


def coord_index(cfg, b, rows):
    """Global coordinate indices e = (b*O + o)*I + i for the given rows of layer b."""
    rows = np.asarray(rows, dtype=np.int64)
    i = np.arange(cfg.in_features, dtype=np.int64)
    return ((b * cfg.out_features + rows)[:, None] * cfg.in_features + i[None, :]).reshape(-1)


def init_layer(cfg, W, scales_init=None, rows=None, batches=None):
    """Initial state of ``gsq_layer_init``: scales, RTN codes, logits, zero moments.

    ``rows`` restricts the state to a subset of the rows of every layer and
    ``batches`` to a subset of the layers (every quantity of the initialisation is
    row-local); noise indices stay global.
    """
    W = np.asarray(W, dtype=np.float64).reshape(cfg.batch, cfg.out_features, cfg.in_features)
    B, O, I, K = cfg.batch, cfg.out_features, cfg.in_features, cfg.K
    rows = np.arange(O) if rows is None else np.asarray(rows)
    batches = np.arange(B) if batches is None else np.asarray(batches)
    W = W[batches][:, rows]
    if scales_init is not None:
        scales_init = np.asarray(scales_init, np.float32).reshape(B, O, I // cfg.gs)[batches][:, rows]
    B = len(batches)
    O = len(rows)
    sb_d = sb_sc = None
    if cfg.layout == "superblock":
        sb_d, sb_sc, scales = superblock_scales(W, cfg)
    elif scales_init is not None:
        scales = np.asarray(scales_init, dtype=np.float32).reshape(B, O, I // cfg.gs).copy()
    else:
        scales = group_absmax_scales(W, cfg)
    q0 = rtn_codes(W, expand_scales(scales, cfg.gs), cfg)
    if cfg.n_grid > 255:
        raise ValueError("grid too large")
    logits = np.empty((B, O, I, K), dtype=np.float32)
    for j, b in enumerate(batches):
        eps = None
        if cfg.init_noise:
            e = coord_index(cfg, b, rows)
            eps = philox.init_normals(cfg.seed, e, K).reshape(O, I, K)
        logits[j] = init_logits(q0[j], cfg, eps)
    z = np.zeros_like(logits)
    zs = np.zeros_like(scales)
    st = State(logits, z, z.copy(), scales.astype(np.float32), zs, zs.copy(), 0, sb_d, sb_sc)
    st.extra["q0"] = q0
    if cfg.relaxation == "shift":
        st.base = q0.astype(np.uint8)
    return st


# ----------------------------------------------------------------------------- one step
def soft_sample(logits, g, tau, kappa):
    """Alg. 1: p_k = exp((kappa l_k + g_k)/tau) / sum_j exp((kappa l_j + g_j)/tau).

    Evaluated in float64 with the maximum subtracted first (the same quotient).
    """
    a = (kappa * np.asarray(logits, np.float64) + g) / np.float64(tau)
    a = a - a.max(axis=-1, keepdims=True)
    e = np.exp(a)
    return e / e.sum(axis=-1, keepdims=True)


def candidates(cfg, base=None):
    """The values each logit stands for.

    Full grid: the levels c_k (the same for every coordinate).  Local shift
    (§3.2, Eq. 6): logit k of a coordinate with initial index j0 stands for the
    grid level of index clip(j0 + delta_k, 0, n - 1) (the paper's 1-based
    clip(j0 + delta, 1, 2^b)), so near the ends of the grid several shifts give
    the same level.  Returns the levels (K,) or an array base.shape + (K,).
    """
    c = cfg.levels64()
    if cfg.relaxation != "shift":
        return c
    j = np.clip(np.asarray(base, np.int64)[..., None] + SHIFTS, 0, cfg.n_grid - 1)
    return c[j]


def forward(cfg, W, logits, s_coord, g, tau, kappa, cand=None):
    """Soft weight and residual of one sample (Alg. 1 return value, scaled per §3.2).

    v = sum_k p_k c_k, W_hat = s * v, R = W - W_hat.  Returns (p, v, R) where R
    is rounded to the contraction's input precision.  ``cand`` holds the values
    of the logits (``candidates``); default: the grid levels.
    """
    p = soft_sample(logits, g, tau, kappa)
    c = cfg.levels64() if cand is None else cand
    v = (p * c).sum(axis=-1)
    R = np.asarray(W, np.float64) - np.asarray(s_coord, np.float64) * v
    return p, v, to_contraction_precision(cfg, R)


def contract(cfg, R, Hs, Hc=None):
    """P = R H and the loss L = sum(R * P) = tr(R H R^T) (Eq. 1 for a linear layer).

    ``Hs`` is the symmetrised float32 H; in the bf16 precision it is rounded to
    bfloat16 first.  Accumulation is float64.  ``Hc``, when given, is that rounded
    operand computed beforehand (long runs round H once; the values are the same).
    """
    if Hc is None:
        Hc = to_contraction_precision(cfg, Hs)
    P = R @ Hc
    return P, float((R * P).sum())


def backward(cfg, G, s_coord, p, v, tau, kappa, cand=None):
    """Gradients of L with respect to the logits and the group scales.

    With W_hat = s v and G = dL/dW_hat:
      dL/dl_k = G s (kappa / tau) p_k (c_k - v)         (softmax Jacobian, App. B proof)
      dL/ds_g = sum_{i in g} G_i v_i
    c_k - v is evaluated as sum_j p_j (c_k - c_j), equal because the p_j sum to
    one; the direct difference cancels to rounding noise once one level holds
    almost all the mass, which is the saturated regime App. B is about.
    """
    c = cfg.levels64() if cand is None else cand
    c = np.broadcast_to(c, p.shape)
    diff = (p[..., None, :] * (c[..., :, None] - c[..., None, :])).sum(axis=-1)   # [.., k] = sum_j p_j (c_k - c_j)
    dlog = (G * s_coord * (kappa / np.float64(tau)))[..., None] * p * diff
    gv = G * v
    B, O, I = gv.shape
    dscale = gv.reshape(B, O, I // cfg.gs, cfg.gs).sum(axis=-1)
    return dlog, dscale


def binary_sample(logit, d, tau, kappa):
    """Alg. 1 on a two-element set with logits {-l, l} (§3): returns (p_first, p_second).

    The softmax of (kappa (-l) + g0, kappa l + g1) / tau depends on the two Gumbel values
    only through d = g1 - g0, a Logistic(0,1) variable; ``d`` is that difference, entered as
    the noise (0, d) of the two elements.
    """
    l = np.asarray(logit, np.float64)
    d = np.asarray(d, np.float64)
    g2 = np.stack([np.zeros_like(d), d], axis=-1)
    p = soft_sample(np.stack([-l, l], axis=-1), g2, tau, kappa)
    return p[..., 0], p[..., 1]


def ternary_forward(cfg, W, logits, s_coord, g, tau, kappa):
    """Ternary sample of Alg. 2: mask m~ = GS({0, 1}, {-l_m, l_m}), sign
    b~ = GS({-1, 1}, {-l_b, l_b}), W_hat = s m~ b~ (Eq. 2).

    ``logits`` (..., 2) holds (l_m, l_b); ``g`` (..., 2) the logistic noise of the mask pair
    then of the sign pair (each the difference of the pair's two Gumbel values, see
    ``binary_sample``).  Returns (p, v, R): p (..., 2, 2) the two pairs of probabilities,
    v = m~ b~ the soft level, R the residual in the contraction precision.
    """
    p0m, p1m = binary_sample(logits[..., 0], g[..., 0], tau, kappa)
    p0b, p1b = binary_sample(logits[..., 1], g[..., 1], tau, kappa)
    m = p1m                                  # 0 * p0 + 1 * p1
    b = p1b - p0b                            # -1 * p0 + 1 * p1
    v = m * b
    R = np.asarray(W, np.float64) - np.asarray(s_coord, np.float64) * v
    p = np.stack([np.stack([p0m, p1m], -1), np.stack([p0b, p1b], -1)], -2)
    return p, v, to_contraction_precision(cfg, R)


def ternary_backward(cfg, G, s_coord, p, tau, kappa):
    """Gradients of the ternary sample.  With u = dL/dW_hat = G:
      dL/dm~ = G s b~,  dL/db~ = G s m~;
    each relaxed value y = sum_k p_k y_k of a pair with logits (-l, l) has
      dy/dl = (kappa / tau) [p_1 (y_1 - y) - p_0 (y_0 - y)]        (softmax Jacobian);
      dL/ds_g = sum_{i in g} G_i m~_i b~_i.
    y_1 - y and y_0 - y are taken as p_0 (y_1 - y_0) and p_1 (y_0 - y_1) (the p's sum
    to one), which keeps full relative accuracy when one value holds almost all the mass.
    Returns dlogits (..., 2) = (d l_m, d l_b) and dscales.
    """
    kt = kappa / np.float64(tau)
    p0m, p1m = p[..., 0, 0], p[..., 0, 1]
    p0b, p1b = p[..., 1, 0], p[..., 1, 1]
    m = p1m
    b = p1b - p0b

    def slope(p0, p1, y0, y1):
        return kt * (p1 * (p0 * (y1 - y0)) - p0 * (p1 * (y0 - y1)))

    dm_dl = slope(p0m, p1m, 0.0, 1.0)
    db_dl = slope(p0b, p1b, -1.0, 1.0)
    u = G * s_coord
    dlog = np.stack([u * b * dm_dl, u * m * db_dl], axis=-1)
    gv = G * m * b
    B, O, I = gv.shape
    return dlog, gv.reshape(B, O, I // cfg.gs, cfg.gs).sum(axis=-1)


def adam(theta, m, v, grad, lr, beta1, beta2, eps, n, wd=0.0):
    """Adam (Kingma & Ba, 2015), bias-corrected at step n >= 1; with wd > 0 the decoupled
    weight decay of AdamW (Loshchilov & Hutter, 2019), the paper's ablation optimiser (App. B).

    Arithmetic in float64 on the float32 state; results stored as float32.
    """
    th = np.asarray(theta, np.float64)
    m1 = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * grad
    v1 = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * grad * grad
    mhat = m1 / (1.0 - beta1 ** n)
    vhat = v1 / (1.0 - beta2 ** n)
    th1 = th - lr * (mhat / (np.sqrt(vhat) + eps) + wd * th)
    return th1.astype(np.float32), m1.astype(np.float32), v1.astype(np.float32)


def lion(theta, m, grad, lr, beta1, beta2, wd=0.0):
    """Lion (Chen et al., 2023), the paper's optimiser (§3.3, App. B): the step is the sign of
    the interpolation beta1 m + (1 - beta1) g, plus decoupled weight decay; the single moment
    then moves with beta2.  sign(0) = 0.  float64 arithmetic, float32 storage.
    """
    th = np.asarray(theta, np.float64)
    m = np.asarray(m, np.float64)
    c = beta1 * m + (1.0 - beta1) * grad
    th1 = th - lr * (np.sign(c) + wd * th)
    m1 = beta2 * m + (1.0 - beta2) * grad
    return th1.astype(np.float32), m1.astype(np.float32)


def update(prm, theta, m, v, grad, lr, n):
    """The chosen optimiser's update of one parameter tensor: (theta, m, v) after the step."""
    if prm.optimizer == "lion":
        th1, m1 = lion(theta, m, grad, lr, prm.beta1, prm.beta2, prm.weight_decay)
        return th1, m1, np.asarray(v, np.float32)
    return adam(theta, m, v, grad, lr, prm.beta1, prm.beta2, prm.eps, n, prm.weight_decay)


def step(cfg, W, Hs, st, prm, rows=None, want=False, batches=None, Hc=None):
    """One GSQ optimisation step on state ``st`` (returns a new state, the loss).

    Order: noise -> soft sample -> residual -> contraction and loss -> gradient
    -> optimiser (Adam / AdamW / Lion) on logits and (if lr_scales > 0) scales; t -> t + 1.
    With prm.samples = M > 1 the noise is drawn M times independently and the gradients
    (and the reported loss) are averaged over the M samples (§3.3, gradient accumulation
    with resampled noise).  The loss is
    taken before the update, averaged over the step's samples.

    ``rows`` restricts the step to a subset of the rows of every layer (rows
    are independent given H) and ``batches`` to a subset of the layers; ``st``
    then holds just those rows and layers, ``Hs`` just those layers' H, and noise
    indices stay the global ones.
    ``want`` returns the intermediates (g, p, v, R, G of the last sample; the averaged
    dlogits, dscales).  ``Hc`` optionally holds ``to_contraction_precision(cfg, Hs)``
    of the same layers, computed once for a run of many steps.
    """
    B, O, I, K = cfg.batch, cfg.out_features, cfg.in_features, cfg.K
    prm = as_f32_params(prm)
    rows = np.arange(O) if rows is None else np.asarray(rows)
    batches = np.arange(B) if batches is None else np.asarray(batches)
    W = np.asarray(W, np.float64).reshape(B, O, I)[batches][:, rows]
    Hs = np.asarray(Hs).reshape(len(batches), I, I)
    n = st.t + 1
    new = st.copy()
    losses = np.zeros(len(batches))
    inter = {k: [] for k in ("g", "p", "v", "R", "G", "dlogits", "dscales")}
    for b, bg in enumerate(batches):
        e = coord_index(cfg, bg, rows)
        lg = st.logits[b]
        sc = st.scales[b]
        s_coord = expand_scales(sc, cfg.gs)
        cand = candidates(cfg, None if st.base is None else st.base[b])
        nz = cfg.n_noise
        dlog = dsc = 0.0
        for smp in range(prm.samples):
            if prm.gumbel_noise and cfg.relaxation == "ternary":
                g = philox.logistic(cfg.seed, e, st.t, nz, smp).reshape(len(rows), I, nz)
            elif prm.gumbel_noise:
                g = philox.gumbel(cfg.seed, e, st.t, nz, smp).reshape(len(rows), I, nz)
            else:
                g = np.zeros((len(rows), I, nz))
            if cfg.relaxation == "ternary":
                p, v, R = ternary_forward(cfg, W[b], lg, s_coord, g, prm.tau, prm.kappa)
            else:
                p, v, R = forward(cfg, W[b], lg, s_coord, g, prm.tau, prm.kappa, cand)
            P, L = contract(cfg, R, Hs[b], None if Hc is None else Hc[b])
            G = -2.0 * P
            if cfg.relaxation == "ternary":
                dl1, ds1 = ternary_backward(cfg, G[None], s_coord[None], p[None], prm.tau, prm.kappa)
            else:
                dl1, ds1 = backward(cfg, G[None], s_coord[None], p[None], v[None], prm.tau,
                                    prm.kappa, None if cand.ndim == 1 else cand[None])
            dlog = dlog + dl1[0]
            dsc = dsc + ds1[0]
            losses[b] += L
        dlog = dlog / prm.samples
        dsc = dsc / prm.samples
        losses[b] /= prm.samples
        th, m1, v1 = update(prm, lg, st.m[b], st.v[b], dlog, prm.lr_logits, n)
        new.logits[b], new.m[b], new.v[b] = th, m1, v1
        if prm.lr_scales > 0:
            ts, ms, vs = update(prm, sc, st.m_s[b], st.v_s[b], dsc, prm.lr_scales, n)
            new.scales[b], new.m_s[b], new.v_s[b] = ts, ms, vs
        if want:
            for k, val in zip(inter, (g, p, v, R, G, dlog, dsc)):
                inter[k].append(val)
    new.t = st.t + 1
    if want:
        return new, losses, {k: np.stack(v) for k, v in inter.items()}
    return new, losses


# ----------------------------------------------------------------------------- hardening
def harden(logits):
    """Hard codes q = argmax_k l_k, ties to the lowest k (the final step of Alg. 2, K-way)."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.uint8)


def hard_codes(cfg, st):
    """Grid codes of the hardened layer, per relaxation.

    grid: argmax of the logits.  shift: clip(j0 + delta*) with delta* the
    argmax shift.  ternary: the thresholds of Alg. 2, mask = [l_m >= 0] and
    sign = +1 if l_b >= 0 else -1 (ties go to active and positive); the code
    indexes (-1, 0, 1), i.e. 1 + mask * sign.
    """
    lg = np.asarray(st.logits)
    if cfg.relaxation == "ternary":
        mask = (lg[..., 0] >= 0).astype(np.int64)
        sign = np.where(lg[..., 1] >= 0, 1, -1)
        return (1 + mask * sign).astype(np.uint8)
    k = harden(lg).astype(np.int64)
    if cfg.relaxation == "shift":
        return np.clip(st.base.astype(np.int64) + SHIFTS[k], 0, cfg.n_grid - 1).astype(np.uint8)
    return k.astype(np.uint8)


def scales_fp16(scales):
    """Deployment scales: float32 -> float16, round-to-nearest-even (16-bit scales of Tab. 1)."""
    return np.asarray(scales, dtype=np.float32).astype(np.float16)


def hard_weights(cfg, codes, scales_eff):
    """W_q = s * c[q] with the stored effective scales (float32 product)."""
    c = np.asarray(cfg.levels, dtype=np.float32)
    s = expand_scales(np.asarray(scales_eff, np.float32), cfg.gs)
    return (s * c[codes]).astype(np.float32)


def hard_loss(cfg, W, Hs, codes, scales_eff):
    """Eq. 1 at the hardened weights: tr(R H R^T) with R = W - s c[q] (contraction precision)."""
    W = np.asarray(W, np.float64).reshape(cfg.batch, cfg.out_features, cfg.in_features)
    Hs = np.asarray(Hs).reshape(cfg.batch, cfg.in_features, cfg.in_features)
    Wq = hard_weights(cfg, codes, scales_eff).astype(np.float64)
    out = np.zeros(cfg.batch)
    for b in range(cfg.batch):
        R = to_contraction_precision(cfg, W[b] - Wq[b])
        out[b] = contract(cfg, R, Hs[b])[1]
    return out


def harden_layer(cfg, W, Hs, st):
    """``gsq_harden``: codes, effective scales (fp16-rounded in the plain layout), hard loss."""
    codes = hard_codes(cfg, st)
    if cfg.layout == "superblock":
        eff = st.scales.astype(np.float32)
    else:
        eff = scales_fp16(st.scales).astype(np.float32)
    return codes, eff, hard_loss(cfg, W, Hs, codes, eff)


def tau_schedule(t, T, tau0=1.0, tau1=0.05):
    """Linear temperature schedule (Tab. 7 anneals tau linearly); last step uses tau1."""
    if T <= 1:
        return tau1
    return tau0 + (tau1 - tau0) * t / (T - 1)
