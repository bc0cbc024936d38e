"""Pins of the oracle's helper functions: bf16 rounding, H symmetrisation, the tau schedule.

Each is checked against something other than itself: torch's own float32 -> bfloat16
conversion (a library routine), Eq. 1 evaluated directly from the calibration inputs X,
finite differences of the loss with an unsymmetrised H, and the endpoints and constant
increments that a linear anneal (Tab. 7) fixes.
"""
import numpy as np
import pytest

from oracle import gsq

torch = pytest.importorskip("torch")


def _torch_bf16(x32):
    t = torch.from_numpy(np.ascontiguousarray(x32, np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy().astype(np.float64)


# ------------------------------------------------------------------ round_bf16
def test_round_bf16_matches_torch_on_random_values():
    rng = np.random.default_rng(0)
    mant = rng.uniform(1, 2, 200_000)
    expo = rng.integers(-140, 120, 200_000)
    sign = rng.choice([-1.0, 1.0], 200_000)
    x = (sign * mant * 2.0 ** expo).astype(np.float32)
    np.testing.assert_array_equal(gsq.round_bf16(x), _torch_bf16(x))


def test_round_bf16_ties_go_to_even_like_torch():
    """Low 16 bits exactly 0x8000: a tie, rounded to the even upper half; one bit either side
    of the tie rounds down / up.  Both parities of the kept bit and both signs."""
    rng = np.random.default_rng(1)
    hi = rng.integers(0x0080, 0x7F00, 4096).astype(np.uint32)   # normal, finite upper halves
    hi = np.concatenate([hi, hi | 0x8000])                       # negative values too
    rows = []
    for low in (0x8000, 0x7FFF, 0x8001, 0x0000, 0xFFFF):
        bits = (hi << 16) | np.uint32(low)
        rows.append(bits.view(np.float32))
    x = np.concatenate(rows)
    got = gsq.round_bf16(x)
    np.testing.assert_array_equal(got, _torch_bf16(x))
    # the tie rule itself, independently of torch: even upper halves stay, odd ones round away
    ties = ((hi << 16) | np.uint32(0x8000)).view(np.float32)
    up = (hi & 1) == 1
    want_bits = np.where(up, hi + 1, hi) << 16
    np.testing.assert_array_equal(gsq.round_bf16(ties), want_bits.astype(np.uint32).view(np.float32))


def test_round_bf16_subnormals_zero_and_carry_into_the_exponent():
    sub = (np.arange(1, 1 << 16, 7, dtype=np.uint32)).view(np.float32)   # float32 subnormals
    big = np.array([0x3F7FFFFF, 0x3FFFFFFF, 0x407FC000, 0x00000000, 0x80000000,
                    0x7F7F7FFF], dtype=np.uint32).view(np.float32)
    x = np.concatenate([sub, -sub, big])
    np.testing.assert_array_equal(gsq.round_bf16(x), _torch_bf16(x))
    assert gsq.round_bf16(np.float32(np.nextafter(np.float32(1), np.float32(0)))) == 1.0
    assert gsq.round_bf16(np.float32(1 + 2 ** -8)) == 1.0           # tie at 1 + half an ulp
    assert gsq.round_bf16(np.float32(1 + 3 * 2 ** -8)) == 1 + 2 ** -6   # tie, odd -> up


def test_round_bf16_is_not_truncation():
    x = np.float32(1 + 2 ** -7 - 2 ** -20)          # just below 1 + one bf16 ulp
    assert gsq.round_bf16(x) == 1 + 2 ** -7
    assert gsq.round_bf16(-x) == -(1 + 2 ** -7)


# ------------------------------------------------------------------ symmetrize
def _layer(rng, O=6, I=32, tokens=48):
    X = rng.standard_normal((tokens, I)) * rng.lognormal(0, 0.5, I)
    W = rng.normal(0, 0.02, (O, I))
    What = W + rng.normal(0, 0.005, (O, I))
    return X, W, What


def test_symmetrize_is_bitwise_symmetric_and_keeps_symmetric_input():
    rng = np.random.default_rng(2)
    A = rng.standard_normal((3, 40, 40)).astype(np.float32)
    S = gsq.symmetrize(A)
    np.testing.assert_array_equal(S, np.swapaxes(S, -1, -2))
    X = rng.standard_normal((80, 40))
    H = (X.T @ X).astype(np.float32)
    np.testing.assert_array_equal(gsq.symmetrize(H), H.astype(np.float64))


def test_loss_through_a_symmetrised_nonsymmetric_H_equals_the_output_error_from_X():
    """Eq. 1 for a linear layer: ||X W_hat^T - X W^T||_F^2 = tr(R H R^T) with H = X^T X.  Add an
    antisymmetric part to H (it leaves the quadratic form unchanged) and a non-symmetric
    perturbation that is removed again: the loss through symmetrize(H') must equal the
    X-direct value; a missing 1/2 doubles it, a transpose-only symmetrisation changes it."""
    rng = np.random.default_rng(3)
    X, W, What = _layer(rng)
    direct = np.sum((X @ What.T - X @ W.T) ** 2)
    H = X.T @ X
    A = rng.standard_normal(H.shape) * np.abs(H).max()
    Hn = H + (A - A.T)                              # non-symmetric, same quadratic form
    assert np.abs(Hn - Hn.T).max() > 0.5 * np.abs(H).max()
    cfg = gsq.Config(W.shape[0], W.shape[1], (-1.0, 0.0, 1.0), 16, precision="fp64")
    R = W - What
    _, loss = gsq.contract(cfg, R, gsq.symmetrize(Hn))
    assert abs(loss - direct) <= 1e-6 * direct
    # the symmetrised matrix itself is X^T X (to float32 rounding of its entries)
    np.testing.assert_allclose(gsq.symmetrize(Hn), H, rtol=0, atol=4e-7 * np.abs(Hn).max())


def test_gradient_through_symmetrize_is_the_derivative_of_the_unsymmetrised_loss():
    """dL/dW_hat of L = tr(R H R^T), R = W - W_hat, for a non-symmetric H is -R (H + H^T); the
    oracle forms G = -2 R symmetrize(H).  Central finite differences of the loss with the raw,
    non-symmetric H pin the factor and the orientation."""
    rng = np.random.default_rng(4)
    X, W, What = _layer(rng, O=3, I=12, tokens=20)
    H = X.T @ X + np.triu(rng.standard_normal((12, 12))) * 3.0
    cfg = gsq.Config(3, 12, (-1.0, 0.0, 1.0), 4, precision="fp64")
    P, _ = gsq.contract(cfg, W - What, gsq.symmetrize(H))
    G = -2.0 * P

    def loss(Wh):
        R = W - Wh
        return np.trace(R @ H @ R.T)

    h = 1e-6
    num = np.zeros_like(What)
    for idx in np.ndindex(What.shape):
        d = np.zeros_like(What)
        d[idx] = h
        num[idx] = (loss(What + d) - loss(What - d)) / (2 * h)
    np.testing.assert_allclose(G, num, rtol=1e-5, atol=1e-6 * np.abs(num).max())


# ------------------------------------------------------------------ tau schedule
@pytest.mark.parametrize("T,tau0,tau1", [(100, 1.0, 0.05), (500, 1.0, 0.05), (300, 2.0, 0.05),
                                         (2, 1.0, 0.05)])
def test_tau_schedule_is_the_linear_anneal_with_both_endpoints(T, tau0, tau1):
    """Tab. 7 anneals tau linearly (2 -> 0.05); the benchmark's layers use 1.0 -> 0.05.  Over T
    steps t = 0 .. T - 1 the first step uses tau0, the last tau1, and consecutive steps differ
    by the same amount (tau1 - tau0) / (T - 1)."""
    taus = np.array([gsq.tau_schedule(t, T, tau0, tau1) for t in range(T)])
    assert taus[0] == tau0
    assert abs(taus[-1] - tau1) <= 1e-15
    np.testing.assert_allclose(np.diff(taus), (tau1 - tau0) / (T - 1), rtol=1e-9, atol=1e-15)
    assert np.all(taus > 0)
    # a schedule that reached tau1 one step late (off by one) would not hit it at t = T - 1
    assert taus[-1] < taus[-2] if T > 1 else True


def test_tau_schedule_single_step_and_defaults():
    assert gsq.tau_schedule(0, 1) == 0.05
    assert gsq.tau_schedule(0, 100) == 1.0
    assert abs(gsq.tau_schedule(99, 100) - 0.05) < 1e-15
    assert abs(gsq.tau_schedule(50, 101) - 0.525) < 1e-15          # the midpoint
