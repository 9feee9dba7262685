"""Pins of the paper-optimiser oracle against facts that do not come from the oracle itself.

  * softplus: special values, the identity softplus(z) - softplus(-z) = z, its derivative;
  * per-token rates and the momentum decay: brute-force scalar loops, and the closed form for a
    segment whose tokens are all equal;
  * the rate-weighted gradient: central finite differences of a brute-force weighted loss, and
    torch.autograd in float64; all-ones rates give the (pinned) plain gradient; a zero rate
    removes exactly that token;
  * the update: with constant rates lr and a vanishing momentum decay, one step equals the
    (pinned) SGD step with every row rescaled to its initial norm; the momentum of the first
    step carries into the second with weight beta; row norms stay at their initial values over
    a whole run; an empty segment changes nothing.
"""
import math

import numpy as np
import pytest

import oracle as orc

SHAPES = [(3, 4, 2, 3), (5, 7, 6, 5), (4, 6, 4, 1)]  # (d, h, D, T)
SOFTPLUS_INV_1 = math.log(math.e - 1.0)  # softplus(SOFTPLUS_INV_1) = 1


def _layer(rng, d, h, D, T):
    x = rng.standard_normal((T, d))
    w1 = rng.standard_normal((h, d)) / math.sqrt(d)
    w2 = rng.standard_normal((D, h)) / math.sqrt(h)
    wkv = rng.standard_normal((D, d)) / math.sqrt(d)
    meta = (rng.standard_normal(d) / math.sqrt(d), 0.3, rng.standard_normal(d) / math.sqrt(d), -0.2)
    return x, w1, w2, wkv, meta


def _brute_loss_weighted(x, w1, w2, wkv, eta):
    """(1/n) sum_j eta_j ||W2 SiLU(W1 x_j) - Wkv x_j||^2 with scalar loops only."""
    n, d = x.shape
    h, D = w1.shape[0], w2.shape[0]
    total = 0.0
    for j in range(n):
        a = []
        for i in range(h):
            z = sum(w1[i, k] * x[j, k] for k in range(d))
            a.append(z / (1.0 + math.exp(-z)))
        lj = 0.0
        for o in range(D):
            y = sum(w2[o, i] * a[i] for i in range(h))
            t = sum(wkv[o, k] * x[j, k] for k in range(d))
            lj += (y - t) ** 2
        total += eta[j] * lj
    return total / n


# ---------------------------------------------------------------- softplus, rates, decay

def test_softplus_special_values_and_identity():
    assert orc.softplus(0.0) == pytest.approx(math.log(2.0), rel=1e-15)
    assert orc.softplus(SOFTPLUS_INV_1) == pytest.approx(1.0, rel=1e-14)
    z = np.linspace(-40, 40, 801)
    np.testing.assert_allclose(orc.softplus(z) - orc.softplus(-z), z, rtol=0, atol=1e-12)
    with np.errstate(over="raise"):
        assert orc.softplus(800.0) == 800.0
        assert 0.0 <= orc.softplus(-800.0) < 1e-300


def test_softplus_derivative_is_logistic():
    z = np.linspace(-8, 8, 33)
    eps = 1e-6
    fd = (orc.softplus(z + eps) - orc.softplus(z - eps)) / (2 * eps)
    np.testing.assert_allclose(fd, 1.0 / (1.0 + np.exp(-z)), rtol=0, atol=1e-9)


def test_token_rates_and_decay_brute_force():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 4))
    u, v = rng.standard_normal(4), rng.standard_normal(4)
    eta = orc.token_rates(x, u, 0.7, 0.05)
    for j in range(5):
        p = sum(u[k] * x[j, k] for k in range(4)) + 0.7
        assert eta[j] == pytest.approx(0.05 * math.log(1.0 + math.exp(p)), rel=1e-13)
    q = sum(sum(v[k] * x[j, k] for k in range(4)) for j in range(5)) / 5 - 0.4
    assert orc.momentum_decay(x, v, -0.4) == pytest.approx(1.0 / (1.0 + math.exp(-q)), rel=1e-13)


def test_decay_of_a_constant_segment_is_the_token_decay():
    rng = np.random.default_rng(2)
    row = rng.standard_normal(6)
    v = rng.standard_normal(6)
    x = np.tile(row, (7, 1))
    want = 1.0 / (1.0 + math.exp(-(row @ v + 0.1)))
    assert orc.momentum_decay(x, v, 0.1) == pytest.approx(want, rel=1e-13)


# ---------------------------------------------------------------- the weighted gradient

@pytest.mark.parametrize("shape", SHAPES)
def test_weighted_grad_matches_finite_differences(shape):
    d, h, D, T = shape
    rng = np.random.default_rng(10 + d)
    x, w1, w2, wkv, _ = _layer(rng, d, h, D, T)
    eta = rng.uniform(0.1, 2.0, T)
    g1, g2, _ = orc.weighted_grad(x, w1, w2, wkv, eta)
    eps = 1e-5
    for w, g in ((w1, g1), (w2, g2)):
        fd = np.zeros_like(w)
        for idx in np.ndindex(w.shape):
            wp, wm = w.copy(), w.copy()
            wp[idx] += eps
            wm[idx] -= eps
            if w is w1:
                lp = _brute_loss_weighted(x, wp, w2, wkv, eta)
                lm = _brute_loss_weighted(x, wm, w2, wkv, eta)
            else:
                lp = _brute_loss_weighted(x, w1, wp, wkv, eta)
                lm = _brute_loss_weighted(x, w1, wm, wkv, eta)
            fd[idx] = (lp - lm) / (2 * eps)
        assert np.linalg.norm(g - fd) <= 1e-7 * max(1.0, np.linalg.norm(fd))


def test_weighted_grad_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    x, w1, w2, wkv, _ = _layer(rng, 6, 5, 4, 7)
    eta = rng.uniform(0.1, 2.0, 7)
    g1, g2, _ = orc.weighted_grad(x, w1, w2, wkv, eta)
    tw1 = torch.tensor(w1, requires_grad=True)
    tw2 = torch.tensor(w2, requires_grad=True)
    tx, tkv, te = torch.tensor(x), torch.tensor(wkv), torch.tensor(eta)
    y = torch.nn.functional.silu(tx @ tw1.T) @ tw2.T
    loss = (te * ((y - tx @ tkv.T) ** 2).sum(dim=1)).mean()
    loss.backward()
    np.testing.assert_allclose(g1, tw1.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(g2, tw2.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_unit_rates_give_the_plain_gradient_and_zero_rate_drops_a_token():
    rng = np.random.default_rng(4)
    x, w1, w2, wkv, _ = _layer(rng, 5, 6, 4, 6)
    g1, g2, _ = orc.weighted_grad(x, w1, w2, wkv, np.ones(6))
    p1, p2, _ = orc.segment_grad(x, w1, w2, wkv)
    np.testing.assert_allclose(g1, p1, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(g2, p2, rtol=1e-13, atol=1e-15)
    # a zero rate on token 2: the gradient of the other 5 tokens, still averaged over 6
    eta = np.ones(6)
    eta[2] = 0.0
    g1, g2, _ = orc.weighted_grad(x, w1, w2, wkv, eta)
    keep = np.delete(x, 2, axis=0)
    q1, q2, _ = orc.segment_grad(keep, w1, w2, wkv)
    np.testing.assert_allclose(g1, q1 * 5 / 6, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g2, q2 * 5 / 6, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------- the update

def _rows_to(w, norms):
    return w * (norms / np.linalg.norm(w, axis=1))[:, None]


@pytest.mark.parametrize("loss", ["mse_sum", "mse_mean"])
def test_constant_rates_without_momentum_are_sgd_then_row_renormalisation(loss):
    rng = np.random.default_rng(5)
    x, w1, w2, wkv, _ = _layer(rng, 6, 8, 4, 5)
    lr = 0.05
    meta = (np.zeros(6), SOFTPLUS_INV_1, np.zeros(6), -80.0)  # eta_j = lr, beta ~ 1e-35
    n0 = (np.linalg.norm(w1, axis=1), np.linalg.norm(w2, axis=1))
    p1, p2, m1, m2, ls, info = orc.paper_step(x, w1, w2, 0 * w1, 0 * w2, wkv, meta, n0, lr, loss)
    s1, s2, ls_sgd = orc.ttl_step(x, w1, w2, wkv, lr, loss)  # pinned SGD step
    np.testing.assert_allclose(p1, _rows_to(s1, n0[0]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(p2, _rows_to(s2, n0[1]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m1, w1 - s1, rtol=1e-12, atol=1e-17)  # the momentum is lr * grad
    assert ls == pytest.approx(ls_sgd, rel=1e-14)


def test_momentum_carries_into_the_next_step_with_weight_beta():
    rng = np.random.default_rng(6)
    x, w1, w2, wkv, _ = _layer(rng, 5, 6, 4, 4)
    lr = 0.1
    n0 = (np.linalg.norm(w1, axis=1), np.linalg.norm(w2, axis=1))
    first = (np.zeros(5), SOFTPLUS_INV_1, np.zeros(5), -80.0)
    a1, a2, m1, m2, _, _ = orc.paper_step(x, w1, w2, 0 * w1, 0 * w2, wkv, first, n0, lr)
    # second step: rates ~ 1e-37 (no new gradient), decay sigmoid(0.4); the weights move
    # again by beta times the first step's lr * gradient, then are renormalised
    second = (np.zeros(5), -85.0, np.zeros(5), 0.4)
    b1, b2, k1, k2, _, info = orc.paper_step(x, a1, a2, m1, m2, wkv, second, n0, lr)
    beta = 1.0 / (1.0 + math.exp(-0.4))
    assert info["beta"] == pytest.approx(beta, rel=1e-14)
    s1, s2, _ = orc.ttl_step(x, w1, w2, wkv, lr)
    np.testing.assert_allclose(b1, _rows_to(a1 - beta * (w1 - s1), n0[0]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(b2, _rows_to(a2 - beta * (w2 - s2), n0[1]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(k1, beta * (w1 - s1), rtol=1e-12, atol=1e-18)


def test_row_norms_stay_at_their_initial_values_over_a_run():
    rng = np.random.default_rng(7)
    d, h, D = 6, 9, 4
    _, w1, w2, wkv, meta = _layer(rng, d, h, D, 1)
    segs = [rng.standard_normal((5, d)) for _ in range(6)]
    r1, r2, m1, m2, losses = orc.paper_run(segs, w1, w2, wkv, meta, 0.2)
    np.testing.assert_allclose(np.linalg.norm(r1, axis=1), np.linalg.norm(w1, axis=1), rtol=1e-13)
    np.testing.assert_allclose(np.linalg.norm(r2, axis=1), np.linalg.norm(w2, axis=1), rtol=1e-13)
    assert np.linalg.norm(r1 - w1) > 1e-3 and np.linalg.norm(m1) > 0  # the run does move
    assert len(losses) == 6


def test_empty_segment_changes_nothing():
    rng = np.random.default_rng(8)
    x, w1, w2, wkv, meta = _layer(rng, 4, 5, 2, 3)
    n0 = (np.linalg.norm(w1, axis=1), np.linalg.norm(w2, axis=1))
    m1, m2 = rng.standard_normal(w1.shape), rng.standard_normal(w2.shape)
    out = orc.paper_step(np.zeros((0, 4)), w1, w2, m1, m2, wkv, meta, n0, 0.1)
    for got, want in zip(out[:4], (w1, w2, m1, m2)):
        assert np.array_equal(got, want)
