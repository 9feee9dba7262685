"""Closed-form pins of the oracle's step, through its own step code.

The oracle's ttl_step/ttl_run also run two test-only memories: the linear memory y = W x (one
matrix) and the 2-layer memory with an identity activation, y = W2 W1 x.  For both, the SGD step
of Eq. update under a squared-error loss has a closed form in terms of the Gram matrix X^T X of the
segment, derived here by hand and never forming per-token residuals:

  * linear, per-token squared error summed over outputs, segment average (Sec. 3.3):
        W' = W - lr (2/T) (W - W_kv) X^T X
    (divided by D for the per-element mean; W' = W + lr (1/T) W_kv X^T X for the negative inner
    product of Eq. mem_loss);
  * repeated steps on one segment: E_k = W_k - W_kv obeys E_{k+1} = E_k (I - lr (2/T) X^T X), so
    with X of full column rank and lr (2/T) lambda_max(X^T X) < 2 the weights converge to W_kv,
    the norm of E shrinking by at most rho = max_i |1 - lr (2/T) lambda_i| per step; beyond 2
    they diverge;
  * identity activation, E = W2 W1 - W_kv, S = X^T X / T:
        dL/dW2 = 2 E S W1^T,   dL/dW1 = 2 W2^T E S;
  * one token (T = 1): both gradients are outer products, written out element by element.

A wrong loss scale, a wrong sign of the residual, the gradient or the update, a swapped operand or
a dropped factor in the backward changes one of these by far more than rounding.
"""
import math

import numpy as np
import pytest

import oracle as orc


def _linear_case(rng, d, D, T):
    x = rng.standard_normal((T, d))
    w = rng.standard_normal((D, d)) / math.sqrt(d)
    wkv = rng.standard_normal((D, d)) / math.sqrt(d)
    return x, w, wkv


@pytest.mark.parametrize("d,D,T", [(3, 2, 1), (4, 3, 7), (6, 5, 4), (5, 8, 12)])
@pytest.mark.parametrize("loss", orc.LOSSES)
def test_linear_memory_single_step_closed_form(d, D, T, loss):
    rng = np.random.default_rng([11, d, D, T])
    x, w, wkv = _linear_case(rng, d, D, T)
    lr = 0.37
    w1_new, w_new, _ = orc.ttl_step(x, None, w, wkv, lr, loss)
    assert w1_new is None
    gram = x.T @ x
    if loss == "mse_sum":
        expect = w - lr * (2.0 / T) * (w - wkv) @ gram
    elif loss == "mse_mean":
        expect = w - lr * (2.0 / (T * D)) * (w - wkv) @ gram
    else:  # negative inner product: dL/dW = -(1/T) W_kv X^T X
        expect = w + lr * (1.0 / T) * wkv @ gram
    np.testing.assert_allclose(w_new, expect, rtol=1e-12, atol=1e-13)


def test_linear_memory_loss_value_closed_form():
    # L_s = (1/T) ||X (W - W_kv)^T||_F^2 = trace(E S E^T) with S = X^T X / T
    rng = np.random.default_rng(5)
    x, w, wkv = _linear_case(rng, 5, 4, 9)
    e = w - wkv
    expect = np.trace(e @ (x.T @ x / 9.0) @ e.T)
    _, _, ls = orc.ttl_step(x, None, w, wkv, 0.0)
    assert ls == pytest.approx(expect, rel=1e-13)


def _contraction(x, lr, T):
    lam = np.linalg.eigvalsh(x.T @ x)
    return lam, np.max(np.abs(1.0 - lr * (2.0 / T) * lam))


@pytest.mark.parametrize("step_frac", [0.3, 1.0, 1.9])
def test_linear_memory_fixed_point_and_rate(step_frac):
    d, D, T = 4, 3, 10
    rng = np.random.default_rng([17, int(step_frac * 10)])
    x, w0, wkv = _linear_case(rng, d, D, T)
    lam = np.linalg.eigvalsh(x.T @ x)
    assert lam[0] > 1e-3  # full column rank
    lr = step_frac / ((2.0 / T) * lam[-1])  # lr (2/T) lambda_max = step_frac
    _, rho = _contraction(x, lr, T)
    assert rho < 1.0
    k = 40
    w1k, wk, losses = orc.ttl_run([x] * k, None, w0, wkv, lr)
    assert w1k is None
    # exact k-step closed form: E_k = E_0 (I - lr (2/T) X^T X)^k
    m = np.eye(d) - lr * (2.0 / T) * (x.T @ x)
    np.testing.assert_allclose(wk - wkv, (w0 - wkv) @ np.linalg.matrix_power(m, k),
                               rtol=1e-9, atol=1e-13)
    # the error contracts by at most rho per step, and the loss falls monotonically
    e_prev = np.linalg.norm(w0 - wkv)
    w = w0
    for _ in range(k):
        _, w, _ = orc.ttl_step(x, None, w, wkv, lr)
        e = np.linalg.norm(w - wkv)
        assert e <= rho * e_prev * (1 + 1e-12) + 1e-15
        e_prev = e
    assert all(b <= a * (1 + 1e-12) for a, b in zip(losses, losses[1:]))
    # long enough, the fixed point is W_kv itself
    _, wlong, _ = orc.ttl_run([x] * 4000, None, w0, wkv, lr)
    np.testing.assert_allclose(wlong, wkv, rtol=0, atol=1e-9)


def test_linear_memory_asymptotic_rate_is_rho():
    # with a well separated dominant mode the ratio of successive errors tends to rho itself
    d, D, T = 3, 2, 6
    x = np.zeros((T, d))
    x[0, 0], x[1, 1], x[2, 2] = 3.0, 1.0, 0.5  # X^T X = diag(9, 1, 0.25)
    x[3:, :] = 0.0
    wkv = np.arange(D * d, dtype=np.float64).reshape(D, d) / 7.0
    w0 = wkv + 1.0
    lr = 0.1 / (2.0 / T)  # lr (2/T) = 0.1: factors 1 - 0.9, 1 - 0.1, 1 - 0.025
    _, rho = _contraction(x, lr, T)
    assert rho == pytest.approx(0.975, abs=1e-15)
    w = w0
    norms = []
    for _ in range(400):
        _, w, _ = orc.ttl_step(x, None, w, wkv, lr)
        norms.append(np.linalg.norm(w - wkv))
    assert norms[-1] / norms[-2] == pytest.approx(rho, rel=1e-10)


def test_linear_memory_diverges_beyond_the_step_bound():
    d, D, T = 4, 3, 10
    rng = np.random.default_rng(23)
    x, w0, wkv = _linear_case(rng, d, D, T)
    lam = np.linalg.eigvalsh(x.T @ x)
    lr = 2.1 / ((2.0 / T) * lam[-1])
    _, w, _ = orc.ttl_run([x] * 200, None, w0, wkv, lr)
    assert np.linalg.norm(w - wkv) > 1e3 * np.linalg.norm(w0 - wkv)


@pytest.mark.parametrize("d,h,D,T", [(3, 4, 2, 1), (4, 6, 5, 7), (5, 3, 4, 9)])
def test_identity_activation_two_layer_closed_form(d, h, D, T):
    rng = np.random.default_rng([29, d, h, D, T])
    x = rng.standard_normal((T, d))
    w1 = rng.standard_normal((h, d)) / math.sqrt(d)
    w2 = rng.standard_normal((D, h)) / math.sqrt(h)
    wkv = rng.standard_normal((D, d)) / math.sqrt(d)
    e = w2 @ w1 - wkv
    s = x.T @ x / T
    gw1, gw2, ls = orc.segment_grad(x, w1, w2, wkv, activation="identity")
    np.testing.assert_allclose(gw2, 2.0 * e @ s @ w1.T, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(gw1, 2.0 * w2.T @ e @ s, rtol=1e-11, atol=1e-13)
    assert ls == pytest.approx(np.trace(e @ s @ e.T), rel=1e-12)
    lr = 0.05
    n1, n2, _ = orc.ttl_step(x, w1, w2, wkv, lr, activation="identity")
    np.testing.assert_allclose(n1, w1 - lr * 2.0 * w2.T @ e @ s, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(n2, w2 - lr * 2.0 * e @ s @ w1.T, rtol=1e-11, atol=1e-13)


def test_identity_activation_converges_to_the_targets_map():
    # repeated steps on one full-rank segment drive the product W2 W1 to W_kv
    d, h, D, T = 3, 5, 2, 12
    rng = np.random.default_rng(31)
    x = rng.standard_normal((T, d))
    w1 = rng.standard_normal((h, d)) / math.sqrt(d)
    w2 = rng.standard_normal((D, h)) / math.sqrt(h)
    wkv = rng.standard_normal((D, d)) / math.sqrt(d)
    o1, o2, losses = orc.ttl_run([x] * 3000, w1, w2, wkv, 0.05, activation="identity")
    np.testing.assert_allclose(o2 @ o1, wkv, rtol=0, atol=1e-8)
    assert losses[-1] < 1e-16 * max(1.0, losses[0]) + 1e-18


def test_single_token_gradients_are_outer_products():
    # T = 1: G = 2 (y - t) is one row, so dL/dW2[o, i] = 2 (y_o - t_o) a_i and
    # dL/dW1[i, c] = (sum_o 2 (y_o - t_o) W2[o, i]) SiLU'(z_i) x_c, written out element by element
    rng = np.random.default_rng(37)
    d, h, D = 3, 4, 2
    x = rng.standard_normal((1, d))
    w1 = rng.standard_normal((h, d))
    w2 = rng.standard_normal((D, h))
    wkv = rng.standard_normal((D, d))
    z = [sum(w1[i, c] * x[0, c] for c in range(d)) for i in range(h)]
    sg = [1.0 / (1.0 + math.exp(-zi)) for zi in z]
    a = [zi * si for zi, si in zip(z, sg)]
    da = [si * (1.0 + zi * (1.0 - si)) for zi, si in zip(z, sg)]
    y = [sum(w2[o, i] * a[i] for i in range(h)) for o in range(D)]
    t = [sum(wkv[o, c] * x[0, c] for c in range(d)) for o in range(D)]
    g = [2.0 * (y[o] - t[o]) for o in range(D)]
    gw2 = np.array([[g[o] * a[i] for i in range(h)] for o in range(D)])
    gw1 = np.array([[sum(g[o] * w2[o, i] for o in range(D)) * da[i] * x[0, c] for c in range(d)]
                    for i in range(h)])
    o1, o2, _ = orc.segment_grad(x, w1, w2, wkv)
    np.testing.assert_allclose(o2, gw2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(o1, gw1, rtol=1e-12, atol=1e-14)
