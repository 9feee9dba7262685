"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test fixes a part of the oracle that a plausible mistake would break:
  * SiLU: a special value, an exact identity, and the closed form of its minimum;
  * forward, targets and loss: brute-force scalar loops on tiny inputs (catches a transposed
    weight, a dropped term or a wrong reduction);
  * gradients: central finite differences of the loss, and torch.autograd on CPU in float64
    (catches a wrong sign, scale or index in backprop);
  * the update: a first-order descent identity (catches a wrong step sign or scale), the
    segment average (duplicating every token leaves the step unchanged) and lr = 0;
  * the TTL chain: segment order matters, a split run equals the one-shot run, layers are
    independent, and a zero residual leaves the weights unchanged.
"""
import math

import numpy as np
import pytest

import oracle as orc

SHAPES = [  # (d, h, D, T)
    (3, 4, 2, 1), (3, 7, 6, 3), (5, 4, 6, 5), (5, 7, 2, 3), (4, 6, 4, 5),
]


def _rand_layer(rng, d, h, D, T, scale=1.0):
    x = rng.standard_normal((T, d))
    w1 = rng.standard_normal((h, d)) * scale / math.sqrt(d)
    w2 = rng.standard_normal((D, h)) * scale / math.sqrt(h)
    wkv = rng.standard_normal((D, d)) / math.sqrt(d)
    return x, w1, w2, wkv


# ---------------------------------------------------------------- SiLU

def test_silu_special_values():
    # SiLU(1) = 1 * logistic(1) = e / (1 + e)
    assert orc.silu(1.0) == pytest.approx(math.e / (1.0 + math.e), rel=1e-15)
    assert orc.silu(0.0) == 0.0
    # SiLU(z) -> z for large z, -> 0 for very negative z; no overflow warnings
    with np.errstate(over="raise"):
        assert orc.silu(800.0) == 800.0
        assert orc.silu(-800.0) == pytest.approx(0.0, abs=1e-300)


def test_silu_reflection_identity():
    # SiLU(-z) = -z * (1 - logistic(z)) = SiLU(z) - z
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(orc.silu(-z), orc.silu(z) - z, rtol=0, atol=1e-13)


def test_silu_minimum_closed_form():
    # At the minimum z*, SiLU'(z*) = 0 <=> 1 + z*(1 - s) = 0, so s = 1 + 1/z* and
    # SiLU(z*) = z* s = z* + 1.  Bisection on SiLU' finds z*; then check SiLU(z*) = z* + 1.
    lo, hi = -2.0, -1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if orc.silu_grad(mid) < 0:  # SiLU decreases left of z*, increases right of it
            lo = mid
        else:
            hi = mid
    zs = 0.5 * (lo + hi)
    assert orc.silu(zs) == pytest.approx(zs + 1.0, abs=1e-14)
    assert zs == pytest.approx(-1.2784645427610738, abs=1e-12)


def test_silu_grad_finite_difference():
    z = np.linspace(-12, 12, 97)
    eps = 1e-5
    fd = (orc.silu(z + eps) - orc.silu(z - eps)) / (2 * eps)
    np.testing.assert_allclose(orc.silu_grad(z), fd, rtol=0, atol=1e-9)


# ---------------------------------------------------------------- forward, targets, loss

def _brute_forward_and_loss(x, w1, w2, wkv, loss):
    T, d = x.shape
    h, D = w1.shape[0], w2.shape[0]
    total = 0.0
    ys = []
    for j in range(T):
        a = []
        for i in range(h):
            z = sum(w1[i][k] * x[j][k] for k in range(d))
            a.append(z / (1.0 + math.exp(-z)))
        y = [sum(w2[o][i] * a[i] for i in range(h)) for o in range(D)]
        t = [sum(wkv[o][k] * x[j][k] for k in range(d)) for o in range(D)]
        if loss == "nip":  # negative inner product with the target row
            lj = -sum(y[o] * t[o] for o in range(D))
        else:
            lj = sum((y[o] - t[o]) ** 2 for o in range(D))
        if loss == "mse_mean":
            lj /= D
        total += lj
        ys.append(y)
    return np.array(ys), total / T


@pytest.mark.parametrize("loss", orc.LOSSES)
@pytest.mark.parametrize("shape", SHAPES[:3])
def test_forward_and_loss_brute_force(shape, loss):
    rng = np.random.default_rng(11)
    x, w1, w2, wkv = _rand_layer(rng, *shape)
    y_ref, l_ref = _brute_forward_and_loss(x, w1, w2, wkv, loss)
    np.testing.assert_allclose(orc.memory_kv(x, w1, w2), y_ref, rtol=1e-13, atol=1e-14)
    assert orc.segment_loss(x, w1, w2, wkv, loss) == pytest.approx(l_ref, rel=1e-13)
    # the loss returned with the gradient is the same quantity
    assert orc.segment_grad(x, w1, w2, wkv, loss)[2] == pytest.approx(l_ref, rel=1e-13)


def test_targets_stack_k_then_v():
    # t_j = [W_k x_j ; W_v x_j]: rows [0, d_kv) of W_kv give K, rows [d_kv, D) give V.
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 5))
    wk, wv = rng.standard_normal((2, 5)), rng.standard_normal((2, 5))
    t = orc.targets(x, np.concatenate([wk, wv]))
    for j in range(4):
        for o in range(2):
            assert t[j, o] == pytest.approx(sum(wk[o, k] * x[j, k] for k in range(5)), rel=1e-14)
            assert t[j, 2 + o] == pytest.approx(sum(wv[o, k] * x[j, k] for k in range(5)),
                                                rel=1e-14)


# ---------------------------------------------------------------- gradients

def _fd_grad(f, w, step_rel=1e-6):
    g = np.zeros_like(w)
    it = np.nditer(w, flags=["multi_index"])
    for _ in it:
        idx = it.multi_index
        hstep = step_rel * max(1.0, abs(w[idx]))
        wp, wm = w.copy(), w.copy()
        wp[idx] += hstep
        wm[idx] -= hstep
        g[idx] = (f(wp) - f(wm)) / (2 * hstep)
    return g


@pytest.mark.parametrize("loss", orc.LOSSES)
@pytest.mark.parametrize("shape", SHAPES)
def test_gradient_finite_differences(shape, loss):
    rng = np.random.default_rng(sum(shape))
    x, w1, w2, wkv = _rand_layer(rng, *shape, scale=2.0)
    gw1, gw2, _ = orc.segment_grad(x, w1, w2, wkv, loss)
    fd1 = _fd_grad(lambda w: orc.segment_loss(x, w, w2, wkv, loss), w1)
    fd2 = _fd_grad(lambda w: orc.segment_loss(x, w1, w, wkv, loss), w2)
    assert np.linalg.norm(gw1 - fd1) <= 1e-7 * np.linalg.norm(fd1)
    assert np.linalg.norm(gw2 - fd2) <= 1e-7 * np.linalg.norm(fd2)


@pytest.mark.parametrize("loss", orc.LOSSES)
def test_steps_match_torch_autograd(loss):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(5)
    d, h, D, T, S, lr = 24, 40, 16, 12, 4, 0.05
    x_segs = [rng.standard_normal((T, d)) for _ in range(S)]
    _, w1, w2, wkv = _rand_layer(rng, d, h, D, T)

    tw1 = torch.tensor(w1, dtype=torch.float64)
    tw2 = torch.tensor(w2, dtype=torch.float64)
    twkv = torch.tensor(wkv, dtype=torch.float64)
    for x in x_segs:
        tx = torch.tensor(x, dtype=torch.float64)
        p1 = tw1.clone().requires_grad_(True)
        p2 = tw2.clone().requires_grad_(True)
        y = F.linear(F.silu(F.linear(tx, p1)), p2)
        tgt = F.linear(tx, twkv)
        if loss == "mse_sum":
            ls = F.mse_loss(y, tgt, reduction="sum") / T
        elif loss == "mse_mean":
            ls = F.mse_loss(y, tgt, reduction="mean")
        else:
            ls = -(y * tgt).sum() / T
        ls.backward()
        with torch.no_grad():
            tw1 = p1 - lr * p1.grad
            tw2 = p2 - lr * p2.grad
    o1, o2, _ = orc.ttl_run(x_segs, w1, w2, wkv, lr, loss)
    np.testing.assert_allclose(o1, tw1.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(o2, tw2.numpy(), rtol=0, atol=1e-13)


# ---------------------------------------------------------------- the update

@pytest.mark.parametrize("loss", orc.LOSSES)
def test_step_is_first_order_descent(loss):
    # L(W - lr g) - L(W) = -lr ||g||^2 + O(lr^2): the ratio tends to 1 as lr -> 0.  A step with
    # the wrong sign gives -1, a wrong scale k gives k, a wrong direction gives |ratio| < 1.
    rng = np.random.default_rng(9)
    x, w1, w2, wkv = _rand_layer(rng, 6, 9, 4, 7)
    gw1, gw2, l0 = orc.segment_grad(x, w1, w2, wkv, loss)
    gsq = np.sum(gw1 ** 2) + np.sum(gw2 ** 2)
    ratios = []
    for lr in (1e-3, 1e-4, 1e-5):
        n1, n2, _ = orc.ttl_step(x, w1, w2, wkv, lr, loss)
        ratios.append((l0 - orc.segment_loss(x, n1, n2, wkv, loss)) / (lr * gsq))
    assert abs(ratios[-1] - 1.0) < 1e-4
    assert abs(ratios[-1] - 1.0) < abs(ratios[0] - 1.0)


def test_segment_average_duplicate_tokens():
    # L_s averages over the segment's tokens, so repeating every token k times changes nothing.
    rng = np.random.default_rng(2)
    x, w1, w2, wkv = _rand_layer(rng, 5, 6, 4, 3)
    a1, a2, la = orc.ttl_step(x, w1, w2, wkv, 0.1)
    b1, b2, lb = orc.ttl_step(np.concatenate([x, x, x]), w1, w2, wkv, 0.1)
    np.testing.assert_allclose(a1, b1, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(a2, b2, rtol=1e-14, atol=1e-15)
    assert la == pytest.approx(lb, rel=1e-14)


def test_mean_reduction_is_sum_over_outputs():
    rng = np.random.default_rng(4)
    x, w1, w2, wkv = _rand_layer(rng, 5, 6, 4, 3)
    s1, s2, ls = orc.segment_grad(x, w1, w2, wkv, "mse_sum")
    m1, m2, lm = orc.segment_grad(x, w1, w2, wkv, "mse_mean")
    np.testing.assert_allclose(m1 * 4, s1, rtol=1e-13)
    np.testing.assert_allclose(m2 * 4, s2, rtol=1e-13)
    assert lm * 4 == pytest.approx(ls, rel=1e-14)


def test_lr_zero_leaves_weights_bitwise():
    rng = np.random.default_rng(6)
    x, w1, w2, wkv = _rand_layer(rng, 5, 6, 4, 3)
    n1, n2, _ = orc.ttl_run([x, x * 2], w1, w2, wkv, 0.0)
    assert np.array_equal(n1, w1) and np.array_equal(n2, w2)


def test_zero_residual_leaves_weights_bitwise():
    # W2 = 0 and W_kv = 0: the memory already outputs the targets (both 0), so G = 0 and both
    # gradients vanish exactly.
    rng = np.random.default_rng(7)
    x, w1, _, _ = _rand_layer(rng, 5, 6, 4, 3)
    w2, wkv = np.zeros((4, 6)), np.zeros((4, 5))
    n1, n2, ls = orc.ttl_step(x, w1, w2, wkv, 0.5)
    assert ls == 0.0
    assert np.array_equal(n1, w1) and np.array_equal(n2, w2)


def test_empty_segment_is_a_no_op():
    rng = np.random.default_rng(8)
    _, w1, w2, wkv = _rand_layer(rng, 5, 6, 4, 3)
    n1, n2, ls = orc.ttl_step(np.zeros((0, 5)), w1, w2, wkv, 0.5)
    assert ls == 0.0 and np.array_equal(n1, w1) and np.array_equal(n2, w2)


# ---------------------------------------------------------------- the TTL chain

def test_segment_order_matters():
    rng = np.random.default_rng(12)
    d, h, D, T = 8, 12, 6, 5
    _, w1, w2, wkv = _rand_layer(rng, d, h, D, T)
    s1, s2 = rng.standard_normal((T, d)), rng.standard_normal((T, d))
    a1, a2, _ = orc.ttl_run([s1, s2], w1, w2, wkv, 0.2)
    b1, b2, _ = orc.ttl_run([s2, s1], w1, w2, wkv, 0.2)
    # W_2 depends on the order: the difference is second order in lr but far above rounding
    assert np.linalg.norm(a1 - b1) > 1e-6 * np.linalg.norm(a1 - w1)
    assert np.linalg.norm(a2 - b2) > 1e-6 * np.linalg.norm(a2 - w2)
    assert np.linalg.norm(a2 - b2) > 1e-9


def test_incremental_extension_equals_one_shot():
    rng = np.random.default_rng(13)
    d, h, D, T = 8, 12, 6, 5
    _, w1, w2, wkv = _rand_layer(rng, d, h, D, T)
    segs = [rng.standard_normal((T, d)) for _ in range(5)]
    o1, o2, lo = orc.ttl_run(segs, w1, w2, wkv, 0.1)
    p1, p2, lp = orc.ttl_run(segs[:2], w1, w2, wkv, 0.1)
    q1, q2, lq = orc.ttl_run(segs[2:], p1, p2, wkv, 0.1)
    assert np.array_equal(o1, q1) and np.array_equal(o2, q2)
    assert lo == lp + lq


def test_layers_are_independent():
    rng = np.random.default_rng(14)
    d, h, D, T = 6, 8, 4, 3
    layers = [_rand_layer(rng, d, h, D, T) for _ in range(3)]
    segs = [[rng.standard_normal((T, d)) for _ in range(2)] for _ in range(3)]
    res = orc.ttl_run_layers(segs, [l[1] for l in layers], [l[2] for l in layers],
                             [l[3] for l in layers], 0.1)
    # perturbing layer 1's inputs changes nothing in layers 0 and 2
    segs2 = [segs[0], [s + 1.0 for s in segs[1]], segs[2]]
    res2 = orc.ttl_run_layers(segs2, [l[1] for l in layers], [l[2] for l in layers],
                              [l[3] for l in layers], 0.1)
    for l in (0, 2):
        assert np.array_equal(res[l][0], res2[l][0]) and np.array_equal(res[l][1], res2[l][1])
    assert not np.array_equal(res[1][0], res2[1][0])
    # each layer alone equals the same layer inside the group
    alone = orc.ttl_run(segs[2], layers[2][1], layers[2][2], layers[2][3], 0.1)
    assert np.array_equal(alone[0], res[2][0]) and np.array_equal(alone[1], res[2][1])


def test_repeated_segment_reduces_loss():
    # Plain gradient descent with a small step on a fixed segment lowers its loss every step.
    rng = np.random.default_rng(15)
    x, w1, w2, wkv = _rand_layer(rng, 8, 16, 4, 32)
    _, _, losses = orc.ttl_run([x] * 20, w1, w2, wkv, 0.05)
    assert all(b < a for a, b in zip(losses, losses[1:]))


def test_memory_kv_is_read_only():
    rng = np.random.default_rng(16)
    x, w1, w2, _ = _rand_layer(rng, 5, 6, 4, 3)
    c1, c2, cx = w1.copy(), w2.copy(), x.copy()
    y1 = orc.memory_kv(x, w1, w2)
    y2 = orc.memory_kv(x, w1, w2)
    assert np.array_equal(y1, y2)
    assert np.array_equal(w1, c1) and np.array_equal(w2, c2) and np.array_equal(x, cx)


def test_negative_inner_product_gradient_of_w2_does_not_depend_on_w2():
    # dL/dY = -T/n does not involve Y, so dL/dW2 = -(1/n) T^T A is the same at any W2, and
    # dL/dW1 is linear in W2
    rng = np.random.default_rng(12)
    x, w1, w2, wkv = _rand_layer(rng, 5, 6, 4, 7)
    g1a, g2a, _ = orc.segment_grad(x, w1, w2, wkv, "nip")
    g1b, g2b, _ = orc.segment_grad(x, w1, 3.0 * w2 + 1.0, wkv, "nip")
    np.testing.assert_allclose(g2a, g2b, rtol=1e-13, atol=1e-15)
    g1c, _, _ = orc.segment_grad(x, w1, 3.0 * w2, wkv, "nip")
    np.testing.assert_allclose(g1c, 3.0 * g1a, rtol=1e-12, atol=1e-15)
