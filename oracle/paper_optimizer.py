"""CPU oracle of MoNe's own update rule -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

Only the test-suite, the package's smoke check and the benchmark's CPU-baseline leg may import
this module; the product path never calls it.

The configuration-mode oracle (mone_oracle) takes a plain SGD step.  The paper's own optimiser
(Sec. 3.3, Eq. update; implementation details in App. A.2) replaces it with:
  * a per-token learning rate, softplus-activated and predicted from the token;
  * momentum whose decay beta_s in (0, 1) is sigmoid-activated and predicted from the hidden
    states of the segment ("chunk");
  * a channel-wise L2 renormalisation of the fast weights after every update.
The paper names these ingredients but not their exact form, so each is a stated reading:
  eta_j  = lr * softplus(u . x_j + b_u)                       (per token j of the segment)
  beta_s = sigmoid(v . xbar_s + b_v),  xbar_s = (1/n) sum_j x_j  (one scalar per layer, segment)
  g      = gradient of (1/n) sum_j eta_j l_j at W_{s-1}        (each token's gradient weighted
                                                               by its own rate)
  mu_s   = beta_s mu_{s-1} + g,   mu_0 = 0                     (Eq. update: W_s = W_{s-1} - mu_s)
  W_s    = rows of (W_{s-1} - mu_s) rescaled to the L2 norms the same rows had in W_0
           (a "channel" is an output unit: a row of W1 [h, d] and of W2 [D, h]; a row of norm 0
           is left as it is)
with u, v in R^d and b_u, b_v scalars per layer: the meta-parameters the paper trains offline
(synthetic values here).  The memory, targets and loss are the configuration-mode ones.

Float64 NumPy; matmul is the library primitive.  Pins: tests/test_oracle_paper_optimizer.py.
"""
from __future__ import annotations

import numpy as np

from .mone_oracle import (_loss_scale, _output_grad, _per_token_loss, memory_forward, sigmoid,
                          silu_grad, targets)


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def softplus(z):
    """softplus(z) = log(1 + e^z), evaluated without overflow."""
    z = _f64(z)
    return np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z)))


def token_rates(x, u, b_u, lr):
    """Per-token learning rates eta_j = lr * softplus(u . x_j + b_u), shape [n]."""
    return float(lr) * softplus(_f64(x) @ _f64(u) + float(b_u))


def momentum_decay(x, v, b_v):
    """beta_s = sigmoid(v . xbar + b_v) with xbar the mean hidden state of the segment."""
    x = _f64(x)
    xbar = x.mean(axis=0)
    return float(sigmoid(xbar @ _f64(v) + float(b_v)))


def row_norms(w):
    """L2 norm of every output channel (row) of a fast weight."""
    w = _f64(w)
    return np.sqrt(np.sum(w * w, axis=1))


def renormalise(w, norms0):
    """Rescale every row of w to the norm norms0 gives for it; rows of norm 0 stay as they are."""
    w = _f64(w)
    nrm = row_norms(w)
    scale = np.where(nrm > 0, _f64(norms0) / np.where(nrm > 0, nrm, 1.0), 1.0)
    return w * scale[:, None]


def weighted_grad(x, w1, w2, wkv, eta, loss: str = "mse_sum"):
    """Gradient of (1/n) sum_j eta_j l_j with respect to this layer's W1 and W2, and the
    unweighted segment loss L_s (for reporting).  With every eta_j = 1 this is segment_grad."""
    x, w1, w2, wkv, eta = _f64(x), _f64(w1), _f64(w2), _f64(wkv), _f64(eta)
    n = x.shape[0]
    z, a, y = memory_forward(x, w1, w2)
    t = targets(x, wkv)
    c = _loss_scale(n, w2.shape[0], loss)
    g = eta[:, None] * _output_grad(y, t, c, loss)
    gw2 = g.T @ a
    dz = (g @ w2) * silu_grad(z)
    gw1 = dz.T @ x
    return gw1, gw2, float(np.sum(_per_token_loss(y, t, loss)) / n)


def paper_step(x, w1, w2, m1, m2, wkv, meta, norms0, lr, loss: str = "mse_sum"):
    """One step of one layer on one segment with the paper's optimiser.

    meta = (u, b_u, v, b_v); norms0 = (row norms of W1_0, row norms of W2_0).
    Returns (W1_s, W2_s, mu1_s, mu2_s, L_s, info) with info = {"eta", "beta", "g1", "g2"}.
    An empty segment changes nothing (no gradient, no momentum decay)."""
    x = _f64(x)
    u, b_u, v, b_v = meta
    if x.shape[0] == 0:
        return _f64(w1), _f64(w2), _f64(m1), _f64(m2), 0.0, {}
    eta = token_rates(x, u, b_u, lr)
    beta = momentum_decay(x, v, b_v)
    g1, g2, ls = weighted_grad(x, w1, w2, wkv, eta, loss)
    m1n = beta * _f64(m1) + g1
    m2n = beta * _f64(m2) + g2
    w1n = renormalise(_f64(w1) - m1n, norms0[0])
    w2n = renormalise(_f64(w2) - m2n, norms0[1])
    return w1n, w2n, m1n, m2n, ls, {"eta": eta, "beta": beta, "g1": g1, "g2": g2}


def paper_run(segments, w1, w2, wkv, meta, lr, loss: str = "mse_sum"):
    """Sequential TTL of one layer with the paper's optimiser, from W_0 = (w1, w2) and zero
    momentum; the renormalisation targets are the row norms of W_0.
    Returns (W1_S, W2_S, mu1_S, mu2_S, [L_1, ..., L_S])."""
    w1, w2 = _f64(w1), _f64(w2)
    norms0 = (row_norms(w1), row_norms(w2))
    m1, m2 = np.zeros_like(w1), np.zeros_like(w2)
    losses = []
    for x in segments:
        w1, w2, m1, m2, ls, _ = paper_step(x, w1, w2, m1, m2, wkv, meta, norms0, lr, loss)
        losses.append(ls)
    return w1, w2, m1, m2, losses
