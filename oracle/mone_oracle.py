"""CPU oracle of MoNe test-time learning (TTL) — TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

Only the test-suite, the package's smoke check and the benchmark's CPU-baseline leg may import
this module.  The product path (the HIP library and its Python binding) never calls it, and it
imports nothing from the product package: its inputs are plain arrays.

What it computes (MoNe, Sec. 3): a long context is split into segments of T tokens (Sec. 3.1).
Every layer l owns a fast-weight memory M(.; W^(l)).  For each segment s in order, and for every
layer independently, the memory takes one gradient step on the associative loss of that segment,
evaluated at W_{s-1} (Sec. 3.4, layer-localised gradient; Eq. update).  After the last segment
the memory is read on query-side inputs without any update (Eq. read).

The memory, loss and optimiser are the configuration-mode ones (a plain, fully specified variant
of the paper's richer defaults; each choice is stated where it is made):
  * M(x) = W2 . SiLU(W1 . x): a 2-layer MLP d -> h -> D with SiLU and no biases.  The paper's
    memory is a SwiGLU MLP per fast-weight head (Eq. swiglu); the configuration keeps its
    structure (input matrix, SiLU, output matrix) without the gate branch.  W1 = W_in is [h, d]
    and W2 = W_out^T is [D, h], both acting on column vectors as in the paper.
  * targets: t_j = [W_k x_j ; W_v x_j] (Eq. proj), frozen projections, raw (no SiLU/L2 norm/RoPE).
  * per-token loss l_j = ||M(x_j) - t_j||^2 summed over the D outputs ("mse_sum"), or divided by
    D ("mse_mean"); or the paper's negative inner product l_j = -t_j . M(x_j) (Eq. mem_loss;
    "nip"), whose value target in this form is the whole [K | V] row t_j; segment loss
    L_s = (1/T) sum_j l_j (the segment-level average of Sec. 3.3).
  * update: W_s = W_{s-1} - lr * grad L_s(W_{s-1})  (Eq. update with mu_s = lr * gradient).

Two test-only memories run through the same step code, so that closed forms can pin it:
  * activation = "identity": M(x) = W2 W1 x, the 2-layer memory with a linear hidden layer;
  * w1 = None: the linear memory M(x) = W2 x with one matrix W2 of shape [D, d].
Neither is part of the method; the kernels implement the SiLU memory only.

Everything is float64 NumPy.  Matrix products use numpy's matmul as a library primitive; there is
no blocking, fusion or reordering beyond the definitions.

Pins (tests in tests/test_oracle_*.py): hand-derived scalar case, central finite differences,
torch.autograd (float64, CPU), brute-force loops, first-order descent, closed forms of the linear
and identity-activation memories (one step in Gram-matrix form, the fixed point W -> W_kv and its
contraction rate), and invariants (lr = 0, zero residual, token duplication under the segment
average, segment order, incremental == one-shot, layer independence).
"""
from __future__ import annotations

import numpy as np

LOSSES = ("mse_sum", "mse_mean", "nip")
ACTIVATIONS = ("silu", "identity")  # "identity" is test-only


def sigmoid(z):
    """Logistic function, evaluated without overflow for large |z|."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(-np.abs(z))
    return np.where(z >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def silu(z):
    """SiLU(z) = z * sigmoid(z) (the activation of Eq. swiglu)."""
    z = np.asarray(z, dtype=np.float64)
    return z * sigmoid(z)


def silu_grad(z):
    """d SiLU / dz = sigmoid(z) * (1 + z * (1 - sigmoid(z)))."""
    z = np.asarray(z, dtype=np.float64)
    s = sigmoid(z)
    return s * (1.0 + z * (1.0 - s))


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def _act(z, activation: str):
    """Hidden-layer activation: SiLU (the method), or the identity (test only)."""
    if activation == "silu":
        return silu(z)
    if activation == "identity":
        return z
    raise ValueError(activation)


def _act_grad(z, activation: str):
    """Derivative of the hidden-layer activation at z."""
    if activation == "silu":
        return silu_grad(z)
    if activation == "identity":
        return np.ones_like(z)
    raise ValueError(activation)


def memory_forward(x, w1, w2, activation: str = "silu"):
    """Memory MLP on the rows of x ([n, d]): returns (Z, A, Y) with
    Z = x W1^T ([n, h]), A = SiLU(Z), Y = A W2^T ([n, D]) -- i.e. y_j = W2 SiLU(W1 x_j).
    With w1 = None (test only) the memory is the linear map y_j = W2 x_j: Z = A = x."""
    x, w2 = _f64(x), _f64(w2)
    if w1 is None:
        z = a = x
    else:
        z = x @ _f64(w1).T
        a = _act(z, activation)
    y = a @ w2.T
    return z, a, y


def targets(x, wkv):
    """Associative targets of Eq. proj, stacked per token: t_j = [W_k x_j ; W_v x_j] = W_kv x_j."""
    return _f64(x) @ _f64(wkv).T


def _loss_scale(n: int, d_out: int, loss: str) -> float:
    """Factor c with dL_s/dY = c * (Y - targets) (mse) or dL_s/dY = -c * targets (nip)."""
    if loss == "mse_sum":
        return 2.0 / n
    if loss == "mse_mean":
        return 2.0 / (n * d_out)
    if loss == "nip":
        return 1.0 / n
    raise ValueError(loss)


def _per_token_loss(y, t, loss: str):
    """l_j for the rows of Y and the targets."""
    if loss == "nip":
        return -np.sum(t * y, axis=1)
    r = y - t
    per_token = np.sum(r * r, axis=1)
    if loss == "mse_mean":
        per_token = per_token / r.shape[1]
    elif loss != "mse_sum":
        raise ValueError(loss)
    return per_token


def _output_grad(y, t, c: float, loss: str):
    """dL_s/dY: c (Y - T) for the squared errors, -c T for the negative inner product."""
    return -c * t if loss == "nip" else c * (y - t)


def segment_loss(x, w1, w2, wkv, loss: str = "mse_sum") -> float:
    """L_s = (1/T) sum_j l_j for the T rows of x (segment-level average, Sec. 3.3)."""
    x = _f64(x)
    n = x.shape[0]
    if n == 0:
        return 0.0
    _, _, y = memory_forward(x, w1, w2)
    return float(np.sum(_per_token_loss(y, targets(x, wkv), loss)) / n)


def segment_grad(x, w1, w2, wkv, loss: str = "mse_sum", activation: str = "silu"):
    """Gradient of L_s with respect to this layer's own fast weights only (Sec. 3.4).

    Returns (dL/dW1 [h, d], dL/dW2 [D, h], L_s).  Backpropagation through the two matrices:
      G  = dL/dY = c (Y - targets)   (squared errors; -c targets for the negative inner product)
      dL/dW2 = G^T A
      dZ = (G W2) * SiLU'(Z)
      dL/dW1 = dZ^T x
    An empty segment has no tokens and contributes a zero gradient.  The test-only linear memory
    (w1 = None) has no first matrix, so its dL/dW1 is None.
    """
    x, w2, wkv = _f64(x), _f64(w2), _f64(wkv)
    n = x.shape[0]
    if n == 0:
        return (None if w1 is None else np.zeros_like(_f64(w1))), np.zeros_like(w2), 0.0
    z, a, y = memory_forward(x, w1, w2, activation)
    t = targets(x, wkv)
    c = _loss_scale(n, w2.shape[0], loss)
    g = _output_grad(y, t, c, loss)
    gw2 = g.T @ a
    gw1 = None
    if w1 is not None:
        dz = (g @ w2) * _act_grad(z, activation)
        gw1 = dz.T @ x
    return gw1, gw2, float(np.sum(_per_token_loss(y, t, loss)) / n)


def ttl_step(x, w1, w2, wkv, lr: float, loss: str = "mse_sum", activation: str = "silu"):
    """One test-time-learning step of one layer on one segment (Eq. update):
    both matrices move along the gradient taken at W_{s-1}.  Returns (W1_s, W2_s, L_s)."""
    gw1, gw2, ls = segment_grad(x, w1, w2, wkv, loss, activation)
    w1_new = None if w1 is None else _f64(w1) - lr * gw1
    return w1_new, _f64(w2) - lr * gw2, ls


def ttl_run(segments, w1, w2, wkv, lr: float, loss: str = "mse_sum", activation: str = "silu"):
    """Sequential TTL of one layer: W_0 -> W_1 -> ... -> W_S over the segments in the given order.
    Returns (W1_S, W2_S, [L_1, ..., L_S])."""
    w1 = None if w1 is None else _f64(w1)
    w2 = _f64(w2)
    losses = []
    for x in segments:
        w1, w2, ls = ttl_step(x, w1, w2, wkv, lr, loss, activation)
        losses.append(ls)
    return w1, w2, losses


def ttl_run_layers(segments_per_layer, w1s, w2s, wkvs, lr: float, loss: str = "mse_sum"):
    """TTL of several layers.  The gradient of layer l's loss with respect to any other layer's
    fast weights is zero (Sec. 3.4), so every layer runs its own chain; nothing crosses layers."""
    out = []
    for segs, w1, w2, wkv in zip(segments_per_layer, w1s, w2s, wkvs):
        out.append(ttl_run(segs, w1, w2, wkv, lr, loss))
    return out


def memory_kv(xq, w1, w2):
    """Read of the final state (Eq. read): the memory's output on the query-side inputs,
    [q, D] with K in columns [0, d_kv) and V in [d_kv, D).  Nothing is updated."""
    return memory_forward(xq, w1, w2)[2]
