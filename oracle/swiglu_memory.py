"""CPU oracle of the paper-form memory (SwiGLU per fast-weight head) -- TEST INFRASTRUCTURE,
NOT PART OF THE PRODUCT.

Only the test-suite, the package's smoke check and the benchmark's CPU-baseline leg may import
this module; the product path never calls it.

The memory of one layer (Sec. 3.2, Eq. swiglu) is H independent heads of width d_h; head e has
three d_h x d_h fast weights and maps a key k_e to
    M_e(k_e) = W_out^T ( SiLU(W_in k_e) * (W_gate k_e) )
(row form, one token per row: z = k W_in^T, g = k W_gate^T, a = SiLU(z) * g, y = a W_out).
During test-time learning (Sec. 3.3) it is trained on the segment's tokens with
  * key / value targets projected from the layer's hidden states (Eq. proj): r_k = x P_k^T,
    r_v = x P_v^T, both of width d = H d_h;
  * key preprocessing (Sec. 3.3, App. A.2): per-channel affine s * r_k + b, SiLU, per-token and
    per-head L2 normalisation, then segment-local RoPE at position j mod T (the token's index in
    its segment);
  * value preprocessing: SiLU;
  * the negative inner product loss of Eq. mem_loss, l_j = -sum_e v_{j,e} . M_e(k_{j,e}),
    averaged over the segment's n tokens;
  * a gradient step (Eq. update) with plain SGD, or with the paper's optimiser: per-token rates,
    momentum with a data-dependent decay, rows renormalised to their initial L2 norms (App. A.2;
    its readings live in paper_optimizer).
Readings (the paper leaves these open):
  * the key and value projections of the targets map the hidden state to the memory's width
    d = H d_h (synthetic frozen weights P_k, P_v);
  * the affine step is a per-channel scale and shift; L2 normalisation divides by
    max(||k_e||, 1e-12);
  * RoPE rotates the channel pairs (c, c + d_h/2) of each head by the angle p * base^(-2c/d_h)
    ("rotate-half" layout), base 10000;
  * a "channel" renormalised by the paper's optimiser is a row of each stored d_h x d_h matrix
    (W_in, W_gate: one hidden unit's input weights; W_out: the output pattern one hidden unit
    writes).

At read time (Eq. read, Eq. attn) the query tokens' hidden states x_q go through the query
projection P_q and the keys' preprocessing (with the query's own affine step; RoPE at positions
0..Q-1, Sec. 3.3), the memory reads them per head, and the output o_e of each head is
RMS-normalised and gated (Sec. 3.2, App. A.2):
    h_{j,e} = RMSNorm(o_{j,e}) * w_rms_e * SiLU(a_e . x_j + c_e),
    RMSNorm(o) = o / sqrt(mean(o^2) + 1e-6);
the memory tokens h are then projected by the backbone's frozen key and value maps, [h W_k^T |
h W_v^T], and join the query tokens' attention (memory_attention).
Readings of the read path: the gate is a learned per-head vector a_e (and bias c_e) on the
query token's hidden state, passed through SiLU (per head, Sec. 3.2; SiLU-gated, App. A.2);
the RMSNorm has a learned per-channel weight w_rms.

Float64 NumPy; plain loops over heads; matmul is the library primitive.
Pins: tests/test_oracle_swiglu_memory.py.
"""
from __future__ import annotations

import numpy as np

from .mone_oracle import sigmoid, silu, silu_grad
from .paper_optimizer import momentum_decay, renormalise, row_norms, token_rates

L2_EPS = 1e-12
ROPE_BASE = 10000.0


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# ------------------------------------------------------------------ preprocessing

def rope(x, pos, base: float = ROPE_BASE):
    """Rotate every row of x [n, d_h] (d_h even) by its position pos[n]: channel pair
    (c, c + d_h/2) turns by pos * base^(-2c/d_h)."""
    x = _f64(x)
    n, dh = x.shape
    half = dh // 2
    theta = float(base) ** (-2.0 * np.arange(half) / dh)
    ang = _f64(pos)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[:, :half], x[:, half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=1)


def l2_normalise(x):
    """Rows of x divided by max(||row||, 1e-12)."""
    x = _f64(x)
    nrm = np.sqrt(np.sum(x * x, axis=1, keepdims=True))
    return x / np.maximum(nrm, L2_EPS)


def preprocess_keys(r, scale, shift, n_heads: int, pos, base: float = ROPE_BASE):
    """Keys from raw projections r [n, H*d_h]: affine, SiLU, per-head L2 norm, per-head RoPE."""
    r = _f64(r)
    k = silu(r * _f64(scale)[None, :] + _f64(shift)[None, :])
    dh = r.shape[1] // n_heads
    out = np.empty_like(k)
    for e in range(n_heads):
        cols = slice(e * dh, (e + 1) * dh)
        out[:, cols] = rope(l2_normalise(k[:, cols]), pos, base)
    return out


def preprocess_values(r):
    return silu(_f64(r))


def layer_keys_values(x, frozen, n_heads: int, pos=None, base: float = ROPE_BASE):
    """Preprocessed keys and values [n, H*d_h] of hidden states x [n, d_in].

    frozen = dict(p_k [d, d_in], p_v [d, d_in], scale [d], shift [d]); pos defaults to the
    segment-local positions 0..n-1."""
    x = _f64(x)
    if pos is None:
        pos = np.arange(x.shape[0])
    k = preprocess_keys(x @ _f64(frozen["p_k"]).T, frozen["scale"], frozen["shift"], n_heads,
                        pos, base)
    v = preprocess_values(x @ _f64(frozen["p_v"]).T)
    return k, v


# ------------------------------------------------------------------ the memory

def swiglu_forward(k, w_in, w_gate, w_out):
    """One head: returns z, g, a, y for keys k [n, d_h] (Eq. swiglu in row form)."""
    k = _f64(k)
    z = k @ _f64(w_in).T
    g = k @ _f64(w_gate).T
    a = silu(z) * g
    y = a @ _f64(w_out)
    return z, g, a, y


def memory_read(k, fast):
    """The memory's output for keys k [n, H*d_h]; fast = (w_in, w_gate, w_out), each
    [H, d_h, d_h]."""
    w_in, w_gate, w_out = (_f64(w) for w in fast)
    n_heads, dh = w_in.shape[0], w_in.shape[1]
    k = _f64(k)
    y = np.empty_like(k)
    for e in range(n_heads):
        cols = slice(e * dh, (e + 1) * dh)
        y[:, cols] = swiglu_forward(k[:, cols], w_in[e], w_gate[e], w_out[e])[3]
    return y


def nip_loss(k, v, fast):
    """Segment loss (1/n) sum_j -v_j . M(k_j) (Eq. mem_loss, summed over heads)."""
    k, v = _f64(k), _f64(v)
    n = k.shape[0]
    if n == 0:
        return 0.0
    return float(-np.sum(v * memory_read(k, fast)) / n)


def weighted_grad(k, v, fast, eta):
    """Gradient of (1/n) sum_j eta_j l_j with respect to every head's (W_in, W_gate, W_out),
    as three [H, d_h, d_h] arrays, and the unweighted segment loss."""
    k, v, eta = _f64(k), _f64(v), _f64(eta)
    w_in, w_gate, w_out = (_f64(w) for w in fast)
    n_heads, dh = w_in.shape[0], w_in.shape[1]
    n = k.shape[0]
    g_in, g_gate, g_out = (np.zeros_like(w_in) for _ in range(3))
    loss = 0.0
    for e in range(n_heads):
        cols = slice(e * dh, (e + 1) * dh)
        ke, ve = k[:, cols], v[:, cols]
        z, g, a, y = swiglu_forward(ke, w_in[e], w_gate[e], w_out[e])
        loss += float(-np.sum(ve * y))
        dy = -(eta[:, None] * ve) / n          # dL/dy of the rate-weighted loss
        g_out[e] = a.T @ dy
        da = dy @ w_out[e].T
        dz = da * g * silu_grad(z)
        dg = da * silu(z)
        g_in[e] = dz.T @ ke
        g_gate[e] = dg.T @ ke
    return (g_in, g_gate, g_out), (loss / n if n else 0.0)


# ------------------------------------------------------------------ the update

def sgd_step(x, fast, frozen, lr, n_heads: int, base: float = ROPE_BASE):
    """One SGD step of one layer on one segment x [n, d_in]: W_s = W_{s-1} - lr grad L_s.
    Returns (fast_s, L_s).  An empty segment changes nothing."""
    x = _f64(x)
    fast = tuple(_f64(w) for w in fast)
    if x.shape[0] == 0:
        return fast, 0.0
    k, v = layer_keys_values(x, frozen, n_heads, base=base)
    grads, ls = weighted_grad(k, v, fast, np.ones(x.shape[0]))
    return tuple(w - float(lr) * g for w, g in zip(fast, grads)), ls


def _heads_renorm(w, norms0):
    return np.stack([renormalise(w[e], norms0[e]) for e in range(w.shape[0])])


def initial_norms(fast):
    """Row norms of every head's three matrices: the paper optimiser's renormalisation targets."""
    return tuple(np.stack([row_norms(w[e]) for e in range(w.shape[0])]) for w in
                 (_f64(f) for f in fast))


def paper_step(x, fast, mom, frozen, meta, norms0, lr, n_heads: int, base: float = ROPE_BASE):
    """One step with the paper's optimiser: eta_j = lr softplus(u . x_j + b_u) weights token j's
    gradient, mu_s = beta_s mu_{s-1} + g_s with beta_s = sigmoid(v . xbar + b_v), W_s = rows of
    (W_{s-1} - mu_s) rescaled to their norms in W_0.  meta = (u, b_u, v, b_v).
    Returns (fast_s, mom_s, L_s, info)."""
    x = _f64(x)
    fast = tuple(_f64(w) for w in fast)
    mom = tuple(_f64(m) for m in mom)
    if x.shape[0] == 0:
        return fast, mom, 0.0, {}
    u, b_u, vv, b_v = meta
    eta = token_rates(x, u, b_u, lr)
    beta = momentum_decay(x, vv, b_v)
    k, v = layer_keys_values(x, frozen, n_heads, base=base)
    grads, ls = weighted_grad(k, v, fast, eta)
    mom_n = tuple(beta * m + g for m, g in zip(mom, grads))
    fast_n = tuple(_heads_renorm(w - m, nz) for w, m, nz in zip(fast, mom_n, norms0))
    return fast_n, mom_n, ls, {"eta": eta, "beta": beta, "grads": grads}


def swiglu_run(segments, fast, frozen, lr, n_heads: int, optimizer: str = "sgd", meta=None,
               base: float = ROPE_BASE):
    """Sequential test-time learning of one layer over its segments from W_0 = fast.
    Returns (fast_S, mom_S or None, [L_1, ..., L_S])."""
    fast = tuple(_f64(w) for w in fast)
    losses = []
    if optimizer == "sgd":
        for x in segments:
            fast, ls = sgd_step(x, fast, frozen, lr, n_heads, base)
            losses.append(ls)
        return fast, None, losses
    if optimizer != "paper":
        raise ValueError(optimizer)
    norms0 = initial_norms(fast)
    mom = tuple(np.zeros_like(w) for w in fast)
    for x in segments:
        fast, mom, ls, _ = paper_step(x, fast, mom, frozen, meta, norms0, lr, n_heads, base)
        losses.append(ls)
    return fast, mom, losses


# ------------------------------------------------------------------ the read

RMS_EPS = 1e-6


def rms_normalise(o):
    """Rows of o divided by sqrt(mean(row^2) + 1e-6)."""
    o = _f64(o)
    return o / np.sqrt(np.mean(o * o, axis=1, keepdims=True) + RMS_EPS)


def memory_tokens(xq, fast, reader, n_heads: int, base: float = ROPE_BASE):
    """Memory tokens h [Q, H*d_h] of query hidden states xq [Q, d_in] at the fast weights fast.

    reader = dict(p_q [d, d_in], q_scale [d], q_shift [d], rms_w [d], gate_w [H, d_in],
    gate_b [H])."""
    xq = _f64(xq)
    q = preprocess_keys(xq @ _f64(reader["p_q"]).T, reader["q_scale"], reader["q_shift"],
                        n_heads, np.arange(xq.shape[0]), base)
    o = memory_read(q, fast)
    dh = o.shape[1] // n_heads
    gate = silu(xq @ _f64(reader["gate_w"]).T + _f64(reader["gate_b"])[None, :])  # [Q, H]
    h = np.empty_like(o)
    w = _f64(reader["rms_w"])
    for e in range(n_heads):
        cols = slice(e * dh, (e + 1) * dh)
        h[:, cols] = rms_normalise(o[:, cols]) * w[None, cols] * gate[:, e:e + 1]
    return h


def memory_kv(h, w_kv):
    """The memory tokens in the backbone's key/value space: [h W_k^T | h W_v^T], with
    w_kv = [W_k ; W_v] of shape [2 d_kv, d]."""
    return _f64(h) @ _f64(w_kv).T


__all__ = ["rope", "l2_normalise", "preprocess_keys", "preprocess_values", "layer_keys_values",
           "swiglu_forward", "memory_read", "nip_loss", "weighted_grad", "sgd_step",
           "initial_norms", "paper_step", "swiglu_run", "sigmoid", "ROPE_BASE", "rms_normalise",
           "memory_tokens", "memory_kv"]
