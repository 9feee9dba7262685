"""CPU oracle of memory injection into attention -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

Only the test-suite, the package's smoke check and the benchmark's CPU-baseline leg may import
this module; the product path never calls it.

At generation time the memory is read on the query tokens (Eq. read) and its output joins the
attention of those tokens as extra key/value entries (Eq. attn), with the standard scaled
softmax attention of Eq. std_attn:
    out = softmax(Q [K || K_mem]^T / sqrt(d_h)) [V || V_mem]      per attention head.
Readings (the paper leaves these open):
  * In the configuration form the memory's output already lives in key/value space: it is
    trained against [W_k x ; W_v x] (Eq. proj), so the memory token of query token j is the
    [K | V] row M(x_j) = [k_mem_j | v_mem_j] (what mone_memory_kv returns).  The per-head RMSNorm
    and gate that the paper applies belong to its x-space memory and are not part of this form.
  * Heads: K, V and the memory K/V have H_kv heads of width d_h = d_kv / H_kv; Q has H_q heads,
    a multiple of H_kv, and query head a reads key/value head a // (H_q / H_kv) (grouped-query
    attention, as the backbone uses).
  * Masking: query token i sees the keys of query tokens 0..i and the memory entries 0..i (the
    memory entry of token j exists once token j has been read), all in one softmax.

Float64 NumPy; plain loops over heads and rows, matmul for the dot products.
Pins: tests/test_oracle_memory_attention.py.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def memory_attention(q, k, v, kv_mem, n_heads: int, n_kv_heads: int):
    """q [Q, n_heads*dh], k and v [Q, n_kv_heads*dh], kv_mem [Q, 2*d_kv] with d_kv =
    n_kv_heads*dh (K columns first).  Returns out [Q, n_heads*dh]."""
    q, k, v, kv_mem = _f64(q), _f64(k), _f64(v), _f64(kv_mem)
    n_q = q.shape[0]
    d_kv = k.shape[1]
    dh = d_kv // n_kv_heads
    group = n_heads // n_kv_heads
    km, vm = kv_mem[:, :d_kv], kv_mem[:, d_kv:]
    out = np.zeros((n_q, n_heads * dh))
    for a in range(n_heads):
        g = a // group
        qa = q[:, a * dh:(a + 1) * dh]
        cols = slice(g * dh, (g + 1) * dh)
        for i in range(n_q):
            keys = np.concatenate([k[:i + 1, cols], km[:i + 1, cols]], axis=0)
            vals = np.concatenate([v[:i + 1, cols], vm[:i + 1, cols]], axis=0)
            s = keys @ qa[i] / np.sqrt(dh)
            w = np.exp(s - s.max())
            out[i, a * dh:(a + 1) * dh] = (w / w.sum()) @ vals
    return out
