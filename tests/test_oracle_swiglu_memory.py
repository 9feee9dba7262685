"""Pins of the paper-form (SwiGLU per head) memory oracle against facts that do not come from it.

  * RoPE: the same rotation written with complex numbers; position 0 is the identity; norms are
    kept; scores depend only on the position difference; d_h = 2 is a plain 2x2 rotation;
  * preprocessing: scalar brute force (affine, logistic, square root, complex rotation); keys of
    unit norm per head; a zero key stays zero; normalising before or after the rotation agrees;
  * forward and loss: scalar brute force;
  * the rate-weighted gradient: central finite differences of a brute-force loss, torch.autograd
    in float64 through the whole path from the hidden states, the W_out-independence of W_out's
    own gradient under this loss, unit rates and a dropped token;
  * the loss equals sum(A * dA) with dA the gradient of the loss with respect to A (the form
    the fused kernels compute it in);
  * the update: a small step lowers the loss; constant rates without momentum are the SGD step
    with rows rescaled to their initial norms; momentum carries with weight beta; row norms
    stay fixed over a run; an empty segment changes nothing.
"""
import cmath
import math

import numpy as np
import pytest

import oracle.swiglu_memory as sw
from oracle import silu, silu_grad

SOFTPLUS_INV_1 = math.log(math.e - 1.0)


def _frozen(rng, d_in, d):
    return dict(p_k=rng.standard_normal((d, d_in)) / math.sqrt(d_in),
                p_v=rng.standard_normal((d, d_in)) / math.sqrt(d_in),
                scale=1.0 + 0.3 * rng.standard_normal(d), shift=0.2 * rng.standard_normal(d))


def _fast(rng, H, dh):
    return tuple(rng.standard_normal((H, dh, dh)) / math.sqrt(dh) for _ in range(3))


# ---------------------------------------------------------------- RoPE

def _rope_complex(x, p, base):
    dh = len(x)
    half = dh // 2
    out = np.zeros(dh)
    for c in range(half):
        w = complex(x[c], x[c + half]) * cmath.exp(1j * p * base ** (-2.0 * c / dh))
        out[c], out[c + half] = w.real, w.imag
    return out


def test_rope_matches_complex_rotation():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 8))
    pos = np.array([0, 1, 7, 100, 511])
    got = sw.rope(x, pos, 10000.0)
    for i in range(5):
        np.testing.assert_allclose(got[i], _rope_complex(x[i], pos[i], 10000.0), rtol=1e-13,
                                   atol=1e-13)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((1, 16)), rng.standard_normal((1, 16))
    np.testing.assert_array_equal(sw.rope(q, [0]), q)
    for p in (3, 250, 511):
        assert np.linalg.norm(sw.rope(q, [p])) == pytest.approx(np.linalg.norm(q), rel=1e-14)
    s = (sw.rope(q, [40]) @ sw.rope(k, [13]).T).item()
    for shift in (1, 17, 400):
        assert (sw.rope(q, [40 + shift]) @ sw.rope(k, [13 + shift]).T).item() == pytest.approx(
            s, rel=1e-10)


def test_rope_two_channels_is_a_plane_rotation():
    x = np.array([[0.6, -1.3]])
    for p in (0.0, 1.0, 2.5, 9.0):
        c, s = math.cos(p), math.sin(p)
        np.testing.assert_allclose(sw.rope(x, [p], 777.0)[0],
                                   [0.6 * c + 1.3 * s, 0.6 * s - 1.3 * c], rtol=1e-14)


# ---------------------------------------------------------------- preprocessing

def _keys_brute(r, scale, shift, H, pos, base):
    n, d = r.shape
    dh = d // H
    out = np.zeros((n, d))
    for j in range(n):
        for e in range(H):
            u = []
            for c in range(dh):
                t = scale[e * dh + c] * r[j, e * dh + c] + shift[e * dh + c]
                u.append(t / (1.0 + math.exp(-t)))
            nrm = math.sqrt(sum(t * t for t in u))
            u = [t / max(nrm, 1e-12) for t in u]
            out[j, e * dh:(e + 1) * dh] = _rope_complex(np.array(u), pos[j], base)
    return out


def test_keys_brute_force_and_unit_norm():
    rng = np.random.default_rng(2)
    H, dh, n = 3, 6, 4
    r = rng.standard_normal((n, H * dh))
    scale, shift = 1 + 0.5 * rng.standard_normal(H * dh), 0.3 * rng.standard_normal(H * dh)
    pos = np.array([0, 5, 9, 31])
    got = sw.preprocess_keys(r, scale, shift, H, pos, 500.0)
    np.testing.assert_allclose(got, _keys_brute(r, scale, shift, H, pos, 500.0), rtol=1e-12,
                               atol=1e-14)
    norms = np.linalg.norm(got.reshape(n, H, dh), axis=2)
    np.testing.assert_allclose(norms, 1.0, rtol=1e-13)


def test_zero_key_stays_zero_and_norm_commutes_with_rope():
    rng = np.random.default_rng(3)
    H, dh = 2, 8
    r = rng.standard_normal((3, H * dh))
    scale = np.ones(H * dh)
    scale[:dh] = 0.0  # head 0: SiLU(0) = 0 everywhere
    got = sw.preprocess_keys(r, scale, np.zeros(H * dh), H, [0, 1, 2])
    assert np.array_equal(got[:, :dh], np.zeros((3, dh)))
    k = silu(r[:, dh:])
    a = sw.rope(sw.l2_normalise(k), [4, 5, 6])
    b = sw.l2_normalise(sw.rope(k, [4, 5, 6]))
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(got[:, dh:], sw.rope(sw.l2_normalise(k), [0, 1, 2]), rtol=1e-13)


# ---------------------------------------------------------------- forward and loss

def _loss_brute(k, v, fast, eta):
    """(1/n) sum_j eta_j sum_e -v_je . W_out^T(SiLU(W_in k) * W_gate k), scalar loops."""
    w_in, w_gate, w_out = fast
    H, dh = w_in.shape[0], w_in.shape[1]
    n = k.shape[0]
    total = 0.0
    for j in range(n):
        for e in range(H):
            ke = k[j, e * dh:(e + 1) * dh]
            a = []
            for i in range(dh):
                z = sum(w_in[e, i, c] * ke[c] for c in range(dh))
                g = sum(w_gate[e, i, c] * ke[c] for c in range(dh))
                a.append(z / (1.0 + math.exp(-z)) * g)
            for o in range(dh):
                y = sum(w_out[e, i, o] * a[i] for i in range(dh))
                total -= eta[j] * v[j, e * dh + o] * y
    return total / n


def test_forward_and_loss_brute_force():
    rng = np.random.default_rng(4)
    H, dh, n = 2, 5, 3
    fast = _fast(rng, H, dh)
    k, v = rng.standard_normal((n, H * dh)), rng.standard_normal((n, H * dh))
    assert sw.nip_loss(k, v, fast) == pytest.approx(_loss_brute(k, v, fast, np.ones(n)),
                                                    rel=1e-12)
    _, ls = sw.weighted_grad(k, v, fast, rng.uniform(0.5, 2, n))
    assert ls == pytest.approx(sw.nip_loss(k, v, fast), rel=1e-13)  # reported loss is unweighted


# ---------------------------------------------------------------- the gradient

@pytest.mark.parametrize("H,dh,n", [(1, 3, 2), (2, 4, 3)])
def test_weighted_grad_matches_finite_differences(H, dh, n):
    rng = np.random.default_rng(10 * H + dh)
    fast = _fast(rng, H, dh)
    k, v = rng.standard_normal((n, H * dh)), rng.standard_normal((n, H * dh))
    eta = rng.uniform(0.2, 2.0, n)
    grads, _ = sw.weighted_grad(k, v, fast, eta)
    eps = 1e-6
    for m in range(3):
        fd = np.zeros_like(fast[m])
        for idx in np.ndindex(fast[m].shape):
            wp, wm = [list(fast) for _ in range(2)]
            wp[m], wm[m] = fast[m].copy(), fast[m].copy()
            wp[m][idx] += eps
            wm[m][idx] -= eps
            fd[idx] = (_loss_brute(k, v, wp, eta) - _loss_brute(k, v, wm, eta)) / (2 * eps)
        assert np.linalg.norm(grads[m] - fd) <= 1e-8 * max(1.0, np.linalg.norm(fd))


def test_grad_through_the_whole_path_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    H, dh, d_in, n = 2, 6, 10, 5
    frozen = _frozen(rng, d_in, H * dh)
    fast = _fast(rng, H, dh)
    x = rng.standard_normal((n, d_in))
    eta = rng.uniform(0.3, 1.7, n)
    k, v = sw.layer_keys_values(x, frozen, H, base=300.0)
    grads, _ = sw.weighted_grad(k, v, fast, eta)

    tx = torch.tensor(x)
    rk = tx @ torch.tensor(frozen["p_k"]).T
    rv = tx @ torch.tensor(frozen["p_v"]).T
    kk = torch.nn.functional.silu(rk * torch.tensor(frozen["scale"]) + torch.tensor(frozen["shift"]))
    kk = kk.reshape(n, H, dh)
    kk = kk / kk.norm(dim=2, keepdim=True).clamp_min(1e-12)
    half = dh // 2
    ang = torch.arange(n, dtype=torch.float64)[:, None] * (
        300.0 ** (-2.0 * torch.arange(half, dtype=torch.float64) / dh))[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    kk = torch.cat([kk[..., :half] * c - kk[..., half:] * s, kk[..., :half] * s + kk[..., half:] * c],
                   dim=2)
    vv = torch.nn.functional.silu(rv).reshape(n, H, dh)
    tw = [torch.tensor(w, requires_grad=True) for w in fast]
    z = torch.einsum("nec,eic->nei", kk, tw[0])
    g = torch.einsum("nec,eic->nei", kk, tw[1])
    y = torch.einsum("nei,eio->neo", torch.nn.functional.silu(z) * g, tw[2])
    loss = (torch.tensor(eta) * -(vv * y).sum(dim=(1, 2))).mean()
    loss.backward()
    for m in range(3):
        np.testing.assert_allclose(grads[m], tw[m].grad.numpy(), rtol=1e-11, atol=1e-14)


def test_out_gradient_does_not_depend_on_w_out_and_rates_weight_tokens():
    rng = np.random.default_rng(6)
    H, dh, n = 2, 4, 5
    fast = _fast(rng, H, dh)
    k, v = rng.standard_normal((n, H * dh)), rng.standard_normal((n, H * dh))
    g1, _ = sw.weighted_grad(k, v, fast, np.ones(n))
    other = (fast[0], fast[1], rng.standard_normal((H, dh, dh)))
    g2, _ = sw.weighted_grad(k, v, other, np.ones(n))
    np.testing.assert_allclose(g1[2], g2[2], rtol=1e-14)
    eta = np.ones(n)
    eta[1] = 0.0
    g3, _ = sw.weighted_grad(k, v, fast, eta)
    g4, _ = sw.weighted_grad(np.delete(k, 1, 0), np.delete(v, 1, 0), fast, np.ones(n - 1))
    for m in range(3):
        np.testing.assert_allclose(g3[m], g4[m] * (n - 1) / n, rtol=1e-12, atol=1e-16)


def test_loss_is_the_hidden_activations_against_their_gradient():
    rng = np.random.default_rng(7)
    H, dh, n = 3, 5, 4
    fast = _fast(rng, H, dh)
    k, v = rng.standard_normal((n, H * dh)), rng.standard_normal((n, H * dh))
    total = 0.0
    for e in range(H):
        cols = slice(e * dh, (e + 1) * dh)
        _, _, a, _ = sw.swiglu_forward(k[:, cols], fast[0][e], fast[1][e], fast[2][e])
        da = (-v[:, cols] / n) @ fast[2][e].T
        total += float(np.sum(a * da))
    assert total == pytest.approx(sw.nip_loss(k, v, fast), rel=1e-12)


# ---------------------------------------------------------------- the update

def test_sgd_step_lowers_the_loss_and_empty_segment_is_a_no_op():
    rng = np.random.default_rng(8)
    H, dh, d_in, n = 2, 8, 12, 6
    frozen, fast = _frozen(rng, d_in, H * dh), _fast(rng, H, dh)
    x = rng.standard_normal((n, d_in))
    k, v = sw.layer_keys_values(x, frozen, H)
    new, ls = sw.sgd_step(x, fast, frozen, 1e-2, H)
    assert ls == pytest.approx(sw.nip_loss(k, v, fast), rel=1e-13)
    assert sw.nip_loss(k, v, new) < ls
    same, l0 = sw.sgd_step(np.zeros((0, d_in)), fast, frozen, 1e-2, H)
    assert l0 == 0.0 and all(np.array_equal(a, b) for a, b in zip(same, fast))


def _rows_to(w, norms):
    return np.stack([w[e] * (norms[e] / np.linalg.norm(w[e], axis=1))[:, None]
                     for e in range(w.shape[0])])


def test_paper_step_without_momentum_is_sgd_then_row_renormalisation():
    rng = np.random.default_rng(9)
    H, dh, d_in, n = 2, 6, 9, 5
    frozen, fast = _frozen(rng, d_in, H * dh), _fast(rng, H, dh)
    x = rng.standard_normal((n, d_in))
    lr = 0.05
    meta = (np.zeros(d_in), SOFTPLUS_INV_1, np.zeros(d_in), -80.0)  # eta_j = lr, beta ~ 1e-35
    n0 = sw.initial_norms(fast)
    zero = tuple(np.zeros_like(w) for w in fast)
    new, mom, ls, info = sw.paper_step(x, fast, zero, frozen, meta, n0, lr, H)
    sgd, ls_sgd = sw.sgd_step(x, fast, frozen, lr, H)
    assert ls == pytest.approx(ls_sgd, rel=1e-14)
    for m in range(3):
        np.testing.assert_allclose(new[m], _rows_to(sgd[m], n0[m]), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(mom[m], fast[m] - sgd[m], rtol=1e-12, atol=1e-15)


def test_paper_momentum_carries_with_beta_and_norms_stay_fixed():
    rng = np.random.default_rng(10)
    H, dh, d_in, n = 2, 4, 7, 4
    frozen, fast = _frozen(rng, d_in, H * dh), _fast(rng, H, dh)
    x = rng.standard_normal((n, d_in))
    lr = 0.1
    n0 = sw.initial_norms(fast)
    zero = tuple(np.zeros_like(w) for w in fast)
    first = (np.zeros(d_in), SOFTPLUS_INV_1, np.zeros(d_in), -80.0)
    a, m1, _, _ = sw.paper_step(x, fast, zero, frozen, first, n0, lr, H)
    second = (np.zeros(d_in), -85.0, np.zeros(d_in), 0.4)  # no new gradient, decay sigmoid(0.4)
    b, m2, _, info = sw.paper_step(x, a, m1, frozen, second, n0, lr, H)
    beta = 1.0 / (1.0 + math.exp(-0.4))
    assert info["beta"] == pytest.approx(beta, rel=1e-14)
    for m in range(3):
        np.testing.assert_allclose(m2[m], beta * m1[m], rtol=1e-12, atol=1e-18)
        np.testing.assert_allclose(b[m], _rows_to(a[m] - beta * m1[m], n0[m]), rtol=1e-12,
                                   atol=1e-15)
    meta = (rng.standard_normal(d_in) / 3, 0.2, rng.standard_normal(d_in) / 3, -0.1)
    segs = [rng.standard_normal((n, d_in)) for _ in range(5)]
    end, mom, losses = sw.swiglu_run(segs, fast, frozen, 0.3, H, "paper", meta)
    for m in range(3):
        np.testing.assert_allclose(np.linalg.norm(end[m], axis=2), np.linalg.norm(fast[m], axis=2),
                                   rtol=1e-13)
    assert np.linalg.norm(end[0] - fast[0]) > 1e-3 and len(losses) == 5


# ---------------------------------------------------------------- the read

def _reader(rng, d_in, H, dh, d_kv):
    d = H * dh
    return dict(p_q=rng.standard_normal((d, d_in)) / math.sqrt(d_in),
                q_scale=1.0 + 0.3 * rng.standard_normal(d), q_shift=0.2 * rng.standard_normal(d),
                rms_w=1.0 + 0.2 * rng.standard_normal(d),
                gate_w=rng.standard_normal((H, d_in)) / math.sqrt(d_in),
                gate_b=0.3 * rng.standard_normal(H),
                w_kv=rng.standard_normal((2 * d_kv, d)) / math.sqrt(d))


def test_memory_tokens_brute_force():
    rng = np.random.default_rng(20)
    H, dh, d_in, Q = 2, 4, 6, 3
    fast, rd = _fast(rng, H, dh), _reader(rng, d_in, H, dh, 4)
    xq = rng.standard_normal((Q, d_in))
    got = sw.memory_tokens(xq, fast, rd, H, base=50.0)
    q = _keys_brute(xq @ rd["p_q"].T, rd["q_scale"], rd["q_shift"], H, list(range(Q)), 50.0)
    for j in range(Q):
        for e in range(H):
            ke = q[j, e * dh:(e + 1) * dh]
            a = []
            for i in range(dh):
                z = sum(fast[0][e, i, c] * ke[c] for c in range(dh))
                g = sum(fast[1][e, i, c] * ke[c] for c in range(dh))
                a.append(z / (1.0 + math.exp(-z)) * g)
            o = [sum(fast[2][e, i, c] * a[i] for i in range(dh)) for c in range(dh)]
            rms = math.sqrt(sum(t * t for t in o) / dh + 1e-6)
            gl = sum(rd["gate_w"][e, k] * xq[j, k] for k in range(d_in)) + rd["gate_b"][e]
            gate = gl / (1.0 + math.exp(-gl))
            for c in range(dh):
                want = o[c] / rms * rd["rms_w"][e * dh + c] * gate
                assert got[j, e * dh + c] == pytest.approx(want, rel=1e-11, abs=1e-14)


def test_memory_tokens_are_scale_free_in_w_out_and_have_unit_rms():
    """RMSNorm per head: scaling one head's W_out leaves its tokens unchanged (up to the 1e-6
    in the norm, negligible once mean(o^2) is large: W_out is scaled up first), and with unit
    norm weights and a gate of SiLU(z) the RMS of a head's token is SiLU(z)."""
    rng = np.random.default_rng(21)
    H, dh, d_in, Q = 3, 8, 5, 4
    fast, rd = _fast(rng, H, dh), _reader(rng, d_in, H, dh, 4)
    fast = (fast[0], fast[1], 1e4 * fast[2])
    xq = rng.standard_normal((Q, d_in))
    h = sw.memory_tokens(xq, fast, rd, H)
    w_out = fast[2].copy()
    w_out[1] *= 7.0
    h2 = sw.memory_tokens(xq, (fast[0], fast[1], w_out), rd, H)
    np.testing.assert_allclose(h2, h, rtol=1e-8)
    rd1 = dict(rd, rms_w=np.ones(H * dh), gate_w=np.zeros((H, d_in)),
               gate_b=np.array([0.5, 1.0, 2.0]))
    h1 = sw.memory_tokens(xq, fast, rd1, H).reshape(Q, H, dh)
    rms = np.sqrt(np.mean(h1 * h1, axis=2))
    want = np.array([0.5, 1.0, 2.0]) / (1.0 + np.exp(-np.array([0.5, 1.0, 2.0])))
    for j in range(Q):
        np.testing.assert_allclose(rms[j], want, rtol=1e-8)


def test_memory_kv_is_the_backbone_projection():
    rng = np.random.default_rng(22)
    h = rng.standard_normal((3, 8))
    w_kv = rng.standard_normal((6, 8))
    got = sw.memory_kv(h, w_kv)
    for j in range(3):
        for o in range(6):
            assert got[j, o] == pytest.approx(sum(h[j, c] * w_kv[o, c] for c in range(8)),
                                               rel=1e-13)
