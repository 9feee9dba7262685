"""Pins of the memory-injection attention oracle against facts that do not come from it.

  * brute force: scalar loops over heads, rows and keys on tiny inputs (catches a wrong scale,
    mask, head grouping or K/V half);
  * a memory whose entries repeat the query-side keys and values leaves ordinary causal
    attention unchanged (every weight is split in two equal halves);
  * the first token sees exactly two entries: a closed-form two-way softmax;
  * memory keys far below the others (scores -> -inf) give ordinary causal attention; memory
    keys far above give the running mean of the memory values.
"""
import math

import numpy as np
import pytest

import oracle as orc


def _brute(q, k, v, kvm, hq, hkv):
    n, dkv = k.shape
    dh = dkv // hkv
    out = np.zeros((n, hq * dh))
    for a in range(hq):
        g = a // (hq // hkv)
        for i in range(n):
            scores, vals = [], []
            for j in range(i + 1):
                scores.append(sum(q[i, a * dh + e] * k[j, g * dh + e] for e in range(dh)) / math.sqrt(dh))
                vals.append([v[j, g * dh + e] for e in range(dh)])
            for j in range(i + 1):
                scores.append(sum(q[i, a * dh + e] * kvm[j, g * dh + e] for e in range(dh)) / math.sqrt(dh))
                vals.append([kvm[j, dkv + g * dh + e] for e in range(dh)])
            m = max(scores)
            w = [math.exp(s - m) for s in scores]
            z = sum(w)
            for e in range(dh):
                out[i, a * dh + e] = sum(w[t] * vals[t][e] for t in range(len(w))) / z
    return out


def _causal(q, k, v, hq, hkv):
    n, dkv = k.shape
    dh = dkv // hkv
    out = np.zeros((n, hq * dh))
    for a in range(hq):
        g = a // (hq // hkv)
        qa, ka, va = q[:, a * dh:(a + 1) * dh], k[:, g * dh:(g + 1) * dh], v[:, g * dh:(g + 1) * dh]
        s = qa @ ka.T / math.sqrt(dh)
        s = np.where(np.tril(np.ones((n, n), bool)), s, -np.inf)
        w = np.exp(s - s.max(axis=1, keepdims=True))
        out[:, a * dh:(a + 1) * dh] = (w / w.sum(axis=1, keepdims=True)) @ va
    return out


@pytest.mark.parametrize("hq,hkv,dh,n", [(1, 1, 3, 4), (4, 2, 2, 3), (6, 3, 4, 5)])
def test_matches_brute_force(hq, hkv, dh, n):
    rng = np.random.default_rng(hq * 10 + n)
    q = rng.standard_normal((n, hq * dh))
    k = rng.standard_normal((n, hkv * dh))
    v = rng.standard_normal((n, hkv * dh))
    kvm = rng.standard_normal((n, 2 * hkv * dh))
    np.testing.assert_allclose(orc.memory_attention(q, k, v, kvm, hq, hkv),
                               _brute(q, k, v, kvm, hq, hkv), rtol=1e-12, atol=1e-13)


def test_memory_repeating_the_keys_leaves_causal_attention():
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((6, w)) for w in (8 * 4, 4 * 4, 4 * 4))
    kvm = np.concatenate([k, v], axis=1)
    np.testing.assert_allclose(orc.memory_attention(q, k, v, kvm, 8, 4), _causal(q, k, v, 8, 4),
                               rtol=1e-12, atol=1e-13)


def test_first_token_is_a_two_way_softmax():
    rng = np.random.default_rng(2)
    dh = 5
    q, k, v = rng.standard_normal((1, dh)), rng.standard_normal((1, dh)), rng.standard_normal((1, dh))
    kvm = rng.standard_normal((1, 2 * dh))
    s1 = float(q[0] @ k[0]) / math.sqrt(dh)
    s2 = float(q[0] @ kvm[0, :dh]) / math.sqrt(dh)
    w1 = 1.0 / (1.0 + math.exp(s2 - s1))
    want = w1 * v[0] + (1.0 - w1) * kvm[0, dh:]
    np.testing.assert_allclose(orc.memory_attention(q, k, v, kvm, 1, 1)[0], want, rtol=1e-13)


def test_extreme_memory_scores():
    rng = np.random.default_rng(3)
    n, dh = 5, 4
    q = np.abs(rng.standard_normal((n, dh))) + 0.5  # positive queries
    k, v = rng.standard_normal((n, dh)), rng.standard_normal((n, dh))
    vm = rng.standard_normal((n, dh))
    low = np.concatenate([-1e4 * np.ones((n, dh)), vm], axis=1)
    np.testing.assert_allclose(orc.memory_attention(q, k, v, low, 1, 1), _causal(q, k, v, 1, 1),
                               rtol=1e-12, atol=1e-13)
    high = np.concatenate([1e4 * np.ones((n, dh)), vm], axis=1)
    running_mean = np.cumsum(vm, axis=0) / np.arange(1, n + 1)[:, None]
    np.testing.assert_allclose(orc.memory_attention(q, k, v, high, 1, 1), running_mean,
                               rtol=1e-12, atol=1e-13)
