"""Shared set-up of the GPU tests: device problems whose checked layers come from the keyed
input generator (so the oracle sees the same numbers) and whose other layers are drawn on the
device (only the GPU path reads them; layers are independent, so they cannot influence the
checked ones)."""
from __future__ import annotations

import numpy as np

from paper_2608_17616_amd import inputs


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))


def local_rel_max(a, b, block=64) -> float:
    """Largest relative L2 error over the rows of a matrix and over its block x block tiles,
    each against its own oracle norm.  A single wrong row, or one wrong column chunk of an
    output tile, moves a whole-tensor norm by only about 1/sqrt(rows), but its own row or tile
    by its full size."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    a2, b2 = a.reshape(-1, a.shape[-1]), b.reshape(-1, b.shape[-1])
    num = np.linalg.norm(a2 - b2, axis=1)
    den = np.linalg.norm(b2, axis=1)
    worst = float(np.max(num / np.where(den > 0, den, 1.0)))
    R, C = a2.shape
    for r0 in range(0, R, block):
        for c0 in range(0, C, block):
            e = rel_l2(a2[r0:r0 + block, c0:c0 + block], b2[r0:r0 + block, c0:c0 + block])
            worst = max(worst, e)
    return worst


# Local (per-row, per-tile) errors may exceed the whole-tensor bar by this factor: a row or a
# 64 x 64 tile averages fewer rounding errors than the whole tensor.
LOCAL_FACTOR = 5.0


class DeviceProblem:
    def __init__(self, cfg, checked, seed_dev=1234, device="cuda"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.checked = list(checked)
        self.device = device
        self.act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed_dev)
        L, d, h, D = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out
        self.w1 = torch.empty(L, h, d, dtype=torch.float32, device=device)
        self.w2 = torch.empty(L, D, h, dtype=torch.float32, device=device)
        self.wkv = torch.empty(L, D, d, dtype=self.act, device=device)
        inputs.device_normal_(self.w1, 1 / np.sqrt(d), self.gen)
        inputs.device_normal_(self.w2, 1 / np.sqrt(h), self.gen)
        inputs.device_normal_(self.wkv, 1 / np.sqrt(d), self.gen)
        self.host = {}
        for l in self.checked:
            w1, w2, wkv = inputs.layer_w1(cfg, l), inputs.layer_w2(cfg, l), inputs.layer_wkv(cfg, l)
            self.host[l] = dict(w1=w1, w2=w2, wkv=wkv, x=[])
            self.w1[l].copy_(torch.from_numpy(w1))
            self.w2[l].copy_(torch.from_numpy(w2))
            self.wkv[l].copy_(torch.from_numpy(wkv))

    def segment(self, s, n_tokens=None, record=True):
        """Device X [L, n, d] of segment s; records the checked layers' host copies.  With
        record=False every layer is drawn on the device and nothing is kept on the host (long
        contexts whose early segments only the GPU runs)."""
        torch = self.torch
        cfg = self.cfg
        n = cfg.seg_len if n_tokens is None else n_tokens
        x = torch.empty(cfg.n_layers, n, cfg.d_model, dtype=self.act, device=self.device)
        inputs.device_normal_(x, 1.0, self.gen)
        if not record:
            return x
        for l in self.checked:
            xs = inputs.segment_x(cfg, l, s, n)
            self.host[l]["x"].append(xs)
            x[l].copy_(torch.from_numpy(xs))
        return x

    def query(self, q=None, index=0):
        torch = self.torch
        cfg = self.cfg
        q = cfg.n_query if q is None else q
        xq = torch.empty(cfg.n_layers, q, cfg.d_model, dtype=self.act, device=self.device)
        inputs.device_normal_(xq, 1.0, self.gen)
        hx = {}
        for l in self.checked:
            hx[l] = inputs.query_x(cfg, l, q, index)
            xq[l].copy_(torch.from_numpy(hx[l]))
        return xq, hx

    def paper_state(self):
        """Optimiser buffers of the paper's optimiser, as the tuple TtlSession takes: rate and
        decay projections and biases (checked layers from the keyed generator, the others on
        the device), and zero momentum.  Records the checked layers' host meta-parameters."""
        torch = self.torch
        cfg = self.cfg
        L, d, h, D = cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_out
        dev = self.device
        u = inputs.device_normal_(torch.empty(L, d, dtype=torch.float32, device=dev),
                                  1 / np.sqrt(d), self.gen)
        v = inputs.device_normal_(torch.empty(L, d, dtype=torch.float32, device=dev),
                                  1 / np.sqrt(d), self.gen)
        bu = torch.full((L,), inputs.B_U, dtype=torch.float32, device=dev)
        bv = torch.full((L,), inputs.B_V, dtype=torch.float32, device=dev)
        for l in self.checked:
            mu, mbu, mv, mbv = inputs.layer_meta(cfg, l)
            self.host[l]["meta"] = (mu.astype(np.float64), float(mbu), mv.astype(np.float64),
                                    float(mbv))
            u[l].copy_(torch.from_numpy(mu))
            v[l].copy_(torch.from_numpy(mv))
            bu[l] = float(mbu)
            bv[l] = float(mbv)
        m1 = torch.zeros(L, h, d, dtype=torch.float32, device=dev)
        m2 = torch.zeros(L, D, h, dtype=torch.float32, device=dev)
        return (u, bu, v, bv, m1, m2)
