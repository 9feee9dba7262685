"""The seeded input generator: keyed streams, distributions, bf16 rounding."""
import numpy as np
import pytest

from paper_2608_17616_amd import configs, inputs


def test_keyed_streams_are_reproducible_and_independent():
    a = inputs.normal(0, inputs.KIND_X, 3, 7, (16, 8), 1.0)
    b = inputs.normal(0, inputs.KIND_X, 3, 7, (16, 8), 1.0)
    c = inputs.normal(0, inputs.KIND_X, 3, 8, (16, 8), 1.0)
    d = inputs.normal(0, inputs.KIND_X, 4, 7, (16, 8), 1.0)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, d)


def test_bf16_rounding_matches_torch_cast():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 3,
                        # exact ties between two bf16 values, both parities
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8],
                                 dtype=np.float32)])
    ours = inputs.bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    np.testing.assert_array_equal(inputs.bf16_widen(ours),
                                  torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_distributions_and_shapes():
    cfg = configs.ONE_B.with_(n_layers=2)
    w1, w2, wkv = inputs.layer_w1(cfg, 1), inputs.layer_w2(cfg, 1), inputs.layer_wkv(cfg, 1)
    assert w1.shape == (2048, 2048) and w2.shape == (1024, 2048) and wkv.shape == (1024, 2048)
    assert abs(w1.std() * np.sqrt(2048) - 1) < 0.01
    assert abs(w2.std() * np.sqrt(2048) - 1) < 0.01
    assert abs(wkv.std() * np.sqrt(2048) - 1) < 0.01
    x = inputs.segment_x(cfg, 0, 5)
    assert x.shape == (512, 2048) and abs(x.std() - 1) < 0.01
    # bf16 mode: the values are bf16-representable
    assert np.array_equal(inputs.bf16_widen(inputs.bf16_bits(x)), x)
    assert np.array_equal(inputs.bf16_widen(inputs.bf16_bits(wkv)), wkv)
    # a shorter segment is a prefix-free draw of its own length
    assert inputs.segment_x(cfg, 0, 5, 100).shape == (100, 2048)


def test_config_table():
    c = configs.EIGHT_B
    assert (c.n_layers, c.d_model, c.d_hidden, c.d_out, c.seg_len, c.n_segments) == \
        (32, 4096, 4096, 2048, 2048, 64)
    assert c.flops_per_token() == 2 ** 32
    assert configs.STRESS.n_segments == 8192 and configs.TINY.n_segments == 8
    assert configs.ONE_B.flops_per_token() == 16 * 33554432


# ---------------------------------------------------------------- the paper-form memory

def test_swiglu_generators_are_keyed_and_independent():
    cfg = configs.SW_TINY
    p0, p1 = inputs.sw_layer_proj(cfg, 0), inputs.sw_layer_proj(cfg, 1)
    assert p0.shape == (2 * cfg.d_model, cfg.d_model) and not np.array_equal(p0, p1)
    assert np.array_equal(p0, inputs.sw_layer_proj(cfg, 0))
    f = inputs.sw_layer_fast(cfg, 1)
    assert all(w.shape == (cfg.n_heads, cfg.d_head, cfg.d_head) for w in f)
    assert not np.array_equal(f[0], f[1]) and not np.array_equal(f[1], f[2])
    s, b = inputs.sw_layer_affine(cfg, 0)
    assert s.dtype == np.float32 and abs(float(s.mean()) - 1.0) < 0.05 and abs(float(b.mean())) < 0.05
    r = inputs.sw_layer_reader(cfg, 0, 64)
    assert r["w_kv"].shape == (128, cfg.d_model) and r["gate_w"].shape == (cfg.n_heads, cfg.d_model)
    bf = configs.SW_TINY.with_(act_dtype="bf16")
    q = inputs.sw_layer_proj(bf, 0)
    assert np.array_equal(q, inputs.act_round(q, "bf16"))  # bf16-representable in bf16 mode


def test_swiglu_flops_formula():
    cfg = configs.SW_PAPER
    d, H, dh = cfg.d_model, cfg.n_heads, cfg.d_head
    # projections (2 * d * 2d) + per head: dA (2 dh^2), the two branches (4 dh^2), the three
    # weight gradients (6 dh^2)
    assert cfg.flops_per_token_layer() == 2 * d * 2 * d + H * (2 + 4 + 6) * dh * dh
    assert cfg.flops_per_token() == cfg.n_layers * cfg.flops_per_token_layer()
    assert cfg.n_segments == 256 and H * dh == d
