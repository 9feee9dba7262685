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
