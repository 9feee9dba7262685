"""Workload configurations of the MoNe test-time-learning (TTL) hot path.

Every configuration is a frozen-backbone shape with a 2-layer SiLU memory MLP per layer,
``d_model -> d_hidden -> 2*d_kv`` producing ``[K | V]``, trained at test time by plain SGD on
an MSE loss against the frozen layer's key/value projections (MoNe, Sec. 3.3-3.4), one step per
segment of ``seg_len`` tokens (Sec. 3.1).

Where a workload leaves a detail open the smaller workloads' stated defaults are inherited:
MSE with the per-token squared error summed over the 2*d_kv output channels and averaged over the
segment's tokens (Sec. 3.3, segment-level average), learning rate 1e-3, seed 0 and a 64-token query
batch for the read step.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class MoneConfig:
    name: str
    n_layers: int      # L: layers with a memory (one independent fast-weight MLP each)
    d_model: int       # d: width of the segment hidden states x (memory input)
    d_hidden: int      # h: memory MLP hidden width
    d_kv: int          # width of K (and of V); the memory output is D = 2*d_kv = [K | V]
    seg_len: int       # T: tokens per segment
    n_context: int     # N: context tokens; S = N / T segments
    act_dtype: str     # "f32" or "bf16": dtype of x, x_q, W_kv and stored intermediates
    lr: float          # learning rate (scales the per-token rates of the paper optimiser)
    loss: str = "mse_sum"   # "mse_sum": c = 2/T ; "mse_mean": c = 2/(T*D) ; "nip": -t.y
    n_query: int = 64  # Q: query tokens for the read step
    seed: int = 0
    optimizer: str = "sgd"  # "sgd" or "paper" (per-token rates, momentum, renormalisation)
    block_tokens: int = 0   # block form of multi-segment calls: 0 automatic, < 0 none, > 0 size

    @property
    def d_out(self) -> int:
        return 2 * self.d_kv

    @property
    def n_segments(self) -> int:
        return self.n_context // self.seg_len

    def flops_per_token_layer(self, with_targets: bool = True) -> int:
        """Algorithmic FLOPs of one TTL step per context token per layer.

        forward 1 (2dh) + forward 2 (2hD; not with the negative inner product) + target
        projection (2dD) + backward to the hidden layer (2hD) + the two weight gradients
        (2hD + 2dh).
        """
        d, h, D = self.d_model, self.d_hidden, self.d_out
        f = 2 * (2 * d * h + 3 * h * D)
        if self.loss == "nip":  # dL/dY = -T/n: the output layer's forward is not needed
            f -= 2 * h * D
        if with_targets:
            f += 2 * d * D
        return f

    def flops_per_token(self, with_targets: bool = True) -> int:
        return self.n_layers * self.flops_per_token_layer(with_targets)

    def with_(self, **kw) -> "MoneConfig":
        return replace(self, **kw)


TINY = MoneConfig("tiny", n_layers=1, d_model=256, d_hidden=512, d_kv=128, seg_len=128,
                  n_context=1024, act_dtype="f32", lr=1e-2)
ONE_B = MoneConfig("1b", n_layers=16, d_model=2048, d_hidden=2048, d_kv=512, seg_len=512,
                   n_context=32768, act_dtype="bf16", lr=1e-3)
THREE_B = MoneConfig("3b", n_layers=28, d_model=3072, d_hidden=3072, d_kv=1024, seg_len=1024,
                     n_context=131072, act_dtype="bf16", lr=1e-3)
EIGHT_B = MoneConfig("8b", n_layers=32, d_model=4096, d_hidden=4096, d_kv=1024, seg_len=2048,
                     n_context=131072, act_dtype="bf16", lr=1e-3)
STRESS = MoneConfig("stress", n_layers=16, d_model=2048, d_hidden=2048, d_kv=512, seg_len=64,
                    n_context=524288, act_dtype="bf16", lr=1e-3)

CONFIGS = {c.name: c for c in (TINY, ONE_B, THREE_B, EIGHT_B, STRESS)}


@dataclass(frozen=True)
class SwigluConfig:
    """The paper-form memory (Eq. swiglu): per layer, H fast-weight heads of width d_h, each a
    SwiGLU MLP of three d_h x d_h matrices, trained on preprocessed keys and values (affine,
    SiLU, L2 norm and segment-local RoPE on keys; SiLU on values) with the negative inner
    product loss (Eq. mem_loss).  The memory's width H d_h equals d_model."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_head: int
    seg_len: int
    n_context: int
    act_dtype: str
    lr: float
    optimizer: str = "sgd"
    rope_base: float = 10000.0
    n_query: int = 64
    seed: int = 0
    prep_segments: int = 0  # preprocessing batch of multi-segment calls (0: library default)

    @property
    def n_segments(self) -> int:
        return self.n_context // self.seg_len

    def flops_per_token_layer(self) -> int:
        """Algorithmic FLOPs of one step per context token per layer: the key and value
        projections (2 d 2d), and per head the hidden activations' gradient (2 d_h^2), the
        two branches' forward (4 d_h^2) and the three weight gradients (6 d_h^2).  The memory's
        output is not formed: the loss gradient at the output does not depend on it."""
        d, dh = self.d_model, self.d_head
        return 4 * d * d + self.n_heads * 12 * dh * dh

    def flops_per_token(self) -> int:
        return self.n_layers * self.flops_per_token_layer()

    def with_(self, **kw) -> "SwigluConfig":
        return replace(self, **kw)


# The paper's own memory on Qwen2.5-0.5B (App. A.2: 24 layers, d_model 896, H = 4 heads of
# d_h = 224, 512-token segments, contexts up to 128K tokens).  The learning rate is synthetic
# (the paper's rates are learned): with unit-norm keys, lr = 1 moves the weights by about 1e-3
# of their norm per segment.
SW_TINY = SwigluConfig("sw_tiny", n_layers=2, d_model=128, n_heads=2, d_head=64, seg_len=128,
                       n_context=512, act_dtype="f32", lr=1.0)
SW_PAPER = SwigluConfig("sw_qwen0.5b", n_layers=24, d_model=896, n_heads=4, d_head=224,
                        seg_len=512, n_context=131072, act_dtype="bf16", lr=1.0)

SW_CONFIGS = {c.name: c for c in (SW_TINY, SW_PAPER)}
