"""The C ABI on the CPU: the library loads, exports what the header declares, and rejects bad
arguments on the host before any HIP call (no GPU is touched here)."""
import ctypes
import os
import re

import pytest

import bench

from paper_2608_17616_amd import configs, mone

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]

pytestmark = pytest.mark.skipif(not os.path.exists(mone.LIB_PATH),
                                reason="libmone_ttl.so not built")


def header_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(mone_\w+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_binding_exports():
    assert header_functions() == sorted(mone.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = mone.lib()
    for name in header_functions():
        assert hasattr(L, name), name


def _cfg(**kw):
    base = dict(n_layers=2, d_model=128, d_hidden=192, d_kv=64, seg_len=100, act_dtype="bf16",
                loss="mse_sum", lr=1e-3)
    base.update(kw)
    return mone.make_config(**base)


def test_workspace_bytes_formula_and_independent_of_context_length():
    c = _cfg()
    n = mone.mone_ttl_workspace_bytes(c)
    L, d, h, D, Tp, E = 2, 128, 192, 128, 256, 2
    act = E * L * (h * d + D * h + 2 * h * D + 3 * Tp * h + 2 * Tp * D + h * Tp + d * Tp)
    split = 4 * 256 * 64 * 256  # split-contraction partial sums: one 64 x 256 tile per CU
    assert act + split <= n <= act + split + 64 * 1024
    # the configs' context lengths never enter: N is not a parameter of any call
    for cfg in configs.CONFIGS.values():
        a = mone.mone_ttl_workspace_bytes(mone.config_from(cfg))
        b = mone.mone_ttl_workspace_bytes(mone.config_from(cfg.with_(n_context=cfg.n_context * 8)))
        assert a == b


@pytest.mark.parametrize("kw,code", [
    (dict(n_layers=0), mone.MONE_EINVAL),
    (dict(seg_len=0), mone.MONE_EINVAL),
    (dict(act_dtype=7), mone.MONE_EINVAL),
    (dict(loss=3), mone.MONE_EINVAL),
    (dict(lr=float("nan")), mone.MONE_EINVAL),
    (dict(d_model=100), mone.MONE_EUNSUPPORTED),
    (dict(d_kv=32), mone.MONE_EUNSUPPORTED),
    (dict(seg_len=70000), mone.MONE_EUNSUPPORTED),
])
def test_invalid_configs_are_rejected(kw, code):
    c = _cfg(**kw)
    assert mone.lib().mone_ttl_workspace_bytes(ctypes.byref(c)) == 0
    assert mone.mone_ttl_last_error()
    h = ctypes.c_void_p(1234)
    rc = mone.lib().mone_ttl_init(ctypes.byref(h), ctypes.byref(c), 16, 16, 16, 256, 1 << 30,
                                  None)
    assert rc == code and h.value is None


def test_init_argument_checks_before_any_hip_call():
    c = _cfg()
    need = mone.mone_ttl_workspace_bytes(c)
    L = mone.lib()
    h = ctypes.c_void_p()
    assert L.mone_ttl_init(None, ctypes.byref(c), 16, 16, 16, 256, need, None) == mone.MONE_EINVAL
    assert L.mone_ttl_init(ctypes.byref(h), None, 16, 16, 16, 256, need, None) == mone.MONE_EINVAL
    assert L.mone_ttl_init(ctypes.byref(h), ctypes.byref(c), None, 16, 16, 256, need,
                           None) == mone.MONE_EINVAL
    assert L.mone_ttl_init(ctypes.byref(h), ctypes.byref(c), 16, 16, 24, 256, need,
                           None) == mone.MONE_EINVAL          # misaligned w2
    assert L.mone_ttl_init(ctypes.byref(h), ctypes.byref(c), 16, 16, 16, 272, need,
                           None) == mone.MONE_EINVAL          # workspace not 256-aligned
    assert L.mone_ttl_init(ctypes.byref(h), ctypes.byref(c), 16, 16, 16, 256, need - 1,
                           None) == mone.MONE_EINVAL          # workspace too small
    assert "workspace" in mone.mone_ttl_last_error()


def test_null_handle_calls_fail_cleanly():
    L = mone.lib()
    assert L.mone_ttl_segment(None, 16, 1, None) == mone.MONE_EINVAL
    assert L.mone_memory_kv(None, 16, 1, 16, 0, None) == mone.MONE_EINVAL
    out = (ctypes.c_float * 1)()
    assert L.mone_ttl_loss(None, out, None) == mone.MONE_EINVAL
    assert L.mone_ttl_destroy(None) == mone.MONE_OK
    assert L.mone_ttl_set_stage_timing(None, 4, mone.MONE_ALL_STAGES) == mone.MONE_EINVAL


def test_library_is_built_from_the_current_sources():
    # A stale libmone_ttl.so would make every other test exercise old kernels.
    from paper_2608_17616_amd import build
    lib_t = os.path.getmtime(mone.LIB_PATH)
    stale = [p for p in build.DEPENDS if os.path.getmtime(p) > lib_t]
    assert not stale, f"rebuild libmone_ttl.so (python -m paper_2608_17616_amd.build): {stale}"


def test_paper_optimizer_workspace_adds_only_its_small_buffers():
    c = _cfg()
    p = _cfg(optimizer="paper")
    n, n_p = mone.mone_ttl_workspace_bytes(c), mone.mone_ttl_workspace_bytes(p)
    L, d, h, D, Tp = 2, 128, 192, 128, 256
    extra = 4 * L * (Tp + Tp // 16 + 1 + h + D + h * (d // 64) + D * (h // 64) + h + D)
    assert extra <= n_p - n <= extra + 9 * 256


def test_optimizer_mismatch_and_paper_init_argument_checks():
    L = mone.lib()
    h = ctypes.c_void_p()
    p = _cfg(optimizer="paper")
    need = mone.mone_ttl_workspace_bytes(p)
    # mone_ttl_init refuses the paper optimiser, mone_ttl_init_paper anything else
    assert L.mone_ttl_init(ctypes.byref(h), ctypes.byref(p), 16, 16, 16, 256, need,
                           None) == mone.MONE_EINVAL
    assert "mone_ttl_init_paper" in mone.mone_ttl_last_error()
    opt = mone.mone_paper_optimizer(16, 16, 16, 16, 16, 16)
    s = _cfg()
    assert L.mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(s), 16, 16, 16, ctypes.byref(opt),
                                 256, need, None) == mone.MONE_EINVAL
    assert L.mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(p), 16, 16, 16, None, 256, need,
                                 None) == mone.MONE_EINVAL
    bad = mone.mone_paper_optimizer(16, 16, 16, 16, None, 16)
    assert L.mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(p), 16, 16, 16, ctypes.byref(bad),
                                 256, need, None) == mone.MONE_EINVAL
    mis = mone.mone_paper_optimizer(16, 16, 24, 16, 16, 16)
    assert L.mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(p), 16, 16, 16, ctypes.byref(mis),
                                 256, need, None) == mone.MONE_EINVAL
    assert "aligned" in mone.mone_ttl_last_error()
    assert L.mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(p), 16, 16, 16, ctypes.byref(opt),
                                 256, need - 1, None) == mone.MONE_EINVAL
    assert "workspace" in mone.mone_ttl_last_error()
    assert h.value is None
    bad_opt = _cfg(optimizer=5)
    assert mone.lib().mone_ttl_workspace_bytes(ctypes.byref(bad_opt)) == 0


def test_memory_attention_null_handle():
    assert mone.lib().mone_memory_attention(None, 16, 16, 16, 16, 0, 4, 4, 2, 16, 0,
                                            None) == mone.MONE_EINVAL


# ---------------------------------------------------------------- paper-form (SwiGLU) memory

def _swcfg(**kw):
    base = dict(n_layers=2, d_model=192, n_heads=2, d_head=96, seg_len=300, act_dtype="bf16",
                optimizer="sgd", lr=1.0)
    base.update(kw)
    return mone.make_swiglu_config(**base)


def test_swiglu_workspace_formula():
    c = _swcfg()
    n = mone.mone_swiglu_workspace_bytes(c)
    L, d, H, dh, dhp, Tp, E = 2, 192, 2, 96, 128, 512, 2
    B = L * H
    act = (E * L * Tp * d + E * B * (2 * Tp * dhp + 4 * dh * Tp + 2 * dh * Tp + 3 * dh * dhp)
           + Tp * (dh // 2) * 8 + 4 * L * Tp * H)
    assert act <= n <= act + 64 * 1024
    p = mone.mone_swiglu_workspace_bytes(_swcfg(optimizer="paper"))
    extra = 4 * (L * Tp + L * (Tp // 16) + L + 3 * B * dh)
    assert extra <= p - n <= extra + 8 * 256
    # the context length is not a parameter of any call
    for cfg in configs.SW_CONFIGS.values():
        a = mone.mone_swiglu_workspace_bytes(mone.swiglu_config_from(cfg))
        b = mone.mone_swiglu_workspace_bytes(
            mone.swiglu_config_from(cfg.with_(n_context=cfg.n_context * 4)))
        assert a == b


@pytest.mark.parametrize("kw,code", [
    (dict(n_layers=0), mone.MONE_EINVAL),
    (dict(n_heads=3), mone.MONE_EINVAL),           # d_model != H * d_h
    (dict(d_model=190, d_head=95), mone.MONE_EINVAL),  # odd head width
    (dict(act_dtype=9), mone.MONE_EINVAL),
    (dict(optimizer=4), mone.MONE_EINVAL),
    (dict(lr=float("inf")), mone.MONE_EINVAL),
    (dict(rope_base=0.0), mone.MONE_EINVAL),
    (dict(d_model=160, d_head=80), mone.MONE_EUNSUPPORTED),  # d_model not a multiple of 64
    (dict(d_model=320, n_heads=1, d_head=320), mone.MONE_EUNSUPPORTED),  # d_head above 256
    (dict(d_model=192, n_heads=8, d_head=24), mone.MONE_EUNSUPPORTED),  # not a multiple of 16
    (dict(d_model=256, n_heads=16, d_head=16, seg_len=70000), mone.MONE_EUNSUPPORTED),
])
def test_swiglu_invalid_configs_are_rejected(kw, code):
    c = _swcfg(**kw)
    assert mone.lib().mone_swiglu_workspace_bytes(ctypes.byref(c)) == 0
    assert mone.mone_ttl_last_error()
    h = ctypes.c_void_p(1234)
    fz = mone.mone_swiglu_frozen(16, 16, 16)
    w = mone.mone_swiglu_weights(16, 16, 16)
    rc = mone.lib().mone_swiglu_init(ctypes.byref(h), ctypes.byref(c), ctypes.byref(fz),
                                     ctypes.byref(w), None, 256, 1 << 30, None)
    assert rc == code and h.value is None


def test_swiglu_init_argument_checks_before_any_hip_call():
    L = mone.lib()
    h = ctypes.c_void_p()
    c, p = _swcfg(), _swcfg(optimizer="paper")
    need = mone.mone_swiglu_workspace_bytes(p)
    fz = mone.mone_swiglu_frozen(16, 16, 16)
    w = mone.mone_swiglu_weights(16, 16, 16)
    opt = mone.mone_swiglu_optimizer(16, 16, 16, 16, 16, 16, 16)
    args = lambda cfg, f, ww, o, ws=256, nb=need: L.mone_swiglu_init(  # noqa: E731
        ctypes.byref(h), ctypes.byref(cfg), f and ctypes.byref(f), ww and ctypes.byref(ww),
        o and ctypes.byref(o), ws, nb, None)
    assert args(c, None, w, None) == mone.MONE_EINVAL
    assert args(c, fz, None, None) == mone.MONE_EINVAL
    assert args(c, mone.mone_swiglu_frozen(16, None, 16), w, None) == mone.MONE_EINVAL
    assert args(c, fz, mone.mone_swiglu_weights(16, 24, 16), None) == mone.MONE_EINVAL
    assert "aligned" in mone.mone_ttl_last_error()
    assert args(c, fz, w, opt) == mone.MONE_EINVAL      # SGD takes no optimiser state
    assert args(p, fz, w, None) == mone.MONE_EINVAL     # the paper optimiser needs it
    assert args(p, fz, w, mone.mone_swiglu_optimizer(16, 16, 16, 16, 16, None, 16)) == \
        mone.MONE_EINVAL
    assert args(p, fz, w, mone.mone_swiglu_optimizer(16, 16, 16, 16, 16, 16, 40)) == \
        mone.MONE_EINVAL
    assert args(p, fz, w, opt, ws=272) == mone.MONE_EINVAL
    assert args(p, fz, w, opt, nb=need - 1) == mone.MONE_EINVAL
    assert "workspace" in mone.mone_ttl_last_error()
    assert h.value is None
    assert L.mone_swiglu_init(None, ctypes.byref(c), ctypes.byref(fz), ctypes.byref(w), None,
                              256, need, None) == mone.MONE_EINVAL


def test_swiglu_null_handle_calls_fail_cleanly():
    L = mone.lib()
    out = (ctypes.c_float * 1)()
    assert L.mone_swiglu_segment(None, 16, 1, None) == mone.MONE_EINVAL
    assert L.mone_swiglu_loss(None, out, None) == mone.MONE_EINVAL
    assert L.mone_swiglu_destroy(None) == mone.MONE_OK
    assert L.mone_swiglu_set_stage_timing(None, 4, mone.MONE_ALL_STAGES) == mone.MONE_EINVAL
    ms = (ctypes.c_double * mone.MONE_SW_N_STAGES)()
    cnt = (ctypes.c_int32 * mone.MONE_SW_N_STAGES)()
    assert L.mone_swiglu_stage_times(None, ms, cnt) == mone.MONE_EINVAL
    rd = mone.mone_swiglu_reader(16, 16, 16, 16, 16, 16, 16, 64)
    assert L.mone_swiglu_read(None, ctypes.byref(rd), 16, 1, 16, 0, None) == mone.MONE_EINVAL
    assert L.mone_swiglu_attention(None, 64, 16, 16, 16, 16, 0, 4, 4, 2, 16, 0,
                                   None) == mone.MONE_EINVAL


def test_noalloc_step_rejects_before_any_hip_call():
    # every check of the no-allocation step precedes its first HIP call, so none touches a GPU
    dummy = 4096  # a 16-byte-aligned non-NULL address that is never used
    big = mone.config_from(configs.ONE_B)  # workspace far beyond the 64 MiB static scratch
    with pytest.raises(mone.MoneError) as e:
        mone.mone_ttl_step_noalloc(big, dummy, dummy, dummy, dummy, 16, 0)
    assert e.value.code == mone.MONE_EUNSUPPORTED and "scratch" in str(e.value)
    paper = _cfg(optimizer="paper")
    with pytest.raises(mone.MoneError) as e:
        mone.mone_ttl_step_noalloc(paper, dummy, dummy, dummy, dummy, 16, 0)
    assert e.value.code == mone.MONE_EUNSUPPORTED
    small = _cfg()
    with pytest.raises(mone.MoneError) as e:
        mone.mone_ttl_step_noalloc(small, None, dummy, dummy, dummy, 16, 0)
    assert e.value.code == mone.MONE_EINVAL
    for n in (-1, 101):
        with pytest.raises(mone.MoneError) as e:
            mone.mone_ttl_step_noalloc(small, dummy, dummy, dummy, dummy, n, 0)
        assert e.value.code == mone.MONE_EINVAL
    with pytest.raises(mone.MoneError) as e:
        mone.mone_ttl_step_noalloc(small, dummy, dummy, dummy, None, 16, 0)
    assert e.value.code == mone.MONE_EINVAL


def test_block_form_workspace_and_config_checks():
    base = dict(n_layers=2, d_model=128, d_hidden=192, d_kv=64, seg_len=64, act_dtype="bf16",
                loss="mse_sum", lr=1e-3)
    ws = lambda **kw: mone.mone_ttl_workspace_bytes(mone.make_config(**dict(base, **kw)))  # noqa
    none = ws(block_tokens=-1)
    assert ws() == none  # small memories: no block form by default
    L, d, h, D, Tp, Bp, E = 2, 128, 192, 128, 256, 512, 2
    extra = L * (4 * Bp * (h + D) + E * (Bp * Bp + 3 * Bp * h + 2 * Bp * D + h * Bp + d * Bp)
                 + 4 * Tp * (D + h) + 2 * E * Tp * Bp)
    assert extra <= ws(block_tokens=512) - none <= extra + 14 * 256
    # the 64-token workload takes the block form by default
    st = configs.STRESS
    assert (mone.mone_ttl_workspace_bytes(mone.config_from(st))
            > mone.mone_ttl_workspace_bytes(mone.config_from(st.with_(block_tokens=-1))))
    # the default block: 8 segments, at most 1024 tokens, for segments of at most 256 tokens
    big = dict(base, n_layers=16, d_model=2048, d_hidden=2048, d_kv=512)
    wsb = lambda **kw: mone.mone_ttl_workspace_bytes(mone.make_config(**dict(big, **kw)))  # noqa
    for T, default in ((64, 512), (128, 1024), (192, 960), (256, 1024)):
        assert wsb(seg_len=T) == wsb(seg_len=T, block_tokens=default) != wsb(seg_len=T,
                                                                           block_tokens=-1)
        assert bench.block_segments(configs.STRESS.with_(seg_len=T)) == default // T
    assert wsb(seg_len=320) == wsb(seg_len=320, block_tokens=-1)
    assert bench.block_segments(configs.STRESS.with_(seg_len=320)) == 1
    for bad in (dict(block_tokens=100), dict(block_tokens=64), dict(block_tokens=8192),
                dict(block_tokens=512, loss="nip"), dict(block_tokens=512, optimizer="paper"),
                dict(block_tokens=500, seg_len=100)):
        with pytest.raises(mone.MoneError):
            ws(**bad)


def test_swiglu_preprocessing_copies_in_the_workspace():
    # prep_segments copies of K' (the raw keys), and above 1 two sets of prep_segments copies of
    # K, K^T, dY0, dY^T: one batch's preprocessing fills a set while the batch before reads the
    # other
    L, d, H, dh, dhp, Tp, E = 2, 192, 2, 96, 128, 512, 2
    B = L * H
    one = mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=512, prep_segments=1))
    raw = E * L * Tp * d
    per_set_copy = E * B * (2 * Tp * dhp + 2 * dh * Tp)
    for g in (2, 4, 16):
        n = mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=512, prep_segments=g))
        extra = (g - 1) * raw + (2 * g - 1) * per_set_copy
        assert extra <= n - one <= extra + 8 * 256
    # the default batches 8 segments of a multiple of 64 tokens, and 1 otherwise
    assert (mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=512))
            == mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=512, prep_segments=8)))
    assert (mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=300))
            == mone.mone_swiglu_workspace_bytes(_swcfg(seg_len=300, prep_segments=1)))
    for bad in (dict(prep_segments=17), dict(prep_segments=-1),
                dict(seg_len=300, prep_segments=2)):
        with pytest.raises(mone.MoneError):
            mone.mone_swiglu_workspace_bytes(_swcfg(**bad))
