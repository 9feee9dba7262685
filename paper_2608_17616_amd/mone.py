"""Python binding of libmone_ttl.so (the C ABI in include/mone_ttl.h and include/mone_swiglu.h).

Argument marshalling only: every function forwards to the C call of the same name.  Device
buffers are passed as torch tensors (their data_ptr()) or as raw integer addresses, streams as
torch.cuda.Stream objects, raw hipStream_t integers, or None for torch's current stream.
PyTorch is used only to own device memory and streams.

The library must have been built (``python -m paper_2608_17616_amd.build``); loading fails
loudly otherwise -- there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmone_ttl.so")

MONE_OK, MONE_EINVAL, MONE_EUNSUPPORTED, MONE_EHIP, MONE_ESTATE = 0, -1, -2, -3, -4
MONE_F32, MONE_BF16 = 0, 1
MONE_LOSS_MSE_SUM, MONE_LOSS_MSE_MEAN, MONE_LOSS_NIP = 0, 1, 2
MONE_OPT_SGD, MONE_OPT_PAPER = 0, 1
MONE_ALL_STAGES = 0xFFFFFFFF
STAGES = ("xt", "fwd1", "fwd2", "bwd", "upd", "kv1", "kv2", "rate", "renorm", "attn", "bfwd",
          "bseq", "bupd")
MONE_N_STAGES = len(STAGES)

SW_STAGES = ("rate", "proj", "keys", "da", "fwd", "upd", "qproj", "qkeys", "qfwd", "qout", "qkv",
             "attn")
MONE_SW_N_STAGES = len(SW_STAGES)

# every symbol include/mone_ttl.h and include/mone_swiglu.h declare
EXPORTS = ("mone_ttl_workspace_bytes", "mone_ttl_init", "mone_ttl_init_paper",
           "mone_ttl_segment", "mone_ttl_segments", "mone_ttl_step_noalloc", "mone_memory_kv",
           "mone_memory_attention",
           "mone_ttl_loss", "mone_ttl_destroy", "mone_ttl_last_error",
           "mone_ttl_set_stage_timing", "mone_ttl_stage_times",
           "mone_swiglu_workspace_bytes", "mone_swiglu_init", "mone_swiglu_segment",
           "mone_swiglu_segments",
           "mone_swiglu_loss", "mone_swiglu_read", "mone_swiglu_attention",
           "mone_swiglu_destroy", "mone_swiglu_set_stage_timing", "mone_swiglu_stage_times")


class MoneError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


class mone_ttl_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("d_hidden", ctypes.c_int32), ("d_kv", ctypes.c_int32),
                ("seg_len", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("loss", ctypes.c_int32), ("lr", ctypes.c_float),
                ("optimizer", ctypes.c_int32), ("block_tokens", ctypes.c_int32)]


class mone_paper_optimizer(ctypes.Structure):
    _fields_ = [("rate_w", ctypes.c_void_p), ("rate_b", ctypes.c_void_p),
                ("decay_w", ctypes.c_void_p), ("decay_b", ctypes.c_void_p),
                ("mom1", ctypes.c_void_p), ("mom2", ctypes.c_void_p)]


class mone_swiglu_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_head", ctypes.c_int32),
                ("seg_len", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("optimizer", ctypes.c_int32), ("lr", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("prep_segments", ctypes.c_int32)]


class mone_swiglu_frozen(ctypes.Structure):
    _fields_ = [("proj", ctypes.c_void_p), ("k_scale", ctypes.c_void_p),
                ("k_shift", ctypes.c_void_p)]


class mone_swiglu_weights(ctypes.Structure):
    _fields_ = [("w_in", ctypes.c_void_p), ("w_gate", ctypes.c_void_p),
                ("w_out", ctypes.c_void_p)]


class mone_swiglu_optimizer(ctypes.Structure):
    _fields_ = [("rate_w", ctypes.c_void_p), ("rate_b", ctypes.c_void_p),
                ("decay_w", ctypes.c_void_p), ("decay_b", ctypes.c_void_p),
                ("mom_in", ctypes.c_void_p), ("mom_gate", ctypes.c_void_p),
                ("mom_out", ctypes.c_void_p)]


class mone_swiglu_reader(ctypes.Structure):
    _fields_ = [("proj_q", ctypes.c_void_p), ("q_scale", ctypes.c_void_p),
                ("q_shift", ctypes.c_void_p), ("rms_w", ctypes.c_void_p),
                ("gate_w", ctypes.c_void_p), ("gate_b", ctypes.c_void_p),
                ("w_kv", ctypes.c_void_p), ("d_kv", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2608_17616_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        cfgp = ctypes.POINTER(mone_ttl_config)
        L.mone_ttl_workspace_bytes.argtypes = [cfgp]
        L.mone_ttl_workspace_bytes.restype = ctypes.c_size_t
        L.mone_ttl_init.argtypes = [ctypes.POINTER(vp), cfgp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.mone_ttl_init_paper.argtypes = [ctypes.POINTER(vp), cfgp, vp, vp, vp,
                                          ctypes.POINTER(mone_paper_optimizer), vp,
                                          ctypes.c_size_t, vp]
        L.mone_ttl_segment.argtypes = [vp, vp, i32, vp]
        L.mone_ttl_segments.argtypes = [vp, vp, ctypes.c_int64, i32, vp]
        L.mone_ttl_step_noalloc.argtypes = [cfgp, vp, vp, vp, vp, i32, vp]
        L.mone_memory_kv.argtypes = [vp, vp, i32, vp, i32, vp]
        L.mone_memory_attention.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, i32, vp]
        L.mone_ttl_loss.argtypes = [vp, ctypes.POINTER(ctypes.c_float), vp]
        L.mone_ttl_destroy.argtypes = [vp]
        L.mone_ttl_last_error.argtypes = []
        L.mone_ttl_last_error.restype = ctypes.c_char_p
        L.mone_ttl_set_stage_timing.argtypes = [vp, i32, ctypes.c_uint32]
        L.mone_ttl_stage_times.argtypes = [vp, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_int32)]
        swp = ctypes.POINTER(mone_swiglu_config)
        L.mone_swiglu_workspace_bytes.argtypes = [swp]
        L.mone_swiglu_workspace_bytes.restype = ctypes.c_size_t
        L.mone_swiglu_init.argtypes = [ctypes.POINTER(vp), swp,
                                       ctypes.POINTER(mone_swiglu_frozen),
                                       ctypes.POINTER(mone_swiglu_weights),
                                       ctypes.POINTER(mone_swiglu_optimizer), vp, ctypes.c_size_t,
                                       vp]
        L.mone_swiglu_segment.argtypes = [vp, vp, i32, vp]
        L.mone_swiglu_segments.argtypes = [vp, vp, ctypes.c_int64, i32, vp]
        L.mone_swiglu_loss.argtypes = [vp, ctypes.POINTER(ctypes.c_float), vp]
        L.mone_swiglu_read.argtypes = [vp, ctypes.POINTER(mone_swiglu_reader), vp, i32, vp, i32,
                                       vp]
        L.mone_swiglu_attention.argtypes = [vp, i32, vp, vp, vp, vp, i32, i32, i32, i32, vp, i32,
                                            vp]
        L.mone_swiglu_destroy.argtypes = [vp]
        L.mone_swiglu_set_stage_timing.argtypes = [vp, i32, ctypes.c_uint32]
        L.mone_swiglu_stage_times.argtypes = [vp, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_int32)]
        for name in EXPORTS:
            if name not in ("mone_ttl_workspace_bytes", "mone_ttl_last_error",
                            "mone_swiglu_workspace_bytes"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != MONE_OK:
        raise MoneError(rc, mone_ttl_last_error())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s) -> int | None:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def make_config(n_layers, d_model, d_hidden, d_kv, seg_len, act_dtype, loss, lr,
                optimizer="sgd", block_tokens=0):
    dt = {"f32": MONE_F32, "bf16": MONE_BF16}.get(act_dtype, act_dtype)
    ls = {"mse_sum": MONE_LOSS_MSE_SUM, "mse_mean": MONE_LOSS_MSE_MEAN,
          "nip": MONE_LOSS_NIP}.get(loss, loss)
    op = {"sgd": MONE_OPT_SGD, "paper": MONE_OPT_PAPER}.get(optimizer, optimizer)
    return mone_ttl_config(int(n_layers), int(d_model), int(d_hidden), int(d_kv), int(seg_len),
                           int(dt), int(ls), float(lr), int(op), int(block_tokens))


def config_from(cfg) -> mone_ttl_config:
    """C config of a configs.MoneConfig."""
    return make_config(cfg.n_layers, cfg.d_model, cfg.d_hidden, cfg.d_kv, cfg.seg_len,
                       cfg.act_dtype, cfg.loss, cfg.lr, cfg.optimizer,
                       getattr(cfg, "block_tokens", 0))


def mone_ttl_last_error() -> str:
    return lib().mone_ttl_last_error().decode()


def mone_ttl_workspace_bytes(cfg: mone_ttl_config) -> int:
    n = lib().mone_ttl_workspace_bytes(ctypes.byref(cfg))
    if n == 0:
        raise MoneError(MONE_EINVAL, mone_ttl_last_error())
    return n


def mone_ttl_init(cfg: mone_ttl_config, wkv, w1, w2, workspace, workspace_bytes: int,
                  stream=None) -> int:
    h = ctypes.c_void_p()
    _check(lib().mone_ttl_init(ctypes.byref(h), ctypes.byref(cfg), _ptr(wkv), _ptr(w1), _ptr(w2),
                               _ptr(workspace), int(workspace_bytes), _stream(stream)))
    return h.value


def mone_ttl_init_paper(cfg: mone_ttl_config, wkv, w1, w2, opt: mone_paper_optimizer,
                        workspace, workspace_bytes: int, stream=None) -> int:
    h = ctypes.c_void_p()
    _check(lib().mone_ttl_init_paper(ctypes.byref(h), ctypes.byref(cfg), _ptr(wkv), _ptr(w1),
                                     _ptr(w2), ctypes.byref(opt) if opt is not None else None,
                                     _ptr(workspace), int(workspace_bytes), _stream(stream)))
    return h.value


def paper_optimizer(rate_w, rate_b, decay_w, decay_b, mom1, mom2) -> mone_paper_optimizer:
    """C struct of the paper optimiser's buffers (device tensors or raw addresses)."""
    return mone_paper_optimizer(*(_ptr(t) for t in (rate_w, rate_b, decay_w, decay_b, mom1, mom2)))


def mone_ttl_segment(handle: int, x, n_tokens: int, stream=None) -> None:
    _check(lib().mone_ttl_segment(handle, _ptr(x), int(n_tokens), _stream(stream)))


def mone_ttl_segments(handle: int, x, layer_stride: int, n_segments: int, stream=None) -> None:
    _check(lib().mone_ttl_segments(handle, _ptr(x), int(layer_stride), int(n_segments),
                                   _stream(stream)))


def mone_ttl_step_noalloc(cfg: mone_ttl_config, wkv, w1, w2, x, n_tokens: int,
                          stream=None) -> None:
    _check(lib().mone_ttl_step_noalloc(ctypes.byref(cfg), _ptr(wkv), _ptr(w1), _ptr(w2), _ptr(x),
                                       int(n_tokens), _stream(stream)))


def mone_memory_kv(handle: int, xq, q: int, kv, kv_dtype: int, stream=None) -> None:
    _check(lib().mone_memory_kv(handle, _ptr(xq), int(q), _ptr(kv), int(kv_dtype),
                                _stream(stream)))


def mone_memory_attention(handle: int, qh, kh, vh, kv_mem, kv_dtype: int, q: int, n_heads: int,
                          n_kv_heads: int, out, out_dtype: int, stream=None) -> None:
    _check(lib().mone_memory_attention(handle, _ptr(qh), _ptr(kh), _ptr(vh), _ptr(kv_mem),
                                       int(kv_dtype), int(q), int(n_heads), int(n_kv_heads),
                                       _ptr(out), int(out_dtype), _stream(stream)))


def mone_ttl_loss(handle: int, n_layers: int, stream=None) -> list[float]:
    out = (ctypes.c_float * n_layers)()
    _check(lib().mone_ttl_loss(handle, out, _stream(stream)))
    return list(out)


def mone_ttl_destroy(handle: int) -> None:
    _check(lib().mone_ttl_destroy(handle))


def mone_ttl_set_stage_timing(handle: int, max_records: int,
                              stage_mask: int = MONE_ALL_STAGES) -> None:
    _check(lib().mone_ttl_set_stage_timing(handle, int(max_records), int(stage_mask)))


def mone_ttl_stage_times(handle: int) -> dict:
    ms = (ctypes.c_double * MONE_N_STAGES)()
    cnt = (ctypes.c_int32 * MONE_N_STAGES)()
    _check(lib().mone_ttl_stage_times(handle, ms, cnt))
    return {name: (ms[i], cnt[i]) for i, name in enumerate(STAGES)}


class TtlSession:
    """Device state of one TTL run: the caller-owned tensors the C ABI borrows, and a handle.

    w1 [L, h, d] fp32, w2 [L, D, h] fp32 and wkv [L, D, d] (activation dtype) are torch tensors
    on the GPU; the workspace is allocated here with torch (the library allocates nothing).
    """

    def __init__(self, cfg, wkv, w1, w2, stream=None, opt=None):
        """opt: for cfg.optimizer == "paper", the tensors (rate_w [L, d], rate_b [L],
        decay_w [L, d], decay_b [L], mom1 [L, h, d], mom2 [L, D, h]), all fp32 on the GPU."""
        import torch
        self.cfg = cfg
        self.ccfg = config_from(cfg)
        self.wkv, self.w1, self.w2 = wkv, w1, w2
        self.opt = opt
        self.ws_bytes = mone_ttl_workspace_bytes(self.ccfg)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=w1.device)
        if cfg.optimizer == "paper":
            self.copt = paper_optimizer(*opt)
            self.handle = mone_ttl_init_paper(self.ccfg, wkv, w1, w2, self.copt, self.workspace,
                                              self.ws_bytes, stream)
        else:
            self.handle = mone_ttl_init(self.ccfg, wkv, w1, w2, self.workspace, self.ws_bytes,
                                        stream)

    def segment(self, x, n_tokens=None, stream=None):
        n = x.shape[1] if n_tokens is None else n_tokens
        mone_ttl_segment(self.handle, x, n, stream)

    def segments(self, x, n_segments=None, stream=None):
        """x: [L, S*T, d] (or a view with that layout: each layer's tokens contiguous, layer
        stride x.stride(0)); runs the first n_segments (default S) segments of T tokens."""
        T = self.cfg.seg_len
        n = x.shape[1] // T if n_segments is None else n_segments
        mone_ttl_segments(self.handle, x, x.stride(0), n, stream)

    def memory_kv(self, xq, kv, stream=None):
        import torch
        dt = MONE_BF16 if kv.dtype == torch.bfloat16 else MONE_F32
        mone_memory_kv(self.handle, xq, xq.shape[1], kv, dt, stream)
        return kv

    def loss(self, stream=None):
        return mone_ttl_loss(self.handle, self.cfg.n_layers, stream)

    def close(self):
        if self.handle:
            mone_ttl_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- paper-form (SwiGLU) memory

def make_swiglu_config(n_layers, d_model, n_heads, d_head, seg_len, act_dtype, optimizer, lr,
                       rope_base=10000.0, prep_segments=0) -> mone_swiglu_config:
    dt = {"f32": MONE_F32, "bf16": MONE_BF16}.get(act_dtype, act_dtype)
    op = {"sgd": MONE_OPT_SGD, "paper": MONE_OPT_PAPER}.get(optimizer, optimizer)
    return mone_swiglu_config(int(n_layers), int(d_model), int(n_heads), int(d_head),
                              int(seg_len), int(dt), int(op), float(lr), float(rope_base),
                              int(prep_segments))


def swiglu_config_from(cfg) -> mone_swiglu_config:
    """C config of a configs.SwigluConfig."""
    return make_swiglu_config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_head, cfg.seg_len,
                              cfg.act_dtype, cfg.optimizer, cfg.lr, cfg.rope_base,
                              getattr(cfg, "prep_segments", 0))


def mone_swiglu_workspace_bytes(cfg: mone_swiglu_config) -> int:
    n = lib().mone_swiglu_workspace_bytes(ctypes.byref(cfg))
    if n == 0:
        raise MoneError(MONE_EINVAL, mone_ttl_last_error())
    return n


def mone_swiglu_init(cfg: mone_swiglu_config, frozen: mone_swiglu_frozen,
                     weights: mone_swiglu_weights, opt, workspace, workspace_bytes: int,
                     stream=None) -> int:
    h = ctypes.c_void_p()
    _check(lib().mone_swiglu_init(ctypes.byref(h), ctypes.byref(cfg),
                                  ctypes.byref(frozen) if frozen is not None else None,
                                  ctypes.byref(weights) if weights is not None else None,
                                  ctypes.byref(opt) if opt is not None else None,
                                  _ptr(workspace), int(workspace_bytes), _stream(stream)))
    return h.value


def mone_swiglu_segment(handle: int, x, n_tokens: int, stream=None) -> None:
    _check(lib().mone_swiglu_segment(handle, _ptr(x), int(n_tokens), _stream(stream)))


def mone_swiglu_segments(handle: int, x, layer_stride: int, n_segments: int,
                         stream=None) -> None:
    _check(lib().mone_swiglu_segments(handle, _ptr(x), int(layer_stride), int(n_segments),
                                      _stream(stream)))


def mone_swiglu_loss(handle: int, n_layers: int, stream=None) -> list[float]:
    out = (ctypes.c_float * n_layers)()
    _check(lib().mone_swiglu_loss(handle, out, _stream(stream)))
    return list(out)


def swiglu_reader(proj_q, q_scale, q_shift, rms_w, gate_w, gate_b, w_kv,
                  d_kv: int) -> mone_swiglu_reader:
    """C struct of the read's frozen parameters (device tensors or raw addresses)."""
    return mone_swiglu_reader(*(_ptr(t) for t in (proj_q, q_scale, q_shift, rms_w, gate_w,
                                                   gate_b, w_kv)), int(d_kv))


def mone_swiglu_read(handle: int, reader: mone_swiglu_reader, xq, q: int, kv, kv_dtype: int,
                     stream=None) -> None:
    _check(lib().mone_swiglu_read(handle, ctypes.byref(reader) if reader is not None else None,
                                  _ptr(xq), int(q), _ptr(kv), int(kv_dtype), _stream(stream)))


def mone_swiglu_attention(handle: int, d_kv: int, qh, kh, vh, kv_mem, kv_dtype: int, q: int,
                          n_heads: int, n_kv_heads: int, out, out_dtype: int,
                          stream=None) -> None:
    _check(lib().mone_swiglu_attention(handle, int(d_kv), _ptr(qh), _ptr(kh), _ptr(vh),
                                       _ptr(kv_mem), int(kv_dtype), int(q), int(n_heads),
                                       int(n_kv_heads), _ptr(out), int(out_dtype),
                                       _stream(stream)))


def mone_swiglu_destroy(handle: int) -> None:
    _check(lib().mone_swiglu_destroy(handle))


def mone_swiglu_set_stage_timing(handle: int, max_records: int,
                                 stage_mask: int = MONE_ALL_STAGES) -> None:
    _check(lib().mone_swiglu_set_stage_timing(handle, int(max_records), int(stage_mask)))


def mone_swiglu_stage_times(handle: int) -> dict:
    ms = (ctypes.c_double * MONE_SW_N_STAGES)()
    cnt = (ctypes.c_int32 * MONE_SW_N_STAGES)()
    _check(lib().mone_swiglu_stage_times(handle, ms, cnt))
    return {name: (ms[i], cnt[i]) for i, name in enumerate(SW_STAGES)}


class SwigluSession:
    """Device state of one paper-form TTL run.

    proj [L, 2d, d] (activation dtype), k_scale and k_shift [L, d] fp32, and the fast weights
    w_in, w_gate, w_out [L, H, d_h, d_h] fp32 are torch tensors on the GPU; opt, for
    cfg.optimizer == "paper", is (rate_w [L, d], rate_b [L], decay_w [L, d], decay_b [L],
    mom_in, mom_gate, mom_out), all fp32.  The workspace is allocated here with torch.
    """

    def __init__(self, cfg, proj, k_scale, k_shift, w_in, w_gate, w_out, opt=None, stream=None):
        import torch
        self.cfg = cfg
        self.ccfg = swiglu_config_from(cfg)
        self.keep = (proj, k_scale, k_shift, w_in, w_gate, w_out, opt)
        self.frozen = mone_swiglu_frozen(_ptr(proj), _ptr(k_scale), _ptr(k_shift))
        self.weights = mone_swiglu_weights(_ptr(w_in), _ptr(w_gate), _ptr(w_out))
        self.copt = mone_swiglu_optimizer(*(_ptr(t) for t in opt)) if opt is not None else None
        self.ws_bytes = mone_swiglu_workspace_bytes(self.ccfg)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=w_in.device)
        self.handle = mone_swiglu_init(self.ccfg, self.frozen, self.weights, self.copt,
                                       self.workspace, self.ws_bytes, stream)

    def segment(self, x, n_tokens=None, stream=None):
        n = x.shape[1] if n_tokens is None else n_tokens
        mone_swiglu_segment(self.handle, x, n, stream)

    def segments(self, x, n_segments=None, stream=None):
        """x: [L, S*T, d] (or a view with that layout, layer stride x.stride(0))."""
        n = x.shape[1] // self.cfg.seg_len if n_segments is None else n_segments
        mone_swiglu_segments(self.handle, x, x.stride(0), n, stream)

    def loss(self, stream=None):
        return mone_swiglu_loss(self.handle, self.cfg.n_layers, stream)

    def read(self, reader: mone_swiglu_reader, xq, kv, stream=None):
        """Memory K/V rows kv [L, q, 2 d_kv] (fp32 or bf16 tensor) of query inputs xq."""
        import torch
        dt = MONE_BF16 if kv.dtype == torch.bfloat16 else MONE_F32
        mone_swiglu_read(self.handle, reader, xq, xq.shape[1], kv, dt, stream)
        return kv

    def close(self):
        if self.handle:
            mone_swiglu_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
