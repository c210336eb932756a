"""ctypes binding of libssd (include/ssd.h): the same entry points, argument marshalling only.

Device pointers may be given as integers or as objects with ``data_ptr()`` (torch tensors); None
is NULL.  Every non-zero return code raises SSDError.  The library must have been built
(``python -m paper_2510_22641_amd.build``); importing this module without it raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libssd.so")

SSD_OK, SSD_ERR_ARG, SSD_ERR_SHAPE, SSD_ERR_CAPACITY, SSD_ERR_HIP, SSD_ERR_STATE, SSD_ERR_DEVICE = \
    0, -1, -2, -3, -4, -5, -6
SSD_ARCH_T5, SSD_ARCH_LLAMA = 0, 1
SSD_F32, SSD_BF16 = 0, 1
SSD_MODE_GREEDY, SSD_MODE_SPECULATIVE, SSD_MODE_SPECULATIVE_DYNAMIC = 0, 1, 2
SSD_DEV_BAD_TOKEN, SSD_DEV_CAPACITY, SSD_DEV_BAD_PAGE = 1, 2, 4


class ssd_dims(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("arch", "n_layers", "d_model", "n_heads", "d_head", "d_ff",
                                       "vocab", "n_visual", "rel_buckets", "rel_max_dist")] + \
               [(n, c_float) for n in ("rope_theta", "norm_eps", "ln_eps")] + \
               [(n, c_int32) for n in ("wdtype", "kvdtype", "draft_layers", "in_hidden",
                                       "in_residual", "max_batch", "max_gamma", "max_seq",
                                       "max_prompt", "page_size", "max_pages")]


LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "xattn_norm", "xq", "xk", "xv", "xo",
                "ffn_norm", "w_gate", "w_up", "w_down")
GLOBAL_FIELDS = ("embed", "lm_head", "final_norm", "rel_bias", "in_ln_w", "in_ln_b", "in_w1",
                 "in_b1", "in_w2", "in_b2")


class ssd_layer_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in LAYER_FIELDS]


class ssd_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in GLOBAL_FIELDS] + [("layers", POINTER(ssd_layer_weights))]


class ssd_kv(ctypes.Structure):
    _fields_ = [("k_pool", c_void_p), ("v_pool", c_void_p), ("n_pages", c_int32),
                ("page_table", c_void_p), ("seq_len", c_void_p), ("xk", c_void_p),
                ("xv", c_void_p)]


class SSDError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {status_string(code)} ({code})")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libssd.so is not built ({LIB_PATH}); run "
                           "`python -m paper_2510_22641_amd.build` (the device path has no "
                           "fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    sig = {
        "ssd_workspace_bytes": (c_size_t, [POINTER(ssd_dims)]),
        "ssd_create": (c_int, [POINTER(ssd_dims), POINTER(ssd_weights), POINTER(ssd_kv), P,
                               c_size_t, P, POINTER(P)]),
        "ssd_create_static": (c_int, [POINTER(ssd_dims), POINTER(ssd_weights), POINTER(ssd_kv),
                                      P, POINTER(P)]),
        "ssd_prefill": (c_int, [P, c_int, c_int, P, P, P, P]),
        "ssd_draft": (c_int, [P, c_int, c_int, P, P, P]),
        "ssd_verify": (c_int, [P, c_int, c_int, P, P, c_int, P, P]),
        "ssd_accept": (c_int, [P, c_int, c_int, P, P, P, P, P, P]),
        "ssd_draft_sample": (c_int, [P, c_int, c_int, P, P, ctypes.c_float, P, P]),
        "ssd_accept_sample": (c_int, [P, c_int, c_int, P, P, P, P, ctypes.c_float, P, P, P, P]),
        "ssd_generate": (c_int, [P, c_int, c_int, P, P, c_int, c_int, c_int, c_int, P,
                                 POINTER(c_int64)]),
        "ssd_draft_confident": (c_int, [P, c_int, c_int, ctypes.c_float, P, P, P, P, P, P,
                                        POINTER(c_int)]),
        "ssd_accept_counts": (c_int, [P, c_int, c_int, P, P, P, P, P, P, P]),
        "ssd_generate_confident": (c_int, [P, c_int, c_int, P, P, c_int, c_int, ctypes.c_float,
                                           c_int, P, POINTER(c_int64)]),
        "ssd_dynamic_gamma": (c_int, [c_int, c_int, c_int]),
        "ssd_set_graphs": (c_int, [P, c_int]),
        "ssd_set_hidden_export": (c_int, [P, P, P, P]),
        "ssd_profile_enable": (c_int, [P, c_int]),
        "ssd_profile_read": (c_int, [P, POINTER(c_int64), POINTER(ctypes.c_double),
                                     POINTER(ctypes.c_double)]),
        "ssd_read_bandwidth": (c_int, [P, c_size_t, P, c_int, P, POINTER(ctypes.c_double)]),
        "ssd_sync_status": (c_int, [P, POINTER(c_int32)]),
        "ssd_status_string": (ctypes.c_char_p, [c_int]),
        "ssd_destroy": (None, [P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
EXPORTS = ("ssd_workspace_bytes", "ssd_create", "ssd_create_static", "ssd_prefill", "ssd_draft", "ssd_verify",
           "ssd_accept", "ssd_draft_sample", "ssd_accept_sample", "ssd_generate", "ssd_draft_confident", "ssd_accept_counts",
           "ssd_generate_confident", "ssd_dynamic_gamma", "ssd_set_graphs", "ssd_set_hidden_export",
           "ssd_profile_enable",
           "ssd_profile_read", "ssd_read_bandwidth", "ssd_sync_status",
           "ssd_status_string", "ssd_destroy")


def _p(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _check(fn, rc):
    if rc != SSD_OK:
        raise SSDError(fn, rc)


def status_string(code: int) -> str:
    return _lib.ssd_status_string(code).decode()


ssd_status_string = status_string


def ssd_workspace_bytes(dims: ssd_dims) -> int:
    return int(_lib.ssd_workspace_bytes(ctypes.byref(dims)))


def ssd_create(dims: ssd_dims, weights: ssd_weights, kv: ssd_kv, d_workspace, workspace_bytes: int,
               stream) -> c_void_p:
    ctx = c_void_p()
    _check("ssd_create", _lib.ssd_create(ctypes.byref(dims), ctypes.byref(weights),
                                         ctypes.byref(kv), _p(d_workspace), workspace_bytes,
                                         _p(stream), ctypes.byref(ctx)))
    return ctx


def ssd_create_static(dims: ssd_dims, weights: ssd_weights, kv: ssd_kv, stream) -> c_void_p:
    """ssd_create with the library's fixed per-device array as the workspace (no allocation)."""
    ctx = c_void_p()
    _check("ssd_create_static", _lib.ssd_create_static(ctypes.byref(dims), ctypes.byref(weights),
                                                       ctypes.byref(kv), _p(stream),
                                                       ctypes.byref(ctx)))
    return ctx


SSD_STATIC_SCRATCH_BYTES = 64 << 20


def ssd_prefill(ctx, B, P, d_prompt, d_visual, d_pending, d_logits=None):
    _check("ssd_prefill", _lib.ssd_prefill(ctx, B, P, _p(d_prompt), _p(d_visual), _p(d_pending),
                                           _p(d_logits)))


def ssd_draft(ctx, B, gamma, d_pending, d_draft, d_draft_logits=None):
    _check("ssd_draft", _lib.ssd_draft(ctx, B, gamma, _p(d_pending), _p(d_draft),
                                       _p(d_draft_logits)))


def ssd_verify(ctx, B, gamma, d_pending, d_draft, reuse_hidden, d_target, d_logits=None):
    _check("ssd_verify", _lib.ssd_verify(ctx, B, gamma, _p(d_pending), _p(d_draft),
                                         int(reuse_hidden), _p(d_target), _p(d_logits)))


def ssd_accept(ctx, B, gamma, d_draft, d_target, d_pending, d_out=None, d_accept_len=None,
               d_active=None):
    _check("ssd_accept", _lib.ssd_accept(ctx, B, gamma, _p(d_draft), _p(d_target), _p(d_pending),
                                         _p(d_out), _p(d_accept_len), _p(d_active)))


def ssd_draft_sample(ctx, B, gamma, d_pending, d_u, temperature, d_draft, d_draft_logits):
    _check("ssd_draft_sample", _lib.ssd_draft_sample(ctx, B, gamma, _p(d_pending), _p(d_u),
                                                     float(temperature), _p(d_draft),
                                                     _p(d_draft_logits)))


def ssd_accept_sample(ctx, B, gamma, d_draft, d_draft_logits, d_target_logits, d_u, temperature,
                      d_pending, d_out=None, d_accept_len=None, d_active=None):
    _check("ssd_accept_sample", _lib.ssd_accept_sample(
        ctx, B, gamma, _p(d_draft), _p(d_draft_logits), _p(d_target_logits), _p(d_u),
        float(temperature), _p(d_pending), _p(d_out), _p(d_accept_len), _p(d_active)))


def ssd_generate(ctx, B, P, d_prompt, d_visual, T, gamma, mode, reuse_hidden, d_tokens):
    stats = (c_int64 * 3)()
    _check("ssd_generate", _lib.ssd_generate(ctx, B, P, _p(d_prompt), _p(d_visual), T, gamma,
                                             mode, int(reuse_hidden), _p(d_tokens), stats))
    return {"rounds": int(stats[0]), "accepted": int(stats[1]), "drafted": int(stats[2])}


def ssd_draft_confident(ctx, B, gamma, threshold, d_pending, d_active, d_draft, d_ndraft,
                        d_conf=None, d_draft_logits=None) -> int:
    """Confidence-stopped drafting; returns the draft steps run."""
    steps = c_int(0)
    _check("ssd_draft_confident", _lib.ssd_draft_confident(
        ctx, B, gamma, float(threshold), _p(d_pending), _p(d_active), _p(d_draft), _p(d_ndraft),
        _p(d_conf), _p(d_draft_logits), ctypes.byref(steps)))
    return int(steps.value)


def ssd_accept_counts(ctx, B, gamma, d_draft, d_ndraft, d_target, d_pending, d_out=None,
                      d_accept_len=None, d_active=None):
    _check("ssd_accept_counts", _lib.ssd_accept_counts(
        ctx, B, gamma, _p(d_draft), _p(d_ndraft), _p(d_target), _p(d_pending), _p(d_out),
        _p(d_accept_len), _p(d_active)))


def ssd_generate_confident(ctx, B, P, d_prompt, d_visual, T, gamma, threshold, reuse_hidden,
                           d_tokens):
    stats = (c_int64 * 3)()
    _check("ssd_generate_confident", _lib.ssd_generate_confident(
        ctx, B, P, _p(d_prompt), _p(d_visual), T, gamma, float(threshold), int(reuse_hidden),
        _p(d_tokens), stats))
    return {"rounds": int(stats[0]), "accepted": int(stats[1]), "drafted": int(stats[2])}


def ssd_dynamic_gamma(t: int, d0: int, n_max: int) -> int:
    return int(_lib.ssd_dynamic_gamma(int(t), int(d0), int(n_max)))


def ssd_set_graphs(ctx, enable: bool):
    _check("ssd_set_graphs", _lib.ssd_set_graphs(ctx, int(bool(enable))))


def ssd_set_hidden_export(ctx, d_phi, d_xk, d_xl):
    _check("ssd_set_hidden_export", _lib.ssd_set_hidden_export(ctx, _p(d_phi), _p(d_xk), _p(d_xl)))


def ssd_profile_enable(ctx, enable: bool):
    _check("ssd_profile_enable", _lib.ssd_profile_enable(ctx, int(bool(enable))))


def ssd_profile_read(ctx):
    """(launches, seconds, bytes) of the profiled kernel since the previous read."""
    n, sec, by = c_int64(0), ctypes.c_double(0), ctypes.c_double(0)
    _check("ssd_profile_read", _lib.ssd_profile_read(ctx, ctypes.byref(n), ctypes.byref(sec),
                                                     ctypes.byref(by)))
    return int(n.value), float(sec.value), float(by.value)


def ssd_read_bandwidth(d_buf, nbytes: int, d_out, reps: int, stream) -> float:
    """Best GB/s of a read-only stream over nbytes of device memory (measurement utility)."""
    g = ctypes.c_double(0)
    _check("ssd_read_bandwidth", _lib.ssd_read_bandwidth(_p(d_buf), int(nbytes), _p(d_out),
                                                         int(reps), _p(stream), ctypes.byref(g)))
    return float(g.value)


def ssd_sync_status(ctx):
    """Returns (return code, device status bits) without raising on SSD_ERR_DEVICE."""
    st = c_int32(0)
    rc = _lib.ssd_sync_status(ctx, ctypes.byref(st))
    if rc not in (SSD_OK, SSD_ERR_DEVICE):
        raise SSDError("ssd_sync_status", rc)
    return rc, int(st.value)


def ssd_destroy(ctx):
    _lib.ssd_destroy(ctx)
