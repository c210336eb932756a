"""Seeded synthetic tensors: decoder weights, visual tokens and prompt ids.

Every tensor has its own generator, seeded from (seed, layer, tensor id) through
numpy's SeedSequence and the SFC64 bit generator, so any tensor can be made on its
own, in any order, on any thread, with identical values.  In "bf16" shapes every
generated value is rounded once to bfloat16 (round to nearest, ties to even) and
handed out as float32 holding that bfloat16 value; in "f32" shapes values stay
float32.  Both the oracle and the device path take exactly these values.

Initialisation (synthetic; the paper's trained weights are not used):
  matrices and embeddings     N(0, 0.02)
  norm gains                  1 + N(0, 0.02)
  imitation-network biases    N(0, 0.02)   (also the LayerNorm shift)
  relative-position bias      N(0, 1)
  visual tokens               N(0, 1)
  prompt ids                  uniform over [0, vocab)
The residual-branch output projections (self-attention out, cross-attention out,
FFN down) of layers >= boundary, and the imitation network's second matrix, are
multiplied by the workload's deep scale s before rounding.

This module holds no arithmetic of the method.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
import os
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

from .configs import Shape, Workload

GLOBAL = 10_000
VISUAL = 20_000
PROMPT = 30_000
UNIFORM = 40_000

# tensor id, name, kind
_GLOBAL_TENSORS = [
    (1, "embed", "matrix"),
    (2, "lm_head", "matrix"),
    (3, "final_norm", "gain"),
    (4, "rel_bias", "relbias"),
    (5, "in_ln_w", "gain"),
    (6, "in_ln_b", "bias"),
    (7, "in_w1", "matrix"),
    (8, "in_b1", "bias"),
    (9, "in_w2", "matrix"),
    (10, "in_b2", "bias"),
]
_LAYER_TENSORS = [
    (20, "attn_norm", "gain"),
    (21, "wq", "matrix"),
    (22, "wk", "matrix"),
    (23, "wv", "matrix"),
    (24, "wo", "matrix"),
    (30, "xattn_norm", "gain"),
    (31, "xq", "matrix"),
    (32, "xk", "matrix"),
    (33, "xv", "matrix"),
    (34, "xo", "matrix"),
    (40, "ffn_norm", "gain"),
    (41, "w_gate", "matrix"),
    (42, "w_up", "matrix"),
    (43, "w_down", "matrix"),
]
_T5_ONLY = {"rel_bias", "xattn_norm", "xq", "xk", "xv", "xo"}
_SCALED = {"wo", "xo", "w_down"}


def tensor_shape(shape: Shape, name: str) -> Tuple[int, ...]:
    d, hd, f, v, h = shape.d_model, shape.hd, shape.d_ff, shape.vocab, shape.in_width
    return {
        "embed": (v, d), "lm_head": (v, d), "final_norm": (d,),
        "rel_bias": (shape.rel_buckets, shape.n_heads),
        "in_ln_w": (d,), "in_ln_b": (d,), "in_w1": (h, d), "in_b1": (h,),
        "in_w2": (d, h), "in_b2": (d,),
        "attn_norm": (d,), "wq": (hd, d), "wk": (hd, d), "wv": (hd, d), "wo": (d, hd),
        "xattn_norm": (d,), "xq": (hd, d), "xk": (hd, d), "xv": (hd, d), "xo": (d, hd),
        "ffn_norm": (d,), "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }[name]


def tensor_list(shape: Shape) -> List[Tuple[str, int, int, str]]:
    """(name, layer or -1, tensor id, kind) for every tensor of the decoder."""
    out = []
    for tid, name, kind in _GLOBAL_TENSORS:
        if name in _T5_ONLY and shape.arch != "t5":
            continue
        out.append((name, -1, tid, kind))
    for layer in range(shape.n_layers):
        for tid, name, kind in _LAYER_TENSORS:
            if name in _T5_ONLY and shape.arch != "t5":
                continue
            out.append((name, layer, tid, kind))
    return out


def _rng(seed: int, layer: int, tid: int) -> np.random.Generator:
    return np.random.Generator(np.random.SFC64(np.random.SeedSequence([seed, layer, tid])))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32. Finite inputs only."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).copy()
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


def make_tensor(shape: Shape, seed: int, name: str, layer: int, tid: int, kind: str,
                deep_scale: float = 1.0, boundary: int = 0) -> np.ndarray:
    dims = tensor_shape(shape, name)
    rng = _rng(seed, GLOBAL if layer < 0 else layer, tid)
    x = rng.standard_normal(dims, dtype=np.float32)
    if kind == "matrix" or kind == "bias":
        x *= np.float32(0.02)
    elif kind == "gain":
        x *= np.float32(0.02)
        x += np.float32(1.0)
    elif kind == "relbias":
        pass
    else:
        raise ValueError(kind)
    scaled = (name in _SCALED and layer >= boundary) or name == "in_w2"
    if scaled and deep_scale != 1.0:
        x *= np.float32(deep_scale)
    if shape.dtype == "bf16":
        x = round_to_bf16(x)
    return x


def make_weights(shape: Shape, seed: int, deep_scale: float, boundary: int,
                 sink: Optional[Callable[[str, int, np.ndarray], None]] = None,
                 threads: Optional[int] = None) -> Optional[Dict]:
    """All decoder tensors.  Returns {"name": arr, ..., "layers": [ {name: arr}, ... ]}
    or, when ``sink`` is given, passes each tensor to sink(name, layer, arr) and keeps none."""
    items = tensor_list(shape)
    threads = threads or min(16, len(os.sched_getaffinity(0)))
    out: Dict = {"layers": [dict() for _ in range(shape.n_layers)]}

    def job(it):
        name, layer, tid, kind = it
        return name, layer, make_tensor(shape, seed, name, layer, tid, kind, deep_scale, boundary)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        for name, layer, arr in ex.map(job, items):
            if sink is not None:
                sink(name, layer, arr)
            elif layer < 0:
                out[name] = arr
            else:
                out["layers"][layer][name] = arr
    return None if sink is not None else out


def workload_weights(wl: Workload, seed: int, **kw):
    return make_weights(wl.shape, seed, wl.deep_scale, wl.boundary, **kw)


def make_visual(shape: Shape, seed: int, batch: int) -> np.ndarray:
    """[batch, n_visual, d_model] visual tokens, N(0,1) (bf16-rounded in bf16 shapes)."""
    out = np.empty((batch, shape.n_visual, shape.d_model), dtype=np.float32)
    for b in range(batch):
        out[b] = _rng(seed, VISUAL + b, 0).standard_normal((shape.n_visual, shape.d_model),
                                                           dtype=np.float32)
    if shape.dtype == "bf16":
        out = round_to_bf16(out)
    return out


def make_prompts(shape: Shape, seed: int, batch: int, prompt_len: int) -> np.ndarray:
    """[batch, prompt_len] int32 token ids, uniform over the vocabulary."""
    out = np.empty((batch, prompt_len), dtype=np.int32)
    for b in range(batch):
        out[b] = _rng(seed, PROMPT + b, 0).integers(0, shape.vocab, prompt_len)
    return out


def make_uniforms(seed: int, batch: int, rounds: int, per_round: int) -> np.ndarray:
    """[batch, rounds, per_round] float32 uniforms in [0, 1): the random draws of sampled
    decoding, an input to both the device path and the oracle."""
    out = np.empty((batch, rounds, per_round), dtype=np.float32)
    for b in range(batch):
        out[b] = _rng(seed, UNIFORM + b, 0).random((rounds, per_round), dtype=np.float32)
    return out
