"""Decoder shapes and decode workloads used throughout the repository.

These are synthetic stand-ins for the paper's models: the paper evaluates
BLIP-2 with a FlanT5-xl decoder and LLaVA-1.5-7B (LLaMA-2 decoder) on COCO,
NoCaps, VisDial, MM-Vet and LLaVA-Wild (Sec. "Experiments"); none of those
weights or datasets are used here.  Each workload instead draws a random-init
decoder of the same shape, N(0,1) visual tokens standing in for the encoder
output z = E(I, T0) (Sec. "SSD Setup for VLMs"), and uniform prompt ids.

The decoder contract itself is only sketched in the paper (x_{l+1} = x_l +
f_l(x_l), o = g(x_L)); the layer internals follow the public T5-v1.1 /
LLaMA-2 definitions and are spelled out in ``oracle/model.py``.

This module holds no arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class Shape:
    """Architecture of one synthetic decoder."""

    name: str
    arch: str  # "t5": pre-norm T5-v1.1 decoder block with cross-attention; "llama": LLaMA-2 block
    n_layers: int
    d_model: int
    n_heads: int
    d_head: int
    d_ff: int
    vocab: int
    n_visual: int  # visual tokens (T5: cross-attention memory; LLaMA: KV prefix rows)
    dtype: str  # "f32" or "bf16": storage precision of every generated tensor
    rel_buckets: int = 32
    rel_max_dist: int = 128
    rope_theta: float = 10000.0
    in_hidden: int = 0  # width of the imitation network's hidden layer; 0 means d_model
    in_residual: bool = True

    @property
    def norm_eps(self) -> float:
        return 1e-6 if self.arch == "t5" else 1e-5

    @property
    def ln_eps(self) -> float:
        return 1e-5

    @property
    def hd(self) -> int:
        return self.n_heads * self.d_head

    @property
    def in_width(self) -> int:
        return self.in_hidden if self.in_hidden else self.d_model

    def prefix_len(self) -> int:
        """Positions that precede the prompt in the decoder's own sequence."""
        return self.n_visual if self.arch == "llama" else 0


@dataclass(frozen=True)
class Workload:
    """One decode job: a shape, a batch of prompts and the speculative settings."""

    name: str
    shape: Shape
    batch: int
    prompt_len: int
    draft_layers: int  # k: the draft is layers 1..k + imitation network + shared LM head
    gamma: int  # draft tokens per round
    new_tokens: int  # T: tokens emitted per sequence (the first comes from prefill)
    deep_scale: float  # s: multiplies the residual-branch output projections of layers k+1..L
    scale_boundary: int = -1  # first scaled layer (0-based); -1 means draft_layers
    seeds: Tuple[int, ...] = (0, 1, 2)

    @property
    def boundary(self) -> int:
        return self.draft_layers if self.scale_boundary < 0 else self.scale_boundary

    def max_seq(self) -> int:
        """KV positions one sequence can need: prefix + prompt + T + a full verify chunk."""
        return self.shape.prefix_len() + self.prompt_len + self.new_tokens + self.gamma + 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# ---- shapes --------------------------------------------------------------------------------

TINY_T5 = Shape("tiny-t5", "t5", n_layers=4, d_model=256, n_heads=4, d_head=64, d_ff=1024,
                vocab=1024, n_visual=32, dtype="f32")
FLANT5_BASE = Shape("flant5-base", "t5", n_layers=12, d_model=768, n_heads=12, d_head=64,
                    d_ff=2048, vocab=32128, n_visual=32, dtype="bf16")
FLANT5_XL = Shape("flant5-xl", "t5", n_layers=24, d_model=2048, n_heads=32, d_head=64,
                  d_ff=5120, vocab=32128, n_visual=32, dtype="bf16")
LLAVA_7B = Shape("llava-1.5-7b", "llama", n_layers=32, d_model=4096, n_heads=32, d_head=128,
                 d_ff=11008, vocab=32000, n_visual=576, dtype="bf16")

# Shrunk copies with the same structure, small enough for the CPU oracle in seconds.
SMALL_T5_BF16 = Shape("small-t5-bf16", "t5", n_layers=6, d_model=128, n_heads=2, d_head=64,
                      d_ff=320, vocab=2000, n_visual=8, dtype="bf16")
SMALL_LLAMA_BF16 = Shape("small-llama-bf16", "llama", n_layers=6, d_model=256, n_heads=2,
                         d_head=128, d_ff=704, vocab=2000, n_visual=24, dtype="bf16")
SMALL_LLAMA_F32 = replace(SMALL_LLAMA_BF16, name="small-llama-f32", dtype="f32")

# ---- workloads ------------------------------------------------------------------------------
# Deep-layer scale s: the configs ask for deep layers damped so that acceptance is
# non-trivial with random weights; the values for the larger shapes were chosen with
# oracle/tune_scale.py (a sweep over s on the CPU oracle's own acceptance).

C1 = Workload("c1-tiny-t5-f32", TINY_T5, batch=1, prompt_len=8, draft_layers=1, gamma=4,
              new_tokens=32, deep_scale=0.1)
C2 = Workload("c2-flant5-base", FLANT5_BASE, batch=1, prompt_len=16, draft_layers=4, gamma=4,
              new_tokens=64, deep_scale=0.2)
C3 = Workload("c3-flant5-xl", FLANT5_XL, batch=1, prompt_len=8, draft_layers=6, gamma=5,
              new_tokens=128, deep_scale=0.04)  # oracle alpha 0.707 at seed 0 (tune_scale)
C5 = Workload("c5-llava-7b", LLAVA_7B, batch=1, prompt_len=32, draft_layers=8, gamma=5,
              new_tokens=256, deep_scale=0.02)  # oracle alpha 0.653 over 64 tokens, seed 0


def c4_points():
    """The FlanT5-xl sweep: batch x draft depth x gamma, one decoder (scaled at k=6)."""
    pts = []
    for b in (1, 8):
        for k in (4, 8, 12):
            for g in (2, 4, 8):
                pts.append(C3.with_(name=f"c4-b{b}-k{k}-g{g}", batch=b, draft_layers=k, gamma=g,
                                    scale_boundary=C3.draft_layers))
    return pts


# Small workloads for oracle self-tests and GPU parity at sizes the oracle finishes in seconds.
S1 = C1.with_(name="s1-tiny-t5-f32")
S_T5 = Workload("s-t5-bf16", SMALL_T5_BF16, batch=1, prompt_len=5, draft_layers=2, gamma=4,
                new_tokens=24, deep_scale=0.2)
S_LLAMA = Workload("s-llama-bf16", SMALL_LLAMA_BF16, batch=1, prompt_len=7, draft_layers=2,
                   gamma=3, new_tokens=24, deep_scale=0.2)
S_LLAMA_F32 = S_LLAMA.with_(name="s-llama-f32", shape=SMALL_LLAMA_F32)

ALL = {w.name: w for w in (C1, C2, C3, C5, S1, S_T5, S_LLAMA, S_LLAMA_F32)}
