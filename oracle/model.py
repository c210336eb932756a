"""The decoder, the imitation network and the shared LM head, float64, position by position.

Paper (Sec. "SSD Setup for VLMs"): the decoder embeds token ids to x_0, each layer updates
x_{l+1} = x_l + f_l(x_l), and an LM head maps x_L to logits o_L = g(x_L).  The encoder output
z = E(I, T0) is an input of the decoder.  Sec. "Self-Speculative Decoding": the draft model is
the first n layers; Sec. "Methodology" (deep representation imitation): the imitation network I
maps the n-th layer output x_n to x_I, and the draft's logits are g(I(x_n)) with the same head g.

Readings used where the paper is silent (each listed in the design doc):
  * g = final RMSNorm followed by the (untied) output matrix.
  * T5 block: RMSNorm -> self-attention with a learned relative-position bias (32 buckets,
    max distance 128, one table shared by all layers, no 1/sqrt(dh)) -> RMSNorm ->
    cross-attention to z (no mask, no bias, no scale) -> RMSNorm -> gated-GELU(tanh) FFN.
    RMSNorm eps 1e-6.  The decoder's own sequence is the prompt; z is the cross-attention memory.
  * LLaMA block: RMSNorm(eps 1e-5) -> causal self-attention with half-split rotary embedding
    (theta 10000) and 1/sqrt(dh) scale -> RMSNorm -> SwiGLU FFN.  The visual tokens are the first
    n_visual positions' x_0 (no projector); the prompt's embeddings follow.
  * Imitation network: two fully connected layers and a LayerNorm, hidden width = model width:
    I(x) = x + W2 gelu_tanh(W1 LN(x) + b1) + b2 (pre-norm, residual; LN eps 1e-5).  The residual can
    be switched off (``in_residual=False``) to get the literal two-layer form.

Every position runs through the same code whether it is prefilled, drafted, verified or decoded
greedily; a block of several positions is only used for prefill.  The KV cache is a plain array
per layer indexed by absolute position; ``seq_len`` counts valid positions.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np

from . import ops


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


@dataclass
class State:
    """Decode state of one sequence."""

    K: np.ndarray  # [L, capacity, H, dh]
    V: np.ndarray
    XK: Optional[np.ndarray]  # [L, n_visual, H, dh] cross-attention keys (T5)
    XV: Optional[np.ndarray]
    seq_len: int = 0


class Decoder:
    """Synthetic VLM language decoder; ``weights`` is the dict made by ``synth.make_weights``."""

    def __init__(self, shape, weights: Dict, draft_layers: int, in_residual: Optional[bool] = None):
        self.shape = shape
        self.k = int(draft_layers)
        if not 1 <= self.k <= shape.n_layers:
            raise ValueError("draft depth must lie in [1, n_layers]")
        self.in_residual = shape.in_residual if in_residual is None else bool(in_residual)
        self.g = {n: _f64(a) for n, a in weights.items() if n != "layers"}
        self.layers: List[Dict[str, np.ndarray]] = [
            {n: _f64(a) for n, a in lw.items()} for lw in weights["layers"]]
        self.t5 = shape.arch == "t5"
        self.H, self.dh = shape.n_heads, shape.d_head
        self.scale = 1.0 if self.t5 else 1.0 / math.sqrt(shape.d_head)

    # ---- state ------------------------------------------------------------------------------
    def new_state(self, capacity: int) -> State:
        L, H, dh = self.shape.n_layers, self.H, self.dh
        K = np.zeros((L, capacity, H, dh))
        V = np.zeros((L, capacity, H, dh))
        if self.t5:
            nv = self.shape.n_visual
            return State(K, V, np.zeros((L, nv, H, dh)), np.zeros((L, nv, H, dh)))
        return State(K, V, None, None)

    def set_visual(self, st: State, z: np.ndarray) -> None:
        """T5: project the visual tokens z [n_visual, d] to each layer's cross-attention K and V."""
        if not self.t5:
            return
        z = _f64(z)
        for l, lw in enumerate(self.layers):
            st.XK[l] = (z @ lw["xk"].T).reshape(-1, self.H, self.dh)
            st.XV[l] = (z @ lw["xv"].T).reshape(-1, self.H, self.dh)

    # ---- one decoder layer over a block of consecutive positions ---------------------------
    def self_bias(self, p: int, n_keys: int) -> Optional[np.ndarray]:
        if not self.t5:
            return None
        rb = self.g["rel_bias"]  # [buckets, H]
        b = [ops.relative_bucket(p - j, self.shape.rel_buckets, self.shape.rel_max_dist)
             for j in range(n_keys)]
        return rb[b].T  # [H, n_keys]

    def layer(self, l: int, x: np.ndarray, positions: List[int], st: State) -> np.ndarray:
        lw, sh = self.layers[l], self.shape
        H, dh, eps = self.H, self.dh, sh.norm_eps
        M = x.shape[0]
        # self-attention
        h = ops.rms_norm(x, lw["attn_norm"], eps)
        q = (h @ lw["wq"].T).reshape(M, H, dh)
        k = (h @ lw["wk"].T).reshape(M, H, dh)
        v = (h @ lw["wv"].T).reshape(M, H, dh)
        if not self.t5:
            q = np.stack([ops.rope(q[i], p, sh.rope_theta) for i, p in enumerate(positions)])
            k = np.stack([ops.rope(k[i], p, sh.rope_theta) for i, p in enumerate(positions)])
        for i, p in enumerate(positions):
            st.K[l, p] = k[i]
            st.V[l, p] = v[i]
        o = np.empty((M, H, dh))
        for i, p in enumerate(positions):
            o[i] = ops.attend(q[i], st.K[l, :p + 1], st.V[l, :p + 1], self.self_bias(p, p + 1),
                              self.scale)
        x = x + o.reshape(M, H * dh) @ lw["wo"].T
        # cross-attention to the visual tokens (T5)
        if self.t5:
            h = ops.rms_norm(x, lw["xattn_norm"], eps)
            q = (h @ lw["xq"].T).reshape(M, H, dh)
            for i in range(M):
                o[i] = ops.attend(q[i], st.XK[l], st.XV[l], None, 1.0)
            x = x + o.reshape(M, H * dh) @ lw["xo"].T
        # feed-forward
        h = ops.rms_norm(x, lw["ffn_norm"], eps)
        act = ops.gelu_tanh if self.t5 else ops.silu
        a = act(h @ lw["w_gate"].T) * (h @ lw["w_up"].T)
        return x + a @ lw["w_down"].T

    def run_layers(self, x: np.ndarray, positions: List[int], st: State, l0: int, l1: int):
        for l in range(l0, l1):
            x = self.layer(l, x, positions, st)
        return x

    # ---- embedding, heads ------------------------------------------------------------------
    def embed(self, tokens) -> np.ndarray:
        return self.g["embed"][np.asarray(tokens, dtype=np.int64)]

    def head(self, x: np.ndarray) -> np.ndarray:
        """g: final RMSNorm then the output matrix -> logits over the vocabulary."""
        return ops.rms_norm(x, self.g["final_norm"], self.shape.norm_eps) @ self.g["lm_head"].T

    def imitation(self, x: np.ndarray) -> np.ndarray:
        """I(x_n): LayerNorm -> FC1 (+b1) -> GELU(tanh) -> FC2 (+b2), plus x when residual."""
        g = self.g
        h = ops.layer_norm(x, g["in_ln_w"], g["in_ln_b"], self.shape.ln_eps)
        u = ops.gelu_tanh(h @ g["in_w1"].T + g["in_b1"])
        y = u @ g["in_w2"].T + g["in_b2"]
        return x + y if self.in_residual else y

    # ---- the three position-level computations of the decode loop ---------------------------
    def full_step(self, st: State, token: int, pos: int):
        """Full decoder at one position: returns (logits g(x_L), x_k)."""
        x = self.embed([token])
        xk = None
        for l in range(self.shape.n_layers):
            x = self.layer(l, x, [pos], st)
            if l == self.k - 1:
                xk = x[0].copy()
        return self.head(x)[0], xk

    def draft_step(self, st: State, token: int, pos: int, use_imitation: bool = True):
        """Draft model at one position: layers 1..k, then I, then g.  Returns (logits, x_k)."""
        x = self.run_layers(self.embed([token]), [pos], st, 0, self.k)
        xk = x[0].copy()
        xi = self.imitation(x) if use_imitation else x
        return self.head(xi)[0], xk
