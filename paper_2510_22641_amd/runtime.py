"""Device memory for one libssd context: weights, paged KV cache, page table, workspace.

PyTorch is used only to allocate device memory and to name the stream; every step of the decode
loop runs in libssd's kernels through the C ABI (``paper_2510_22641_amd.ssd``).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np
import torch

from . import ssd as abi


def _t(arr: np.ndarray, dtype, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(arr)).to(dtype).to(device)


@dataclass
class Capacity:
    max_batch: int
    max_gamma: int
    max_seq: int
    max_prompt: int
    page_size: int = 16
    spare_pages: int = 0  # pool pages beyond those the page table can reach at once


class DeviceDecoder:
    """A decoder resident in HBM plus its libssd context.

    ``shape`` is a ``synth.Shape``; tensors come either from a dict (``synth.make_weights``) or
    streamed through ``load(name, layer, array)`` before ``create()``.
    """

    MATRICES = {"embed", "lm_head", "in_w1", "in_w2", "wq", "wk", "wv", "wo", "xq", "xk", "xv",
                "xo", "w_gate", "w_up", "w_down"}

    def __init__(self, shape, draft_layers: int, cap: Capacity, device: str = "cuda",
                 kv_dtype: Optional[str] = None, page_seed: Optional[int] = None,
                 in_residual: Optional[bool] = None):
        self.shape = shape
        self.k = draft_layers
        self.cap = cap
        self.device = torch.device(device)
        self.wdtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        # KV cache in float32 by default: rounding cached keys and values to bf16 alone moves the
        # logits of the 12-layer FlanT5-base shape by about twice 2e-2 x their spread (T5
        # attention is unscaled and adds a unit-variance position bias); "bf16" is available
        kvd = kv_dtype or "f32"
        self.kvdtype = torch.bfloat16 if kvd == "bf16" else torch.float32
        self.page_seed = page_seed
        self.in_residual = shape.in_residual if in_residual is None else in_residual
        self.g: Dict[str, torch.Tensor] = {}
        self.layers = [dict() for _ in range(shape.n_layers)]
        self.ctx = None

    # ---- weights ---------------------------------------------------------------------------
    def load(self, name: str, layer: int, arr: np.ndarray) -> None:
        dt = self.wdtype if name in self.MATRICES else torch.float32
        t = _t(arr, dt, self.device)
        if layer < 0:
            self.g[name] = t
        else:
            self.layers[layer][name] = t

    def load_dict(self, w: Dict) -> "DeviceDecoder":
        for n, a in w.items():
            if n != "layers":
                self.load(n, -1, a)
        for l, lw in enumerate(w["layers"]):
            for n, a in lw.items():
                self.load(n, l, a)
        return self

    # ---- context ---------------------------------------------------------------------------
    def dims(self) -> abi.ssd_dims:
        sh, cap = self.shape, self.cap
        d = abi.ssd_dims()
        d.arch = abi.SSD_ARCH_T5 if sh.arch == "t5" else abi.SSD_ARCH_LLAMA
        d.n_layers, d.d_model, d.n_heads, d.d_head = sh.n_layers, sh.d_model, sh.n_heads, sh.d_head
        d.d_ff, d.vocab, d.n_visual = sh.d_ff, sh.vocab, sh.n_visual
        d.rel_buckets, d.rel_max_dist = sh.rel_buckets, sh.rel_max_dist
        d.rope_theta, d.norm_eps, d.ln_eps = sh.rope_theta, sh.norm_eps, sh.ln_eps
        d.wdtype = abi.SSD_BF16 if self.wdtype == torch.bfloat16 else abi.SSD_F32
        d.kvdtype = abi.SSD_BF16 if self.kvdtype == torch.bfloat16 else abi.SSD_F32
        d.draft_layers, d.in_hidden, d.in_residual = self.k, sh.in_width, int(self.in_residual)
        d.max_batch, d.max_gamma, d.max_seq = cap.max_batch, cap.max_gamma, cap.max_seq
        d.max_prompt, d.page_size = cap.max_prompt, cap.page_size
        d.max_pages = (cap.max_seq + cap.page_size - 1) // cap.page_size
        return d

    def create(self, static: bool = False) -> "DeviceDecoder":
        """Allocate the KV cache and the workspace, and create the context; with static=True the
        context is made by ssd_create_static and uses the library's own fixed device array as
        its workspace (no workspace tensor is allocated)."""
        sh, cap, dev = self.shape, self.cap, self.device
        dims = self.dims()
        self._dims = dims
        H, dh, L = sh.n_heads, sh.d_head, sh.n_layers
        n_table = cap.max_batch * dims.max_pages
        n_pages = n_table + cap.spare_pages
        self.k_pool = torch.zeros((L, n_pages, H, cap.page_size, dh), dtype=self.kvdtype, device=dev)
        self.v_pool = torch.zeros_like(self.k_pool)
        pages = np.arange(n_pages, dtype=np.int32)
        if self.page_seed is not None:  # scatter sequences over the pool to exercise the table
            pages = np.random.default_rng(self.page_seed).permutation(pages).astype(np.int32)
        pages = pages[:n_table]
        self.page_table = torch.from_numpy(pages.reshape(cap.max_batch, dims.max_pages)).to(dev)
        self.seq_len = torch.zeros(cap.max_batch, dtype=torch.int32, device=dev)
        if sh.arch == "t5":
            self.xk = torch.zeros((L, cap.max_batch, H, sh.n_visual, dh), dtype=self.kvdtype, device=dev)
            self.xv = torch.zeros_like(self.xk)
        else:
            self.xk = self.xv = None
        nbytes = abi.ssd_workspace_bytes(dims)
        if nbytes == 0:
            raise ValueError("libssd rejected the dimensions")
        if not static:
            self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
            ws_ptr = (self.workspace.data_ptr() + 255) // 256 * 256

        self._layer_structs = (abi.ssd_layer_weights * L)()
        for l in range(L):
            ls = self._layer_structs[l]
            for f in abi.LAYER_FIELDS:
                t = self.layers[l].get(f)
                setattr(ls, f, t.data_ptr() if t is not None else None)
        w = abi.ssd_weights()
        for f in abi.GLOBAL_FIELDS:
            t = self.g.get(f)
            setattr(w, f, t.data_ptr() if t is not None else None)
        w.layers = ctypes.cast(self._layer_structs, ctypes.POINTER(abi.ssd_layer_weights))
        kv = abi.ssd_kv()
        kv.k_pool, kv.v_pool, kv.n_pages = self.k_pool.data_ptr(), self.v_pool.data_ptr(), n_pages
        kv.page_table, kv.seq_len = self.page_table.data_ptr(), self.seq_len.data_ptr()
        kv.xk = self.xk.data_ptr() if self.xk is not None else None
        kv.xv = self.xv.data_ptr() if self.xv is not None else None
        # a stream of its own (default priority): the null stream cannot be captured into graphs
        self.stream = torch.cuda.Stream(dev)
        torch.cuda.current_stream(dev).synchronize()
        if static:
            self.ctx = abi.ssd_create_static(dims, w, kv, self.stream.cuda_stream)
        else:
            self.ctx = abi.ssd_create(dims, w, kv, ws_ptr, nbytes, self.stream.cuda_stream)
        self._w_struct, self._kv_struct = w, kv
        return self

    def close(self):
        if self.ctx is not None:
            abi.ssd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- the four steps and the loop ---------------------------------------------------------
    def ivec(self, *shape) -> torch.Tensor:
        return torch.zeros(shape, dtype=torch.int32, device=self.device)

    def fvec(self, *shape) -> torch.Tensor:
        return torch.zeros(shape, dtype=torch.float32, device=self.device)

    def buf(self, name: str, shape, dtype=torch.int32) -> torch.Tensor:
        """A device buffer reused across calls (stable pointers keep captured graphs valid)."""
        if not hasattr(self, "_bufs"):
            self._bufs = {}
        key = (name, tuple(shape), dtype)
        t = self._bufs.get(key)
        if t is None:
            t = self._bufs[key] = torch.zeros(tuple(shape), dtype=dtype, device=self.device)
        return t

    def _call(self, fn, *args):
        """Run a library call on the context's stream, ordered after and before torch's stream."""
        cur = torch.cuda.current_stream(self.device)
        self.stream.wait_stream(cur)
        out = fn(*args)
        cur.wait_stream(self.stream)
        return out

    def upload_inputs(self, prompts: np.ndarray, visual: np.ndarray):
        p = torch.from_numpy(np.ascontiguousarray(prompts, dtype=np.int32)).to(self.device)
        v = _t(visual, self.wdtype, self.device)
        return p, v

    def prefill(self, prompt: torch.Tensor, visual: torch.Tensor, logits: bool = False):
        """Returns (pending [B], logits [B, V] or None); pending is a reused buffer."""
        B, P = prompt.shape
        pending = self.buf("pending", (B,))
        lg = self.buf("prefill_logits", (B, self.shape.vocab), torch.float32) if logits else None
        self._call(abi.ssd_prefill, self.ctx, B, P, prompt, visual, pending, lg)
        return pending, lg

    def draft(self, pending: torch.Tensor, gamma: int, logits: bool = False):
        B = pending.shape[0]
        d = self.buf("draft", (B, gamma))
        lg = self.buf("draft_logits", (B, gamma, self.shape.vocab), torch.float32) if logits else None
        self._call(abi.ssd_draft, self.ctx, B, gamma, pending, d, lg)
        return d, lg

    def verify(self, pending, draft, gamma: int, reuse: bool = False, logits: bool = False):
        B = pending.shape[0]
        t = self.buf("target", (B, gamma + 1))
        lg = self.buf("verify_logits", (B, gamma + 1, self.shape.vocab), torch.float32) if logits else None
        self._call(abi.ssd_verify, self.ctx, B, gamma, pending, draft, reuse, t, lg)
        return t, lg

    def accept(self, draft, target, pending, gamma: int, active=None):
        """Advances seq_len and overwrites ``pending`` in place; returns (out, accept_len)."""
        B = pending.shape[0]
        out = self.buf("accept_out", (B, gamma + 1))
        alen = self.buf("accept_len", (B,))
        self._call(abi.ssd_accept, self.ctx, B, gamma, draft, target, pending, out, alen, active)
        return out, alen

    def draft_confident(self, pending: torch.Tensor, gamma: int, threshold: float, active=None,
                        logits: bool = False):
        """Confidence-stopped drafting; returns (draft [B, steps], ndraft [B], conf [B, gamma],
        draft logits [B, gamma, V] or None, steps)."""
        B = pending.shape[0]
        d = self.buf("draft_conf", (B * gamma,))
        nd = self.buf("ndraft", (B,))
        cf = self.buf("conf", (B, gamma), torch.float32)
        lg = self.buf("draft_logits", (B, gamma, self.shape.vocab), torch.float32) if logits else None
        steps = self._call(abi.ssd_draft_confident, self.ctx, B, gamma, threshold, pending, active,
                           d, nd, cf, lg)
        return d[:B * steps].view(B, steps), nd, cf, lg, steps

    def accept_counts(self, draft, ndraft, target, pending, gamma: int, active=None):
        B = pending.shape[0]
        out = self.buf("accept_out", (B, gamma + 1))
        alen = self.buf("accept_len", (B,))
        self._call(abi.ssd_accept_counts, self.ctx, B, gamma, draft, ndraft, target, pending, out,
                   alen, active)
        return out, alen

    def generate_confident(self, prompt, visual, T: int, gamma: int, threshold: float,
                           reuse: bool = True):
        B, P = prompt.shape
        tokens = self.ivec(B, T)
        stats = self._call(abi.ssd_generate_confident, self.ctx, B, P, prompt, visual, T, gamma,
                           threshold, reuse, tokens)
        return tokens, stats

    def draft_sample(self, pending: torch.Tensor, gamma: int, u: torch.Tensor, temperature: float):
        """Sampled drafts (u [B, gamma] float32 uniforms); returns (draft, draft logits)."""
        B = pending.shape[0]
        d = self.buf("draft", (B, gamma))
        lg = self.buf("draft_logits", (B, gamma, self.shape.vocab), torch.float32)
        self._call(abi.ssd_draft_sample, self.ctx, B, gamma, pending, u, temperature, d, lg)
        return d, lg

    def accept_sample(self, draft, draft_logits, target_logits, u: torch.Tensor,
                      temperature: float, pending, gamma: int, active=None):
        """Speculative-sampling acceptance (u [B, gamma + 1]); overwrites ``pending`` in place and
        returns (out, accept_len)."""
        B = pending.shape[0]
        out = self.buf("accept_out", (B, gamma + 1))
        alen = self.buf("accept_len", (B,))
        self._call(abi.ssd_accept_sample, self.ctx, B, gamma, draft, draft_logits, target_logits,
                   u, temperature, pending, out, alen, active)
        return out, alen

    def generate(self, prompt, visual, T: int, gamma: int, speculative: bool = True,
                 reuse: bool = True, dynamic: bool = False):
        """ssd_generate; with dynamic=True gamma is d(0) of the context-length schedule."""
        B, P = prompt.shape
        tokens = self.ivec(B, T)
        mode = abi.SSD_MODE_GREEDY if not speculative else (
            abi.SSD_MODE_SPECULATIVE_DYNAMIC if dynamic else abi.SSD_MODE_SPECULATIVE)
        stats = self._call(abi.ssd_generate, self.ctx, B, P, prompt, visual, T, gamma, mode, reuse, tokens)
        return tokens, stats

    def set_graphs(self, enable: bool):
        abi.ssd_set_graphs(self.ctx, enable)

    def sync_status(self):
        torch.cuda.current_stream(self.device).synchronize()
        return abi.ssd_sync_status(self.ctx)


def from_workload(wl, seed: int, device: str = "cuda", max_batch: Optional[int] = None,
                  max_gamma: Optional[int] = None, extra_seq: int = 0, page_seed: Optional[int] = None,
                  kv_dtype: Optional[str] = None, weights: Optional[Dict] = None,
                  draft_layers: Optional[int] = None, spare_pages: int = 0,
                  static: bool = False) -> DeviceDecoder:
    """Build a DeviceDecoder for a synth workload, streaming its seeded tensors to the device
    (static=True: the context takes the library's fixed workspace, ssd_create_static)."""
    import synth
    sh = wl.shape
    mg = max_gamma if max_gamma is not None else max(wl.gamma, 1)
    cap = Capacity(max_batch=max_batch or wl.batch, max_gamma=mg,
                   max_seq=sh.prefix_len() + wl.prompt_len + wl.new_tokens + mg + 1 + extra_seq,
                   max_prompt=wl.prompt_len, spare_pages=spare_pages)
    dd = DeviceDecoder(sh, draft_layers or wl.draft_layers, cap, device=device, kv_dtype=kv_dtype,
                       page_seed=page_seed)
    if weights is not None:
        dd.load_dict(weights)
    else:
        synth.make_weights(sh, seed, wl.deep_scale, wl.boundary, sink=dd.load)
    return dd.create(static=static)
