"""Fit the imitation network's output layer on the decoder's own hidden states.

The paper trains the imitation network I (two fully connected layers and a layer norm) so that
I(x_k), computed from the draft's layer-k state, imitates the full model's deep representation
(cosine-similarity and distillation losses on captioning data; Sec. "Deep Representation
Imitation").  The workloads here are random-init decoders with no data, so this module fits I's
second layer in closed form instead, a data-free stand-in for that training:

  * the decoder's own decoding supplies, for every drafted position, I's hidden features
    phi = gelu(W1 LN(x_k) + b1) and the layer-k row x_k (both computed by the device in the draft
    step) and the full model's last residual row x_L at the same position (from the verify);
  * W2, b2 minimise the ridge-regularised squared error of x_k + W2 phi + b2 against x_L (with the
    residual form of I; the target is x_L itself for the literal two-layer form);
  * W1, b1 and the layer norm keep their values.

Collection runs through the C ABI (ssd_set_hidden_export); the regression is a host-side float64
solve of an in_hidden x in_hidden system; nothing here is on the decode path.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np
import torch

from . import ssd as abi


def collect(dd, prompt_t: torch.Tensor, visual_t: torch.Tensor, T: int, gamma: int,
            reuse: bool = True) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Decode one sequence (prompt_t [1, P], visual_t [1, Nv, d]) for T tokens speculatively and
    return the rows (phi [N, in_hidden], x_k [N, d], x_L [N, d]) of every drafted position."""
    assert prompt_t.shape[0] == 1, "one sequence per call"
    sh = dd.shape
    H = sh.in_width
    dev = prompt_t.device
    phi = torch.zeros(1, gamma, H, dtype=torch.float32, device=dev)
    xk = torch.zeros(1, gamma, sh.d_model, dtype=torch.float32, device=dev)
    xl = torch.zeros(1, gamma + 1, sh.d_model, dtype=torch.float32, device=dev)
    abi.ssd_set_hidden_export(dd.ctx, phi, xk, xl)
    rows_p, rows_k, rows_l = [], [], []
    try:
        pending, _ = dd.prefill(prompt_t, visual_t)
        emitted = 1
        while emitted < T:
            d, _ = dd.draft(pending, gamma)
            p_np, k_np = phi[0].cpu().numpy().copy(), xk[0].cpu().numpy().copy()
            t, _ = dd.verify(pending, d, gamma, reuse=reuse)
            l_np = xl[0, :gamma].cpu().numpy().copy()
            _, alen = dd.accept(d, t, pending, gamma)
            rows_p.append(p_np)
            rows_k.append(k_np)
            rows_l.append(l_np)
            emitted += int(alen[0]) + 1
    finally:
        abi.ssd_set_hidden_export(dd.ctx, None, None, None)
    return (np.concatenate(rows_p).astype(np.float64), np.concatenate(rows_k).astype(np.float64),
            np.concatenate(rows_l).astype(np.float64))


def fit(phi: np.ndarray, xk: np.ndarray, xl: np.ndarray, residual: bool = True,
        ridge: float = 1e-3) -> Tuple[np.ndarray, np.ndarray]:
    """Least squares for I's second layer: W2 [d, in_hidden], b2 [d] minimising
    sum_n |(x_k + ) W2 phi_n + b2 - x_L|^2 + lam |W2|^2, lam = ridge * trace(Pc^T Pc) / in_hidden
    with Pc the centred features (the bias absorbs the means)."""
    y = xl - xk if residual else xl
    mp, my = phi.mean(axis=0), y.mean(axis=0)
    pc, yc = phi - mp, y - my
    gram = pc.T @ pc
    lam = ridge * float(np.trace(gram)) / gram.shape[0]
    w2t = np.linalg.solve(gram + lam * np.eye(gram.shape[0]), pc.T @ yc)  # [in_hidden, d]
    w2 = w2t.T
    b2 = my - w2 @ mp
    return w2, b2


def mse(phi: np.ndarray, xk: np.ndarray, xl: np.ndarray, w2, b2, residual: bool = True) -> float:
    """Mean squared imitation error of I's output rows against x_L."""
    out = phi @ np.asarray(w2, np.float64).T + np.asarray(b2, np.float64)
    if residual:
        out = out + xk
    return float(np.mean(np.square(out - xl)))


def fit_validated(phi, xk, xl, w2_now, b2_now, residual: bool = True,
                  ridges=(1e-3, 1e-2, 1e-1, 1.0, 10.0, 100.0, 1000.0), val_frac: float = 0.2,
                  seed: int = 0):
    """fit() with the ridge chosen on held-out rows (a random val_frac of them), refitted on all
    rows.  Returns (w2, b2, info); w2 / b2 are None when no ridge beats the current layer
    (w2_now, b2_now) on the held-out rows, which then stays."""
    n = phi.shape[0]
    idx = np.random.default_rng(seed).permutation(n)
    nv = max(1, int(n * val_frac))
    va, tr = idx[:nv], idx[nv:]
    now = mse(phi[va], xk[va], xl[va], w2_now, b2_now, residual)
    scores = {}
    for r in ridges:
        w2, b2 = fit(phi[tr], xk[tr], xl[tr], residual, r)
        scores[r] = mse(phi[va], xk[va], xl[va], w2, b2, residual)
    best = min(scores, key=scores.get)
    info = {"rows": int(n), "val_rows": int(nv), "ridge": best, "val_mse": scores[best],
            "val_mse_configured": now}
    if scores[best] >= now:
        return None, None, info
    w2, b2 = fit(phi, xk, xl, residual, best)
    return w2, b2, info


def install(dd, w2: np.ndarray, b2: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Write the fitted layer into the decoder's device weights (in place, so the context's
    pointers stay valid), rounded as every generated tensor is: the matrix to the weight type,
    the bias to bf16-representable float32 in bf16 workloads.  Returns the rounded arrays (the
    values the device now holds, for a host-side model of the same decoder)."""
    import synth
    bf16 = dd.shape.dtype == "bf16"
    w2r = synth.round_to_bf16(w2.astype(np.float32)) if bf16 else w2.astype(np.float32)
    b2r = synth.round_to_bf16(b2.astype(np.float32)) if bf16 else b2.astype(np.float32)
    dd.g["in_w2"].copy_(torch.from_numpy(w2r).to(dd.g["in_w2"].dtype))
    dd.g["in_b2"].copy_(torch.from_numpy(b2r))
    torch.cuda.synchronize()
    return w2r, b2r
