"""Choose the deep-layer scale s of a synthetic workload from the oracle's own acceptance rate.

With random weights the deep layers would overwrite whatever the first k layers computed and
the draft would almost never agree with the full model; the workloads damp the residual-branch
output projections of layers k+1..L by s.  This script measures, for candidate values of s, the
acceptance rate alpha = accepted drafts / drafted tokens that Algorithm 1 reaches, and prints it.

The rate needs only one full-model greedy pass: while a round's drafts agree with the full model,
the draft sees exactly the greedy prefix and reads the same layer-1..k KV entries, so the draft's
token at position p is g(I(x_k(p))) of the greedy pass; a round starting at l accepts the longest
run of positions l+i (i < gamma) where that token equals the full model's.

Usage:  python -m oracle.tune_scale c3-flant5-xl 0.05 0.1 0.15 [--seeds 0 1] [--tokens 128]
"""
from __future__ import annotations

import argparse
import time

import numpy as np

import synth
from synth.generate import make_tensor, tensor_list

from .decode import argmax, prefill
from .model import Decoder


def greedy_with_draft_tokens(dec: Decoder, prompt, visual, T: int):
    """Greedy decode; returns (full tokens t_p, draft tokens d_p) for each decoded position p."""
    cap = dec.shape.prefix_len() + len(prompt) + T + 1
    st, y, _ = prefill(dec, prompt, visual, cap)
    full, draft = [], []
    while len(full) < T - 1:
        lg, xk = dec.full_step(st, y, st.seq_len)
        st.seq_len += 1
        y = argmax(lg)
        full.append(y)
        draft.append(argmax(dec.head(dec.imitation(xk[None]))[0]))
    return full, draft


def simulate_alpha(full, draft, gamma: int) -> float:
    """Acceptance rate of Algorithm 1 given per-position full and draft predictions."""
    i, acc, drafted = 0, 0, 0
    n = len(full)
    while i < n:
        a = 0
        while a < gamma and i + a < n and draft[i + a] == full[i + a]:
            a += 1
        acc += a
        drafted += gamma
        i += a + 1
    return acc / drafted if drafted else 0.0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("workload")
    ap.add_argument("scales", type=float, nargs="+")
    ap.add_argument("--seeds", type=int, nargs="+", default=[0])
    ap.add_argument("--tokens", type=int, default=0)
    ap.add_argument("--gamma", type=int, default=0)
    args = ap.parse_args(argv)
    wl = synth.ALL[args.workload]
    T = args.tokens or wl.new_tokens
    gamma = args.gamma or wl.gamma
    for seed in args.seeds:
        t0 = time.time()
        w = synth.make_weights(wl.shape, seed, 1.0, wl.boundary)
        dec = Decoder(wl.shape, w, wl.draft_layers)
        del w
        print(f"{wl.name} seed={seed}: decoder ready ({time.time() - t0:.0f}s)", flush=True)
        z = synth.make_visual(wl.shape, seed, 1)[0]
        pr = synth.make_prompts(wl.shape, seed, 1, wl.prompt_len)[0]
        scaled = [(n, l, tid, kind) for n, l, tid, kind in tensor_list(wl.shape)
                  if n == "in_w2" or (n in ("wo", "xo", "w_down") and l >= wl.boundary)]
        for s in args.scales:
            for n, l, tid, kind in scaled:
                arr = np.asarray(make_tensor(wl.shape, seed, n, l, tid, kind, s, wl.boundary),
                                 dtype=np.float64)
                if l < 0:
                    dec.g[n] = arr
                else:
                    dec.layers[l][n] = arr
            full, draft = greedy_with_draft_tokens(dec, pr, z, T)
            alpha = simulate_alpha(full, draft, gamma)
            agree = np.mean(np.array(full) == np.array(draft))
            print(f"{wl.name} seed={seed} s={s:g} gamma={gamma} T={T} alpha={alpha:.3f} "
                  f"per-position agreement={agree:.3f} ({time.time() - t0:.0f}s)", flush=True)


if __name__ == "__main__":
    main()
