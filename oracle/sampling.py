"""Speculative sampling on the self-speculative decoder (oracle; TEST INFRASTRUCTURE ONLY).

The paper's loop is greedy (Algorithm 1); it notes that the decoder's next token may also be
sampled from its distribution (Sec. "SSD Setup for VLMs").  This module is the reference for the
sampling variant of the loop, using the standard speculative-sampling rule, which keeps the
output distribution of the full model:

  * each draft token x_i is sampled from the draft's distribution q_i (layers 1..k, I, g);
  * the full model's distributions p_0..p_gamma come from the verification pass over
    [pending, x_1..x_gamma]; x_i is compared with p_{i-1}, the full model's distribution for the
    same position;
  * x_i is accepted when u * q_i(x_i) < p_{i-1}(x_i) (probability min(1, p/q)); at the first
    rejection the round emits a sample from the normalised residual max(0, p_{i-1} - q_i)
    instead (p_{i-1} itself if the residual vanishes); when all gamma drafts are accepted it also
    emits a sample from p_gamma;
  * distributions at temperature tau: softmax(logits / tau), float64.

All randomness is an input.  Per round and sequence, 2*gamma + 1 uniforms in [0, 1):
  u[0 .. gamma-1]           the draft samples,
  u[gamma .. 2 gamma - 1]   the acceptance tests,
  u[2 gamma]                the residual sample at the first rejection, or the extra sample.
A sample from weights w with uniform u is the inverse CDF: the smallest k with
w_0 + ... + w_k > u * (w_0 + ... + w_{V-1}).

The prefill's token stays the greedy argmax (the round structure starts from a pending token).

Pins: tests/test_oracle_sampling.py (inverse CDF on a uniform grid; the first emitted token of a
round follows p_0 exactly, checked by Monte Carlo against rules with plausible mistakes; a
vanishing temperature reduces the loop to greedy Algorithm 1; a draft equal to the full model
accepts every draft).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from . import decode
from .model import Decoder


def distribution(logits: np.ndarray, tau: float) -> np.ndarray:
    """softmax(logits / tau) in float64."""
    z = (np.asarray(logits, dtype=np.float64) - np.max(logits)) / float(tau)
    w = np.exp(z)
    return w / w.sum()


def sample_index(weights: np.ndarray, u: float) -> int:
    """Inverse CDF: the smallest k with w_0 + ... + w_k > u * sum(w)."""
    c = np.cumsum(np.asarray(weights, dtype=np.float64))
    k = int(np.searchsorted(c, float(u) * c[-1], side="right"))
    if k >= len(c):  # u * sum rounded up to the total: the last entry of positive weight
        k = int(np.flatnonzero(np.asarray(weights) > 0)[-1])
    return k


def accept_round(p_rows: Sequence[np.ndarray], q_rows: Sequence[np.ndarray],
                 drafts: Sequence[int], u: Sequence[float], gamma: int):
    """The speculative-sampling rule for one round: returns (accepted count a, emitted token)."""
    for i in range(gamma):
        x = int(drafts[i])
        if float(u[gamma + i]) * q_rows[i][x] < p_rows[i][x]:
            continue
        resid = np.maximum(p_rows[i] - q_rows[i], 0.0)
        if not resid.sum() > 0:
            resid = p_rows[i]
        return i, sample_index(resid, u[2 * gamma])
    return gamma, sample_index(p_rows[gamma], u[2 * gamma])


@dataclass
class SampledRound:
    l: int
    drafts: List[int]
    accepted: int
    token: int  # the emitted token after the accepted drafts
    draft_logits: List[np.ndarray] = field(default_factory=list)
    target_logits: List[np.ndarray] = field(default_factory=list)


@dataclass
class SampledRun:
    tokens: List[int]
    rounds: List[SampledRound] = field(default_factory=list)


def ssd_sample(dec: Decoder, prompt, visual, T: int, gamma: int, tau: float,
               uniforms: np.ndarray, capacity: Optional[int] = None,
               use_imitation: bool = True) -> SampledRun:
    """Self-speculative decoding with speculative sampling; uniforms [rounds][2 gamma + 1]."""
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + T + gamma + 1)
    st, y, _ = decode.prefill(dec, prompt, visual, capacity)
    run = SampledRun(tokens=[y])
    r = 0
    while len(run.tokens) < T:
        u = uniforms[r]
        l = st.seq_len
        inp, drafts, dlog, q_rows = [y], [], [], []
        for i in range(gamma):
            lg, _ = dec.draft_step(st, inp[i], l + i, use_imitation)
            q = distribution(lg, tau)
            t = sample_index(q, u[i])
            drafts.append(t)
            dlog.append(lg)
            q_rows.append(q)
            inp.append(t)
        tlog = [dec.full_step(st, inp[i], l + i)[0] for i in range(gamma + 1)]
        p_rows = [distribution(lg, tau) for lg in tlog]
        a, tok = accept_round(p_rows, q_rows, drafts, u, gamma)
        for t in drafts[:a] + [tok]:
            if len(run.tokens) < T:
                run.tokens.append(t)
        st.seq_len = l + a + 1
        y = tok
        run.rounds.append(SampledRound(l, drafts, a, tok, dlog, tlog))
        r += 1
    return run


def sample_full(dec: Decoder, prompt, visual, T: int, tau: float, uniforms: Sequence[float],
                capacity: Optional[int] = None) -> List[int]:
    """Plain sampling from the full model, one uniform per token after the prefill's token."""
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + T + 1)
    st, y, _ = decode.prefill(dec, prompt, visual, capacity)
    out = [y]
    while len(out) < T:
        lg, _ = dec.full_step(st, y, st.seq_len)
        st.seq_len += 1
        y = sample_index(distribution(lg, tau), uniforms[len(out) - 1])
        out.append(y)
    return out


def replay_sampled(dec: Decoder, prompt, visual, pending0: int, rounds, gamma: int,
                   capacity: Optional[int] = None, use_imitation: bool = True):
    """Follow a device run: ``rounds`` is a sequence of (drafts[gamma], accepted a, token); the
    oracle feeds the device's tokens, returns its own draft and full logits for them and advances
    exactly as the device did.  Returns a list of SampledRound (with the oracle's logits)."""
    n_tok = sum(gamma + 1 for _ in rounds)
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + n_tok + gamma + 2)
    st, _, _ = decode.prefill(dec, prompt, visual, capacity)
    y = int(pending0)
    out = []
    for drafts, a, tok in rounds:
        drafts = [int(t) for t in drafts]
        l = st.seq_len
        inp = [y] + drafts
        dlog = [dec.draft_step(st, inp[i], l + i, use_imitation)[0] for i in range(gamma)]
        tlog = [dec.full_step(st, inp[i], l + i)[0] for i in range(gamma + 1)]
        st.seq_len = l + int(a) + 1
        y = int(tok)
        out.append(SampledRound(l, drafts, int(a), int(tok), dlog, tlog))
    return out
