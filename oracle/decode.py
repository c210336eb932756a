"""Prefill, full-model greedy decoding and Algorithm 1 (greedy self-speculative imitation decoding).

Algorithm 1 of the paper, with the readings used where it is ambiguous (listed in the design doc):
  * a round drafts exactly ``gamma`` tokens (the loop bound as printed runs d+1 times, the text
    says d tokens y^{t+1}..y^{t+d});
  * the loop runs while fewer than T tokens have been emitted and no <eos> was emitted; the
    workloads disable <eos> (eos_id = -1) and emit exactly T tokens, the last round truncated;
  * when every draft is accepted the full model's next token is emitted too, so a round emits
    a+1 tokens with a in [0, gamma];
  * the KV cache is shared by draft and verify (Sec. "KV cache"); a rejection rolls it back by
    resetting the valid length to l + a + 1, stale entries beyond it are never read;
  * the prefill's argmax is emitted token #1 and is the "pending" token: the full model's next
    token whose KV is not yet computed.

Verification is "a single forward pass" over the drafted tokens (Sec. "Self-Speculative
Decoding"); here the causal pass is evaluated one position at a time, which is the same
mathematics, so every position's arithmetic is identical in greedy and speculative mode and the
two produce bit-identical tokens and logits (the self-check in tests/test_oracle_decode.py).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence

import numpy as np

from .model import Decoder, State


def argmax(logits: np.ndarray) -> int:
    """Greedy choice; equal maxima resolve to the lowest index."""
    return int(np.argmax(logits))


def dynamic_draft_length(t: int, d0: int, n_max: int) -> int:
    """Draft length at context length t (appendix on the choice of d): d(0) plus the floor of ten
    times the logistic function of 0.01 (t - N/2), N the maximum sequence length."""
    x = -0.01 * (t - n_max / 2.0)
    e = math.exp(x) if x < 700.0 else math.inf  # IEEE: 1 / (1 + inf) = 0 far below N/2
    return d0 + math.floor(10.0 / (1.0 + e))


def confidence(logits: np.ndarray) -> float:
    """The confidence of a prediction: the largest softmax probability over the vocabulary,
    max_v softmax(logits)_v = 1 / sum_v exp(logits_v - max logits) (the paper's C_l, appendix on
    the choice of n)."""
    lg = np.asarray(logits, dtype=np.float64)
    return float(1.0 / np.sum(np.exp(lg - np.max(lg))))


def accept_length(drafts: Sequence[int], targets: Sequence[int]) -> int:
    """Longest prefix of drafts that matches the full model: a = max{j : draft_i = target_{i-1}, i<=j}.

    drafts[i] is the draft's token for position l+i+1, targets[i] the full model's token for the
    same position (computed from the verified prefix up to l+i).
    """
    a = 0
    while a < len(drafts) and drafts[a] == targets[a]:
        a += 1
    return a


@dataclass
class Round:
    seq_len: int  # l at the start of the round
    inputs: List[int]  # u_0 (pending) .. u_gamma
    drafts: List[int]
    targets: List[int]
    accepted: int  # a
    draft_logits: List[np.ndarray] = field(default_factory=list)
    target_logits: List[np.ndarray] = field(default_factory=list)
    confidences: List[float] = field(default_factory=list)  # of each draft (confidence stop)


@dataclass
class Run:
    tokens: List[int]
    prefill_logits: np.ndarray
    rounds: List[Round] = field(default_factory=list)
    step_logits: List[np.ndarray] = field(default_factory=list)  # greedy mode

    def acceptance_rate(self) -> float:
        drafted = sum(len(r.drafts) for r in self.rounds)
        return sum(r.accepted for r in self.rounds) / drafted if drafted else 0.0


def prefill(dec: Decoder, prompt: Sequence[int], visual: np.ndarray, capacity: int):
    """Run the full decoder over the context; returns (state, pending token, its logits).

    T5: the prompt ids are positions 0..P-1 and z is the cross-attention memory.
    LLaMA: the visual rows are x_0 of positions 0..Nv-1, the prompt follows.
    """
    st = dec.new_state(capacity)
    if dec.t5:
        dec.set_visual(st, visual)
        x = dec.embed(prompt)
    else:
        x = np.concatenate([np.asarray(visual, dtype=np.float64), dec.embed(prompt)], axis=0)
    positions = list(range(x.shape[0]))
    x = dec.run_layers(x, positions, st, 0, dec.shape.n_layers)
    st.seq_len = len(positions)
    logits = dec.head(x[-1:])[0]
    return st, argmax(logits), logits


def greedy(dec: Decoder, prompt, visual, T: int, capacity: Optional[int] = None) -> Run:
    """Full-model greedy decoding: each step runs all L layers on the pending token."""
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + T + 1)
    st, y, lg = prefill(dec, prompt, visual, capacity)
    run = Run(tokens=[y], prefill_logits=lg)
    while len(run.tokens) < T:
        lg, _ = dec.full_step(st, y, st.seq_len)
        st.seq_len += 1
        y = argmax(lg)
        run.tokens.append(y)
        run.step_logits.append(lg)
    return run


def _poison(st: State) -> None:
    st.K[:, st.seq_len:] = np.nan
    st.V[:, st.seq_len:] = np.nan


def ssd(dec: Decoder, prompt, visual, T: int, gamma: int, capacity: Optional[int] = None,
        draft_policy: Optional[Callable[[int, int, np.ndarray], int]] = None,
        poison: bool = False, use_imitation: bool = True, eos_id: int = -1,
        max_rounds: Optional[int] = None,
        gamma_fn: Optional[Callable[[int], int]] = None,
        confidence_stop: Optional[float] = None) -> Run:
    """Algorithm 1: draft gamma tokens with layers 1..k + I + g, verify them with the full decoder,
    keep the longest matching prefix plus the full model's token at the first mismatch.

    ``draft_policy(round, i, logits) -> token`` replaces the draft's argmax (host-forced drafts);
    ``poison`` overwrites every KV entry beyond the valid length with NaN after each acceptance;
    ``max_rounds`` stops early (a bounded sample of the loop, for timing);
    ``gamma_fn(l) -> d`` drafts d tokens in a round that starts at context length l (the dynamic
    draft length; ``gamma`` then only sizes the cache);
    ``confidence_stop`` = tau stops a round's drafting after the first draft whose confidence (the
    draft's largest softmax probability) is below tau, that draft still proposed (the Draft &
    Verify rule the paper compares with, Sec. "Experiments", baselines): a round then drafts
    between 1 and gamma tokens.
    """
    if gamma < 0:
        raise ValueError("gamma must be >= 0")
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + T + gamma + 1)
    st, y, lg = prefill(dec, prompt, visual, capacity)
    run = Run(tokens=[y], prefill_logits=lg)
    done = (y == eos_id)
    while len(run.tokens) < T and not done:
        if max_rounds is not None and len(run.rounds) >= max_rounds:
            break
        l = st.seq_len
        g = gamma if gamma_fn is None else int(gamma_fn(l))
        # drafting stage: u_0 = pending, u_{i+1} = draft's argmax at position l+i
        u = [y]
        drafts, dlog, conf = [], [], []
        for i in range(g):
            lg, _ = dec.draft_step(st, u[i], l + i, use_imitation)
            t = argmax(lg) if draft_policy is None else int(draft_policy(len(run.rounds), i, lg))
            drafts.append(t)
            dlog.append(lg)
            u.append(t)
            if confidence_stop is not None:
                conf.append(confidence(lg))
                if conf[-1] < confidence_stop:
                    break
        # verification stage: the full decoder over u_0..u_n at positions l..l+n (n drafts)
        g = len(drafts)
        targets, tlog = [], []
        for i in range(g + 1):
            lg, _ = dec.full_step(st, u[i], l + i)
            targets.append(argmax(lg))
            tlog.append(lg)
        # acceptance and rollback
        a = accept_length(drafts, targets)
        emitted = drafts[:a] + [targets[a]]
        for t in emitted:
            if len(run.tokens) < T and not done:
                run.tokens.append(t)
                done = (t == eos_id)
        st.seq_len = l + a + 1
        y = targets[a]
        run.rounds.append(Round(l, u, drafts, targets, a, dlog, tlog, conf))
        if poison:
            _poison(st)
    return run


def replay(dec: Decoder, prompt, visual, pending0: int, rounds, gamma: int,
           capacity: Optional[int] = None, use_imitation: bool = True):
    """Follow a device run's token stream and return the oracle's logits at every step.

    ``rounds`` is a sequence of (drafts[n], targets[n+1]) produced by the device (n = gamma, or
    fewer for a round whose drafting stopped early).  The oracle feeds the device's tokens as
    inputs (u_0 = pending, u_i = device draft i), computes its own draft and full logits for them
    (and the confidence of each draft), applies its own acceptance rule to the device's drafts
    and targets, and advances exactly as the device did.  Returns (prefill logits, list of
    Round).
    """
    n_tok = sum(gamma + 1 for _ in rounds)
    capacity = capacity or (dec.shape.prefix_len() + len(prompt) + n_tok + gamma + 2)
    st, _, lg0 = prefill(dec, prompt, visual, capacity)
    y = int(pending0)
    out = []
    for drafts, targets in rounds:
        drafts = [int(t) for t in drafts]
        targets = [int(t) for t in targets]
        n = len(drafts)
        l = st.seq_len
        u = [y] + drafts
        dlog = [dec.draft_step(st, u[i], l + i, use_imitation)[0] for i in range(n)]
        tlog = [dec.full_step(st, u[i], l + i)[0] for i in range(n + 1)]
        a = accept_length(drafts, targets)
        st.seq_len = l + a + 1
        y = targets[a]
        out.append(Round(l, u, drafts, targets, a, dlog, tlog, [confidence(lg) for lg in dlog]))
    return lg0, out
