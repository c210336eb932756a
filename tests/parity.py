"""Helpers of the device-vs-oracle parity tests (no tests here).

Tolerances (per step, over the vocabulary):
  f32 workloads   max |device logit - oracle logit| <= 1e-4
  bf16 workloads  max |device logit - oracle logit| <= 2e-2 * std(oracle logits of that step)
Tokens follow the replay protocol: the oracle follows the device's token stream; where a device
token differs from the oracle's argmax, the oracle's own logits must put it within the tolerance
of the top; the accepted length per round must be bit-exact given the device's drafts and
targets.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import synth
from oracle import decode
from oracle.model import Decoder


def tolerance(shape, ref_logits) -> float:
    return 1e-4 if shape.dtype == "f32" else 2e-2 * float(np.std(ref_logits))


def check_logits(dev, ref, shape, what: str) -> float:
    tol = tolerance(shape, ref)
    err = float(np.max(np.abs(np.asarray(dev, dtype=np.float64) - ref)))
    assert np.isfinite(err) and err <= tol, f"{what}: max-abs {err:.3g} > tol {tol:.3g}"
    return err / tol


def check_token(dev_tok: int, ref_logits, shape, what: str) -> bool:
    """True when the device token is the oracle's argmax; False for an accepted near-tie."""
    top = int(np.argmax(ref_logits))
    if int(dev_tok) == top:
        return True
    gap = float(ref_logits[top] - ref_logits[int(dev_tok)])
    tol = tolerance(shape, ref_logits)
    assert gap <= tol, (f"{what}: device token {dev_tok} vs oracle {top}: oracle gap {gap:.3g} "
                        f"> tol {tol:.3g}")
    return False


@dataclass
class DevRound:
    drafts: np.ndarray  # [B, gamma]
    targets: np.ndarray  # [B, gamma+1]
    accepted: np.ndarray  # [B]
    active: np.ndarray  # [B] bool: the sequence took part
    draft_logits: Optional[np.ndarray] = None  # [B, gamma, V]
    target_logits: Optional[np.ndarray] = None  # [B, gamma+1, V]


@dataclass
class DevRun:
    pending0: np.ndarray
    prefill_logits: Optional[np.ndarray]
    rounds: List[DevRound] = field(default_factory=list)
    tokens: List[List[int]] = field(default_factory=list)


def poison_stale_kv(dd) -> None:
    """Overwrite every KV entry at or beyond each sequence's valid length with NaN."""
    import torch
    sl = dd.seq_len.cpu().numpy()
    pt = dd.page_table.cpu().numpy()
    ps = dd.cap.page_size
    for b in range(pt.shape[0]):
        for p in range(int(sl[b]), pt.shape[1] * ps):
            page, slot = int(pt[b, p // ps]), p % ps
            dd.k_pool[:, page, :, slot, :] = float("nan")
            dd.v_pool[:, page, :, slot, :] = float("nan")
    torch.cuda.synchronize()


def device_run(dd, prompt_t, visual_t, T: int, gamma: int, reuse: bool = False,
               logits: bool = True, poison: bool = False, forced=None,
               max_rounds: Optional[int] = None) -> DevRun:
    """Step through prefill / draft / verify / accept via the C ABI and record everything
    (at most ``max_rounds`` rounds when given)."""
    import torch
    B = prompt_t.shape[0]
    pending, lg0 = dd.prefill(prompt_t, visual_t, logits=logits)
    run = DevRun(pending.cpu().numpy().copy(), lg0.cpu().numpy().copy() if logits else None)
    run.tokens = [[int(t)] for t in run.pending0]
    active = dd.buf("active_mask", (B,))
    active.fill_(1)
    if poison:
        poison_stale_kv(dd)
    for rnd in range(T if max_rounds is None else min(T, max_rounds)):
        act = np.array([len(t) < T for t in run.tokens])
        if not act.any():
            break
        active.copy_(torch.from_numpy(act.astype(np.int32)))
        if gamma > 0:
            d, dl = dd.draft(pending, gamma, logits=logits)
            if forced is not None:
                d.copy_(torch.from_numpy(forced(rnd, d.cpu().numpy()).astype(np.int32)))
        else:
            d, dl = dd.buf("no_draft", (B, 1)), None
        t, tl = dd.verify(pending, d, gamma, reuse=reuse, logits=logits)
        out, alen = dd.accept(d, t, pending, gamma, active)
        r = DevRound(d.cpu().numpy()[:, :gamma].copy(), t.cpu().numpy().copy(),
                     alen.cpu().numpy().copy(), act,
                     dl.cpu().numpy().copy() if dl is not None else None,
                     tl.cpu().numpy().copy() if tl is not None else None)
        run.rounds.append(r)
        o = out.cpu().numpy()
        for b in range(B):
            if act[b]:
                run.tokens[b].extend(int(x) for x in o[b, : r.accepted[b] + 1])
        if poison:
            poison_stale_kv(dd)
    run.tokens = [t[:T] for t in run.tokens]
    return run


def check_run_against_oracle(dec: Decoder, shape, prompt, visual, run: DevRun, b: int, gamma: int,
                             use_imitation: bool = True, max_rounds: Optional[int] = None):
    """Replay sequence b of a device run (its first ``max_rounds`` rounds when given) through
    the oracle; returns the count of near-ties."""
    rounds = [r for r in run.rounds if r.active[b]][:max_rounds]
    lg0, orounds = decode.replay(dec, prompt, visual, int(run.pending0[b]),
                                 [(r.drafts[b], r.targets[b]) for r in rounds], gamma,
                                 use_imitation=use_imitation)
    ties = 0
    if run.prefill_logits is not None:
        check_logits(run.prefill_logits[b], lg0, shape, f"seq {b} prefill logits")
    ties += not check_token(run.pending0[b], lg0, shape, f"seq {b} prefill token")
    for k, (r, o) in enumerate(zip(rounds, orounds)):
        for i in range(gamma):
            if r.draft_logits is not None:
                check_logits(r.draft_logits[b, i], o.draft_logits[i], shape, f"seq {b} round {k} draft {i} logits")
            ties += not check_token(r.drafts[b, i], o.draft_logits[i], shape, f"seq {b} round {k} draft {i}")
        for j in range(gamma + 1):
            if r.target_logits is not None:
                check_logits(r.target_logits[b, j], o.target_logits[j], shape, f"seq {b} round {k} verify {j} logits")
            ties += not check_token(r.targets[b, j], o.target_logits[j], shape, f"seq {b} round {k} verify {j}")
        assert int(r.accepted[b]) == o.accepted, f"seq {b} round {k}: accepted {r.accepted[b]} != {o.accepted}"
    return ties


def oracle_full_logits_along(dec: Decoder, prompt, visual, tokens, i: int) -> np.ndarray:
    """The oracle's full-model logits that choose emitted token i of a stream whose tokens
    0..i-1 are ``tokens[:i]`` (token 0 comes from the prefill)."""
    cap = dec.shape.prefix_len() + len(prompt) + i + 2
    st, _, lg = decode.prefill(dec, prompt, visual, cap)
    for t in tokens[:i]:
        if i == 0:
            break
        lg, _ = dec.full_step(st, int(t), st.seq_len)
        st.seq_len += 1
    return lg


def check_streams_agree_until_near_tie(dec: Decoder, shape, prompt, visual, a, b,
                                       what: str) -> int:
    """Two device token streams of the same sequence (speculative and greedy decoding) must be
    identical up to their first difference, and there the oracle's logits along the common
    prefix must put both tokens within the tolerance of its top.  Returns the index of the first
    difference (len(a) when none)."""
    a, b = [int(t) for t in a], [int(t) for t in b]
    assert len(a) == len(b), what
    first = next((i for i, (x, y) in enumerate(zip(a, b)) if x != y), len(a))
    if first < len(a):
        lg = oracle_full_logits_along(dec, prompt, visual, a, first)
        check_token(a[first], lg, shape, f"{what}: token {first} of the first stream")
        check_token(b[first], lg, shape, f"{what}: token {first} of the second stream")
    return first


# ---- confidence-stopped drafting ------------------------------------------------------------

@dataclass
class ConfDevRound:
    steps: int                # draft steps the device ran
    drafts: np.ndarray        # [B, steps]
    ndraft: np.ndarray        # [B] drafts proposed
    conf: np.ndarray          # [B, steps] device confidences
    targets: np.ndarray       # [B, steps + 1]
    accepted: np.ndarray      # [B]
    active: np.ndarray        # [B]
    draft_logits: np.ndarray  # [B, steps, V]
    target_logits: np.ndarray  # [B, steps + 1, V]


def device_run_confident(dd, prompt_t, visual_t, T: int, gamma: int, tau: float,
                         reuse: bool = True):
    """Stepwise confidence-stopped decoding through the C ABI (ssd_draft_confident, ssd_verify,
    ssd_accept_counts); returns (pending0, prefill logits, rounds, tokens per sequence)."""
    import torch
    B = prompt_t.shape[0]
    pending, lg0 = dd.prefill(prompt_t, visual_t, logits=True)
    pend0, lg0 = pending.cpu().numpy().copy(), lg0.cpu().numpy().copy()
    tokens = [[int(t)] for t in pend0]
    active = dd.buf("active_mask", (B,))
    rounds = []
    for _ in range(T):
        act = np.array([len(t) < T for t in tokens])
        if not act.any():
            break
        active.copy_(torch.from_numpy(act.astype(np.int32)))
        d, nd, cf, dl, steps = dd.draft_confident(pending, gamma, tau, active, logits=True)
        t, tl = dd.verify(pending, d, steps, reuse=reuse, logits=True)
        out, alen = dd.accept_counts(d, nd, t, pending, steps, active)
        r = ConfDevRound(steps, d.cpu().numpy().copy(), nd.cpu().numpy().copy(),
                         cf.cpu().numpy()[:, :steps].copy(), t.cpu().numpy().copy(),
                         alen.cpu().numpy().copy(), act, dl.cpu().numpy()[:, :steps].copy(),
                         tl.cpu().numpy().copy())
        rounds.append(r)
        o = out.cpu().numpy()
        for b in range(B):
            if act[b]:
                tokens[b].extend(int(x) for x in o[b, : r.accepted[b] + 1])
    return pend0, lg0, rounds, [t[:T] for t in tokens]


def check_confident_run(dec: Decoder, shape, prompt, visual, pend0, lg0, rounds, b: int,
                        gamma: int, tau: float) -> int:
    """Replay sequence b of a confidence-stopped device run through the oracle.  Logits within
    the usual tolerance; each device confidence within the band that the logit tolerance allows
    (log-confidence moves by at most twice the largest logit error); every stop decision the
    device took on its own confidence, and the oracle's on its own except within that band; the
    accepted length bit-exact.  Returns the count of decisions taken inside the band."""
    mine = [r for r in rounds if r.active[b]]
    orounds_in = [(r.drafts[b, :r.ndraft[b]], r.targets[b, :r.ndraft[b] + 1]) for r in mine]
    o0, orounds = decode.replay(dec, prompt, visual, int(pend0[b]), orounds_in, gamma)
    check_logits(lg0[b], o0, shape, f"seq {b} prefill logits")
    near = 0
    for k, (r, o) in enumerate(zip(mine, orounds)):
        n = int(r.ndraft[b])
        assert 1 <= n <= min(gamma, r.steps), f"seq {b} round {k}: {n} drafts of {r.steps} steps"
        for i in range(n):
            check_logits(r.draft_logits[b, i], o.draft_logits[i], shape, f"seq {b} r{k} draft {i}")
            check_token(r.drafts[b, i], o.draft_logits[i], shape, f"seq {b} r{k} draft {i}")
            band = 2.0 * tolerance(shape, o.draft_logits[i])
            dc, oc = float(r.conf[b, i]), o.confidences[i]
            assert abs(np.log(dc) - np.log(oc)) <= band + 1e-6, (
                f"seq {b} r{k} draft {i}: confidence {dc:.6g} vs oracle {oc:.6g}")
            stopped_here = i == n - 1 and n < gamma
            # the device's own decision on its own confidence: exact
            assert (dc < tau) == stopped_here or (i == n - 1 and n == gamma), (
                f"seq {b} r{k} draft {i}: device conf {dc:.6g} vs tau {tau:.6g}, stopped "
                f"{stopped_here}")
            if i < n - 1 or stopped_here:
                if (oc < tau) != stopped_here:
                    assert abs(np.log(oc) - np.log(tau)) <= band + 1e-6, (
                        f"seq {b} r{k} draft {i}: oracle conf {oc:.6g} on the other side of "
                        f"tau {tau:.6g}")
                    near += 1
        for j in range(n + 1):
            check_logits(r.target_logits[b, j], o.target_logits[j], shape, f"seq {b} r{k} verify {j}")
            check_token(r.targets[b, j], o.target_logits[j], shape, f"seq {b} r{k} verify {j}")
        assert int(r.accepted[b]) == o.accepted, f"seq {b} r{k}: {r.accepted[b]} != {o.accepted}"
    return near


def workload_inputs(wl, seed: int, batch: Optional[int] = None):
    B = batch or wl.batch
    w = synth.workload_weights(wl, seed, threads=4)
    z = synth.make_visual(wl.shape, seed, B)
    pr = synth.make_prompts(wl.shape, seed, B, wl.prompt_len)
    return w, z, pr


# ---- the sampling variant (speculative sampling) --------------------------------------------

@dataclass
class SampledDevRound:
    drafts: np.ndarray        # [gamma]
    accepted: int
    token: int
    draft_logits: np.ndarray  # [gamma, V]
    target_logits: np.ndarray  # [gamma+1, V]


@dataclass
class SampledDevRun:
    pending0: int
    rounds: List[SampledDevRound] = field(default_factory=list)
    tokens: List[int] = field(default_factory=list)


def device_run_sampled(dd, prompt_t, visual_t, T: int, gamma: int, tau: float, uniforms,
                       reuse: bool = True) -> SampledDevRun:
    """One sequence through prefill / ssd_draft_sample / ssd_verify / ssd_accept_sample with
    uniforms [rounds, 2 gamma + 1] (draft samples, acceptance tests, the extra sample)."""
    import torch
    pending, _ = dd.prefill(prompt_t, visual_t)
    run = SampledDevRun(int(pending.cpu().numpy()[0]))
    run.tokens = [run.pending0]
    r = 0
    while len(run.tokens) < T:
        u = np.asarray(uniforms[r], dtype=np.float32)
        ud = torch.from_numpy(u[None, :gamma].copy()).to(pending.device)
        ua = torch.from_numpy(u[None, gamma:].copy()).to(pending.device)
        d, dl = dd.draft_sample(pending, gamma, ud, tau)
        t, tl = dd.verify(pending, d, gamma, reuse=reuse, logits=True)
        out, alen = dd.accept_sample(d, dl, tl, ua, tau, pending, gamma)
        a = int(alen.cpu().numpy()[0])
        o = out.cpu().numpy()[0]
        run.rounds.append(SampledDevRound(d.cpu().numpy()[0].copy(), a, int(o[a]),
                                          dl.cpu().numpy()[0].copy(), tl.cpu().numpy()[0].copy()))
        run.tokens.extend(int(x) for x in o[: a + 1])
        r += 1
    run.tokens = run.tokens[:T]
    return run


def _check_cdf_pick(k: int, weights, u: float, ftol: float, what: str) -> bool:
    """The device's inverse-CDF pick k from weights with uniform u, where the oracle's cumulative
    distribution may be off by ftol: u must lie within ftol of k's interval.  True when k is
    exactly the oracle's pick."""
    from oracle import sampling
    w = np.asarray(weights, dtype=np.float64)
    c = np.cumsum(w) / w.sum()
    lo = c[k - 1] if k > 0 else 0.0
    assert w[k] > 0 or ftol > 0, f"{what}: picked a zero-weight entry {k}"
    assert lo - ftol <= u <= c[k] + ftol, (f"{what}: device picked {k}, u {u:.6f} outside "
                                          f"[{lo:.6f}, {c[k]:.6f}] +- {ftol:.2g}")
    return k == sampling.sample_index(w, u)


def check_sampled_run(dec, shape, prompt, visual, run: SampledDevRun, gamma: int, tau: float,
                      uniforms) -> int:
    """Replay a sampled device run through the oracle; returns the count of decisions taken
    within the tolerance band (where the oracle's own decision differs)."""
    from oracle import sampling
    orounds = sampling.replay_sampled(dec, prompt, visual, run.pending0,
                                      [(r.drafts, r.accepted, r.token) for r in run.rounds], gamma)
    close = 0
    for k, (r, o) in enumerate(zip(run.rounds, orounds)):
        u = np.asarray(uniforms[k], dtype=np.float64)
        q_rows, p_rows, ftols = [], [], []
        for i in range(gamma):
            check_logits(r.draft_logits[i], o.draft_logits[i], shape, f"round {k} draft {i} logits")
            q_rows.append(sampling.distribution(o.draft_logits[i], tau))
        for j in range(gamma + 1):
            check_logits(r.target_logits[j], o.target_logits[j], shape, f"round {k} verify {j} logits")
            p_rows.append(sampling.distribution(o.target_logits[j], tau))
            ftols.append(4.0 * tolerance(shape, o.target_logits[j]) / tau + 1e-6)
        ftol = max(ftols + [4.0 * tolerance(shape, lg) / tau + 1e-6 for lg in o.draft_logits])
        for i in range(gamma):
            close += not _check_cdf_pick(int(r.drafts[i]), q_rows[i], u[i], ftol,
                                         f"round {k} draft {i}")
        # acceptance decisions: the oracle's, except within the tolerance band
        for i in range(min(r.accepted + 1, gamma)):
            x = int(r.drafts[i])
            lhs, rhs = u[gamma + i] * q_rows[i][x], p_rows[i][x]
            dev_accept = i < r.accepted
            if (lhs < rhs) != dev_accept:
                assert abs(np.log(max(lhs, 1e-300)) - np.log(max(rhs, 1e-300))) <= 2 * ftol, (
                    f"round {k} draft {i}: device {'accepted' if dev_accept else 'rejected'}, "
                    f"oracle u q = {lhs:.3g} vs p = {rhs:.3g}")
                close += 1
        a = r.accepted
        if a < gamma:
            w = np.maximum(p_rows[a] - q_rows[a], 0.0)
            if not w.sum() > 0:
                w = p_rows[a]
        else:
            w = p_rows[gamma]
        close += not _check_cdf_pick(int(r.token), w, u[2 * gamma], 2 * ftol, f"round {k} token")
    return close
