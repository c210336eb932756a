"""Pins of the speculative-sampling oracle (oracle/sampling.py) against what the mathematics fixes.

* The inverse CDF on a grid of uniforms hits every index with its exact weight, never a zero one.
* The first token a round emits follows the full model's distribution p_0 exactly, whatever the
  draft's distribution q (the defining property of the rule): Monte Carlo over random uniforms,
  with a tolerance of 5 standard deviations; the same check rejects the rule with plausible
  mistakes (acceptance min(1, q/p), residual max(0, q - p)).
* A vanishing temperature turns every distribution into a point mass on the argmax, and the loop
  into greedy Algorithm 1: the same tokens as the oracle's greedy decoding.
* A draft model equal to the full model (deep layers zeroed, the imitation network the identity)
  accepts every draft.
"""
import numpy as np
import pytest

import synth
from oracle import decode, sampling
from oracle.model import Decoder


def test_inverse_cdf_on_a_uniform_grid():
    w = np.array([0.0, 3.0, 0.0, 1.0, 4.0, 0.0])
    n = 80_000
    u = (np.arange(n) + 0.5) / n
    counts = np.bincount([sampling.sample_index(w, x) for x in u], minlength=len(w))
    assert np.allclose(counts / n, w / w.sum(), atol=2.0 / n)
    assert counts[0] == counts[2] == counts[5] == 0


def _first_token_freq(rule, p, q, gamma, n, seed):
    rng = np.random.default_rng(seed)
    V = len(p)
    counts = np.zeros(V)
    for _ in range(n):
        u = rng.random(2 * gamma + 1)
        drafts = [sampling.sample_index(q, u[i]) for i in range(gamma)]
        a, tok = rule([p] * (gamma + 1), [q] * gamma, drafts, u, gamma)
        first = drafts[0] if a > 0 else tok
        counts[first] += 1
    return counts / n


def _bad_ratio(p_rows, q_rows, drafts, u, gamma):
    for i in range(gamma):
        x = drafts[i]
        if u[gamma + i] * p_rows[i][x] < q_rows[i][x]:  # min(1, q/p): wrong
            continue
        return i, sampling.sample_index(np.maximum(p_rows[i] - q_rows[i], 0), u[2 * gamma])
    return gamma, sampling.sample_index(p_rows[gamma], u[2 * gamma])


def _bad_residual(p_rows, q_rows, drafts, u, gamma):
    for i in range(gamma):
        x = drafts[i]
        if u[gamma + i] * q_rows[i][x] < p_rows[i][x]:
            continue
        r = np.maximum(q_rows[i] - p_rows[i], 0)  # wrong sign
        return i, sampling.sample_index(r if r.sum() > 0 else p_rows[i], u[2 * gamma])
    return gamma, sampling.sample_index(p_rows[gamma], u[2 * gamma])


@pytest.mark.parametrize("gamma", [1, 3])
def test_first_emitted_token_follows_the_full_model(gamma):
    p = np.array([0.55, 0.05, 0.25, 0.15])
    q = np.array([0.10, 0.60, 0.05, 0.25])
    n = 30_000
    tol = 5 * np.sqrt(p * (1 - p) / n)
    f = _first_token_freq(sampling.accept_round, p, q, gamma, n, seed=gamma)
    assert np.all(np.abs(f - p) <= tol), (f, p)
    for bad in (_bad_ratio, _bad_residual):
        fb = _first_token_freq(bad, p, q, gamma, n, seed=gamma)
        assert np.any(np.abs(fb - p) > tol), bad.__name__


@pytest.mark.parametrize("wl", [synth.S1, synth.S_T5], ids=lambda w: w.name)
def test_vanishing_temperature_is_greedy(wl):
    w = synth.workload_weights(wl, 0)
    z = synth.make_visual(wl.shape, 0, 1)[0]
    pr = synth.make_prompts(wl.shape, 0, 1, wl.prompt_len)[0]
    dec = Decoder(wl.shape, w, wl.draft_layers)
    u = synth.make_uniforms(0, 1, wl.new_tokens, 2 * wl.gamma + 1)[0]
    run = sampling.ssd_sample(dec, pr, z, wl.new_tokens, wl.gamma, 1e-6, u)
    assert run.tokens == decode.greedy(dec, pr, z, wl.new_tokens).tokens


def test_identical_draft_accepts_every_draft():
    wl = synth.S1
    w = synth.workload_weights(wl, 1)
    for lw in w["layers"][wl.draft_layers:]:
        for k in ("wo", "xo", "w_down"):
            lw[k] = np.zeros_like(lw[k])
    w["in_w2"] = np.zeros_like(w["in_w2"])
    w["in_b2"] = np.zeros_like(w["in_b2"])
    z = synth.make_visual(wl.shape, 1, 1)[0]
    pr = synth.make_prompts(wl.shape, 1, 1, wl.prompt_len)[0]
    dec = Decoder(wl.shape, w, wl.draft_layers)
    u = synth.make_uniforms(1, 1, wl.new_tokens, 2 * wl.gamma + 1)[0]
    run = sampling.ssd_sample(dec, pr, z, wl.new_tokens, wl.gamma, 0.7, u)
    assert all(r.accepted == wl.gamma for r in run.rounds[:-1])
