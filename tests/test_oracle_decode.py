"""Pins of the oracle's decode loop (Algorithm 1) against full-model greedy decoding and the
special cases that fix the acceptance count."""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from oracle import decode

SMALL = [synth.S1, synth.S_T5, synth.S_LLAMA]


def _setup(wl, seed=0, mutate=None, k=None):
    w = synth.workload_weights(wl, seed, threads=2)
    if mutate:
        mutate(w)
    z = synth.make_visual(wl.shape, seed, 1)[0]
    pr = synth.make_prompts(wl.shape, seed, 1, wl.prompt_len)[0]
    return Decoder(wl.shape, w, k or wl.draft_layers), pr, z


def test_accept_length_cases():
    assert decode.accept_length([5, 6, 7], [5, 6, 9, 4]) == 2
    assert decode.accept_length([5, 6, 7], [5, 6, 7, 4]) == 3
    assert decode.accept_length([5, 6, 7], [1, 6, 7, 4]) == 0
    assert decode.accept_length([], [3]) == 0


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
@pytest.mark.parametrize("seed", [0, 1])
def test_ssd_equals_greedy_bit_exact(wl, seed):
    dec, pr, z = _setup(wl, seed)
    g = decode.greedy(dec, pr, z, wl.new_tokens)
    for gamma in (1, wl.gamma, 7):
        s = decode.ssd(dec, pr, z, wl.new_tokens, gamma)
        assert s.tokens == g.tokens
        assert np.array_equal(s.prefill_logits, g.prefill_logits)
        # every verified position's logits equal the greedy step's logits bit for bit
        pos_logits = {}
        for r in s.rounds:
            for i, lg in enumerate(r.target_logits[: r.accepted + 1]):
                pos_logits[r.seq_len + i] = lg
        base = s.rounds[0].seq_len
        for j, lg in enumerate(g.step_logits):
            if base + j in pos_logits:
                assert np.array_equal(pos_logits[base + j], lg)
        # accepted length per round in [0, gamma], emitted count exactly T
        assert all(0 <= r.accepted <= gamma for r in s.rounds)
        assert len(s.tokens) == wl.new_tokens
        assert 1 + sum(r.accepted + 1 for r in s.rounds) >= wl.new_tokens
        assert 1 + sum(r.accepted + 1 for r in s.rounds[:-1]) < wl.new_tokens


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_other_draft_depths(wl):
    for k in (1, wl.shape.n_layers):
        dec, pr, z = _setup(wl, 2, k=k)
        g = decode.greedy(dec, pr, z, 16)
        assert decode.ssd(dec, pr, z, 16, 3).tokens == g.tokens


def _kill_deep(wl):
    def m(w):
        for lw in w["layers"][wl.draft_layers:]:
            lw["wo"][:] = 0
            lw["w_down"][:] = 0
            if "xo" in lw:
                lw["xo"][:] = 0
        w["in_w2"][:] = 0
        w["in_b2"][:] = 0
    return m


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_zero_deep_layers_accept_everything(wl):
    # s = 0 and an identity imitation network: the draft equals the full model exactly
    dec, pr, z = _setup(wl, 0, _kill_deep(wl))
    s = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma)
    assert all(r.accepted == wl.gamma for r in s.rounds)
    assert s.acceptance_rate() == 1.0
    for r in s.rounds:
        for i in range(wl.gamma):
            assert np.array_equal(r.draft_logits[i], r.target_logits[i])


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_forced_wrong_drafts_accept_nothing(wl):
    dec, pr, z = _setup(wl, 1)
    g = decode.greedy(dec, pr, z, wl.new_tokens)
    vocab = wl.shape.vocab
    s = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma,
                   draft_policy=lambda r, i, lg: (int(np.argmax(lg)) + 1) % vocab)
    # a wrong draft can still match by chance only if argmax+1 is the full model's token
    assert sum(r.accepted for r in s.rounds) <= 2
    assert s.tokens == g.tokens
    always_bad = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, draft_policy=lambda r, i, lg: -1)
    assert all(r.accepted == 0 for r in always_bad.rounds)
    assert always_bad.tokens == g.tokens
    assert len(always_bad.rounds) == wl.new_tokens - 1


def test_gamma_zero_is_greedy():
    dec, pr, z = _setup(synth.S1, 0)
    g = decode.greedy(dec, pr, z, 20)
    s = decode.ssd(dec, pr, z, 20, 0)
    assert s.tokens == g.tokens and all(r.accepted == 0 for r in s.rounds)


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_stale_kv_is_never_read(wl):
    dec, pr, z = _setup(wl, 3)
    clean = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma)
    poisoned = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, poison=True)
    assert poisoned.tokens == clean.tokens
    for a, b in zip(clean.rounds, poisoned.rounds):
        assert a.accepted == b.accepted
        assert all(np.array_equal(x, y) for x, y in zip(a.target_logits, b.target_logits))


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_draft_without_imitation_still_yields_greedy_output(wl):
    dec, pr, z = _setup(wl, 4)
    g = decode.greedy(dec, pr, z, wl.new_tokens)
    s = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, use_imitation=False)
    assert s.tokens == g.tokens


def test_eos_stops_the_loop():
    dec, pr, z = _setup(synth.S1, 0)
    g = decode.greedy(dec, pr, z, 24)
    eos = g.tokens[5]
    s = decode.ssd(dec, pr, z, 24, 4, eos_id=eos)
    first = g.tokens.index(eos)
    assert s.tokens == g.tokens[: first + 1]


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_replay_of_own_stream_reproduces_logits(wl):
    dec, pr, z = _setup(wl, 5)
    s = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma)
    lg0, rounds = decode.replay(dec, pr, z, s.tokens[0], [(r.drafts, r.targets) for r in s.rounds],
                                wl.gamma)
    assert np.array_equal(lg0, s.prefill_logits)
    for a, b in zip(s.rounds, rounds):
        assert a.accepted == b.accepted
        assert all(np.array_equal(x, y) for x, y in zip(a.draft_logits, b.draft_logits))
        assert all(np.array_equal(x, y) for x, y in zip(a.target_logits, b.target_logits))


def test_dynamic_draft_length_closed_forms():
    """d(t) = d0 + floor(10 * sigmoid(0.01 (t - N/2))): d0 + 5 at the midpoint, d0 far below it,
    at most d0 + 9 for every t <= N (the logistic stays below 1 there), d0 + 10 only where the
    double-precision logistic rounds to exactly 1 (t - N/2 > ~3700), non-decreasing, hand values."""
    f = decode.dynamic_draft_length
    assert f(71, 5, 142) == 10
    assert f(-100000, 5, 142) == 5 and f(100000, 5, 142) == 15
    for n_max in (142, 512, 4096):
        assert max(f(t, 5, n_max) for t in range(0, n_max + 1)) <= 14
    # t = 0, N = 142: 10 / (1 + e^0.71) = 3.296...
    assert f(0, 5, 142) == 8 and f(0, 1, 142) == 4
    vals = [f(t, 5, 512) for t in range(0, 4000)]
    assert all(b >= a for a, b in zip(vals, vals[1:])) and set(vals) == set(range(5, 16))
    # the logistic crosses 0.9 at x = ln 9: one step below and above the boundary
    x9 = 100.0 * np.log(9.0) + 256.0
    assert f(int(np.floor(x9)), 0, 512) == 8 and f(int(np.ceil(x9)), 0, 512) == 9


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA], ids=lambda w: w.name)
def test_dynamic_draft_length_ssd_equals_greedy(wl):
    """With the context-length schedule each round drafts d(l) tokens, and the output is still
    the full model's greedy output bit for bit."""
    dec, pr, z = _setup(wl, seed=3)
    n_max = wl.max_seq() + 9
    fn = lambda l: decode.dynamic_draft_length(l, 2, n_max)  # noqa: E731
    run = decode.ssd(dec, pr, z, wl.new_tokens, 11, gamma_fn=fn)
    g = decode.greedy(dec, pr, z, wl.new_tokens)
    assert run.tokens == g.tokens
    for r in run.rounds:
        assert len(r.drafts) == fn(r.seq_len)
        assert 0 <= r.accepted <= len(r.drafts)


def test_confidence_closed_forms():
    # the largest softmax probability: 1/V for equal logits, 1/2 for two equal maxima far above
    # the rest, -> 1 for one dominant logit, and invariant to a shift of every logit
    V = 1000
    assert decode.confidence(np.zeros(V)) == pytest.approx(1.0 / V, rel=1e-12)
    lg = np.full(V, -800.0)
    lg[[3, 700]] = 5.0
    assert decode.confidence(lg) == pytest.approx(0.5, rel=1e-12)
    lg = np.zeros(V)
    lg[17] = 50.0
    assert decode.confidence(lg) == pytest.approx(1.0 / (1.0 + (V - 1) * np.exp(-50.0)), rel=1e-12)
    r = np.random.default_rng(1).standard_normal(V)
    assert decode.confidence(r + 123.0) == pytest.approx(decode.confidence(r), rel=1e-12)
    # brute force: the probability of the argmax under softmax computed term by term
    e = [float(np.exp(x)) for x in r]
    assert decode.confidence(r) == pytest.approx(max(e) / sum(e), rel=1e-12)


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_confidence_stop_rule(wl):
    """Threshold 0 never stops (the fixed-gamma run, bit for bit); threshold 1 stops after the
    first draft of every round; any threshold keeps the greedy output; and in every round the
    number of drafts is 1 + the leading drafts at or above the threshold, capped at gamma."""
    dec, pr, z = _setup(wl, 4)
    g = decode.greedy(dec, pr, z, wl.new_tokens)
    fixed = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma)
    zero = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, confidence_stop=0.0)
    assert zero.tokens == fixed.tokens
    assert [r.accepted for r in zero.rounds] == [r.accepted for r in fixed.rounds]
    for a, b in zip(zero.rounds, fixed.rounds):
        assert a.drafts == b.drafts and len(a.confidences) == wl.gamma
        assert all(np.array_equal(x, y) for x, y in zip(a.target_logits, b.target_logits))
    one = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, confidence_stop=1.0)
    assert all(len(r.drafts) == 1 for r in one.rounds)
    assert one.tokens == g.tokens
    confs = sorted(c for r in zero.rounds for c in r.confidences)
    for q in (0.2, 0.5, 0.8):
        tau = confs[int(q * (len(confs) - 1))]
        s = decode.ssd(dec, pr, z, wl.new_tokens, wl.gamma, confidence_stop=tau)
        assert s.tokens == g.tokens
        for r in s.rounds:
            lead = 0
            while lead < len(r.confidences) and r.confidences[lead] >= tau:
                lead += 1
            assert len(r.drafts) == min(wl.gamma, lead + 1) == len(r.confidences)
            assert len(r.targets) == len(r.drafts) + 1
            assert 0 <= r.accepted <= len(r.drafts)
            # each recorded confidence is that of the draft logits it came with
            for c, lg in zip(r.confidences, r.draft_logits):
                p = np.exp(lg - lg.max())
                assert c == pytest.approx(p.max() / p.sum(), rel=1e-12)
