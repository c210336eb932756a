"""Confidence-stopped drafting (the Draft & Verify rule the paper compares with) on the device
against the oracle: draft and verify logits, the confidence of every draft, every stop decision,
the per-round draft counts and accepted lengths; threshold 0 is the fixed-gamma loop, threshold 1
drafts one token a round; ssd_generate_confident equals the stepwise calls; the output is the
full model's greedy output."""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu

WLS = [synth.S1, synth.S_T5, synth.S_LLAMA]


def _setup(wl, seed, batch=1):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed, batch)
    dd = runtime.from_workload(wl, seed, weights=w, max_batch=batch, page_seed=3,
                               extra_seq=wl.gamma)
    pt, vt = dd.upload_inputs(pr, z)
    return dd, Decoder(wl.shape, w, wl.draft_layers), pr, z, pt, vt


def _median_conf(dd, pt, vt, gamma):
    """The median draft confidence of two rounds at threshold 0 (device values)."""
    pend0, lg0, rounds, _ = parity.device_run_confident(dd, pt, vt, 3 * (gamma + 1), gamma, 0.0)
    c = np.concatenate([r.conf[r.active].ravel() for r in rounds])
    return float(np.median(c))


@pytest.mark.parametrize("wl", WLS, ids=lambda w: w.name)
def test_confidence_stop_matches_oracle(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, 5)
    tau = _median_conf(dd, pt, vt, wl.gamma)
    pend0, lg0, rounds, toks = parity.device_run_confident(dd, pt, vt, wl.new_tokens, wl.gamma,
                                                           tau)
    assert dd.sync_status() == (0, 0)
    near = parity.check_confident_run(dec, wl.shape, pr[0], z[0], pend0, lg0, rounds, 0,
                                      wl.gamma, tau)
    assert near <= 2
    counts = [int(r.ndraft[0]) for r in rounds]
    assert min(counts) < wl.gamma or max(counts) == wl.gamma  # stops happen at the median
    assert len(toks[0]) == wl.new_tokens
    # the loop equals the stepwise calls: tokens, rounds, accepted and proposed drafts
    gtoks, st = dd.generate_confident(pt, vt, wl.new_tokens, wl.gamma, tau)
    assert gtoks.cpu().numpy()[0].tolist() == toks[0]
    assert st["rounds"] == len(rounds)
    assert st["accepted"] == sum(int(r.accepted[0]) for r in rounds)
    assert st["drafted"] == sum(int(r.ndraft[0]) for r in rounds)
    # and the output is the full model's greedy output up to a near-tie
    greedy, _ = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=False)
    parity.check_streams_agree_until_near_tie(dec, wl.shape, pr[0], z[0], toks[0],
                                              greedy.cpu().numpy()[0].tolist(),
                                              f"{wl.name} confident vs greedy")
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA], ids=lambda w: w.name)
def test_threshold_zero_and_one(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, 6)
    # threshold 0: never stops, the fixed-gamma loop token for token and round for round
    t0, s0 = dd.generate_confident(pt, vt, wl.new_tokens, wl.gamma, 0.0)
    tf, sf = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert t0.cpu().numpy().tolist() == tf.cpu().numpy().tolist()
    assert s0 == sf
    # threshold 1: every round proposes exactly one draft after one step
    pend0, lg0, rounds, toks = parity.device_run_confident(dd, pt, vt, wl.new_tokens, wl.gamma,
                                                           1.0)
    assert all(r.steps == 1 and int(r.ndraft[0]) == 1 for r in rounds)
    parity.check_confident_run(dec, wl.shape, pr[0], z[0], pend0, lg0, rounds, 0, wl.gamma, 1.0)
    t1, s1 = dd.generate_confident(pt, vt, wl.new_tokens, wl.gamma, 1.0)
    assert t1.cpu().numpy()[0].tolist() == toks[0] and s1["drafted"] == s1["rounds"]
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_ragged_batch_confidence_stop(wl):
    """Three sequences that stop drafting at different steps of the same rounds (the steps run
    while one still drafts) and finish in different rounds: each follows the oracle, and the loop
    equals the stepwise calls."""
    B = 3
    dd, dec, pr, z, pt, vt = _setup(wl, 7, batch=B)
    tau = _median_conf(dd, pt, vt, wl.gamma)
    pend0, lg0, rounds, toks = parity.device_run_confident(dd, pt, vt, wl.new_tokens, wl.gamma,
                                                           tau)
    assert dd.sync_status() == (0, 0)
    ragged = sum(1 for r in rounds if len(set(r.ndraft[r.active].tolist())) > 1)
    assert ragged >= 1
    for b in range(B):
        parity.check_confident_run(dec, wl.shape, pr[b], z[b], pend0, lg0, rounds, b, wl.gamma,
                                   tau)
        assert len(toks[b]) == wl.new_tokens
    gtoks, st = dd.generate_confident(pt, vt, wl.new_tokens, wl.gamma, tau)
    assert gtoks.cpu().numpy().tolist() == toks
    assert st["rounds"] == len(rounds)
    assert dd.sync_status() == (0, 0)


def test_argument_checks():
    from paper_2510_22641_amd import ssd as abi
    wl = synth.S1
    dd, dec, pr, z, pt, vt = _setup(wl, 8)
    pend = dd.buf("p_conf", (1,))
    with pytest.raises(abi.SSDError) as e:
        dd.draft_confident(pend, wl.gamma, 0.5)  # before prefill
    assert e.value.code == abi.SSD_ERR_STATE
    pending, _ = dd.prefill(pt, vt)
    with pytest.raises(abi.SSDError) as e:
        dd.draft_confident(pending, wl.gamma + 1, 0.5)
    assert e.value.code == abi.SSD_ERR_SHAPE
    with pytest.raises(abi.SSDError) as e:
        dd.draft_confident(pending, wl.gamma, float("nan"))
    assert e.value.code == abi.SSD_ERR_ARG
    # a verify reusing the layer-k states must use the steps that were run
    d, nd, cf, lg, steps = dd.draft_confident(pending, wl.gamma, 1.0)
    assert steps == 1
    with pytest.raises(abi.SSDError) as e:
        dd.verify(pending, d, wl.gamma, reuse=True)
    assert e.value.code == abi.SSD_ERR_STATE
    t, _ = dd.verify(pending, d, steps, reuse=True)
    dd.accept_counts(d, nd, t, pending, steps)
    assert dd.sync_status() == (0, 0)
