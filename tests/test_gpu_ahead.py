"""Drafting the next round ahead on a second stream (SSD_MODE_SPECULATIVE_AHEAD), through the
C ABI.

The two-stream schedule computes Algorithm 1 unchanged: its tokens and its per-round acceptance
must equal those of the one-stream loop with the layer-k reuse (itself checked against the oracle
in test_gpu_parity.py) bit for bit, for single sequences, ragged batches, with and without HIP
graphs, and on a decoder whose draft equals the full model (every drafted-ahead round is used).
"""
import numpy as np
import pytest

import synth
from oracle import decode
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu

SMALL = [synth.S1, synth.S_T5, synth.S_LLAMA, synth.S_LLAMA_F32]


def _setup(wl, seed=0, batch=None, weights=None, extra_seq=None):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed, batch)
    if weights is not None:
        weights(w)
    # drafts made ahead reach 2 gamma positions past a round's start
    dd = runtime.from_workload(wl, seed, weights=w, max_batch=batch or wl.batch,
                               extra_seq=wl.gamma if extra_seq is None else extra_seq,
                               page_seed=3)
    pt, vt = dd.upload_inputs(pr, z)
    return dd, w, pr, z, pt, vt


def _both(dd, pt, vt, wl):
    plain, ps = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    plain = plain.cpu().numpy().tolist()
    ahead, st = dd.generate(pt, vt, wl.new_tokens, wl.gamma, ahead=True)
    ahead = ahead.cpu().numpy().tolist()
    assert dd.sync_status() == (0, 0)
    return plain, ps, ahead, st


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_ahead_equals_one_stream_loop(wl):
    dd, w, pr, z, pt, vt = _setup(wl, seed=4)
    plain, ps, ahead, st = _both(dd, pt, vt, wl)
    assert ahead == plain
    assert st == ps
    # and the run again on the same context (graphs replayed, buffers reused)
    again, st2 = dd.generate(pt, vt, wl.new_tokens, wl.gamma, ahead=True)
    assert again.cpu().numpy().tolist() == plain and st2 == ps


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_ahead_without_graphs(wl):
    dd, w, pr, z, pt, vt = _setup(wl, seed=5)
    plain, ps, _, _ = _both(dd, pt, vt, wl)
    dd.set_graphs(False)
    ahead, st = dd.generate(pt, vt, wl.new_tokens, wl.gamma, ahead=True)
    assert ahead.cpu().numpy().tolist() == plain and st == ps
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_ahead_ragged_batch(wl):
    """Sequences finish in different rounds; drafts made ahead are used only when every sequence
    still active accepted all drafts and its extra token was the one they started from."""
    B = 3
    dd, w, pr, z, pt, vt = _setup(wl, seed=6, batch=B)
    plain, ps, ahead, st = _both(dd, pt, vt, wl)
    assert ahead == plain and st == ps
    for b in range(B):
        one, _ = dd.generate(pt[b:b + 1], vt[b:b + 1], wl.new_tokens, wl.gamma, ahead=True)
        assert one.cpu().numpy()[0].tolist() == plain[b]
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA], ids=lambda w: w.name)
def test_ahead_when_every_draft_passes(wl):
    """Deep layers and the imitation network switched off (zero output projections): the draft
    model is the full model, every draft passes and the full model's extra token is the draft's
    next token, so after the first round every round runs on drafts made ahead.  The tokens are
    the oracle's greedy tokens."""

    def kill(w):
        for lw in w["layers"][wl.draft_layers:]:
            lw["wo"][:] = 0
            lw["w_down"][:] = 0
            if "xo" in lw:
                lw["xo"][:] = 0
        w["in_w2"][:] = 0
        w["in_b2"][:] = 0

    dd, w, pr, z, pt, vt = _setup(wl, seed=7, weights=kill)
    plain, ps, ahead, st = _both(dd, pt, vt, wl)
    assert ahead == plain and st == ps
    assert st["accepted"] == st["drafted"]
    g = decode.greedy(Decoder(wl.shape, w, wl.draft_layers), pr[0], z[0], wl.new_tokens)
    dev = ahead[0]
    if dev != g.tokens:
        first = next(i for i, (a, b) in enumerate(zip(dev, g.tokens)) if a != b)
        lg = g.prefill_logits if first == 0 else g.step_logits[first - 1]
        parity.check_token(dev[first], lg, wl.shape, f"greedy token {first}")


def test_ahead_needs_room_for_two_rounds_of_drafts():
    from paper_2510_22641_amd import ssd as abi
    wl = synth.S_T5
    dd, w, pr, z, pt, vt = _setup(wl, seed=8, extra_seq=0)
    with pytest.raises(abi.SSDError) as e:
        dd.generate(pt, vt, wl.new_tokens, wl.gamma, ahead=True)
    assert e.value.code == abi.SSD_ERR_CAPACITY
    # the one-stream loop still fits the minimal cache
    toks, _ = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert len(toks.cpu().numpy()[0]) == wl.new_tokens
    assert dd.sync_status() == (0, 0)


def test_ahead_refuses_the_hidden_state_export():
    from paper_2510_22641_amd import ssd as abi
    import torch
    wl = synth.S_T5
    dd, w, pr, z, pt, vt = _setup(wl, seed=9)
    sh = wl.shape
    phi = torch.zeros((1, wl.gamma, sh.in_width), dtype=torch.float32, device="cuda")
    xk = torch.zeros((1, wl.gamma, sh.d_model), dtype=torch.float32, device="cuda")
    xl = torch.zeros((1, wl.gamma + 1, sh.d_model), dtype=torch.float32, device="cuda")
    abi.ssd_set_hidden_export(dd.ctx, phi, xk, xl)
    with pytest.raises(abi.SSDError) as e:
        dd.generate(pt, vt, wl.new_tokens, wl.gamma, ahead=True)
    assert e.value.code == abi.SSD_ERR_STATE
    abi.ssd_set_hidden_export(dd.ctx, None, None, None)
    assert dd.sync_status() == (0, 0)


def test_c3_flant5_xl_ahead_equals_one_stream_loop():
    """The benchmark's workload (FlanT5-xl shape, 128 tokens): the two-stream schedule gives the
    one-stream loop's tokens and acceptance."""
    wl = synth.C3
    dd, w, pr, z, pt, vt = _setup(wl, seed=0)
    del w
    plain, ps, ahead, st = _both(dd, pt, vt, wl)
    assert ahead == plain and st == ps
    assert np.array(plain).shape == (1, wl.new_tokens)
