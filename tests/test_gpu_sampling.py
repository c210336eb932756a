"""The sampling variant of the loop (speculative sampling) on the device, through the C ABI,
against the oracle with the same uniforms: per-step draft and verify logits within the parity
tolerance; every sampled token and acceptance decision equal to the oracle's, except within the
tolerance band the logit tolerance implies; a vanishing temperature reproduces greedy decoding."""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu

SMALL = [synth.S1, synth.S_T5, synth.S_LLAMA, synth.S_LLAMA_F32]


def _setup(wl, seed):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed)
    dd = runtime.from_workload(wl, seed, weights=w, page_seed=4)
    pt, vt = dd.upload_inputs(pr, z)
    return w, z, pr, dd, pt, vt


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
@pytest.mark.parametrize("scale", [1.0, 0.25], ids=["tau-std", "tau-quarter-std"])
def test_sampled_rounds_match_oracle(wl, scale):
    w, z, pr, dd, pt, vt = _setup(wl, 3)
    _, lg0 = dd.prefill(pt, vt, logits=True)
    tau = scale * float(np.std(lg0.cpu().numpy()))
    u = synth.make_uniforms(3, 1, wl.new_tokens, 2 * wl.gamma + 1)[0]
    run = parity.device_run_sampled(dd, pt, vt, wl.new_tokens, wl.gamma, tau, u)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    close = parity.check_sampled_run(dec, wl.shape, pr[0], z[0], run, wl.gamma, tau, u)
    assert len(run.tokens) == wl.new_tokens
    assert all(0 <= r.accepted <= wl.gamma for r in run.rounds)
    assert close <= 3
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA_F32], ids=lambda w: w.name)
def test_vanishing_temperature_is_greedy(wl):
    """At a temperature far below the logit gaps every distribution is a point mass on its argmax:
    the sampled loop emits the greedy tokens."""
    w, z, pr, dd, pt, vt = _setup(wl, 5)
    u = synth.make_uniforms(5, 1, wl.new_tokens, 2 * wl.gamma + 1)[0]
    run = parity.device_run_sampled(dd, pt, vt, wl.new_tokens, wl.gamma, 1e-6, u)
    greedy, _ = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=False)
    assert run.tokens == [int(t) for t in greedy.cpu().numpy()[0]]
    assert dd.sync_status() == (0, 0)


def test_argument_checks():
    from paper_2510_22641_amd import ssd as abi
    w, z, pr, dd, pt, vt = _setup(synth.S1, 0)
    pending, _ = dd.prefill(pt, vt)
    import torch
    u = torch.zeros(1, 4, dtype=torch.float32, device=pending.device)
    d = dd.buf("draft", (1, 4))
    lg = dd.buf("draft_logits", (1, 4, synth.S1.shape.vocab), torch.float32)
    for bad_tau in (0.0, -1.0, float("inf")):
        with pytest.raises(abi.SSDError):
            abi.ssd_draft_sample(dd.ctx, 1, 4, pending, u, bad_tau, d, lg)
    with pytest.raises(abi.SSDError):
        abi.ssd_draft_sample(dd.ctx, 1, 4, pending, u, 1.0, d, None)
    assert dd.sync_status() == (0, 0)
