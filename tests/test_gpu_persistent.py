"""The persistent one-row pass (one launch per draft step, greedy step and the one-row part of a
reusing verify) against the chain of kernels it replaces and against the CPU oracle, through the
C ABI: both paths follow the oracle, and while their token streams agree their per-step draft and
target logits agree within the parity tolerance."""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu

SMALL = [synth.S1, synth.S_T5, synth.S_LLAMA, synth.S_LLAMA_F32]


def _run(wl, persistent: bool, seed: int, reuse: bool, extra_seq: int = 0, kv_dtype=None):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed)
    kw = {} if kv_dtype is None else {"kv_dtype": kv_dtype}
    dd = runtime.from_workload(wl, seed, weights=w, page_seed=7, extra_seq=extra_seq, **kw)
    active = dd.set_persistent(persistent)
    assert active == persistent, "the persistent pass should exist for this shape"
    pt, vt = dd.upload_inputs(pr, z)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=reuse)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    assert dd.sync_status() == (0, 0)
    greedy = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], greedy, 0, 0, max_rounds=6)
    assert dd.sync_status() == (0, 0)
    return run, greedy


def _compare(a, b, shape):
    compared = 0
    for i, (ra, rb) in enumerate(zip(a.rounds, b.rounds)):
        if not (np.array_equal(ra.drafts, rb.drafts) and np.array_equal(ra.targets, rb.targets)):
            break
        if ra.draft_logits is not None:
            for j in range(ra.draft_logits.shape[1]):
                parity.check_logits(ra.draft_logits[0, j], rb.draft_logits[0, j].astype(np.float64),
                                    shape, f"round {i} draft {j}")
        for j in range(ra.target_logits.shape[1]):
            parity.check_logits(ra.target_logits[0, j], rb.target_logits[0, j].astype(np.float64),
                                shape, f"round {i} verify {j}")
        compared += 1
    return compared


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
@pytest.mark.parametrize("reuse", [False, True], ids=["recompute", "reuse"])
def test_persistent_matches_chain_and_oracle(wl, reuse):
    (sp, gp), (sc, gc) = (_run(wl, True, 5, reuse), _run(wl, False, 5, reuse))
    assert _compare(sp, sc, wl.shape) >= 1
    assert _compare(gp, gc, wl.shape) >= 1


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA_F32], ids=lambda w: w.name)
def test_persistent_long_context_merges_many_splits(wl):
    """A cache of several hundred positions splits each head's keys over more partials than the
    staging merge takes, so a separate merge phase runs before the output projection."""
    run, _ = _run(wl, True, 9, True, extra_seq=400)
    assert len(run.tokens[0]) == wl.new_tokens


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_persistent_bf16_kv(wl):
    run, _ = _run(wl, True, 3, True, kv_dtype="bf16")
    assert len(run.tokens[0]) == wl.new_tokens


def test_persistent_generate_equals_greedy_and_repeats():
    """ssd_generate through graphs of persistent launches: identical tokens on a repeat call (the
    barrier flags carry over between launches) and equal to its own greedy decode."""
    from paper_2510_22641_amd import runtime
    wl = synth.S_LLAMA
    w, z, pr = parity.workload_inputs(wl, 2)
    dd = runtime.from_workload(wl, 2, weights=w, page_seed=1)
    assert dd.set_persistent(True)
    pt, vt = dd.upload_inputs(pr, z)
    toks = [dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)[0].cpu()
            for _ in range(3)]
    g, _ = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=False)
    assert all(np.array_equal(toks[0].numpy(), t.numpy()) for t in toks[1:])
    assert np.array_equal(toks[0].numpy(), g.cpu().numpy())
    assert dd.sync_status() == (0, 0)
