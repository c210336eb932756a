"""Device path vs the CPU oracle at the workloads' full sizes, in the launch configuration the
benchmark times (HIP graphs on, verify reusing the draft's layer-k states).

FlanT5-base (c2): the whole 64-token job, every draft and verify logit.  FlanT5-xl (c3): the
whole 128-token job on the device, its first rounds replayed through the oracle logit by logit,
and the benchmark's ``ssd_generate`` loop equal to the stepwise calls token for token.
LLaVA-1.5-7B shape (c5): prefill over the 576-row visual prefix + 32 ids, then the first rounds
(the float64 oracle holds 54 GB of weights and needs tens of seconds per prefill there).
"""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu


def _setup(wl, seed=0):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed)
    dd = runtime.from_workload(wl, seed, weights=w)
    pt, vt = dd.upload_inputs(pr, z)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    del w
    return dd, dec, pr, z, pt, vt


def _check(wl, max_rounds=None, device_rounds=None):
    dd, dec, pr, z, pt, vt = _setup(wl)
    print(f"[{wl.name}] device run", flush=True)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True,
                            max_rounds=device_rounds)
    assert dd.sync_status() == (0, 0)
    print(f"[{wl.name}] {len(run.rounds)} device rounds; oracle replay", flush=True)
    ties = parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma,
                                           max_rounds=max_rounds)
    checked = len(run.rounds) if max_rounds is None else min(max_rounds, len(run.rounds))
    assert ties <= max(2, checked // 4), f"{ties} near-ties in {checked} rounds"
    assert all(0 <= r.accepted[0] <= wl.gamma for r in run.rounds)
    return dd, run, pt, vt


def test_c2_flant5_base_whole_job():
    wl = synth.C2
    dd, run, pt, vt = _check(wl)
    assert len(run.tokens[0]) == wl.new_tokens
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy()[0].tolist() == run.tokens[0]
    assert stats["rounds"] == len(run.rounds)


def test_c3_flant5_xl_bench_configuration():
    wl = synth.C3
    dd, run, pt, vt = _check(wl, max_rounds=8)
    assert len(run.tokens[0]) == wl.new_tokens
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy()[0].tolist() == run.tokens[0]
    assert stats["accepted"] == sum(int(r.accepted[0]) for r in run.rounds)


@pytest.mark.timeout(900)
def test_c5_llava_7b_prefill_and_first_rounds():
    wl = synth.C5
    _check(wl, max_rounds=2, device_rounds=2)


def test_c4_batch8_ragged_point():
    """A point of the FlanT5-xl sweep at batch 8 (k 4, gamma 8): the verify chunk is 72 rows
    (tile MFMA path) and every sequence keeps its own length.  Two sequences are replayed through
    the oracle for their first rounds; all eight are checked against the device's own batch-1
    runs token for token where no near-tie intervenes (first divergence must be a near-tie)."""
    from paper_2510_22641_amd import runtime
    wl = next(p for p in synth.c4_points() if p.batch == 8 and p.draft_layers == 4 and p.gamma == 8)
    w, z, pr = parity.workload_inputs(wl, 0)
    # stepwise calls on a ragged batch: gamma positions of slack for finished sequences
    dd = runtime.from_workload(wl, 0, weights=w, extra_seq=wl.gamma)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    del w
    pt, vt = dd.upload_inputs(pr, z)
    print(f"[{wl.name}] device run", flush=True)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    assert all(len(t) == wl.new_tokens for t in run.tokens)
    lens = {len([r for r in run.rounds if r.active[b]]) for b in range(wl.batch)}
    print(f"[{wl.name}] rounds per sequence {sorted(lens)}; oracle replay", flush=True)
    for b in (0, 5):
        parity.check_run_against_oracle(dec, wl.shape, pr[b], z[b], run, b, wl.gamma, max_rounds=3)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy().tolist() == run.tokens
    assert dd.sync_status() == (0, 0)
