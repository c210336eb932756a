"""Device path vs the CPU oracle, through the C ABI, at sizes the oracle finishes in seconds
(several tiles and ragged tails: d 128..256, vocab 1024..2000, heads of 64 and 128 dims)."""
import numpy as np
import pytest

import synth
from oracle.model import Decoder
from oracle import decode
from tests import parity

pytestmark = pytest.mark.gpu

SMALL = [synth.S1, synth.S_T5, synth.S_LLAMA, synth.S_LLAMA_F32]


def _setup(wl, seed=0, batch=None, page_seed=None, weights=None, max_batch=None, extra_seq=0):
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed, batch)
    if weights is not None:
        weights(w)
    dd = runtime.from_workload(wl, seed, weights=w, max_batch=max_batch or batch or wl.batch,
                               page_seed=page_seed, extra_seq=extra_seq)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    pt, vt = dd.upload_inputs(pr, z)
    return dd, dec, pr, z, pt, vt


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
@pytest.mark.parametrize("reuse", [False, True], ids=["recompute", "reuse"])
def test_speculative_rounds_match_oracle(wl, reuse):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=0, page_seed=11)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=reuse)
    ties = parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    assert len(run.tokens[0]) == wl.new_tokens
    assert all(0 <= r.accepted[0] <= wl.gamma for r in run.rounds)
    assert ties <= 2
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_greedy_steps_match_oracle(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=1)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, 0)
    assert all(r.accepted[0] == 0 for r in run.rounds)


@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_generate_loop_equals_stepwise_and_greedy(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=2)
    step = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True, logits=False)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy()[0].tolist() == step.tokens[0]
    # every round the loop queues without a read-back is one the stepwise run needed
    assert stats["rounds"] == len(step.rounds)
    assert stats["drafted"] == wl.gamma * stats["rounds"]
    assert stats["accepted"] == sum(int(r.accepted[0]) for r in step.rounds)
    gtoks, gstats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=False)
    assert gstats["rounds"] == wl.new_tokens - 1
    # self-speculative output is the full model's greedy output: the device's two streams agree
    # token for token up to a near-tie of the oracle's logits (none expected in float32)
    ssd_t, gr_t = toks.cpu().numpy()[0].tolist(), gtoks.cpu().numpy()[0].tolist()
    first = parity.check_streams_agree_until_near_tie(dec, wl.shape, pr[0], z[0], ssd_t, gr_t,
                                                      f"{wl.name} ssd vs greedy")
    if wl.shape.dtype == "f32":
        assert first == wl.new_tokens
    # and the device's greedy stream is the oracle's up to a near-tie
    g = decode.greedy(dec, pr[0], z[0], wl.new_tokens)
    parity.check_streams_agree_until_near_tie(dec, wl.shape, pr[0], z[0], gr_t, g.tokens,
                                              f"{wl.name} device vs oracle greedy")


def test_generate_reports_device_status():
    """A prompt id outside the vocabulary sets the device status word during the prefill: the
    loop stops at its first read-back and ssd_generate returns SSD_ERR_DEVICE; the word stays set
    for ssd_sync_status, which reports and clears it."""
    from paper_2510_22641_amd import ssd as abi
    wl = synth.S1
    dd, dec, pr, z, pt, vt = _setup(wl, seed=9)
    bad = pt.clone()
    bad[0, 2] = wl.shape.vocab + 3
    with pytest.raises(abi.SSDError) as e:
        dd.generate(bad, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert e.value.code == abi.SSD_ERR_DEVICE
    rc, st = dd.sync_status()
    assert rc == abi.SSD_ERR_DEVICE and st & abi.SSD_DEV_BAD_TOKEN
    assert dd.sync_status() == (0, 0)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.shape[1] == wl.new_tokens and stats["rounds"] >= 1


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_graphs_equal_eager(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=3)
    a = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    dd.set_graphs(False)
    b = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert a.tokens == b.tokens
    for ra, rb in zip(a.rounds, b.rounds):
        assert np.array_equal(ra.target_logits, rb.target_logits)
        assert np.array_equal(ra.draft_logits, rb.draft_logits)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA], ids=lambda w: w.name)
def test_stale_kv_poison_changes_nothing(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=4)
    clean = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    dirty = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True, poison=True)
    assert clean.tokens == dirty.tokens
    for ra, rb in zip(clean.rounds, dirty.rounds):
        assert np.array_equal(ra.target_logits, rb.target_logits)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_T5], ids=lambda w: w.name)
def test_forced_drafts_acceptance_rule(wl):
    dd, dec, pr, z, pt, vt = _setup(wl, seed=5)
    V = wl.shape.vocab
    rng = np.random.default_rng(0)
    forced = lambda rnd, d: (d + 1 + rng.integers(0, V - 1, d.shape)) % V if rnd % 2 else d
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, forced=forced)
    for r in run.rounds:
        n = 0
        while n < wl.gamma and r.drafts[0, n] == r.targets[0, n]:
            n += 1
        assert r.accepted[0] == n
    # the verified stream is the full model's whatever the drafts: replay verify and accept only
    rounds = [(r.drafts[0], r.targets[0]) for r in run.rounds]
    lg0, orounds = decode.replay(dec, pr[0], z[0], int(run.pending0[0]), rounds, wl.gamma)
    for k, (r, o) in enumerate(zip(run.rounds, orounds)):
        for j in range(wl.gamma + 1):
            parity.check_logits(r.target_logits[0, j], o.target_logits[j], wl.shape, f"r{k} v{j}")
        assert r.accepted[0] == o.accepted


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_ragged_batch_each_sequence_matches_oracle(wl):
    B = 3
    # stepwise calls on a ragged batch: finished sequences are still drafted at their last
    # length, so the cache holds gamma more positions
    dd, dec, pr, z, pt, vt = _setup(wl, seed=6, batch=B, page_seed=7, extra_seq=wl.gamma)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    accepted = set()
    for b in range(B):
        parity.check_run_against_oracle(dec, wl.shape, pr[b], z[b], run, b, wl.gamma)
        assert len(run.tokens[b]) == wl.new_tokens
        accepted.add(tuple(int(r.accepted[b]) for r in run.rounds if r.active[b]))
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy().tolist() == run.tokens
    assert stats["rounds"] == len(run.rounds)
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_ragged_batch_with_key_splits_matches_oracle(wl):
    """A ragged batch in a cache of 256 positions or more: each head's keys are split into fixed
    ranges of ceil(capacity / splits), so while the contexts are short the later splits of every
    sequence are empty (their partials carry no weight in the merge), and the sequences reach
    their split boundaries in different rounds.  Every sequence follows the oracle."""
    B = 3
    dd, dec, pr, z, pt, vt = _setup(wl, seed=6, batch=B, page_seed=7, extra_seq=250 + wl.gamma)
    assert dd.cap.max_seq >= 256
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    for b in range(B):
        parity.check_run_against_oracle(dec, wl.shape, pr[b], z[b], run, b, wl.gamma)
        assert len(run.tokens[b]) == wl.new_tokens
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy().tolist() == run.tokens
    assert stats["rounds"] == len(run.rounds)
    assert dd.sync_status() == (0, 0)


def test_generate_ragged_batch_fits_the_minimal_cache():
    """ssd_generate on a batch whose sequences finish in different rounds needs no slack: a
    finished sequence keeps only its emitted positions."""
    wl = synth.S_LLAMA
    B = 4
    dd, dec, pr, z, pt, vt = _setup(wl, seed=8, batch=B)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert dd.sync_status() == (0, 0)
    one, rounds = [], []
    for b in range(B):
        t1, s1 = dd.generate(pt[b:b + 1], vt[b:b + 1], wl.new_tokens, wl.gamma,
                             speculative=True, reuse=True)
        one.append(t1.cpu().numpy()[0].tolist())
        rounds.append(s1["rounds"])
    assert dd.sync_status() == (0, 0)
    assert toks.cpu().numpy().tolist() == one
    # the batch runs in lock step until its slowest sequence is done: no round more
    assert stats["rounds"] == max(rounds)


def test_zero_deep_layers_accept_every_draft():
    wl = synth.S_T5

    def kill(w):
        for lw in w["layers"][wl.draft_layers:]:
            lw["wo"][:] = 0
            lw["xo"][:] = 0
            lw["w_down"][:] = 0
        w["in_w2"][:] = 0
        w["in_b2"][:] = 0

    dd, dec, pr, z, pt, vt = _setup(wl, seed=7, weights=kill)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert stats["accepted"] == stats["drafted"]


def test_lm_head_ties_resolve_to_lowest_index():
    wl = synth.S1

    def plant(w):
        u = w["lm_head"][5].copy()
        w["lm_head"][:] = 0
        for j in (7, 300, 1000):
            w["lm_head"][j] = u

    dd, dec, pr, z, pt, vt = _setup(wl, seed=8, weights=plant)
    run = parity.device_run(dd, pt, vt, 12, wl.gamma)
    toks = [run.pending0[0]] + [t for r in run.rounds for t in r.targets[0]]
    assert set(int(t) for t in toks) <= {0, 7}
    assert set(int(t) for r in run.rounds for t in r.drafts[0]) <= {0, 7}


def test_error_codes_and_device_status():
    from paper_2510_22641_amd import ssd as abi
    wl = synth.S1
    dd, dec, pr, z, pt, vt = _setup(wl, seed=9)
    pend = dd.buf("p_err", (1,))
    drafts = dd.buf("d_err", (1, wl.gamma))
    with pytest.raises(abi.SSDError) as e:
        dd.draft(pend, wl.gamma)  # before prefill
    assert e.value.code == abi.SSD_ERR_STATE
    pending, _ = dd.prefill(pt, vt)
    with pytest.raises(abi.SSDError) as e:
        abi.ssd_draft(dd.ctx, 2, wl.gamma, pending, drafts, None)
    assert e.value.code == abi.SSD_ERR_SHAPE
    with pytest.raises(abi.SSDError) as e:
        abi.ssd_draft(dd.ctx, 1, wl.gamma + 1, pending, drafts, None)
    assert e.value.code == abi.SSD_ERR_SHAPE
    with pytest.raises(abi.SSDError) as e:
        dd.verify(pending, drafts, wl.gamma, reuse=True)  # no preceding draft
    assert e.value.code == abi.SSD_ERR_STATE
    # a token id outside the vocabulary is reported, not read
    bad = pt.clone()
    bad[0, 3] = wl.shape.vocab + 5
    dd.prefill(bad, vt)
    rc, st = dd.sync_status()
    assert rc == abi.SSD_ERR_DEVICE and st & abi.SSD_DEV_BAD_TOKEN
    assert dd.sync_status() == (0, 0)


def test_positions_past_the_cache_are_reported_not_written():
    """Greedy steps fill the cache to its last position; a draft of gamma tokens then reaches
    past it: the KV stores beyond max_seq are skipped and the device status says so.  Rounds
    that stay inside the cache never raise the bit, including a final round that ends at the
    last position."""
    from paper_2510_22641_amd import ssd as abi
    wl = synth.S1
    dd, dec, pr, z, pt, vt = _setup(wl, seed=4)
    max_seq = dd.cap.max_seq
    pending, _ = dd.prefill(pt, vt)
    nd = dd.buf("no_draft", (1, 1))
    while int(dd.seq_len[0].item()) < max_seq - 1:
        t, _ = dd.verify(pending, nd, 0)
        dd.accept(nd, t, pending, 0)
    assert dd.sync_status() == (0, 0)
    k_before = dd.k_pool.clone()
    dd.draft(pending, wl.gamma)
    rc, st = dd.sync_status()
    assert rc == abi.SSD_ERR_DEVICE and st == abi.SSD_DEV_CAPACITY
    # only the one in-range position (max_seq - 1) of layers 1..k was written
    changed = (dd.k_pool != k_before).reshape(dd.k_pool.shape[0], -1).any(dim=1).cpu().numpy()
    assert changed[: wl.draft_layers].all() and not changed[wl.draft_layers:].any()
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_bf16_kv_cache_option(wl):
    """The bf16 KV cache (kv_dtype="bf16", not the default) also stays within the tolerance at
    these sizes: every logit of a speculative run against the oracle."""
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, 5)
    dd = runtime.from_workload(wl, 5, weights=w, kv_dtype="bf16", page_seed=2)
    assert dd.k_pool.dtype.itemsize == 2
    dec = Decoder(wl.shape, w, wl.draft_layers)
    pt, vt = dd.upload_inputs(pr, z)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S1, synth.S_LLAMA_F32], ids=lambda w: w.name)
def test_dynamic_draft_length_generate_matches_oracle(wl):
    """ssd_generate with the context-length schedule (d(0) = 2, up to 11 drafts a round): the
    tokens, round count, accepted and drafted totals equal the oracle's Algorithm 1 with the same
    schedule (float32 workloads: no near-ties at these sizes)."""
    from paper_2510_22641_amd import runtime
    from oracle import decode as odec
    d0 = 2
    w, z, pr = parity.workload_inputs(wl, 3)
    dd = runtime.from_workload(wl, 3, weights=w, max_gamma=d0 + 9)
    dec = Decoder(wl.shape, w, wl.draft_layers)
    pt, vt = dd.upload_inputs(pr, z)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, d0, speculative=True, reuse=True, dynamic=True)
    n_max = dd.cap.max_seq
    ref = odec.ssd(dec, pr[0], z[0], wl.new_tokens, d0 + 9,
                   gamma_fn=lambda l: odec.dynamic_draft_length(l, d0, n_max))
    assert toks.cpu().numpy()[0].tolist() == ref.tokens
    assert stats["rounds"] == len(ref.rounds)
    assert stats["accepted"] == sum(r.accepted for r in ref.rounds)
    assert stats["drafted"] == sum(len(r.drafts) for r in ref.rounds)
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_long_capacity_splits_attention_keys(wl):
    """A cache of 256 positions or more splits each head's keys over several blocks whose partial
    (max, sum, output) are merged by a second kernel: the whole run still matches the oracle."""
    dd, dec, pr, z, pt, vt = _setup(wl, seed=12, page_seed=5, extra_seq=250)
    assert dd.cap.max_seq >= 256
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    assert dd.sync_status() == (0, 0)


def test_kv_pool_beyond_2gib_matches_small_pool():
    """Layer pools of more than 2 GiB (sequences scattered over 200k spare pages, about a third
    of them past the 2 GiB offset): the attention addresses them with 64-bit pointers instead of
    32-bit buffer offsets, and the run equals the one on a small pool token for token and in its
    acceptance (the same values enter the same arithmetic)."""
    import torch
    from paper_2510_22641_amd import runtime
    wl = synth.S_LLAMA_F32
    sh = wl.shape
    runs = []
    for spare in (0, 200_000):
        w, z, pr = parity.workload_inputs(wl, 13)
        dd = runtime.from_workload(wl, 13, weights=w, page_seed=5, extra_seq=250,
                                   spare_pages=spare)
        layer_bytes = dd.k_pool[0].numel() * dd.k_pool.element_size()
        assert (layer_bytes > 2 ** 31) == (spare > 0)
        assert dd.cap.max_seq >= 256  # key splits too
        pt, vt = dd.upload_inputs(pr, z)
        toks, st = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
        runs.append((toks.cpu().numpy().tolist(), st))
        assert dd.sync_status() == (0, 0)
        dd.close()
        del dd
        torch.cuda.empty_cache()
    assert runs[0] == runs[1]
    assert sh.d_head == 128 and sh.dtype == "f32"


@pytest.mark.parametrize("wl", [synth.S1, synth.S_T5], ids=lambda w: w.name)
def test_folded_cross_attention_matches_unfolded_and_oracle(wl):
    """A one-sequence T5 context folds the cross-attention into two float32 matrices per layer,
    used by its one-row steps; a two-sequence context keeps the query projection, attention launch
    and output projection.  Both runs follow the oracle, and while their token streams agree their
    per-step draft and target logits agree within the tolerance."""
    runs = []
    for mb in (1, 2):
        dd, dec, pr, z, pt, vt = _setup(wl, seed=4, page_seed=3, max_batch=mb)
        run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
        parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
        assert dd.sync_status() == (0, 0)
        runs.append(run)
    folded, unfolded = runs
    parity.check_logits(folded.prefill_logits[0], unfolded.prefill_logits[0].astype(np.float64),
                        wl.shape, "prefill")
    compared = 0
    for i, (ra, rb) in enumerate(zip(folded.rounds, unfolded.rounds)):
        if not (np.array_equal(ra.drafts, rb.drafts) and np.array_equal(ra.targets, rb.targets)):
            break
        for j in range(ra.draft_logits.shape[1]):
            parity.check_logits(ra.draft_logits[0, j], rb.draft_logits[0, j].astype(np.float64),
                                wl.shape, f"round {i} draft {j}")
        compared += 1
    assert compared >= 1

def test_wide_ffn_rows_take_the_k_split_gemv():
    """A LLaMA-style decoder whose FFN is 6208 wide: the one-row down projection (K = 6208, four
    2048-element pieces, the last one ragged) runs on the K-split GEMV without a norm, as the
    LLaMA-7B shape's K = 11008 does.  Drafts, verify logits and greedy steps follow the oracle."""
    from dataclasses import replace
    wide = replace(synth.SMALL_LLAMA_BF16, name="small-llama-wide-ffn", n_layers=3, d_ff=6208)
    wl = synth.S_LLAMA.with_(name="s-llama-wide-ffn", shape=wide, new_tokens=16)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=12, page_seed=5)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    greedy = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], greedy, 0, 0)
    assert dd.sync_status() == (0, 0)


def test_folded_scores_from_layer_input_at_d2048():
    """A T5-style decoder of FlanT5-xl width (d 2048, 32 heads of 64, 32 visual tokens), three
    layers: the one-row steps of layers 1..k take the output projection and the folded
    cross-attention scores from [x; o] in one launch (the scores matrix F and its product with
    W_o, built at prefill) and apply 1 / rms of the new residual inside the next launch's softmax.
    Drafts, verify logits and greedy steps follow the oracle, and the run agrees with an
    unfolded two-sequence context within the tolerance while the token streams agree."""
    from dataclasses import replace
    wide = replace(synth.SMALL_T5_BF16, name="t5-d2048", n_layers=3, d_model=2048, n_heads=32,
                   d_head=64, d_ff=2048, vocab=2000, n_visual=32)
    wl = synth.S_T5.with_(name="s-t5-d2048", shape=wide, draft_layers=2, new_tokens=20)
    runs = []
    for mb in (1, 2):
        dd, dec, pr, z, pt, vt = _setup(wl, seed=14, page_seed=4, max_batch=mb)
        run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
        parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
        if mb == 1:
            greedy = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
            parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], greedy, 0, 0)
        assert dd.sync_status() == (0, 0)
        runs.append(run)
    folded, unfolded = runs
    for i, (ra, rb) in enumerate(zip(folded.rounds, unfolded.rounds)):
        if not (np.array_equal(ra.drafts, rb.drafts) and np.array_equal(ra.targets, rb.targets)):
            break
        for j in range(ra.draft_logits.shape[1]):
            parity.check_logits(ra.draft_logits[0, j], rb.draft_logits[0, j].astype(np.float64),
                                wl.shape, f"round {i} draft {j}")


@pytest.mark.parametrize("heads,d_head", [(2, 128), (4, 64)], ids=["dh128", "dh64"])
def test_long_prefix_prefill_splits_residual_projections_over_k(heads, d_head):
    """A LLaMA-style decoder with a 300-row visual prefix: the prefill's context block (307 rows)
    is past the skinny capacity, so its projections take the tile GEMM, and the residual
    projections (W_o, down) with few 128 x 128 tiles run over four ranges of K whose partial
    products are added to the residual in range order; its causal self-attention takes the MFMA
    kernel (five 64-row query tiles, keys in 64-key tiles, the last one ragged).  Prefill logits,
    drafts, verify logits and greedy steps follow the oracle."""
    from dataclasses import replace
    long = replace(synth.SMALL_LLAMA_BF16, name="small-llama-long-prefix", n_visual=300,
                   n_heads=heads, d_head=d_head)
    wl = synth.S_LLAMA.with_(name="s-llama-long-prefix", shape=long, new_tokens=12)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=15, page_seed=6)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    greedy = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], greedy, 0, 0)
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("width", [256, 2048], ids=["d256", "d2048"])
def test_one_token_prompt_with_folded_cross_attention(width):
    """A one-sequence T5 context prefilled from a one-token prompt: the prompt's pass through the
    decoder is a single row, the case the one-row folded paths serve, while the folded
    cross-attention (and, at d 2048, the folded-scores products) are still being formed on the
    prefill's second stream; that pass must read the cross K/V instead.  Prefill logits, drafts,
    verify logits and greedy steps follow the oracle."""
    from dataclasses import replace
    sh = replace(synth.SMALL_T5_BF16, name=f"t5-d{width}-p1", n_layers=3, d_model=width,
                 n_heads=width // 64, d_head=64, d_ff=width, vocab=2000, n_visual=32)
    wl = synth.S_T5.with_(name=f"s-t5-d{width}-p1", shape=sh, draft_layers=2, new_tokens=14,
                          prompt_len=1)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=16, page_seed=2, max_batch=1)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    greedy = parity.device_run(dd, pt, vt, wl.new_tokens, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], greedy, 0, 0)
    assert dd.sync_status() == (0, 0)


def test_verify_chunks_past_the_skinny_capacity_take_the_tile_path():
    """Batch 8 with gamma = 16: a verify chunk is 8 x 17 = 136 rows, past the skinny path's 128, so
    the verify's projections run on the tile GEMM (the residual ones over ranges of K) and each
    sequence's 17-row causal self-attention on the MFMA kernel, its keys starting at that
    sequence's cached length.  Every sequence's drafts and verify logits follow the oracle round
    by round, with the accepted lengths bit-exact."""
    wl = synth.S_LLAMA.with_(name="s-llama-b8-g16", gamma=16, new_tokens=40)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=17, batch=8, page_seed=7, extra_seq=wl.gamma)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    for s in range(8):
        parity.check_run_against_oracle(dec, wl.shape, pr[s], z[s], run, s, wl.gamma)


@pytest.mark.parametrize("arch,batch,d_ff", [("t5", 1, 8704), ("t5", 1, 5120), ("llama", 1, 8704),
                                             ("llama", 2, 8704), ("llama", 3, 8704)],
                         ids=["t5-b1", "t5-b1-ff5120", "llama-b1", "llama-b2", "llama-b3"])
def test_wide_skinny_projections_share_input_loads_over_tiles(arch, batch, d_ff):
    """Decoders 1536 wide: at a chunk of at most 8 rows on a 256-unit device the QKV projection
    (288 tiles of 16 features) takes three half tiles a block (QKV epilogue with rotary or
    without), a gated FFN 8704 wide (544 tiles) three whole tiles, one 5120 wide (320 tiles) three
    half tiles of both matrices, and W_o, the cross-attention projections and the down projection
    (96 tiles) one half tile.  Batch 2 also runs the draft steps (2 rows) on those paths; batch 3
    verifies 12-row chunks on the two-plane form with several tiles a block.  Every sequence's
    drafts, verify logits and accepted lengths follow the oracle."""
    from dataclasses import replace
    if arch == "t5":
        sh = replace(synth.SMALL_T5_BF16, name="t5-wide-skinny", n_layers=3, d_model=1536,
                     n_heads=24, d_head=64, d_ff=d_ff, vocab=2000, n_visual=16)
        wl = synth.S_T5.with_(name="s-t5-wide-skinny", shape=sh, draft_layers=2, gamma=5,
                              new_tokens=16)
    else:
        sh = replace(synth.SMALL_LLAMA_BF16, name="llama-wide-skinny", n_layers=3, d_model=1536,
                     n_heads=12, d_head=128, d_ff=d_ff, vocab=2000, n_visual=24)
        wl = synth.S_LLAMA.with_(name="s-llama-wide-skinny", shape=sh, draft_layers=2, gamma=3,
                                 new_tokens=16)
    # stepwise rounds keep drafting a finished sequence at its last length: gamma more positions
    dd, dec, pr, z, pt, vt = _setup(wl, seed=21, batch=batch, page_seed=9, extra_seq=wl.gamma)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    for s in range(batch):
        parity.check_run_against_oracle(dec, wl.shape, pr[s], z[s], run, s, wl.gamma)


@pytest.mark.parametrize("n_visual", [8, 16, 32], ids=["nv8", "nv16", "nv32"])
def test_verify_chunk_folded_cross_attention(n_visual):
    """A one-sequence T5 context (8 heads, n_visual 8, 16 or 32 visual keys): the verify chunk's
    cross-attention runs folded on half tiles, the scores fold_q . rmsnorm(x) with the float32
    matrix split into bf16 hi / lo in the kernel, then x += fold_o . softmax(scores), the softmax
    over groups of n_visual taken in the second launch's input loads.  A two-sequence context of
    the same decoder keeps the query projection, attention launch and output projection.  Both
    runs follow the oracle, and while their token streams agree their verify logits agree within
    the tolerance."""
    from dataclasses import replace
    sh = replace(synth.SMALL_T5_BF16, name=f"t5-fold-chunk-nv{n_visual}", n_layers=4, d_model=512,
                 n_heads=8, d_head=64, d_ff=1024, vocab=2000, n_visual=n_visual)
    wl = synth.S_T5.with_(name=f"s-t5-fold-chunk-nv{n_visual}", shape=sh, draft_layers=2,
                          gamma=5, new_tokens=20)
    runs = []
    for mb in (1, 2):
        dd, dec, pr, z, pt, vt = _setup(wl, seed=23, page_seed=6, max_batch=mb)
        run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
        parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
        assert dd.sync_status() == (0, 0)
        runs.append(run)
    folded, unfolded = runs
    compared = 0
    for i, (ra, rb) in enumerate(zip(folded.rounds, unfolded.rounds)):
        if not (np.array_equal(ra.drafts, rb.drafts) and np.array_equal(ra.targets, rb.targets)):
            break
        for j in range(ra.target_logits.shape[1]):
            parity.check_logits(ra.target_logits[0, j], rb.target_logits[0, j].astype(np.float64),
                                wl.shape, f"round {i} verify {j}")
        compared += 1
    assert compared >= 1


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_longest_draft_and_one_token_jobs(wl):
    """gamma = 32, the largest draft length a context accepts: the verify chunk is 33 rows, three
    16-row groups of the two-plane skinny path with a one-row tail, and a round drafts 32 tokens
    through the captured draft step.  Every draft and verify logit follows the oracle, the
    accepted lengths are bit-exact and the generate loop equals the stepwise calls.  A job of one
    token (T = 1) is the prefill's token alone: no round runs."""
    wl = wl.with_(name=wl.name + "-g32", gamma=32, new_tokens=40)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=21, page_seed=4)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    parity.check_run_against_oracle(dec, wl.shape, pr[0], z[0], run, 0, wl.gamma)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy()[0].tolist() == run.tokens[0]
    assert stats["rounds"] == len(run.rounds)
    assert stats["drafted"] == wl.gamma * stats["rounds"]
    one, st1 = dd.generate(pt, vt, 1, wl.gamma, speculative=True, reuse=True)
    assert one.cpu().numpy()[0].tolist() == run.tokens[0][:1]
    assert st1["rounds"] == 0 and st1["drafted"] == 0
    assert dd.sync_status() == (0, 0)


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_verify_chunk_at_the_skinny_capacity(wl):
    """Batch 32 with gamma = 3: the verify chunk is 32 x 4 = 128 rows, the most the skinny MFMA
    path takes (eight 16-row groups of the two-plane form), and the draft steps are 32-row skinny
    launches; the T5 cross-attention runs unfolded (more than one sequence).  Every sequence's
    drafts and verify logits follow the oracle round by round, with the accepted lengths
    bit-exact, and the generate loop equals the stepwise calls."""
    wl = wl.with_(name=wl.name + "-b32", gamma=3, new_tokens=10)
    dd, dec, pr, z, pt, vt = _setup(wl, seed=23, batch=32, page_seed=9, extra_seq=wl.gamma)
    run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
    assert dd.sync_status() == (0, 0)
    for s in range(32):
        parity.check_run_against_oracle(dec, wl.shape, pr[s], z[s], run, s, wl.gamma)
    toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    assert toks.cpu().numpy().tolist() == run.tokens
    assert stats["rounds"] == len(run.rounds)
    assert dd.sync_status() == (0, 0)
