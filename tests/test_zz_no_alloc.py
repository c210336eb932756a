"""ssd_create_static: a context whose workspace is the library's fixed per-device array, for
callers that cannot allocate.  Its decode output is checked against a context made by ssd_create
(caller-allocated workspace) on the same weights and inputs, on two contexts in a row on one GPU,
the second with a smaller input (it inherits the first one's leftovers in the shared array)."""
import ctypes

import numpy as np
import pytest

import synth
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu


def _run_pair(wl, seed, batch, page_seed):
    """The same stepwise decode on a regular and a static context; returns both runs, the
    static context's generate tokens and the oracle decoder."""
    from paper_2510_22641_amd import runtime
    w, z, pr = parity.workload_inputs(wl, seed, batch)
    runs = {}
    for static in (False, True):
        print(f"[no-alloc] {wl.name} batch {batch} static={static}", flush=True)
        dd = runtime.from_workload(wl, seed, weights=w, max_batch=batch, page_seed=page_seed,
                                   extra_seq=wl.gamma, static=static)
        assert hasattr(dd, "workspace") != static
        pt, vt = dd.upload_inputs(pr, z)
        run = parity.device_run(dd, pt, vt, wl.new_tokens, wl.gamma, reuse=True)
        assert dd.sync_status() == (0, 0)
        toks, stats = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
        assert dd.sync_status() == (0, 0)
        runs[static] = (run, toks.cpu().numpy().tolist(), stats)
        dd.close()
    return runs, Decoder(wl.shape, w, wl.draft_layers), pr, z


def _compare(wl, runs, dec, pr, z, batch):
    (reg, reg_gen, reg_st), (sta, sta_gen, sta_st) = runs[False], runs[True]
    assert sta_gen == sta.tokens  # the loop equals the stepwise calls on the static context
    for b in range(batch):
        parity.check_run_against_oracle(dec, wl.shape, pr[b], z[b], sta, b, wl.gamma)
        parity.check_streams_agree_until_near_tie(dec, wl.shape, pr[b], z[b], sta.tokens[b],
                                                  reg.tokens[b], f"{wl.name} seq {b}")
    parity.check_logits(sta.prefill_logits[0], reg.prefill_logits[0].astype(np.float64),
                        wl.shape, "prefill")
    for i, (ra, rb) in enumerate(zip(sta.rounds, reg.rounds)):
        if not (np.array_equal(ra.drafts, rb.drafts) and np.array_equal(ra.targets, rb.targets)):
            break
        for b in range(batch):
            if not ra.active[b]:
                continue
            for j in range(wl.gamma):
                parity.check_logits(ra.draft_logits[b, j], rb.draft_logits[b, j].astype(np.float64),
                                    wl.shape, f"round {i} seq {b} draft {j}")
            for j in range(wl.gamma + 1):
                parity.check_logits(ra.target_logits[b, j],
                                    rb.target_logits[b, j].astype(np.float64), wl.shape,
                                    f"round {i} seq {b} verify {j}")


def test_static_context_matches_regular_twice():
    # first: a ragged LLaMA-style batch of three (the same kernels as the regular context)
    first = synth.S_LLAMA
    runs, dec, pr, z = _run_pair(first, 3, 3, 7)
    _compare(first, runs, dec, pr, z, 3)
    assert runs[True][1] == runs[False][1]  # no folding difference here: the same tokens
    # second, smaller: one T5-style sequence with fewer tokens (the static context keeps the
    # cross-attention unfolded, the regular one folds it)
    second = synth.S_T5.with_(new_tokens=14)
    assert (1 * second.shape.d_model * second.max_seq() <
            3 * first.shape.d_model * first.max_seq())
    runs, dec, pr, z = _run_pair(second, 4, 1, 5)
    _compare(second, runs, dec, pr, z, 1)


def test_static_context_refusals():
    from paper_2510_22641_amd import runtime, ssd as abi
    # a LLaVA-7B-sized context needs far more than the fixed array: refused before any device
    # work (the descriptors are only checked for null pointers)
    big = runtime.DeviceDecoder(synth.LLAVA_7B, 8,
                                runtime.Capacity(max_batch=1, max_gamma=5, max_seq=870,
                                                 max_prompt=32))
    dims = big.dims()
    assert abi.ssd_workspace_bytes(dims) > abi.SSD_STATIC_SCRATCH_BYTES
    one = ctypes.c_void_p(256)
    layers = (abi.ssd_layer_weights * dims.n_layers)()
    for l in range(dims.n_layers):
        for f in abi.LAYER_FIELDS:
            setattr(layers[l], f, one)
    w = abi.ssd_weights()
    for f in abi.GLOBAL_FIELDS:
        setattr(w, f, one)
    w.layers = ctypes.cast(layers, ctypes.POINTER(abi.ssd_layer_weights))
    kv = abi.ssd_kv()
    kv.k_pool = kv.v_pool = kv.page_table = kv.seq_len = one
    kv.n_pages = 1
    ctx = ctypes.c_void_p()
    rc = abi._lib.ssd_create_static(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(kv), None,
                                    ctypes.byref(ctx))
    assert rc == abi.SSD_ERR_CAPACITY and not ctx.value
    # one live static context per device
    wl = synth.S1.with_(new_tokens=6)
    dd = runtime.from_workload(wl, 0, static=True)
    dd2 = runtime.DeviceDecoder(wl.shape, wl.draft_layers, dd.cap)
    dd2.load_dict(synth.workload_weights(wl, 0, threads=4))
    with pytest.raises(abi.SSDError) as e:
        dd2.create(static=True)
    assert e.value.code == abi.SSD_ERR_STATE
    dd.close()
    dd2.create(static=True)  # free again once the first is destroyed
    dd2.close()
