"""Hidden-state export and the fitted imitation network (a data-free stand-in for the paper's
imitation training, Sec. "Deep Representation Imitation"), through the C ABI.

* The exported rows are the decoder's own states: x_k and x_L of the first round against the
  oracle stepped over the same tokens, phi against the oracle's first layer of I applied to x_k.
* Fitting I's second layer on states of other sequences lowers the imitation error on a held-out
  sequence, and decoding with the fitted network still follows the oracle (built with the same
  rounded weights) and still equals greedy decoding token for token.
"""
import copy

import numpy as np
import pytest

import synth
from oracle import decode, ops
from oracle.model import Decoder
from tests import parity

pytestmark = pytest.mark.gpu


def _close(dev, ref, what, rtol=2e-3):
    scale = float(np.sqrt(np.mean(np.square(ref)))) + 1e-12
    err = float(np.max(np.abs(dev - ref)))
    assert err <= rtol * scale, f"{what}: max-abs {err:.3g} > {rtol} x rms {scale:.3g}"


def _device(wl, seed, w):
    from paper_2510_22641_amd import runtime
    dd = runtime.from_workload(wl, seed, weights=w, page_seed=2)
    return dd


@pytest.mark.parametrize("wl", [synth.S_T5, synth.S_LLAMA], ids=lambda w: w.name)
def test_exported_rows_are_the_decoders_states(wl):
    from paper_2510_22641_amd import imitation
    w, z, pr = parity.workload_inputs(wl, 0)
    dd = _device(wl, 0, w)
    pt, vt = dd.upload_inputs(pr, z)
    g = wl.gamma
    phi, xk, xl = imitation.collect(dd, pt[:1], vt[:1], 2, g)  # one round
    assert phi.shape[0] == g and xk.shape == (g, wl.shape.d_model) and xl.shape == xk.shape
    # the oracle stepped over the same tokens: pending, then the device's drafts
    dec = Decoder(wl.shape, w, wl.draft_layers)
    ell = len(pr[0]) + wl.shape.prefix_len()
    st, pending, _ = decode.prefill(dec, pr[0], z[0], ell + g + 1)
    toks = [pending]
    # the collected round's drafts: a second context replays the same first round
    dd2 = _device(wl, 0, w)
    pt2, vt2 = dd2.upload_inputs(pr, z)
    pend, _ = dd2.prefill(pt2[:1], vt2[:1])
    dr, _ = dd2.draft(pend, g)
    toks += [int(t) for t in dr.cpu().numpy()[0, : g - 1]]
    for i, tok in enumerate(toks):
        x = dec.embed([tok])
        x = dec.run_layers(x, [ell + i], st, 0, dec.k)
        _close(xk[i], x[0], f"x_k row {i}")
        gw = dec.g
        h = ops.layer_norm(x, gw["in_ln_w"], gw["in_ln_b"], wl.shape.ln_eps)
        _close(phi[i], ops.gelu_tanh(h @ gw["in_w1"].T + gw["in_b1"])[0], f"phi row {i}")
        x = dec.run_layers(x, [ell + i], st, dec.k, wl.shape.n_layers)
        _close(xl[i], x[0], f"x_L row {i}")
    assert dd.sync_status() == (0, 0) and dd2.sync_status() == (0, 0)


@pytest.mark.parametrize("wl,n_fit", [(synth.S_T5, 16), (synth.S_LLAMA, 24)], ids=["s-t5", "s-llama"])
def test_fitted_imitation_network(wl, n_fit):
    from paper_2510_22641_amd import imitation
    sh = wl.shape
    w, z0, pr0 = parity.workload_inputs(wl, 0)
    dd = _device(wl, 0, w)
    # training states: other sequences (prompts and visual tokens of seeds 100..)
    rows = [[], [], []]
    for s in range(100, 100 + n_fit):
        z = synth.make_visual(sh, s, 1)
        pr = synth.make_prompts(sh, s, 1, wl.prompt_len)
        pt, vt = dd.upload_inputs(pr, z)
        for r, a in zip(rows, imitation.collect(dd, pt, vt, wl.new_tokens, wl.gamma)):
            r.append(a)
    phi, xk, xl = (np.concatenate(r) for r in rows)
    # held-out states: the benchmark sequence itself
    pt0, vt0 = dd.upload_inputs(pr0, z0)
    hphi, hxk, hxl = imitation.collect(dd, pt0, vt0, wl.new_tokens, wl.gamma)
    w2, b2 = imitation.fit(phi, xk, xl, residual=dd.in_residual)

    def err(W2, B2):
        return float(np.mean(np.square(hxk + hphi @ np.asarray(W2, np.float64).T + B2 - hxl)))

    before = err(w["in_w2"], w["in_b2"])
    w2r, b2r = imitation.install(dd, w2, b2)
    after = err(w2r, b2r)
    assert after < 0.5 * before, (before, after)
    # decoding with the fitted network: parity with the oracle, SSD equals greedy
    w_fit = copy.copy(w)
    w_fit["in_w2"], w_fit["in_b2"] = w2r, b2r
    run = parity.device_run(dd, pt0, vt0, wl.new_tokens, wl.gamma, reuse=True)
    dec = Decoder(sh, w_fit, wl.draft_layers)
    parity.check_run_against_oracle(dec, sh, pr0[0], z0[0], run, 0, wl.gamma)
    ssd, st = dd.generate(pt0, vt0, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
    greedy, _ = dd.generate(pt0, vt0, wl.new_tokens, wl.gamma, speculative=False)
    assert np.array_equal(ssd.cpu().numpy(), greedy.cpu().numpy())
    assert dd.sync_status() == (0, 0)
