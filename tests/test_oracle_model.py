"""Pins of the oracle decoder: closed forms of degenerate layers, causality, the relative form of
the rotary scores, bias direction, imitation-network special cases."""
from dataclasses import replace

import numpy as np
import pytest

import synth
from oracle import ops
from oracle.model import Decoder
from oracle.decode import prefill

T5 = replace(synth.SMALL_T5_BF16, name="t5-tiny", n_layers=3, d_model=32, n_heads=2, d_head=8,
             d_ff=24, vocab=50, n_visual=3, dtype="f32")
LL = replace(synth.SMALL_LLAMA_BF16, name="llama-tiny", n_layers=3, d_model=32, n_heads=2,
             d_head=8, d_ff=24, vocab=50, n_visual=4, dtype="f32")


def _weights(shape, seed=0, scale=1.0):
    return synth.make_weights(shape, seed, scale, 1, threads=1)


@pytest.mark.parametrize("shape", [T5, LL])
def test_zero_branches_leave_the_residual_untouched(shape):
    w = _weights(shape)
    for lw in w["layers"]:
        lw["wo"][:] = 0
        lw["w_down"][:] = 0
        if "xo" in lw:
            lw["xo"][:] = 0
    dec = Decoder(shape, w, 1)
    st = dec.new_state(16)
    z = synth.make_visual(shape, 0, 1)[0]
    dec.set_visual(st, z)
    x0 = dec.embed([7, 3, 9])
    x = dec.run_layers(x0.copy(), [0, 1, 2], st, 0, shape.n_layers)
    assert np.array_equal(x, x0)
    g = w["final_norm"].astype(np.float64)
    e = x0[1]
    want = w["lm_head"].astype(np.float64) @ (g * e / np.sqrt(np.mean(e * e) + shape.norm_eps))
    assert np.allclose(dec.head(x[1:2])[0], want, atol=1e-13)


@pytest.mark.parametrize("shape", [T5, LL])
def test_first_position_attention_collapses_to_value(shape):
    # one key: self-attention output is W_o W_v h regardless of bias or scale; with a single visual
    # token the cross-attention output is W_xo W_xv z
    shape = replace(shape, n_visual=1)
    w = _weights(shape, seed=3)
    dec = Decoder(shape, w, 1)
    st = dec.new_state(4)
    z = synth.make_visual(shape, 3, 1)[0]
    dec.set_visual(st, z)
    lw = dec.layers[0]
    x = dec.embed([11])
    eps = shape.norm_eps
    h = ops.rms_norm(x, lw["attn_norm"], eps)
    y = x + (lw["wv"] @ h[0]) @ lw["wo"].T
    if shape.arch == "t5":
        y = y + (lw["xv"] @ z[0].astype(np.float64)) @ lw["xo"].T
    h2 = ops.rms_norm(y, lw["ffn_norm"], eps)
    act = ops.gelu_tanh if shape.arch == "t5" else ops.silu
    y = y + (act(h2 @ lw["w_gate"].T) * (h2 @ lw["w_up"].T)) @ lw["w_down"].T
    assert np.allclose(dec.layer(0, x, [0], st), y, atol=1e-12)


@pytest.mark.parametrize("shape", [T5, LL])
def test_block_equals_position_serial(shape):
    w = _weights(shape, seed=5)
    dec = Decoder(shape, w, 2)
    z = synth.make_visual(shape, 5, 1)[0]
    toks = [4, 8, 15, 16, 23, 42]
    a = dec.new_state(8)
    dec.set_visual(a, z)
    xa = dec.run_layers(dec.embed(toks), list(range(6)), a, 0, shape.n_layers)
    b = dec.new_state(8)
    dec.set_visual(b, z)
    xb = np.concatenate([dec.run_layers(dec.embed([t]), [p], b, 0, shape.n_layers)
                         for p, t in enumerate(toks)])
    assert np.allclose(xa, xb, atol=1e-12)
    assert np.allclose(a.K[:, :6], b.K[:, :6], atol=1e-12)


@pytest.mark.parametrize("shape", [T5, LL])
def test_causality(shape):
    w = _weights(shape, seed=6)
    dec = Decoder(shape, w, 2)
    z = synth.make_visual(shape, 6, 1)[0]
    outs = []
    for tail in ([1, 2, 3], [30, 31, 49]):
        st = dec.new_state(8)
        dec.set_visual(st, z)
        outs.append(dec.run_layers(dec.embed([5, 6] + tail), list(range(5)), st, 0,
                                   shape.n_layers))
    assert np.array_equal(outs[0][:2], outs[1][:2])
    assert not np.allclose(outs[0][2:], outs[1][2:])


def test_llama_scores_use_relative_rotation():
    # at position 1 the two scores are rope(q, 1 - j) . k_j / sqrt(dh) for keys j = 0, 1, with q and
    # k the unrotated projections (relative form of the rotary identity)
    w = _weights(LL, seed=7)
    dec = Decoder(LL, w, 1)
    st = dec.new_state(4)
    lw = dec.layers[0]
    x = dec.embed([17, 29])
    h = ops.rms_norm(x, lw["attn_norm"], LL.norm_eps)
    H, dh = LL.n_heads, LL.d_head
    q = (h @ lw["wq"].T).reshape(2, H, dh)
    k = (h @ lw["wk"].T).reshape(2, H, dh)
    v = (h @ lw["wv"].T).reshape(2, H, dh)
    o = np.empty((H, dh))
    for hh in range(H):
        s = np.array([ops.rope(q[1, hh], 1 - j, LL.rope_theta) @ k[j, hh] for j in (0, 1)])
        s /= np.sqrt(dh)
        p = np.exp(s - s.max())
        p /= p.sum()
        o[hh] = p[0] * v[0, hh] + p[1] * v[1, hh]
    y = dec.layer(0, x, [0, 1], st)
    attn = x[1] + o.reshape(-1) @ lw["wo"].T
    h2 = ops.rms_norm(attn, lw["ffn_norm"], LL.norm_eps)
    want = attn + (ops.silu(h2 @ lw["w_gate"].T) * (h2 @ lw["w_up"].T)) @ lw["w_down"].T
    assert np.allclose(y[1], want, atol=1e-12)


def test_t5_bias_direction_selects_previous_position():
    # a dominant bias on bucket 1 (distance 1) makes every position p >= 1 attend to p-1,
    # on bucket 0 to itself
    w = _weights(T5, seed=8)
    dec = Decoder(T5, w, 1)
    st = dec.new_state(8)
    dec.set_visual(st, synth.make_visual(T5, 8, 1)[0])
    lw = dec.layers[0]
    x = dec.embed([5, 9, 13, 2])
    h = ops.rms_norm(x, lw["attn_norm"], T5.norm_eps)
    v = (h @ lw["wv"].T).reshape(4, T5.n_heads, T5.d_head)
    q = (h @ lw["wq"].T).reshape(4, T5.n_heads, T5.d_head)
    k = (h @ lw["wk"].T).reshape(4, T5.n_heads, T5.d_head)
    for bucket, shift in ((1, 1), (0, 0)):
        dec.g["rel_bias"] = np.full((32, T5.n_heads), -1e4)
        dec.g["rel_bias"][bucket] = 1e4
        st.K[0, :4], st.V[0, :4] = k, v
        for p in range(1, 4):
            o = ops.attend(q[p], st.K[0, :p + 1], st.V[0, :p + 1], dec.self_bias(p, p + 1), 1.0)
            assert np.allclose(o, v[p - shift], atol=1e-12)


def test_imitation_network_special_cases():
    w = _weights(T5, seed=9)
    dec = Decoder(T5, w, 1)
    x = np.random.default_rng(0).standard_normal((2, T5.d_model))
    dec.g["in_w2"][:] = 0
    dec.g["in_b2"][:] = 0
    assert np.array_equal(dec.imitation(x), x)
    dec = Decoder(T5, w, 1)
    dec.g["in_w1"][:] = 0
    c = dec.g["in_b1"]
    want = x + dec.g["in_w2"] @ ops.gelu_tanh(c) + dec.g["in_b2"]
    assert np.allclose(dec.imitation(x), want, atol=1e-13)
    lit = Decoder(T5, w, 1, in_residual=False)
    lit.g["in_w1"][:] = 0
    assert np.allclose(lit.imitation(x), want - x, atol=1e-13)


def test_llama_prefix_uses_visual_rows_as_inputs():
    w = _weights(LL, seed=10)
    dec = Decoder(LL, w, 1)
    z = synth.make_visual(LL, 10, 1)[0]
    st, y, lg = prefill(dec, [1, 2], z, 16)
    assert st.seq_len == LL.n_visual + 2
    st2 = dec.new_state(16)
    x = np.concatenate([z.astype(np.float64), dec.embed([1, 2])])
    x = dec.run_layers(x, list(range(LL.n_visual + 2)), st2, 0, LL.n_layers)
    assert np.array_equal(dec.head(x[-1:])[0], lg)
    assert y == int(np.argmax(lg))


def test_draft_logits_are_head_of_imitation_of_layer_k():
    w = _weights(T5, seed=11)
    dec = Decoder(T5, w, 2)
    z = synth.make_visual(T5, 11, 1)[0]
    a = dec.new_state(8)
    dec.set_visual(a, z)
    lg, xk = dec.draft_step(a, 7, 0)
    b = dec.new_state(8)
    dec.set_visual(b, z)
    full, xk_full = dec.full_step(b, 7, 0)
    assert np.array_equal(xk, xk_full)
    assert np.array_equal(lg, dec.head(dec.imitation(xk[None]))[0])
    assert np.array_equal(dec.draft_step(a, 7, 0, use_imitation=False)[0], dec.head(xk[None])[0])


def _golden_bucket_of():
    """distance -> bucket from the integer thresholds in tests/golden/t5_buckets.txt"""
    import os
    firsts = []
    with open(os.path.join(os.path.dirname(__file__), "golden", "t5_buckets.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, n = map(int, line.split())
                firsts.append((n, b))

    def bucket(n):
        return max(b for first, b in firsts if first <= n)
    return bucket


def test_t5_layer_by_explicit_loops():
    # One whole T5 decoder layer over positions 0..4 (with 3 visual tokens), written out with
    # scalar loops over heads, keys and visual tokens, independent of ops.attend and of the
    # oracle's bucket function.  The relative-bias table holds a distinct N(0,1) value per
    # (bucket, head) and the attention projections are scaled so that q.k is O(1): a dropped
    # bias, a 1/sqrt(dh) scale on self- or cross-attention scores, or the cross keys taken from
    # W_xv instead of W_xk each move the output far beyond the tolerance.
    import math
    shape = T5
    w = _weights(shape, seed=12)
    rng = np.random.default_rng(12)
    w["rel_bias"] = rng.standard_normal((shape.rel_buckets, shape.n_heads))
    for name in ("wq", "wk", "xq", "xk"):
        w["layers"][0][name] = w["layers"][0][name] * 8.0
    dec = Decoder(shape, w, 1)
    z = synth.make_visual(shape, 12, 1)[0].astype(np.float64)
    st = dec.new_state(8)
    dec.set_visual(st, z)
    toks = [3, 41, 17, 8, 29]
    x = dec.embed(toks)
    got = dec.layer(0, x.copy(), list(range(len(toks))), st)

    lw = {n: np.asarray(a, dtype=np.float64) for n, a in w["layers"][0].items()}
    H, dh, eps, nv = shape.n_heads, shape.d_head, shape.norm_eps, shape.n_visual
    bucket = _golden_bucket_of()
    table = np.asarray(w["rel_bias"], dtype=np.float64)

    def rms(row, gain):
        ms = sum(float(v) * float(v) for v in row) / len(row)
        return np.array([gain[i] * row[i] / math.sqrt(ms + eps) for i in range(len(row))])

    def softmax_list(s):
        m = max(s)
        e = [math.exp(v - m) for v in s]
        t = sum(e)
        return [v / t for v in e]

    P = len(toks)
    hs = [rms(x[p], lw["attn_norm"]) for p in range(P)]
    qs = [lw["wq"] @ hs[p] for p in range(P)]
    ks = [lw["wk"] @ hs[p] for p in range(P)]
    vs = [lw["wv"] @ hs[p] for p in range(P)]
    zk = [lw["xk"] @ z[j] for j in range(nv)]
    zv = [lw["xv"] @ z[j] for j in range(nv)]
    want = np.empty_like(x)
    for p in range(P):
        o = np.zeros(H * dh)
        for h in range(H):
            sl = slice(h * dh, (h + 1) * dh)
            s = []
            for j in range(p + 1):
                dot = sum(qs[p][sl][e] * ks[j][sl][e] for e in range(dh))
                s.append(dot + table[bucket(p - j), h])  # unscaled, plus the relative bias
            pr = softmax_list(s)
            for j in range(p + 1):
                o[sl] += pr[j] * vs[j][sl]
        y = x[p] + lw["wo"] @ o
        hq = rms(y, lw["xattn_norm"])
        xq = lw["xq"] @ hq
        o = np.zeros(H * dh)
        for h in range(H):
            sl = slice(h * dh, (h + 1) * dh)
            s = [sum(xq[sl][e] * zk[j][sl][e] for e in range(dh)) for j in range(nv)]
            pr = softmax_list(s)  # no scale, no bias, no mask
            for j in range(nv):
                o[sl] += pr[j] * zv[j][sl]
        y = y + lw["xo"] @ o
        hf = rms(y, lw["ffn_norm"])
        g = lw["w_gate"] @ hf
        u = lw["w_up"] @ hf
        c = math.sqrt(2.0 / math.pi)
        a = np.array([0.5 * g[i] * (1.0 + math.tanh(c * (g[i] + 0.044715 * g[i] ** 3))) * u[i]
                      for i in range(len(g))])
        want[p] = y + lw["w_down"] @ a
    # the scores matter: the bias and the q.k products both move the attention weights by O(1)
    assert np.max(np.abs(want - got)) < 1e-12 * max(1.0, np.max(np.abs(want)))
