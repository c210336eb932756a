"""The seeded input generators: bf16 rounding against torch's conversion, determinism, ranges."""
import numpy as np
import torch

import synth
from synth.generate import make_tensor


def test_round_to_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-8, 8, 100000).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, -0.0], np.float32)])
    ours = synth.round_to_bf16(x)
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(ours.view(np.uint32), want.view(np.uint32))
    # ties go to even: 1 + 2^-8 sits halfway between 1 and 1 + 2^-7
    assert ours[-5] == 1.0 and ours[-4] == np.float32(1.0 + 2 ** -6)


def test_tensors_are_deterministic_and_independent_of_order():
    sh = synth.SMALL_T5_BF16
    a = synth.make_weights(sh, 3, 0.5, 2, threads=1)
    b = synth.make_weights(sh, 3, 0.5, 2, threads=4)
    for n in ("embed", "lm_head", "in_w2"):
        assert np.array_equal(a[n], b[n])
    for la, lb in zip(a["layers"], b["layers"]):
        for n in la:
            assert np.array_equal(la[n], lb[n])
    c = synth.make_weights(sh, 4, 0.5, 2, threads=1)
    assert not np.array_equal(a["embed"], c["embed"])


def test_deep_scale_applies_to_output_projections_beyond_boundary():
    sh = synth.SMALL_T5_BF16
    one = synth.make_weights(sh, 1, 1.0, 2, threads=1)
    half = synth.make_weights(sh, 1, 0.5, 2, threads=1)
    for l in range(sh.n_layers):
        for n in ("wo", "xo", "w_down"):
            ratio = 0.5 if l >= 2 else 1.0
            # bf16 rounding commutes with multiplication by a power of two
            assert np.array_equal(half["layers"][l][n], one["layers"][l][n] * np.float32(ratio))
        assert np.array_equal(half["layers"][l]["wq"], one["layers"][l]["wq"])
    assert np.array_equal(half["in_w2"], one["in_w2"] * np.float32(0.5))


def test_value_ranges():
    sh = synth.SMALL_LLAMA_BF16
    p = synth.make_prompts(sh, 0, 3, 500)
    assert p.dtype == np.int32 and p.min() >= 0 and p.max() < sh.vocab and p.shape == (3, 500)
    z = synth.make_visual(sh, 0, 2)
    assert z.shape == (2, sh.n_visual, sh.d_model) and abs(z.std() - 1) < 0.05
    assert np.array_equal(synth.round_to_bf16(z), z)
    g = make_tensor(sh, 0, "attn_norm", 0, 20, "gain")
    assert abs(g.mean() - 1) < 0.01
