"""bench.py's algorithmic byte counts, checked against hand sums at the FlanT5-xl and LLaVA shapes."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
import synth  # noqa: E402


def test_draft_step_bytes_flant5_xl():
    sh = synth.FLANT5_XL
    d, f, V, ctx, k = 2048, 5120, 32128, 72, 6
    # per layer: QKVO + cross Q/O at bf16, gated FFN at bf16, three fp32 norm gains
    layer = (4 * d * d + 2 * d * d + 3 * d * f) * 2 + 3 * d * 4 + d * 4
    # KV read at fp32 for ctx positions and the 32 visual keys, one position written
    kv = 2 * ctx * d * 4 + 2 * d * 4 + 2 * 32 * d * 4
    imit = 2 * d * d * 2 + (d + 3 * d) * 4
    head = V * d * 2 + d * 4
    assert bench.draft_step_bytes(sh, k, ctx) == k * (layer + kv) + imit + head
    # the figure the design notes quote (~834 MB at the median context)
    assert 8.2e8 < bench.draft_step_bytes(sh, k, ctx) < 8.5e8


def test_draft_step_bytes_flant5_xl_folded_cross_attention():
    sh = synth.FLANT5_XL
    d, f, V, ctx, k, H, nv = 2048, 5120, 32128, 72, 6, 32, 32
    assert bench.cross_folded(sh, 1) and not bench.cross_folded(sh, 8)
    assert not bench.cross_folded(synth.LLAVA_7B, 1)
    # the cross query / output weights and visual K/V give way to two float32 [H*nv][d] matrices
    layer = (4 * d * d + 3 * d * f) * 2 + 3 * d * 4 + 2 * H * nv * d * 4 + d * 4
    kv = 2 * ctx * d * 4 + 2 * d * 4
    imit = 2 * d * d * 2 + (d + 3 * d) * 4
    head = V * d * 2 + d * 4
    assert bench.draft_step_bytes(sh, k, ctx, 4, True) == k * (layer + kv) + imit + head


def test_verify_bytes_llava():
    sh = synth.LLAVA_7B
    d, f, V, L, ctx, g = 4096, 11008, 32000, 32, 700, 5
    layer = (4 * d * d + 3 * d * f) * 2 + 3 * d * 4
    kv = (2 * ctx * d + 2 * (g + 1) * d) * 4
    assert bench.verify_bytes(sh, 1, g, ctx) == L * (layer + kv) + V * d * 2 + d * 4
    assert 1.3e10 < bench.verify_bytes(sh, 1, g, ctx) < 1.5e10


def test_gpus_other_than_one_exit_with_a_message(capsys, monkeypatch):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    try:
        bench.main()
    except SystemExit as e:
        assert e.code == 2
    assert "one GPU" in capsys.readouterr().err


def test_prefill_flops_llava_matches_the_parameter_count():
    """LLaVA-1.5-7B shape, 576 visual + 32 prompt rows: 2 flops per weight per row over the
    6.48e9 parameters the 32 layers touch, plus causal attention (QK and PV over the lower
    triangle) and the head for the last row, about 7.97 TFLOP."""
    sh = synth.LLAVA_7B
    d, f, V, L, rows = 4096, 11008, 32000, 32, 608
    params = L * (4 * d * d + 3 * d * f)
    attn = L * 2 * rows * rows * d  # 2 (QK, PV) x 2 flops x rows^2 / 2 x (H x dh = d)
    expect = 2.0 * params * rows + attn + 2.0 * V * d
    got = bench.prefill_flops(sh, 1, 32)
    assert abs(got - expect) / expect < 1e-12
    assert 7.9e12 < got < 8.05e12


def test_prefill_flops_flant5_xl_counts_the_visual_projections():
    """FlanT5-xl, 8 prompt rows and 32 visual rows: the prompt through the self-attention and FFN
    projections and the cross query / output, the visual rows through the cross K / V
    projections, self-attention over the prompt and cross-attention to the visual rows."""
    sh = synth.FLANT5_XL
    d, f, V, L, P, nv = 2048, 5120, 32128, 24, 8, 32
    per_layer = (2.0 * (4 * d * d + 3 * d * f) * P + 2.0 * P * P * d
                 + 2.0 * 2 * d * d * nv + 2.0 * 2 * d * d * P + 4.0 * P * nv * d)
    assert bench.prefill_flops(sh, 1, P) == L * per_layer + 2.0 * V * d
