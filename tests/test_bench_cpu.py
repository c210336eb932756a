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
