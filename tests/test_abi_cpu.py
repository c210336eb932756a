"""Host-side checks of the C ABI that need no GPU: the library loads, exports every function the
header declares, sizes workspaces and rejects invalid dimensions before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _built():
    lib = os.path.join(ROOT, "paper_2510_22641_amd", "libssd.so")
    if not os.path.exists(lib):
        import __graft_entry__
        __graft_entry__.build()
    return lib


def _declared():
    src = open(os.path.join(ROOT, "include", "ssd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ssd_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(_built())
    names = _declared()
    assert "ssd_prefill" in names and "ssd_draft" in names and "ssd_verify" in names
    assert "ssd_accept" in names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_the_header():
    _built()
    from paper_2510_22641_amd import ssd as abi
    assert sorted(abi.EXPORTS) == _declared()
    assert ctypes.sizeof(abi.ssd_dims) == 24 * 4


def _dims(**kw):
    from paper_2510_22641_amd import ssd as abi
    d = abi.ssd_dims()
    vals = dict(arch=0, n_layers=4, d_model=256, n_heads=4, d_head=64, d_ff=1024, vocab=1024,
                n_visual=32, rel_buckets=32, rel_max_dist=128, rope_theta=1e4, norm_eps=1e-6,
                ln_eps=1e-5, wdtype=0, kvdtype=0, draft_layers=1, in_hidden=256, in_residual=1,
                max_batch=1, max_gamma=4, max_seq=64, max_prompt=8, page_size=16, max_pages=4)
    vals.update(kw)
    for k, v in vals.items():
        setattr(d, k, v)
    return d


def test_workspace_and_dimension_checks():
    _built()
    from paper_2510_22641_amd import ssd as abi
    assert abi.ssd_workspace_bytes(_dims()) > 0
    assert abi.ssd_workspace_bytes(_dims(max_batch=8)) > abi.ssd_workspace_bytes(_dims())
    for bad in (dict(d_model=200), dict(d_head=96), dict(draft_layers=0), dict(draft_layers=5),
                dict(max_pages=3), dict(max_seq=4096), dict(arch=2), dict(max_prompt=100),
                dict(d_ff=1000)):
        assert abi.ssd_workspace_bytes(_dims(**bad)) == 0, bad
    ctx = ctypes.c_void_p()
    rc = abi._lib.ssd_create(ctypes.byref(_dims(d_head=96)), ctypes.byref(abi.ssd_weights()),
                             ctypes.byref(abi.ssd_kv()), 256, 1 << 20, None, ctypes.byref(ctx))
    assert rc == abi.SSD_ERR_SHAPE
    rc = abi._lib.ssd_create(ctypes.byref(_dims()), ctypes.byref(abi.ssd_weights()),
                             ctypes.byref(abi.ssd_kv()), 256, 1 << 20, None, ctypes.byref(ctx))
    assert rc == abi.SSD_ERR_ARG  # null weight pointers, detected before any device call
    assert abi.status_string(abi.SSD_ERR_CAPACITY) == "capacity exceeded"
    with pytest.raises(abi.SSDError):
        abi.ssd_prefill(None, 1, 1, 0, 0, 0)


def test_dynamic_draft_length_matches_the_oracle():
    """The library's host-side schedule (ssd_dynamic_gamma) equals the oracle's d(t)."""
    from oracle import decode
    lib = ctypes.CDLL(_built())
    f = lib.ssd_dynamic_gamma
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    for n_max in (142, 512, 870, 4096):
        for d0 in (1, 5):
            for t in range(0, 5000, 7):
                assert f(t, d0, n_max) == decode.dynamic_draft_length(t, d0, n_max), (t, d0, n_max)
