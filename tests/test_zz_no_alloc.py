"""hspec_paged_attn_static (the attention core on the library's fixed device array, for callers
that cannot allocate) against hspec_paged_attn with a caller workspace: bitwise equal outputs
on two calls in a row, the second with a smaller input, and within the tolerance of the float64
oracle.  Runs alone in a fresh process or after the other GPU tests."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from gpu_util import assert_close, dev, empty, host  # noqa: E402
from paper_2609_24197_amd import hspec, inputs as I  # noqa: E402

pytestmark = pytest.mark.gpu


def _cfg(**kw):
    base = dict(name="na", B=5, k=16, d_model=256, H=4, P=64, N=16, G=1, chunk=16, Hq=32, Hkv=8, D=128,
                lengths="list:3000,0,77,1500,700", dtype="bf16", split_tokens=512)
    base.update(kw)
    return I.StepConfig(**base)


def _both(cfg, seed):
    x = I.make_attn_inputs(cfg, seed=seed, extra_pages=2)
    d = dev(x)
    maxL = int(max(x["ctx_lens"]))
    need = hspec.paged_attn_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL)
    assert need <= hspec.STATIC_WS_BYTES
    o_ref = empty((cfg.B, cfg.k, cfg.Hq, cfg.D))
    ws = hspec.workspace(need)
    hspec.paged_attn(cfg, d, o_ref, ws, maxL)
    o = empty((cfg.B, cfg.k, cfg.Hq, cfg.D))
    o.fill_(float("nan"))
    st = empty((1,), "i32")
    st.fill_(-1)
    hspec.paged_attn_static(cfg, d, o, maxL, status=st)
    return x, host(o), host(o_ref), int(host(st)[0]), hspec.read_status(ws)


def test_static_workspace_matches_caller_workspace():
    big = _cfg()
    small = _cfg(B=2, lengths="list:130,40", split_tokens=0, Hq=16, Hkv=4)
    for cfg, seed in ((big, 41), (small, 42)):
        print(f"[paged_attn_static] {cfg}", flush=True)
        x, o, o_ref, st, st_ref = _both(cfg, seed)
        assert st == 0 and st_ref == 0
        assert np.array_equal(o, o_ref), "static-workspace output differs from the caller-workspace output"
        ref = O.paged_attention(x["q"], x["k_blk"], x["v_blk"], x["k_cache"], x["v_cache"], x["page_table"],
                                x["ctx_lens"], page_size=cfg.page_size)
        assert_close(o, ref, "static workspace")


def test_static_workspace_rejects_oversize():
    """An attention whose workspace exceeds the fixed array is refused before any launch."""
    cfg = I.CONFIGS[5]
    ac = hspec.attn_cfg(cfg, 1024, 300000)
    import ctypes as C
    s = hspec.lib().hspec_paged_attn_static(C.byref(ac), *([C.c_void_p(1 << 20)] * 7), 16384,
                                            C.c_void_p(1 << 20), None, None)
    assert s == 5 and b"HSPEC_STATIC_WS_BYTES" in hspec.lib().hspec_last_error()
