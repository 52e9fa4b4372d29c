"""The whole drafter forward on the GPU (hspec_drafter_forward) against the float64 oracle:
3 x (Mamba, attention, MLP) + 1 x (Mamba, MLP), |M| = 5 fused target layers, one shared
initial state, three target caches on one page table (Sec. 3.3; App. B.1)."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from gpu_util import assert_close, dev, empty, host  # noqa: E402
from paper_2609_24197_amd import hspec, inputs as I  # noqa: E402

pytestmark = pytest.mark.gpu


def _dev_layers(L):
    out = []
    for W in L:
        d = {k: (hspec.to_device(v) if isinstance(v, np.ndarray) else v) for k, v in W.items()}
        out.append(d)
    return out


def _run(cfg, shared, L, x, pack=False):
    X = dev({k: v for k, v in x.items() if k != "caches"})
    X["caches"] = [dev(c) for c in x["caches"]]
    S = dev(shared)
    if pack:
        S["W_dS_packed"] = hspec.pack_w_ds(S.pop("W_dS"), cfg.d_S, cfg.rank)
    maxL = int(x["ctx_lens"].max())
    ws = hspec.workspace(hspec.drafter_forward_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    out = empty((cfg.B, cfg.k, cfg.d_model))
    hspec.drafter_forward(cfg, S, _dev_layers(L), X, out, ws, maxL)
    return host(out), hspec.read_status(ws)


CASES = {
    "bf16_ragged": I.StepConfig(name="f", B=3, k=16, d_model=256, H=4, P=64, N=64, G=1, chunk=16, Hq=32, Hkv=8,
                                D=128, lengths="list:600,0,77", n_fuse=5, ff=768),
    "f32_tiny": I.CONFIGS[1].replace(n_fuse=5, ff=512),
    "bf16_k7_window": I.StepConfig(name="f", B=2, k=7, d_model=512, H=8, P=64, N=128, G=1, chunk=8, Hq=16, Hkv=4,
                                   D=128, lengths="list:3000,40", n_fuse=5, ff=1024, window=256, block_causal=True),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_drafter_forward(name):
    cfg = CASES[name]
    print(f"[drafter_forward] {name} {cfg}", flush=True)
    shared, L = I.make_drafter_weights(cfg, seed=21)
    x = I.make_drafter_inputs(cfg, seed=21, n_caches=3, extra_pages=2)
    out, st = _run(cfg, shared, L, x)
    assert st == 0
    assert_close(out, O.drafter_forward(L, shared, x, x["caches"], cfg), name)


def test_drafter_forward_full_size():
    """8b-serving-b64 shapes (B 64, k 16, d_model 4096, Mamba H 128 x 64 x 128, Hq 32 / Hkv 8,
    ff 12288, |M| = 5, packed W_dS); the oracle checks requests 0 and 63."""
    cfg = I.CONFIGS[3].replace(n_fuse=I.DRAFTER_FUSE, ff=12288)
    shared, L = I.make_drafter_weights(cfg, seed=22)
    x = I.make_drafter_inputs(cfg, seed=22, n_caches=3)
    out, st = _run(cfg, shared, L, x, pack=True)
    assert st == 0
    idx = [0, cfg.B - 1]
    ref = O.drafter_forward(L, shared, x, x["caches"], cfg, requests=idx)
    assert_close(out[idx], ref[idx], "full-size drafter")
