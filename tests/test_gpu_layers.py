"""GPU parity of the layer-level calls and the drafting step against the float64 oracle."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from gpu_util import assert_close, dev, empty, host  # noqa: E402
from paper_2609_24197_amd import hspec, inputs as I  # noqa: E402

pytestmark = pytest.mark.gpu

SMALL = {
    "cfg1": I.CONFIGS[1],
    "small_bf16": I.StepConfig(name="s", B=3, k=16, d_model=512, H=8, P=64, N=128, G=1, chunk=16, Hq=32, Hkv=8,
                               D=128, lengths="list:300,0,77"),
    "k7_chunk4_g2": I.StepConfig(name="s", B=2, k=7, d_model=256, H=4, P=64, N=16, G=2, chunk=4, Hq=8, Hkv=2,
                                 D=128, lengths="list:45,200"),
    "window_causal": I.StepConfig(name="s", B=2, k=16, d_model=256, H=4, P=64, N=128, G=1, chunk=8, Hq=32, Hkv=8,
                                  D=128, lengths="list:900,100", window=256, block_causal=True),
    # B*k = 160 rows: the pipelined dense GEMMs, the fused Q/K/V product with a ragged last tile
    "m160_fused_qkv": I.StepConfig(name="s", B=10, k=16, d_model=320, H=5, P=64, N=32, G=1, chunk=16, Hq=8,
                                   Hkv=2, D=128, lengths="uniform:1:700"),
    # B*k = 640 rows: the 256 x 256 products, with k-split last tiles (in_proj, out_proj with
    # hi/lo inputs; Q/K/V over weight segments of 4096 and 1024 rows; O projection)
    "m640_large_tiles": I.StepConfig(name="s", B=40, k=16, d_model=512, H=8, P=64, N=16, G=1, chunk=16, Hq=32,
                                     Hkv=8, D=128, lengths="uniform:0:300"),
    # fp32 storage with the 4-tap conv (token-parallel conv kernel, fp32 weights), ragged k
    "f32_conv4": I.StepConfig(name="s", B=2, k=5, d_model=256, H=4, P=64, N=16, G=1, chunk=4, Hq=8, Hkv=2,
                              D=128, lengths="list:33,150", dtype="f32"),
    # head dim 64 (8 lanes per head in the q/k norm and rotation)
    "d64_k7": I.StepConfig(name="s", B=2, k=7, d_model=256, H=4, P=64, N=16, G=1, chunk=4, Hq=4, Hkv=2,
                           D=64, lengths="list:10,90"),
    # a 3-tap conv (the serial conv kernel)
    "conv3_k5": I.StepConfig(name="s", B=2, k=5, d_model=256, H=4, P=64, N=32, G=2, chunk=5, Hq=8, Hkv=2,
                             D=128, lengths="list:0,60", conv_w=3),
    # hi/lo attention I/O, block keys in fp32 in the reduction (as in the whole drafter)
    "precise_io": I.StepConfig(name="s", B=3, k=16, d_model=512, H=8, P=64, N=128, G=1, chunk=16, Hq=32, Hkv=8,
                               D=128, lengths="list:300,0,77", precise_io=True),
    # the drafting step's grouped scan (4 heads of a request per workgroup) over several B/C
    # groups: N = 64 with 2 groups of 4 heads, N = 32 with 4 groups of 4 heads
    "grp_n64_g2": I.StepConfig(name="s", B=3, k=16, d_model=512, H=8, P=64, N=64, G=2, chunk=16, Hq=32, Hkv=8,
                               D=128, lengths="list:300,0,77"),
    "grp_n32_g4": I.StepConfig(name="s", B=2, k=16, d_model=256, H=16, P=64, N=32, G=4, chunk=16, Hq=8, Hkv=2,
                               D=128, lengths="list:120,40"),
    # the grouped scan with a block shorter than its 16-token tile (lanes past the block read
    # token 0 and drop it)
    "grp_k5": I.StepConfig(name="s", B=2, k=5, d_model=256, H=8, P=64, N=64, G=2, chunk=8, Hq=8, Hkv=2,
                           D=128, lengths="list:50,300"),
    # the drafter reuses 4 of the target's 8 KV heads (16 query heads)
    "kv_subset": I.StepConfig(name="s", B=3, k=16, d_model=512, H=8, P=64, N=128, G=1, chunk=16, Hq=16, Hkv=4,
                              D=128, lengths="list:300,0,77", Hkv_target=8, kv_heads=(0, 2, 4, 6)),
}


def _weights(cfg, seed=0):
    W = I.make_weights(cfg, seed)
    return W, dev(W)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_mamba_block_scan(name):
    cfg = SMALL[name]
    print(f"[mamba_block_scan] {name}", flush=True)
    W, Wd = _weights(cfg, 1)
    x = I.make_inputs(cfg, seed=1)
    d = dev(dict(h_last=x["h_last"], u=x["block_emb"]))
    ws = hspec.workspace(hspec.mamba_block_scan_workspace(cfg))
    out = empty((cfg.B, cfg.k, cfg.d_model))
    Sf = empty((cfg.B, cfg.H, cfg.P, cfg.N))
    hspec.mamba_block_scan(cfg, Wd, d["h_last"], d["u"], out, ws, S_final=Sf)
    S0, _ = O.state_init(x["h_last"], W["W_r"], W["W_dS"], cfg.H, cfg.P, cfg.N)
    ref, parts = O.mamba_mixer(O.f64(x["block_emb"]), S0, W, cfg, return_parts=True)
    assert_close(host(out), ref, "out")
    assert_close(host(Sf), parts["S_final"], "S_final")


@pytest.mark.parametrize("name", sorted(SMALL))
def test_target_kv_block_attn(name):
    cfg = SMALL[name]
    print(f"[target_kv_block_attn] {name}", flush=True)
    W, Wd = _weights(cfg, 2)
    x = I.make_inputs(cfg, seed=2, extra_pages=2)
    xin = I.normal("attn_x", (cfg.B, cfg.k, cfg.d_model), 1.0, 2, cfg.dtype)
    d = dev(dict(x, xin=xin))
    maxL = int(max(x["ctx_lens"]))
    ws = hspec.workspace(hspec.target_kv_block_attn_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    out = empty((cfg.B, cfg.k, cfg.d_model))
    hspec.target_kv_block_attn(cfg, Wd, d["xin"], d, out, ws, maxL)
    ref = O.attention_layer(O.f64(xin), W, x, cfg)
    assert_close(host(out), ref, "out")
    assert hspec.read_status(ws) == 0


def _draft(cfg, W, Wd, x, maxL=None):
    d = dev(x)
    maxL = int(max(x["ctx_lens"])) if maxL is None else maxL
    ws = hspec.workspace(hspec.draft_step_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    out = empty((cfg.B, cfg.k, cfg.d_model))
    hspec.draft_step(cfg, Wd, d, out, ws, maxL)
    return host(out), hspec.read_status(ws)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_draft_step_small(name):
    cfg = SMALL[name]
    print(f"[draft_step] {name}", flush=True)
    W, Wd = _weights(cfg, 3)
    x = I.make_inputs(cfg, seed=3)
    out, st = _draft(cfg, W, Wd, x)
    assert st == 0
    assert_close(out, O.draft_step(W, x, cfg), "out")


@pytest.mark.parametrize("name", ["small_bf16", "window_causal"])
def test_draft_step_packed(name):
    """The drafting step with W_dS in the packed layout gives the same outputs."""
    cfg = SMALL[name]
    W, Wd = _weights(cfg, 6)
    x = I.make_inputs(cfg, seed=6)
    Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    out, st = _draft(cfg, W, Wd, x)
    assert st == 0
    assert_close(out, O.draft_step(W, x, cfg), "out")


def test_draft_step_zero_inputs():
    """e = 0 and h_last = 0: out = W_o mean(V over cache and block) per query head."""
    cfg = SMALL["small_bf16"]
    W, Wd = _weights(cfg, 4)
    x = I.make_inputs(cfg, seed=4)
    x["h_last"] = np.zeros_like(x["h_last"])
    x["block_emb"] = np.zeros_like(x["block_emb"])
    out, _ = _draft(cfg, W, Wd, x)
    assert_close(out, O.draft_step(W, x, cfg), "out")


def test_draft_step_deterministic():
    cfg = SMALL["small_bf16"]
    W, Wd = _weights(cfg, 5)
    x = I.make_inputs(cfg, seed=5)
    a, _ = _draft(cfg, W, Wd, x)
    b, _ = _draft(cfg, W, Wd, x)
    assert np.array_equal(a, b)


@pytest.mark.slow
@pytest.mark.timeout(900)
@pytest.mark.parametrize("num", [2, 3, 4, 5])
def test_draft_step_full_config(num):
    """The full-size workloads, in the launch configuration the benchmark times, every request
    of the batch compared element by element with the oracle (so every split-count class of the
    KV sweep, the requests clipped at the longest length, and the shortest ones)."""
    import torch
    cfg = I.CONFIGS[num]
    print(f"[draft_step full] config {num}: {cfg}", flush=True)
    W = I.make_weights(cfg, 0)
    x = I.make_inputs(cfg, 0)
    Wd = dev(W)
    if cfg.dtype == "bf16":   # the benchmark streams the packed W_dS
        Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    out, st = _draft(cfg, W, Wd, x)
    assert st == 0
    del Wd
    torch.cuda.empty_cache()
    L = x["ctx_lens"]
    print(f"  oracle on all {cfg.B} requests (lengths {int(L.min())}..{int(L.max())})", flush=True)
    ref = O.draft_step(W, x, cfg, progress=lambda s: print(f"  oracle: {s} done", flush=True))
    worst = max(range(cfg.B), key=lambda b: float(np.max(np.abs(out[b] - ref[b]))))
    print(f"  worst request {worst} (length {int(L[worst])})", flush=True)
    assert_close(out, ref, f"config {num}")


@pytest.mark.slow
@pytest.mark.timeout(900)
@pytest.mark.parametrize("causal", [False, True])
def test_draft_step_window_full(causal):
    """8b-serving-b64 under the sliding window of 2048 (Sec. 3.3.2 attention masks), with and
    without the block-causal mask: the swept range starts at L - 2047, so requests shorter than
    the window, longer ones (split at their visible range) and the window edge inside a block
    are all in the batch; every request compared."""
    cfg = I.CONFIGS[3].replace(window=2048, block_causal=causal)
    W = I.make_weights(cfg, 0)
    x = I.make_inputs(cfg, 0)
    Wd = dev(W)
    Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    out, st = _draft(cfg, W, Wd, x)
    assert st == 0
    del Wd
    ref = O.draft_step(W, x, cfg, progress=lambda s: print(f"  oracle: {s} done", flush=True))
    assert_close(out, ref, f"config 3, window 2048, block-causal {causal}")


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_draft_step_kv_subset_full():
    """8b-serving-b64 with partial target-KV-head reuse: the drafter's 4 KV heads (16 query
    heads) read heads 0, 2, 4, 6 of the target's 8-head cache; every request compared."""
    cfg = I.CONFIGS[3].replace(Hq=16, Hkv=4, Hkv_target=8, kv_heads=(0, 2, 4, 6))
    W = I.make_weights(cfg, 0)
    x = I.make_inputs(cfg, 0)
    Wd = dev(W)
    Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    out, st = _draft(cfg, W, Wd, x)
    assert st == 0
    del Wd
    ref = O.draft_step(W, x, cfg, progress=lambda s: print(f"  oracle: {s} done", flush=True))
    assert_close(out, ref, "config 3, 4 of 8 KV heads")
