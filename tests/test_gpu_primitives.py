"""GPU parity of the primitives (GEMM, gather, KV sweep, SSD scan, state projection) against
the float64 oracle, through the C ABI."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from gpu_util import assert_close, dev, empty, host  # noqa: E402
from paper_2609_24197_amd import hspec, inputs as I  # noqa: E402

pytestmark = pytest.mark.gpu


def _small_attn_cfg(**kw):
    base = dict(name="t", B=3, k=16, d_model=256, H=4, P=64, N=16, G=1, chunk=16, Hq=32, Hkv=8, D=128,
                lengths="list:130,0,77", dtype="bf16")
    base.update(kw)
    return I.StepConfig(**base)


# ------------------------------------------------------------------------------- GEMM

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("M,N,K", [(4, 256, 256), (64, 1000, 512), (100, 384, 264), (128, 512, 1024),
                                   (300, 700, 4096), (1, 4096, 4096), (48, 5000, 4096), (20, 3000, 1024),
                                   (8, 300, 264), (64, 200000, 160),
                                   # 65..128 rows: 128-row weight streaming
                                   (65, 4096, 1024), (128, 16768, 512), (96, 300, 512), (127, 1000, 2048),
                                   # 256 x 256 tiles: whole tiles, k-split last tiles, ragged M and N
                                   (512, 768, 256), (1024, 2304, 1024), (777, 1000, 512), (1536, 4096, 512),
                                   (600, 300, 4096),
                                   # 256..511 rows: one or two row tiles, most columns k-split
                                   (256, 16768, 512), (384, 4096, 1024), (257, 1000, 2048)])
def test_linear(dtype, M, N, K):
    print(f"[linear] dtype={dtype} M={M} N={N} K={K}", flush=True)
    A = I.normal("lin_A", (M, K), 1.0, 0, dtype)
    W = I.normal("lin_W", (N, K), K ** -0.5, 0, dtype)
    R = I.normal("lin_R", (M, N), 1.0, 0, "f32")
    d = dev(dict(A=A, W=W, R=R))
    code = hspec.F32 if dtype == "f32" else hspec.BF16
    ws = hspec.workspace(hspec.linear_workspace(code, M, N, K))
    out = empty((M, N))
    hspec.linear(code, d["A"], d["W"], out, ws, R=d["R"])
    ref = O.f64(A) @ O.f64(W).T + R
    assert_close(host(out), ref, "C")


# ----------------------------------------------------------------------------- gather

def test_gather_slots_bit_exact():
    cfg = _small_attn_cfg(B=5, lengths="list:1,16,17,300,0")
    x = I.make_inputs(cfg, seed=1, extra_pages=5, pad_pages=2)
    d = dev(dict(page_table=x["page_table"], ctx_lens=x["ctx_lens"]))
    maxL = 320
    slots = empty((cfg.B, maxL), "i32")
    st = empty((1,), "i32")
    st.zero_()
    hspec.gather_slots(d["page_table"], d["ctx_lens"], cfg.page_size, x["num_pages"], maxL, slots, st)
    ref = O.gather_slots(x["page_table"], x["ctx_lens"], cfg.page_size, maxL)
    assert np.array_equal(host(slots), ref)
    assert int(host(st)[0]) == 0


def test_gather_slots_flags_bad_page():
    pt = np.array([[0, 7, 1]], np.int32)        # page id 7 is outside a pool of 3 pages
    d = dev(dict(page_table=pt, ctx_lens=np.array([40], np.int32)))
    slots = empty((1, 48), "i32")
    st = empty((1,), "i32")
    st.zero_()
    hspec.gather_slots(d["page_table"], d["ctx_lens"], 16, 3, 48, slots, st)
    s = host(slots)[0]
    assert np.array_equal(s[:16], np.arange(16)) and np.all(s[16:32] == -1)
    assert np.array_equal(s[32:40], 16 + np.arange(8)) and np.all(s[40:] == -1)
    assert int(host(st)[0]) & hspec.DEV_BAD_PAGE


# ------------------------------------------------------------------------- KV sweep

def _run_attn(cfg, x, max_ctx_len=None, split=0):
    cfg = cfg.replace(split_tokens=split)
    d = dev(x)
    maxL = int(max(x["ctx_lens"])) if max_ctx_len is None else max_ctx_len
    ws = hspec.workspace(hspec.paged_attn_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    o = empty((cfg.B, cfg.k, cfg.Hq, cfg.D))
    hspec.paged_attn(cfg, d, o, ws, maxL)
    return host(o), hspec.read_status(ws)


def _ref_attn(cfg, x):
    return O.paged_attention(x["q"], x["k_blk"], x["v_blk"], x["k_cache"], x["v_cache"], x["page_table"],
                             x["ctx_lens"], page_size=cfg.page_size, window=cfg.window,
                             block_causal=cfg.block_causal, kv_heads=cfg.kv_heads)


ATTN_CASES = {
    "cfg1_f32": I.CONFIGS[1],
    "bf16_ragged": _small_attn_cfg(),
    "k7_g4": _small_attn_cfg(k=7, lengths="list:1000,37,16"),
    "g8_128rows": _small_attn_cfg(Hq=64, lengths="list:500,1,260"),
    "d64_mha": _small_attn_cfg(Hq=4, Hkv=4, D=64, k=5, lengths="list:33,64,200"),
    "window": _small_attn_cfg(window=100, lengths="list:1000,5,333"),
    "causal": _small_attn_cfg(block_causal=True),
    "causal_window": _small_attn_cfg(block_causal=True, window=64, lengths="list:700,64,65"),
    "empty_ctx": _small_attn_cfg(B=2, lengths="list:0,0"),
    # block keys in fp32 inside the reduction, every split through partials
    "precise_ragged": _small_attn_cfg(precise_io=True),
    "precise_causal_window": _small_attn_cfg(block_causal=True, window=64, lengths="list:700,64,65", precise_io=True),
    "precise_empty_ctx": _small_attn_cfg(B=2, lengths="list:0,0", precise_io=True),
    "precise_d64_k7": _small_attn_cfg(Hq=4, Hkv=4, D=64, k=7, lengths="list:33,64,200", precise_io=True),
    "precise_f32": I.CONFIGS[1].replace(precise_io=True),
    # partial target-KV-head reuse: 4 of the cache's 8 KV heads, in a shuffled order
    "kv_subset": _small_attn_cfg(Hq=16, Hkv=4, Hkv_target=8, kv_heads=(6, 1, 3, 4), lengths="list:700,0,130"),
    "kv_subset_precise": _small_attn_cfg(Hq=8, Hkv=2, Hkv_target=8, kv_heads=(7, 0), lengths="list:300,40,0",
                                         precise_io=True),
}


@pytest.mark.parametrize("name", sorted(ATTN_CASES))
def test_paged_attn(name):
    cfg = ATTN_CASES[name]
    print(f"[paged_attn] {name} {cfg}", flush=True)
    x = I.make_attn_inputs(cfg, seed=2, extra_pages=3)
    o, st = _run_attn(cfg, x)
    assert st == 0
    assert_close(o, _ref_attn(cfg, x), name)


def test_paged_attn_split_invariance():
    """Every split size meets the tolerance, is bitwise deterministic, and the split sizes agree
    with each other to the bf16 rounding of the probabilities (which depends on each split's
    running maximum)."""
    cfg = _small_attn_cfg(B=2, lengths="list:1000,450")
    x = I.make_attn_inputs(cfg, seed=3)
    ref = _ref_attn(cfg, x)
    outs = {}
    for split in (64, 128, 448, 1024):
        o, st = _run_attn(cfg, x, split=split)
        o2, _ = _run_attn(cfg, x, split=split)
        assert np.array_equal(o, o2), f"split {split} not deterministic"
        assert_close(o, ref, f"split={split}")
        outs[split] = o
    base = outs[1024]
    for s, o in outs.items():
        assert_close(o, base, f"split {s} vs whole context", max_abs=2e-3, rel_l2=3e-3)


def test_paged_attn_many_work_units():
    """More (request, split) entries than the sweep keeps in LDS (512): the sweep then reads each
    claimed item's entry from the work list in memory.  Ragged lengths, 64-key splits."""
    lens = [1100 - 13 * i for i in range(40)]
    split = 64
    assert sum(-(-L // split) for L in lens) > 512
    cfg = _small_attn_cfg(B=len(lens), lengths="list:" + ",".join(map(str, lens)))
    print(f"[paged_attn] many work units {cfg}", flush=True)
    x = I.make_attn_inputs(cfg, seed=5)
    o, st = _run_attn(cfg, x, split=split)
    assert st == 0
    assert_close(o, _ref_attn(cfg, x), "many work units")


def test_paged_attn_workspace_reuse():
    """Consecutive calls on one workspace with different queries, caches and tables: the split
    partials a call combines inside the sweep are its own (stores and loads coherent across
    the XCDs' caches), never a previous call's left in a cache."""
    cfg = _small_attn_cfg(B=4, lengths="list:3000,2500,700,1900")
    ws = None
    for seed, split in ((11, 512), (12, 512), (13, 256), (14, 0)):
        print(f"[paged_attn reuse] seed {seed} split {split}", flush=True)
        c = cfg.replace(split_tokens=split)
        x = I.make_attn_inputs(c, seed=seed, extra_pages=1)
        d = dev(x)
        maxL = int(max(x["ctx_lens"]))
        need = hspec.paged_attn_workspace(c, x["page_table"].shape[1], x["num_pages"], maxL)
        if ws is None or ws.numel() < need:
            ws = hspec.workspace(max(need, 64 << 20))
        o = empty((c.B, c.k, c.Hq, c.D))
        hspec.paged_attn(c, d, o, ws, maxL)
        assert hspec.read_status(ws) == 0
        assert_close(host(o), _ref_attn(c, x), f"seed {seed}")


def test_paged_attn_window_splits():
    """Under a sliding window the splits tile only the positions some query can see,
    starting at ctx_len - window + 1 (not page- or tile-aligned): lengths around the window,
    several splits inside it, and a length short of it."""
    cfg = _small_attn_cfg(B=6, window=300, lengths="list:1000,299,300,301,5,777")
    x = I.make_attn_inputs(cfg, seed=8)
    ref = _ref_attn(cfg, x)
    for split in (64, 128, 0):
        print(f"[paged_attn window] split {split}", flush=True)
        o, st = _run_attn(cfg, x, split=split)
        o2, _ = _run_attn(cfg, x, split=split)
        assert st == 0
        assert np.array_equal(o, o2), f"split {split} not deterministic"
        assert_close(o, ref, f"window 300, split {split}")
    causal = cfg.replace(block_causal=True, B=2, lengths="list:4100,2049", window=2048)
    xc = I.make_attn_inputs(causal, seed=9)
    o, st = _run_attn(causal, xc, split=256)
    assert st == 0
    assert_close(o, _ref_attn(causal, xc), "window 2048 causal, split 256")


@pytest.mark.parametrize("precise", [False, True], ids=["block_in_sweep", "block_in_reduction"])
def test_paged_attn_phases_bitwise(precise):
    """The work list, sweep and reduction launched one call each give the one-call result."""
    cfg = _small_attn_cfg(B=3, lengths="list:1000,37,450", precise_io=precise).replace(split_tokens=256)
    x = I.make_attn_inputs(cfg, seed=6)
    whole, _ = _run_attn(cfg, x, split=256)
    d = dev(x)
    maxL = int(max(x["ctx_lens"]))
    ws = hspec.workspace(hspec.paged_attn_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    o = empty((cfg.B, cfg.k, cfg.Hq, cfg.D))
    for ph in (hspec.PHASE_WORKLIST, hspec.PHASE_SWEEP, hspec.PHASE_REDUCE):
        hspec.paged_attn(cfg, d, o, ws, maxL, phases=ph)
    assert hspec.read_status(ws) == 0
    assert np.array_equal(host(o), whole)


def test_paged_attn_page_permutation_bitwise():
    cfg = _small_attn_cfg()
    x = I.make_attn_inputs(cfg, seed=4, extra_pages=4)
    a, _ = _run_attn(cfg, x)
    perm = np.random.default_rng(0).permutation(x["num_pages"])
    y = dict(x)
    for key in ("k_cache", "v_cache"):
        arr = np.empty_like(x[key])
        arr[perm] = x[key]
        y[key] = arr
    y["page_table"] = np.where(x["page_table"] >= 0, perm[np.maximum(x["page_table"], 0)], -1).astype(np.int32)
    b, _ = _run_attn(cfg, y)
    assert np.array_equal(a, b)


def test_paged_attn_poisoned_slots():
    """NaN/inf in unreferenced pages and in slots at or past ctx_len change nothing."""
    cfg = _small_attn_cfg(lengths="list:130,3,77")
    x = I.make_attn_inputs(cfg, seed=5, extra_pages=6)
    a, _ = _run_attn(cfg, x)
    y = dict(x)
    kc, vc = x["k_cache"].copy(), x["v_cache"].copy()
    used = np.zeros(x["num_pages"], bool)
    for b, L in enumerate(x["ctx_lens"]):
        n = (int(L) + 15) // 16
        pages = x["page_table"][b, :n]
        used[pages] = True
        if L % 16:
            last = pages[-1]
            kc[last, L % 16:] = 0x7FC0   # bf16 NaN
            vc[last, L % 16:] = 0x7F80   # bf16 +inf
    kc[~used] = 0x7FC0
    vc[~used] = 0xFF80
    y["k_cache"], y["v_cache"] = kc, vc
    b_, _ = _run_attn(cfg, y)
    assert np.array_equal(a, b_)


def test_paged_attn_single_key_and_mean():
    """P1 on the GPU: ctx_len 0 and k = 1 returns v_blk; identical keys return the mean of V."""
    cfg = _small_attn_cfg(B=1, k=1, lengths="list:0")
    x = I.make_attn_inputs(cfg, seed=6)
    o, _ = _run_attn(cfg, x)
    vb = O.f64(x["v_blk"])[0, 0]
    assert np.allclose(o[0, 0], np.repeat(vb, cfg.g, axis=0), rtol=0, atol=1e-6)
    cfg = _small_attn_cfg(B=1, k=4, lengths="list:37")
    x = I.make_attn_inputs(cfg, seed=7)
    x["k_cache"][:] = x["k_cache"][0, 0]
    x["k_blk"][:] = x["k_cache"][0, 0]
    o, _ = _run_attn(cfg, x)
    assert_close(o, _ref_attn(cfg, x), "identical keys")


def test_paged_attn_flags_bad_inputs():
    """Out-of-pool page ids and over-long context lengths are flagged, not faulted on."""
    cfg = _small_attn_cfg(B=2, lengths="list:40,20")
    x = I.make_attn_inputs(cfg, seed=8)
    x["page_table"] = x["page_table"].copy()
    x["page_table"][0, 1] = x["num_pages"] + 100
    _, st = _run_attn(cfg, x)
    assert st & hspec.DEV_BAD_PAGE
    x = I.make_attn_inputs(cfg, seed=8)
    x["ctx_lens"] = np.array([40, 20000], np.int32)
    _, st = _run_attn(cfg, x, max_ctx_len=48)
    assert st & hspec.DEV_BAD_CTX_LEN


# ------------------------------------------------------------------------------- scan

SCAN_CASES = [
    # B, T, H, N, G, chunk, dtype, with S0, final state
    (2, 16, 8, 128, 1, 16, "bf16", True, False),
    (2, 16, 8, 128, 1, 16, "bf16", True, True),
    (1, 4, 8, 16, 1, 4, "f32", True, True),
    (2, 7, 4, 128, 2, 4, "bf16", True, True),
    (2, 32, 4, 128, 1, 8, "bf16", True, True),
    (1, 16, 4, 16, 1, 1, "bf16", False, True),
    (3, 5, 6, 64, 3, 2, "f32", True, False),
    (2, 16, 4, 32, 1, 16, "bf16", False, False),
    # one chunk without a final state (the drafting step's path) in fp32 planes, with T < chunk
    (2, 16, 8, 128, 1, 16, "f32", True, False),
    (3, 7, 4, 64, 2, 8, "bf16", True, False),
    (1, 1, 2, 16, 1, 16, "f32", True, False),
    # several chunks at N = 32 (state update in one 32-column block), and a ragged last chunk
    (2, 24, 4, 32, 1, 8, "bf16", True, True),
    (2, 13, 4, 128, 1, 5, "bf16", True, True),
]


@pytest.mark.parametrize("case", SCAN_CASES, ids=[str(c) for c in SCAN_CASES])
def test_ssd_scan(case):
    B, T, H, N, G, chunk, dtype, with_s0, fin = case
    print(f"[ssd_scan] {case}", flush=True)
    s = I.make_scan_inputs(B, T, H, 64, N, G, seed=T + H, dtype=dtype, s0=with_s0)
    d = dev({k: v for k, v in s.items() if v is not None})
    code = hspec.F32 if dtype == "f32" else hspec.BF16
    ws = hspec.workspace(hspec.ssd_scan_workspace(B, T, H, 64, N, G, code))
    y = empty((B, T, H, 64))
    Sf = empty((B, H, 64, N)) if fin else None
    hspec.ssd_scan(B, T, H, 64, N, G, chunk, code, d["x"], d["dt"], d["A"], d["Bm"], d["Cm"], d["Dskip"],
                   d.get("S0"), y, Sf, ws)
    yr, Sr = O.ssd_sequential(s["x"], s["dt"], s["A"], s["Bm"], s["Cm"], s["Dskip"], s["S0"])
    assert_close(host(y), yr, "y")
    if fin:
        assert_close(host(Sf), Sr, "S_final")


def test_ssd_scan_zero_input_zero_state():
    """x = 0 and S0 = 0 give y = 0 and S_final = 0 exactly, for any dt, B, C."""
    B, T, H, N, G = 2, 16, 4, 128, 1
    s = I.make_scan_inputs(B, T, H, 64, N, G, seed=1)
    s["x"] = np.zeros_like(s["x"])
    d = dev({k: v for k, v in s.items() if v is not None})
    ws = hspec.workspace(hspec.ssd_scan_workspace(B, T, H, 64, N, G, hspec.BF16))
    y = empty((B, T, H, 64))
    Sf = empty((B, H, 64, N))
    hspec.ssd_scan(B, T, H, 64, N, G, 16, hspec.BF16, d["x"], d["dt"], d["A"], d["Bm"], d["Cm"], d["Dskip"],
                   None, y, Sf, ws)
    assert not np.any(host(y)) and not np.any(host(Sf))


# -------------------------------------------------------------------- state projection

def _pack_host(W, r):
    """The packed W_dS layout as the header describes it: 16-row tiles in groups of 32 (the
    last group holding what is left), block (s, t) at (32 g S + s gs + t mod 32) * 1024 bytes
    for group g = t // 32 of gs tiles, row 16t+i, columns 32s+8c..+7 at (i + 16c) * 16 bytes
    inside the block, each element the fp16 value of 256 x W (bit patterns; numpy rounds to
    nearest even, as the device does)."""
    d_S = W.shape[0]
    T, S = d_S // 16, r // 32
    with np.errstate(over="ignore"):
        w16 = (I.bf16_bits_to_f32(W).astype(np.float64) * 256.0).astype(np.float16).view(np.uint16)
    blk = w16.reshape(T, 16, S, 4, 8)            # [t, i, s, c, e]
    out = []
    for g0 in range(0, T, 32):                   # a group: its k-steps in order, each its tiles
        grp = blk[g0:g0 + 32]                    # [gs, i, s, c, e]
        out.append(np.ascontiguousarray(grp.transpose(2, 0, 3, 1, 4)).reshape(-1))   # [s, t, c, i, e]
    return np.concatenate(out)


@pytest.mark.parametrize("d_S,r", [(16, 64), (4096, 256), (2048, 192), (640, 128), (1040, 64)])
def test_pack_w_ds_layout(d_S, r):
    """Packing is data movement and an exact fp16 conversion: bit-exact against the host
    re-layout, over weights spanning 2^-25 .. 2^7 in magnitude, plus the ends of the range:
    zeros and bf16 subnormals (to +-0), magnitudes below 2^-25 (rounded to fp16 subnormals),
    above 255.875 up to the largest bf16 and infinities (to +-inf)."""
    W = I.normal("pack_W", (d_S, r), 1.0, 0, "bf16")
    # a spread of exponents, both signs (bf16 bit patterns: sign, 8-bit exponent, 7-bit fraction)
    e = np.random.default_rng(5).integers(127 - 25, 127 + 8, size=W.shape, dtype=np.int64)
    fr = np.random.default_rng(6).integers(0, 128, size=W.shape, dtype=np.int64)
    sg = np.random.default_rng(7).integers(0, 2, size=W.shape, dtype=np.int64)
    # the first row: special exponents (0: zero or subnormal; 255 with fraction 0: inf)
    special = np.array([0, 0, 127 - 40, 127 - 30, 127 - 26, 127 + 8, 127 + 15, 127 + 16, 127 + 120, 254, 255])
    e[0, :special.size] = special
    fr[0, 0] = 0
    fr[0, special.size - 1] = 0
    W = ((sg << 15) | (e << 7) | fr).astype(np.uint16).view(W.dtype)
    d = dev(dict(W=W))
    packed = hspec.pack_w_ds(d["W"], d_S, r)
    got = packed.view(dtype=__import__("torch").int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, _pack_host(W, r))


@pytest.mark.parametrize("B", [1, 5, 40, 64, 65, 100, 128, 130])
def test_state_init_packed(B):
    """Proj_dS from the packed W_dS (the layout the benchmark streams) against the oracle."""
    cfg = _small_attn_cfg(B=B, d_model=512, H=8, N=128, lengths="fixed:16")
    W = I.make_weights(cfg, seed=7, skip=("W_in", "W_out", "W_q", "W_k", "W_v", "W_o"))
    x = I.make_inputs(cfg, seed=7)
    d = dev(dict(W_r=W["W_r"], W_dS=W["W_dS"], h_last=x["h_last"]))
    Wd = dict(W_r=d["W_r"], W_dS_packed=hspec.pack_w_ds(d["W_dS"], cfg.d_S, cfg.rank))
    ws = hspec.workspace(hspec.state_init_workspace(cfg))
    S0 = empty((cfg.B, cfg.H, cfg.P, cfg.N))
    hspec.state_init(cfg, Wd, d["h_last"], S0, ws)
    ref, _ = O.state_init(x["h_last"], W["W_r"], W["W_dS"], cfg.H, cfg.P, cfg.N)
    assert_close(host(S0), ref, "S0")


@pytest.mark.parametrize("cfg", [I.CONFIGS[1], _small_attn_cfg(B=5, d_model=512, H=8, N=128, lengths="fixed:16"),
                                 _small_attn_cfg(B=70, d_model=256, H=4, N=128, lengths="fixed:16")],
                         ids=["cfg1", "b5", "b70"])
def test_state_init(cfg):
    W = I.make_weights(cfg, seed=3, skip=("W_in", "W_out", "W_q", "W_k", "W_v", "W_o"))
    x = I.make_inputs(cfg, seed=3)
    d = dev(dict(W_r=W["W_r"], W_dS=W["W_dS"], h_last=x["h_last"]))
    Wd = dict(d, W_in=None, conv_w=None, conv_b=None, dt_bias=None, A_log=None, D=None, gnorm_w=None, W_out=None)
    ws = hspec.workspace(hspec.state_init_workspace(cfg))
    S0 = empty((cfg.B, cfg.H, cfg.P, cfg.N))
    hspec.state_init(cfg, Wd, d["h_last"], S0, ws)
    ref, _ = O.state_init(x["h_last"], W["W_r"], W["W_dS"], cfg.H, cfg.P, cfg.N)
    assert_close(host(S0), ref, "S0")
