"""Benchmark of one H-Spec block-drafting step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3]
    python bench.py --counters      # one launch of each measured kernel, for rocprofv3 --pmc

A step is one call of hspec_draft_step over the whole batch: state projection from the
last-token hidden state, the Mamba-2 layer with its chunked scan, and the attention layer
over the paged target cache plus the block.  Inputs are synthetic, seeded, and resident in
HBM before timing starts.  Prints one JSON line with the drafted-tokens/s throughput, the
roofline of the dominant kernel (the state projection, which streams W_dS), the roofline of
the target-KV sweep, and the float64 CPU oracle timed on a bounded sample of the same
workload on this host.  Each kernel of a roofline figure is timed with HIP events around its
own launches, each launch right after one drafting step, so that it runs at the clock and
cache state it has inside the step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from paper_2609_24197_amd import hspec, inputs as I, roofline as RL  # noqa: E402

METRIC = "drafted tokens/s per draft step at B=64; achieved HBM GB/s vs MI355X peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2609_24197_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_for(name: str, src_hash: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if taken on this source and
    on this workload (else None)."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    e = t.get(name)
    if not e or e.get("source_hash") != src_hash or e.get("workload") != workload:
        return None
    return e.get("bytes_per_launch")


def time_in_step(fn, n: int, warmup: int, context, torch) -> float:
    """Average duration (s) of fn's launches, each preceded by `context()` (one drafting step),
    HIP events on the launch stream around fn: the kernels are timed at the clock and cache
    state they see inside a step."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for i in range(warmup + n):
        context()
        if i < warmup:
            fn()
            continue
        s, e = ev[i - warmup]
        s.record()
        fn()
        e.record()
    torch.cuda.synchronize()
    return sum(s.elapsed_time(e) for s, e in ev) / 1e3 / n


def time_attention(cfg, Ad, o, aws, maxL, n: int, warmup: int, context, torch):
    """Average durations (s) of the attention core's kernels, each attention call preceded by
    `context()`, one drafting step, so that its kernels run at the clock and cache state they see
    inside a step (the same kernel runs measurably slower back to back, or right after a long
    weight stream).  HIP events on the launch stream bracket the KV-sweep launch and the
    cross-split reduction launch.  The work list is built before the step, as the step itself
    builds it inside its q/k-norm + RoPE launch, ahead of the sweep; its own launch is timed
    separately, back to back.  Returns (work list, sweep, reduction)."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
    for i in range(warmup + n):
        hspec.paged_attn(cfg, Ad, o, aws, maxL, phases=hspec.PHASE_WORKLIST)
        context()
        if i < warmup:
            hspec.paged_attn(cfg, Ad, o, aws, maxL, phases=hspec.PHASE_SWEEP | hspec.PHASE_REDUCE)
            continue
        e = ev[i - warmup]
        e[0].record()
        hspec.paged_attn(cfg, Ad, o, aws, maxL, phases=hspec.PHASE_SWEEP)
        e[1].record()
        hspec.paged_attn(cfg, Ad, o, aws, maxL, phases=hspec.PHASE_REDUCE)
        e[2].record()
    torch.cuda.synchronize()
    t_sweep = sum(e[0].elapsed_time(e[1]) for e in ev) / 1e3 / n
    t_red = sum(e[1].elapsed_time(e[2]) for e in ev) / 1e3 / n
    pl = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for s_, e_ in pl:
        s_.record()
        hspec.paged_attn(cfg, Ad, o, aws, maxL, phases=hspec.PHASE_WORKLIST)
        e_.record()
    torch.cuda.synchronize()
    t_plan = sum(s_.elapsed_time(e_) for s_, e_ in pl) / 1e3 / n
    return t_plan, t_sweep, t_red


def head_figures(cfg, out, step, args, torch):
    """Timing of hspec_draft_head on the drafting step's output, each call after one step, and
    of its LM-head product ([B*k, d_model] x [d_model, V], bf16) launched alone."""
    V, R = I.HEAD_VOCAB, I.HEAD_RANK
    HW = {k: hspec.to_device(v) for k, v in I.make_head_weights(cfg, args.seed).items()}
    prev = hspec.to_device(I.make_head_inputs(cfg, args.seed)["prev_tok"])
    hc = hspec.head_cfg(cfg, V, R)
    hws = hspec.workspace(hspec.draft_head_workspace(hc))
    tok = torch.empty((cfg.B, cfg.k), dtype=torch.int32, device="cuda")
    t_head = time_in_step(lambda: hspec.draft_head(hc, HW, out, prev, tok, hws), args.steps, args.warmup, step, torch)
    assert hspec.read_status(hws) == 0
    M = cfg.B * cfg.k
    A = torch.randn(M, cfg.d_model, device="cuda").to(torch.bfloat16)
    C = torch.empty(M, V, device="cuda")
    lws = hspec.workspace(hspec.linear_workspace(hspec.BF16, M, V, cfg.d_model))
    t_lm = time_in_step(lambda: hspec.linear(hspec.BF16, A, HW["W_lm"], C, lws), args.steps, args.warmup, step, torch)
    flops = 2 * M * V * cfg.d_model
    log(f"draft head: {t_head * 1e6:.1f} us (LM-head GEMM alone {t_lm * 1e6:.1f} us, {flops / t_lm / 1e12:.0f} TFLOP/s)")
    return {"avg_us": round(t_head * 1e6, 2), "vocab": V, "markov_rank": R, "tokens": "greedy",
            "lm_head_gemm_us": round(t_lm * 1e6, 2), "lm_head_tflops": round(flops / t_lm / 1e12, 1),
            "lm_head_frac_of_bf16_peak": round(flops / t_lm / 1e12 / RL.MFMA_BF16_PEAK_TFLOPS, 4)}


def scan_figures(cfg, step, args, torch):
    """The SSD scan launched alone at the step's shapes (B requests, k positions, H heads of
    P x N), each call after one drafting step: the one-chunk kernel the step runs (S0 as bf16
    hi/lo planes here) and the multi-chunk kernel, which carries the state across chunks and
    writes S_final, at chunk = k and chunk = k/2."""
    B, T, H, N, G = cfg.B, cfg.k, cfg.H, cfg.N, cfg.G
    s = I.make_scan_inputs(B, T, H, cfg.P, N, G, seed=args.seed, dtype=cfg.dtype, s0=True)
    d = {k: hspec.to_device(v) for k, v in s.items() if v is not None}
    code = hspec.F32 if cfg.dtype == "f32" else hspec.BF16
    ws = hspec.workspace(hspec.ssd_scan_workspace(B, T, H, cfg.P, N, G, code))
    y = torch.empty((B, T, H, cfg.P), dtype=torch.float32, device="cuda")
    Sf = torch.empty((B, H, cfg.P, N), dtype=torch.float32, device="cuda")
    res = {}
    for name, chunk, fin in (("one_chunk_us", T, False), ("with_final_state_us", T, True),
                             ("two_chunks_with_final_state_us", max(1, T // 2), True)):
        f = lambda: hspec.ssd_scan(B, T, H, cfg.P, N, G, chunk, code, d["x"], d["dt"], d["A"], d["Bm"],  # noqa: E731
                                   d["Cm"], d["Dskip"], d["S0"], y, Sf if fin else None, ws)
        res[name] = round(time_in_step(f, args.steps, args.warmup, step, torch) * 1e6, 2)
    log(f"ssd scan alone: {res}")
    return res


def forward_figures(cfg, Wd, Xd, x, args, torch):
    """Timing of hspec_drafter_forward (3 x (Mamba, attention, MLP) + 1 x (Mamba, MLP), |M| = 5,
    MLP hidden 3 d_model) on the same batch: the step's packed W_dS (the same seeded values), a
    W_r over the five fused layers, and two more target caches on the same page table."""
    fc = cfg.replace(n_fuse=I.DRAFTER_FUSE, ff=3 * cfg.d_model)
    _, L = I.make_drafter_weights(fc, args.seed, skip_state=True)
    shared = {"W_r": hspec.to_device(I.make_weights(fc, args.seed, skip=tuple(
        k for k in ("W_dS", "W_in", "conv_w", "conv_b", "D", "gnorm_w", "W_out", "norm1_w", "norm2_w", "W_q", "W_k",
                    "W_v", "W_o", "q_norm_w", "k_norm_w")))["W_r"]), "W_dS_packed": Wd["W_dS_packed"]}
    Ld = [{k: (hspec.to_device(v) if isinstance(v, np.ndarray) else v) for k, v in W.items()} for W in L]
    shape = x["k_cache"].shape
    X = dict(Xd, h_last=hspec.to_device(I.normal("h_last", (cfg.B, fc.d_h), 1.0, args.seed, cfg.dtype)),
             caches=[dict(k_cache=Xd["k_cache"], v_cache=Xd["v_cache"])] + [
                 dict(k_cache=hspec.to_device(I.normal(f"k_cache{c}", shape, 1.0, args.seed, cfg.dtype)),
                      v_cache=hspec.to_device(I.normal(f"v_cache{c}", shape, 1.0, args.seed, cfg.dtype)))
                 for c in (1, 2)])
    maxL = int(x["ctx_lens"].max())
    fws = hspec.workspace(hspec.drafter_forward_workspace(fc, x["page_table"].shape[1], x["num_pages"], maxL))
    out = torch.empty((cfg.B, cfg.k, cfg.d_model), dtype=torch.float32, device="cuda")
    fwd = lambda: hspec.drafter_forward(fc, shared, Ld, X, out, fws, maxL)  # noqa: E731
    for _ in range(args.warmup):
        fwd()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(args.steps):
        fwd()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / args.steps
    assert hspec.read_status(fws) == 0 and bool(torch.isfinite(out).all())
    log(f"drafter forward (4 layers): {ms:.3f} ms, {cfg.B * cfg.k / ms * 1e3:,.0f} drafted tok/s")
    return {"ms": round(ms, 4), "drafted_tok_s": round(cfg.B * cfg.k / ms * 1e3, 1), "layers": "3 x MAF + 1 x MF",
            "fused_target_layers": I.DRAFTER_FUSE, "mlp_hidden": fc.d_ff, "target_caches": 3}


def compare_systems(args, torch):
    """The hybrid drafter against a block-diffusion drafter with drafter-side KV injection, per
    draft step (the runtime-scaling study of Sec. 4 and the injection cost of Fig. 3), on
    synthetic random weights and caches drawn on the device (timing only; parity is tested
    separately):
      hybrid: hspec_drafter_forward, 3 x (Mamba, attention, MLP) + 1 x (Mamba, MLP), the Mamba
              state projected from |M| = 5 fused target layers;
      block diffusion: hspec_kv_inject of the k new positions into 5 drafter-side caches, then
              5 x (attention, MLP) over those caches (hspec_drafter_forward without Mamba).
    Shapes: the App. B.1 drafter for an 8B target (48 Mamba heads of 64, 4 groups, r = 4096,
    d_state 16: the smallest the scan takes, App. B.1 uses 4), Qwen3-8B attention (32 / 8 / 128),
    MLP hidden 12,288, k = 16, the 2,048-token window of App. B.2."""
    dev = "cuda"
    bf = torch.bfloat16

    def rnd(*shape, std=1.0, dtype=bf):
        return (torch.randn(*shape, device=dev) * std).to(dtype)

    base = I.StepConfig(name="cmp", B=8, k=16, d_model=4096, H=48, P=64, N=16, G=4, chunk=16, Hq=32, Hkv=8, D=128,
                        lengths="fixed:1040", n_fuse=I.DRAFTER_FUSE, ff=12288, window=2048)
    dm, di, ff, kv = base.d_model, base.d_inner, base.d_ff, base.Hkv * base.D

    def attn_w():
        return dict(W_q=rnd(base.Hq * base.D, dm, std=dm ** -0.5), W_k=rnd(kv, dm, std=dm ** -0.5),
                    W_v=rnd(kv, dm, std=dm ** -0.5), W_o=rnd(dm, base.Hq * base.D, std=(base.Hq * base.D) ** -0.5),
                    q_norm_w=torch.ones(base.D, device=dev), k_norm_w=torch.ones(base.D, device=dev),
                    norm2_w=torch.ones(dm, device=dev))

    def mlp_w():
        return dict(W_gate=rnd(ff, dm, std=dm ** -0.5), W_up=rnd(ff, dm, std=dm ** -0.5),
                    W_down=rnd(dm, ff, std=ff ** -0.5), norm3_w=torch.ones(dm, device=dev))

    def mamba_w():
        return dict(W_in=rnd(base.d_in_proj, dm, std=dm ** -0.5), conv_w=rnd(base.conv_dim, base.conv_w, std=0.5),
                    conv_b=rnd(base.conv_dim, std=0.5), dt_bias=torch.full((base.H,), -4.0, device=dev),
                    A_log=torch.zeros(base.H, device=dev), D=torch.ones(base.H, device=dev),
                    gnorm_w=torch.ones(di, device=dev), W_out=rnd(dm, di, std=di ** -0.5),
                    norm1_w=torch.ones(dm, device=dev))

    hyb = [dict(mamba_w(), **attn_w(), **mlp_w(), cache=i) for i in range(3)] + [dict(mamba_w(), **mlp_w(), cache=None)]
    shared = {"W_r": rnd(base.rank, base.d_h, std=base.d_h ** -0.5),
              "W_dS_packed": hspec.pack_w_ds(rnd(base.d_S, base.rank, std=base.rank ** -0.5), base.d_S, base.rank)}
    bd = [dict(attn_w(), **mlp_w(), cache=i) for i in range(5)]
    IW = {"W_fc": rnd(dm, base.d_h, std=base.d_h ** -0.5),
          "layers": [dict(W_k=rnd(kv, dm, std=dm ** -0.5), W_v=rnd(kv, dm, std=dm ** -0.5),
                          k_norm_w=torch.ones(base.D, device=dev)) for _ in range(5)]}

    def timed(fn, n=10, warm=3):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(n):
            fn()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / n

    def point(C, L):
        cfg = base.replace(B=C, lengths=f"fixed:{L}")
        table, num_pages = I.make_page_table(cfg.replace(lengths=f"fixed:{L + cfg.k}"),
                                             np.full(C, L + cfg.k, np.int32), seed=0)
        pt = torch.from_numpy(table).to(dev)
        lens = torch.full((C,), L, dtype=torch.int32, device=dev)
        caches = [dict(k_cache=rnd(num_pages, 16, base.Hkv, base.D), v_cache=rnd(num_pages, 16, base.Hkv, base.D))
                  for _ in range(5)]
        X = dict(page_table=pt, ctx_lens=lens, block_emb=rnd(C, cfg.k, dm), h_last=rnd(C, base.d_h), caches=caches)
        h_new = rnd(C, cfg.k, base.d_h)
        ws_h = hspec.workspace(hspec.drafter_forward_workspace(cfg, table.shape[1], num_pages, L))
        ws_i = hspec.workspace(hspec.kv_inject_workspace(cfg, table.shape[1], num_pages))
        out = torch.empty((C, cfg.k, dm), dtype=torch.float32, device=dev)
        t_h = timed(lambda: hspec.drafter_forward(cfg, shared, hyb, X, out, ws_h, L))
        t_i = timed(lambda: hspec.kv_inject(cfg, IW, h_new, caches, pt, lens, ws_i))
        t_b = timed(lambda: hspec.drafter_forward(cfg, {}, bd, X, out, ws_h, L))
        assert hspec.read_status(ws_h) == 0 and hspec.read_status(ws_i) == 0
        row = {"C": C, "ctx": L, "hybrid_ms": round(t_h, 4), "inject_ms": round(t_i, 4),
               "block_diffusion_ms": round(t_b, 4), "block_diffusion_with_inject_ms": round(t_i + t_b, 4),
               "hybrid_speedup": round((t_i + t_b) / t_h - 1.0, 4)}
        log(f"C={C:4d} ctx={L:5d}: hybrid {t_h:.3f} ms; block diffusion {t_b:.3f} + injection {t_i:.3f} ms; "
            f"hybrid faster by {row['hybrid_speedup'] * 100:+.1f} %")
        return row

    conc = [point(C, 1040) for C in (4, 8, 16, 32, 64, 128)]
    ctx = [point(128, L) for L in (256, 512, 768, 1024, 1536, 2048, 3072, 4096)]
    print(json.dumps({"metric": "draft-step forward time, hybrid vs block diffusion with KV injection",
                      "unit": "ms", "data": "synthetic", "dtype": "bf16",
                      "shapes": {"d_model": dm, "mamba": "H48 P64 N16 G4", "Hq": base.Hq, "Hkv": base.Hkv,
                                 "D": base.D, "ff": ff, "k": base.k, "fused_layers": base.n_fuse, "window": 2048},
                      "concurrency": conc, "context_at_C128": ctx}), flush=True)


def cpu_baseline(cfg, W, x, n_req: int):
    """The float64 oracle on the first n_req requests of the same workload (all positions)."""
    import oracle.hspec_oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        affinity = os.cpu_count() or 1
    pool = O._threads()      # worker threads of the oracle's blocked state projection
    t0 = time.perf_counter()
    O.draft_step(W, x, cfg, requests=list(range(n_req)))
    dt = time.perf_counter() - t0
    return {"value": n_req * cfg.k / dt, "unit": "drafted tokens/s", "cores": int(min(affinity, max(pool, blas))),
            "kind": "oracle", "affinity_cores": int(affinity), "host_cpus": int(os.cpu_count() or 1),
            "blas_threads": int(blas), "oracle_pool_threads": int(pool),
            "sample": f"{n_req} of {cfg.B} requests of {cfg.name} (all {cfg.k} positions, full W_dS "
                      f"projection), {dt:.1f} s wall; value = {n_req} x {cfg.k} drafted tokens / wall time"}


def sweep_inputs(cfg, Xd, x, seed, torch):
    """Block queries/keys/values for the KV sweep over the same cache, table and lengths."""
    Ad = dict(Xd)
    for k, name, heads in (("q", "attn_q", cfg.Hq), ("k_blk", "attn_kblk", cfg.Hkv), ("v_blk", "attn_vblk", cfg.Hkv)):
        Ad[k] = hspec.to_device(I.normal(name, (cfg.B, cfg.k, heads, cfg.D), 1.0, seed, cfg.dtype))
    maxL = int(x["ctx_lens"].max())
    aws = hspec.workspace(hspec.paged_attn_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    o = torch.empty((cfg.B, cfg.k, cfg.Hq, cfg.D), dtype=torch.float32, device="cuda")
    return Ad, aws, o


def counters(cfg, seed, torch):
    """One launch each of a 1 GiB device copy (to calibrate the byte counters), the state
    projection and the attention core, then two whole drafting steps, for counter collection
    under rocprofv3 (FETCH_SIZE / WRITE_SIZE, or SQ counters per kernel of the step)."""
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    log("copy: 1 GiB")
    W = I.make_weights(cfg, seed, skip=("W_in", "W_out", "W_q", "W_k", "W_v", "W_o"))
    x = I.make_inputs(cfg, seed)
    Wd = {k: hspec.to_device(W[k]) for k in ("W_r", "W_dS")}
    if cfg.dtype == "bf16":
        Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    S0 = torch.empty((cfg.B, cfg.H, cfg.P, cfg.N), dtype=torch.float32, device="cuda")
    sws = hspec.workspace(hspec.state_init_workspace(cfg))
    hspec.state_init(cfg, Wd, hspec.to_device(x["h_last"]), S0, sws)
    torch.cuda.synchronize()
    log("state projection: 1 launch")
    del Wd, S0, sws
    Xd = {k: hspec.to_device(v) if isinstance(v, np.ndarray) else v for k, v in x.items()
          if k not in ("h_last", "block_emb")}
    Ad, aws, o = sweep_inputs(cfg, Xd, x, seed, torch)
    hspec.paged_attn(cfg, Ad, o, aws, int(x["ctx_lens"].max()))
    torch.cuda.synchronize()
    log("KV sweep: 1 launch")
    del Ad, aws, o
    W = I.make_weights(cfg, seed)
    Wd = {k: hspec.to_device(v) for k, v in W.items()}
    if cfg.dtype == "bf16":
        Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    Xd["h_last"] = hspec.to_device(x["h_last"])
    Xd["block_emb"] = hspec.to_device(x["block_emb"])
    maxL = int(x["ctx_lens"].max())
    ws = hspec.workspace(hspec.draft_step_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    out = torch.empty((cfg.B, cfg.k, cfg.d_model), dtype=torch.float32, device="cuda")
    for _ in range(2):
        hspec.draft_step(cfg, Wd, Xd, out, ws, maxL)
    torch.cuda.synchronize()
    log("draft step: 2 launches")
    del Wd, Xd, ws, out
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--cpu-requests", type=int, default=0,
                    help="requests the CPU oracle drafts for cpu_baseline (default: the whole batch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--window", type=int, default=None,
                    help="sliding window of the drafter attention in tokens (the paper's drafters use "
                         "2048); default: the workload's own (full context)")
    ap.add_argument("--block-causal", action="store_true",
                    help="causal attention inside the drafted block instead of bidirectional")
    ap.add_argument("--kv-heads", type=int, default=0,
                    help="partial target-KV-head reuse: the drafter attends with this many of the "
                         "target's KV heads (evenly spaced), keeping the GQA group size")
    ap.add_argument("--compare", action="store_true",
                    help="time the hybrid drafter against a block-diffusion drafter with KV injection "
                         "across concurrency and context length, print one JSON line and exit")
    ap.add_argument("--counters", action="store_true",
                    help="launch each measured kernel once (for rocprofv3 --pmc) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): this build has no multi-GPU path; "
              "the drafting step is measured on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    cfg = I.CONFIGS[args.config]
    if args.window is not None:
        cfg = cfg.replace(window=args.window)
    if args.block_causal:
        cfg = cfg.replace(block_causal=True)
    if args.kv_heads:
        n = args.kv_heads
        if not 0 < n <= cfg.Hkv:
            sys.exit(f"--kv-heads must be in 1..{cfg.Hkv}")
        cfg = cfg.replace(Hkv=n, Hq=cfg.g * n, Hkv_target=cfg.Hkv,
                          kv_heads=tuple(i * cfg.Hkv // n for i in range(n)))
    if args.counters:
        counters(cfg, args.seed, torch)
        return
    if args.compare:
        compare_systems(args, torch)
        return
    t0 = time.perf_counter()
    W = I.make_weights(cfg, args.seed)
    x = I.make_inputs(cfg, args.seed)
    log(f"generated inputs in {time.perf_counter() - t0:.1f} s")
    t0 = time.perf_counter()
    Wd = {k: hspec.to_device(v) for k, v in W.items()}
    Xd = {k: hspec.to_device(v) if isinstance(v, np.ndarray) else v for k, v in x.items()}
    if cfg.dtype == "bf16":   # load-time re-layout of W_dS (hspec_pack_w_ds), outside the timed region
        Wd["W_dS_packed"] = hspec.pack_w_ds(Wd.pop("W_dS"), cfg.d_S, cfg.rank)
    torch.cuda.synchronize()
    log(f"uploaded in {time.perf_counter() - t0:.1f} s")
    L = x["ctx_lens"]
    maxL = int(L.max())
    ws = hspec.workspace(hspec.draft_step_workspace(cfg, x["page_table"].shape[1], x["num_pages"], maxL))
    out = torch.empty((cfg.B, cfg.k, cfg.d_model), dtype=torch.float32, device="cuda")

    def step():
        hspec.draft_step(cfg, Wd, Xd, out, ws, maxL)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # one event between consecutive steps: the first and last bracket the K timed steps, the
    # differences give each step's duration (median and p10/p90 beside the mean)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t_wall = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    step_dist = {"mean": round(ms, 4), "median": round(float(np.median(per_step)), 4),
                 "p10": round(float(np.percentile(per_step, 10)), 4),
                 "p90": round(float(np.percentile(per_step, 90)), 4),
                 "min": round(float(per_step.min()), 4), "max": round(float(per_step.max()), 4)}
    assert hspec.read_status(ws) == 0
    assert bool(torch.isfinite(out).all())
    tok_s = cfg.B * cfg.k / (ms / 1e3)
    log(f"draft step: {ms:.3f} ms/step (median {step_dist['median']:.3f}, p10 {step_dist['p10']:.3f}, "
        f"p90 {step_dist['p90']:.3f}; {t_wall / args.steps * 1e3:.3f} ms wall), {tok_s:,.0f} drafted tok/s")

    # dominant kernel: the state projection (Proj_r then Proj_dS), timed as its own launches
    sws = hspec.workspace(hspec.state_init_workspace(cfg))
    S0 = torch.empty((cfg.B, cfg.H, cfg.P, cfg.N), dtype=torch.float32, device="cuda")
    state = lambda: hspec.state_init(cfg, Wd, Xd["h_last"], S0, sws)  # noqa: E731
    t_state = time_in_step(state, args.steps, args.warmup, step, torch)
    b_state = RL.state_proj_bytes(cfg, 2, 4) + cfg.rank * cfg.d_h * 2

    # the target-KV sweep and its split reduction, same cache, table and lengths: the sweep kernel
    # alone, and the whole attention core (work list + sweep + split reduction)
    Ad, aws, o = sweep_inputs(cfg, Xd, x, args.seed, torch)
    t_plan, t_sweep, t_red = time_attention(cfg, Ad, o, aws, maxL, args.steps, args.warmup, step, torch)
    t_core = t_sweep + t_red
    b_sweep = RL.sweep_bytes(cfg, L)
    del S0, sws
    log(f"state projection: {t_state * 1e6:.1f} us, {b_state / t_state / 1e9:.0f} GB/s; "
        f"KV sweep kernel: {t_sweep * 1e6:.1f} us, {b_sweep / t_sweep / 1e9:.0f} GB/s; "
        f"with the split reduction: {t_core * 1e6:.1f} us, {b_sweep / t_core / 1e9:.0f} GB/s "
        f"(work list launched alone: {t_plan * 1e6:.1f} us)")

    h_state = kernel_hash(["gemm.hip"])
    h_sweep = kernel_hash(["attn.hip"])
    roof = {"bound": "hbm", "achieved": round(b_state / t_state / 1e9, 1), "peak": RL.HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(b_state / t_state / 1e9 / RL.HBM_PEAK_GBS, 4),
            "traffic": traffic_for("state_proj", h_state, cfg.name), "kernel": "state projection (Proj_r + Proj_dS GEMMs)",
            "algorithmic_bytes": int(b_state), "avg_launch_us": round(t_state * 1e6, 2)}
    # headline: the attention core on the step's path (split-K sweep + cross-split reduction;
    # the work list rides in the step's q/k-norm + RoPE launch); the sweep alone is a sub-field
    roof_sweep = {"bound": "hbm", "achieved": round(b_sweep / t_core / 1e9, 1), "peak": RL.HBM_PEAK_GBS,
                  "unit": "GB/s", "frac": round(b_sweep / t_core / 1e9 / RL.HBM_PEAK_GBS, 4),
                  "traffic": traffic_for("kv_sweep", h_sweep, cfg.name),
                  "kernel": "target-KV attention core: split-K sweep + cross-split reduction",
                  "algorithmic_bytes": int(b_sweep), "avg_us": round(t_core * 1e6, 2),
                  "reduction_us": round(t_red * 1e6, 2),
                  "work_list": {"where": "extra workgroup of the draft step's q/k-norm + RoPE launch",
                                "standalone_launch_us": round(t_plan * 1e6, 2)},
                  "tflops": round(RL.sweep_flops(cfg, L) / t_core / 1e12, 1),
                  "sweep_kernel_only": {"avg_launch_us": round(t_sweep * 1e6, 2),
                                        "achieved": round(b_sweep / t_sweep / 1e9, 1),
                                        "frac": round(b_sweep / t_sweep / 1e9 / RL.HBM_PEAK_GBS, 4)}}
    del Ad, aws, o

    # the draft head after the step (final norm, LM head over the pruned vocabulary, Markov
    # correction, greedy tokens) on the step's own output, and its LM-head GEMM alone
    head = head_figures(cfg, out, step, args, torch)
    scan = scan_figures(cfg, step, args, torch)
    fwd = forward_figures(cfg, Wd, Xd, x, args, torch) if cfg.dtype == "bf16" else None

    cpu = None
    if not args.no_cpu_baseline:
        del Wd, Xd, ws, out
        torch.cuda.empty_cache()
        n_req = min(cfg.B, args.cpu_requests) if args.cpu_requests > 0 else cfg.B
        log(f"cpu baseline: oracle on {n_req} request(s) ...")
        cpu = cpu_baseline(cfg, W, x, n_req)
        log(f"cpu baseline: {cpu['value']:.2f} tok/s on {cpu['cores']} threads")

    rec = {
        "metric": METRIC, "value": round(tok_s, 1), "unit": "drafted tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "step_ms": step_dist,
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cfg.name, "B": cfg.B, "k": cfg.k, "ctx_lens": cfg.lengths,
                   "sum_ctx_tokens": int(L.sum()), "Hq": cfg.Hq, "Hkv": cfg.Hkv, "D": cfg.D,
                   "d_model": cfg.d_model, "mamba": f"H{cfg.H} P{cfg.P} N{cfg.N} G{cfg.G} chunk{cfg.chunk}",
                   "page_size": cfg.page_size, "window": cfg.window, "block_causal": cfg.block_causal,
                   "kv_heads_reused": list(cfg.kv_map), "target_kv_heads": cfg.Hkv_cache,
                   "W_dS_layout": "packed" if cfg.dtype == "bf16" else "row-major",
                   "parallelism": "single GPU"},
        "roofline": roof,
        "roofline_kv_sweep": roof_sweep,
        "cpu_baseline": cpu,
        "ssd_scan": scan,
        "draft_head": dict(head, drafted_tok_s_with_head=round(cfg.B * cfg.k / (ms / 1e3 + head["avg_us"] / 1e6), 1)),
        "drafter_forward": None if fwd is None else dict(
            fwd, with_head_drafted_tok_s=round(cfg.B * cfg.k / (fwd["ms"] / 1e3 + head["avg_us"] / 1e6), 1)),
        "step_bytes_ideal": int(RL.step_bytes(cfg, L)),
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
    # main's device tensors are released by now; leave nothing for exit-time teardown (which
    # runs after a profiler's own finalisation when the program is profiled)
    import torch as _t
    if _t.cuda.is_available():
        _t.cuda.synchronize()
        _t.cuda.empty_cache()
