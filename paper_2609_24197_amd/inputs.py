"""Seeded synthetic inputs for the H-Spec block-drafting step.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the method's arithmetic, so both the HIP path and the
float64 oracle can consume exactly the same values.

Shapes follow the drafter of the paper (H-Spec, Sec. 3.3 and App. B.1):
a Mamba-2 mixer whose initial state comes from the fused last-token hidden
state, and a Qwen3-style attention layer that reuses one target layer's
paged K/V cache in place.  The workload configurations are synthetic stand-ins
for the paper's 8B-class targets (32 query / 8 KV heads of dimension 128,
hidden size 4096) and its larger shape (64/8 heads, hidden 5120).

Storage convention: bf16 tensors are numpy ``uint16`` arrays holding the bf16
bit pattern (round-to-nearest-even from float32); fp32 tensors are
``float32``.  Per-head / per-channel parameters (dt_bias, A_log, D and the
norm gains) are always fp32.

Every tensor is drawn block by block from its own PCG64 stream keyed by
``(seed, crc32(name), block)``, so any tensor can be regenerated in parallel
and independently of the others.
"""
from __future__ import annotations

import dataclasses
import math
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

BLOCK = 1 << 22  # elements per independent random stream


@dataclass(frozen=True)
class StepConfig:
    """Dimensions of one block-drafting step (notation of the paper, App. B.1)."""

    name: str
    B: int            # concurrent requests
    k: int            # draft block length
    d_model: int      # drafter hidden size (= target hidden size)
    H: int            # Mamba heads
    P: int            # Mamba head dim
    N: int            # Mamba state dim (d_state)
    G: int            # B/C groups
    chunk: int        # SSD chunk length
    Hq: int           # query heads (= target's)
    Hkv: int          # KV heads the drafter attends with (= target's, or a subset of them)
    D: int            # attention head dim
    lengths: str      # context-length recipe, see ``make_lengths``
    dtype: str = "bf16"   # storage dtype: "bf16" or "f32"
    conv_w: int = 4   # depthwise causal conv width
    page_size: int = 16
    window: int = 0   # sliding window in tokens, 0 = full context
    block_causal: bool = False
    precise_io: bool = False   # attention I/O as hi/lo planes, block keys in fp32 (stacked layers)
    eps: float = 1e-6
    rope_theta: float = 1e6
    n_fuse: int = 1   # |M|, number of fused target layers
    ff: int = 0       # MLP hidden size of the full drafter, 0 = 3 * d_model
    r: int = 0        # fusion rank, 0 = d_model
    split_tokens: int = 0  # split-K size for the KV sweep, 0 = automatic
    Hkv_target: int = 0    # KV heads per slot of the target cache, 0 = Hkv
    kv_heads: tuple = ()   # target KV head read by each drafter KV head, () = 0 .. Hkv-1

    @property
    def d_h(self) -> int:
        return self.n_fuse * self.d_model

    @property
    def d_ff(self) -> int:
        return self.ff or 3 * self.d_model

    @property
    def rank(self) -> int:
        return self.r or self.d_model

    @property
    def d_inner(self) -> int:
        return self.H * self.P

    @property
    def d_S(self) -> int:
        return self.H * self.P * self.N

    @property
    def conv_dim(self) -> int:
        return self.d_inner + 2 * self.G * self.N

    @property
    def d_in_proj(self) -> int:
        return 2 * self.d_inner + 2 * self.G * self.N + self.H

    @property
    def g(self) -> int:
        return self.Hq // self.Hkv

    @property
    def Hkv_cache(self) -> int:
        return self.Hkv_target or self.Hkv

    @property
    def kv_map(self) -> tuple:
        return tuple(self.kv_heads) if self.kv_heads else tuple(range(self.Hkv))

    def replace(self, **kw) -> "StepConfig":
        return dataclasses.replace(self, **kw)


_8B = dict(d_model=4096, H=128, P=64, N=128, G=1, chunk=16, Hq=32, Hkv=8, D=128)

CONFIGS = {
    1: StepConfig(name="tiny-f32", B=1, k=4, d_model=256, H=8, P=64, N=16, G=1, chunk=4,
                  Hq=4, Hkv=1, D=64, lengths="fixed:64", dtype="f32"),
    2: StepConfig(name="8b-single", B=1, k=16, lengths="fixed:2048", **_8B),
    3: StepConfig(name="8b-serving-b64", B=64, k=16, lengths="uniform:512:8192", **_8B),
    4: StepConfig(name="8b-longctx-b8", B=8, k=16, lengths="fixed:32768", **_8B),
    5: StepConfig(name="large-b128", B=128, k=16, d_model=5120, H=160, P=64, N=128, G=1,
                  chunk=16, Hq=64, Hkv=8, D=128, lengths="lognormal:2048:1.0:256:16384"),
}


def _stream(seed: int, name: str, block: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([int(seed), zlib.crc32(name.encode()), int(block)])
    return np.random.Generator(np.random.PCG64(ss))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (input plumbing only)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal(name: str, shape, std: float, seed: int, dtype: str, mean: float = 0.0) -> np.ndarray:
    """N(mean, std^2) drawn in float32 and rounded to the storage dtype."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    nblk = (n + BLOCK - 1) // BLOCK

    def fill(i):
        lo, hi = i * BLOCK, min(n, (i + 1) * BLOCK)
        v = _stream(seed, name, i).standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        if mean != 0.0:
            v += np.float32(mean)
        out[lo:hi] = f32_to_bf16_bits(v) if dtype == "bf16" else v

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
    return out.reshape(shape)


def make_lengths(cfg: StepConfig, seed: int = 0) -> np.ndarray:
    """Per-request context lengths.

    Recipes: ``fixed:L``; ``uniform:lo:hi`` (integers, inclusive);
    ``lognormal:median:sigma:lo:hi`` (ln L ~ N(ln median, sigma^2), clipped,
    rounded to the nearest integer); ``list:a,b,c`` (explicit).
    """
    kind, *a = cfg.lengths.split(":")
    rng = _stream(seed, "ctx_lens")
    if kind == "fixed":
        L = np.full(cfg.B, int(a[0]))
    elif kind == "uniform":
        L = rng.integers(int(a[0]), int(a[1]) + 1, size=cfg.B)
    elif kind == "lognormal":
        med, sig, lo, hi = float(a[0]), float(a[1]), int(a[2]), int(a[3])
        L = np.clip(np.rint(np.exp(rng.normal(math.log(med), sig, size=cfg.B))), lo, hi)
    elif kind == "list":
        L = np.array([int(v) for v in a[0].split(",")])
        assert L.size == cfg.B
    else:
        raise ValueError(cfg.lengths)
    return L.astype(np.int32)


def make_page_table(cfg: StepConfig, lengths: np.ndarray, seed: int = 0, extra_pages: int = 0,
                    pad_pages: int = 0):
    """One shared physical pool; each request's logical pages land on a shuffled set.

    Returns ``(page_table [B, max_pages] int32, num_pages)``.  Entries past a
    request's last page are -1; ``extra_pages`` unreferenced pages are added to
    the pool and ``pad_pages`` extra columns to the table.
    """
    ps = cfg.page_size
    npg = [(int(L) + ps - 1) // ps for L in lengths]
    num_pages = int(sum(npg)) + int(extra_pages)
    perm = _stream(seed, "page_perm").permutation(max(num_pages, 1)).astype(np.int32)
    max_pages = max(1, max(npg) if npg else 1) + int(pad_pages)
    table = np.full((cfg.B, max_pages), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(npg):
        table[b, :n] = perm[off:off + n]
        off += n
    return table, max(num_pages, 1)


def make_weights(cfg: StepConfig, seed: int = 0, skip=(), prefix: str = "") -> dict:
    """Synthetic drafter weights: W ~ N(0, 1/fan_in), stored as [out, in].  ``prefix`` keys the
    random streams (one set of weights per drafter layer); the dict keys stay the same."""
    dt = cfg.dtype
    H, dm, di = cfg.H, cfg.d_model, cfg.d_inner
    w = {}

    def add(name, shape, std, store=dt, mean=0.0):
        if name not in skip:
            w[name] = normal(prefix + name, shape, std, seed, store, mean)

    add("W_r", (cfg.rank, cfg.d_h), cfg.d_h ** -0.5)
    add("W_dS", (cfg.d_S, cfg.rank), cfg.rank ** -0.5)
    add("W_in", (cfg.d_in_proj, dm), dm ** -0.5)
    add("conv_w", (cfg.conv_dim, cfg.conv_w), cfg.conv_w ** -0.5)
    add("conv_b", (cfg.conv_dim,), cfg.conv_w ** -0.5)
    # dt bias: inverse softplus of dt0, log-uniform in [1e-3, 1e-1] (Mamba-2 initialisation)
    u = _stream(seed, prefix + "dt_bias").uniform(math.log(1e-3), math.log(1e-1), size=H)
    dt0 = np.exp(u)
    w["dt_bias"] = (dt0 + np.log(-np.expm1(-dt0))).astype(np.float32)
    w["A_log"] = _stream(seed, prefix + "A_log").uniform(-2.0, 1.0, size=H).astype(np.float32)
    add("D", (H,), 1.0, "f32")
    add("gnorm_w", (di,), 0.1, "f32", 1.0)
    add("W_out", (dm, di), di ** -0.5)
    add("norm1_w", (dm,), 0.1, "f32", 1.0)
    add("norm2_w", (dm,), 0.1, "f32", 1.0)
    add("W_q", (cfg.Hq * cfg.D, dm), dm ** -0.5)
    add("W_k", (cfg.Hkv * cfg.D, dm), dm ** -0.5)
    add("W_v", (cfg.Hkv * cfg.D, dm), dm ** -0.5)
    add("W_o", (dm, cfg.Hq * cfg.D), (cfg.Hq * cfg.D) ** -0.5)
    add("q_norm_w", (cfg.D,), 0.1, "f32", 1.0)
    add("k_norm_w", (cfg.D,), 0.1, "f32", 1.0)
    return w


def make_inputs(cfg: StepConfig, seed: int = 0, extra_pages: int = 0, pad_pages: int = 0) -> dict:
    """Activations, the paged target cache and its page table."""
    L = make_lengths(cfg, seed)
    table, num_pages = make_page_table(cfg, L, seed, extra_pages, pad_pages)
    x = {
        "ctx_lens": L,
        "page_table": table,
        "num_pages": num_pages,
        "h_last": normal("h_last", (cfg.B, cfg.d_h), 1.0, seed, cfg.dtype),
        "block_emb": normal("block_emb", (cfg.B, cfg.k, cfg.d_model), 1.0, seed, cfg.dtype),
        "k_cache": normal("k_cache", (num_pages, cfg.page_size, cfg.Hkv_cache, cfg.D), 1.0, seed, cfg.dtype),
        "v_cache": normal("v_cache", (num_pages, cfg.page_size, cfg.Hkv_cache, cfg.D), 1.0, seed, cfg.dtype),
    }
    return x


def make_scan_inputs(B, T, H, P, N, G, seed=0, dtype="bf16", dt_range=(1e-3, 1e-1), s0=True):
    """Direct inputs of the SSD scan primitive (post-conv x, B, C; post-softplus dt)."""
    rng = _stream(seed, "scan_dt")
    dt = np.exp(rng.uniform(math.log(dt_range[0]), math.log(dt_range[1]), size=(B, T, H)))
    out = {
        "x": normal("scan_x", (B, T, H, P), 1.0, seed, dtype),
        "dt": dt.astype(np.float32),
        "A": (-np.exp(_stream(seed, "scan_A").uniform(-2.0, 1.0, size=H))).astype(np.float32),
        "Bm": normal("scan_B", (B, T, G, N), 1.0, seed, dtype),
        "Cm": normal("scan_C", (B, T, G, N), 1.0, seed, dtype),
        "Dskip": normal("scan_D", (H,), 1.0, seed, "f32"),
    }
    out["S0"] = normal("scan_S0", (B, H, P, N), 1.0, seed, dtype) if s0 else None
    return out


def make_attn_inputs(cfg: StepConfig, seed=0, extra_pages=0, pad_pages=0):
    """Direct inputs of the paged-attention primitive (post-norm, post-RoPE q and block k)."""
    x = make_inputs(cfg, seed, extra_pages, pad_pages)
    del x["h_last"], x["block_emb"]
    x["q"] = normal("attn_q", (cfg.B, cfg.k, cfg.Hq, cfg.D), 1.0, seed, cfg.dtype)
    x["k_blk"] = normal("attn_kblk", (cfg.B, cfg.k, cfg.Hkv, cfg.D), 1.0, seed, cfg.dtype)
    x["v_blk"] = normal("attn_vblk", (cfg.B, cfg.k, cfg.Hkv, cfg.D), 1.0, seed, cfg.dtype)
    return x


DRAFTER_LAYERS = ("MAF", "MAF", "MAF", "MF")   # App. B.1: 3 x (Mamba, attention, MLP) + 1 x (Mamba, MLP)
DRAFTER_FUSE = 5                                # |M|: five target layers fused into the state


def make_drafter_weights(cfg: StepConfig, seed: int = 0, layers=DRAFTER_LAYERS, skip_state: bool = False):
    """Weights of the whole drafter: ``shared`` (W_r [r, |M| d_model], W_dS) and one dict per
    layer with its Mamba, attention (layers spelled with "A"; key "cache" = the index of the
    target cache it reads, in order) and SwiGLU MLP weights ([ff, d_model] gate and up,
    [d_model, ff] down) and the three pre-norm gains."""
    shared = {} if skip_state else make_weights(cfg, seed, skip=("W_in", "conv_w", "conv_b", "D", "gnorm_w", "W_out",
                                                                 "norm1_w", "norm2_w", "W_q", "W_k", "W_v", "W_o",
                                                                 "q_norm_w", "k_norm_w"))
    shared.pop("dt_bias", None)
    shared.pop("A_log", None)
    out, n_attn = [], 0
    for l, spec in enumerate(layers):
        pre = f"L{l}."
        attn = () if "A" in spec else ("W_q", "W_k", "W_v", "W_o", "q_norm_w", "k_norm_w", "norm2_w")
        mamba = () if "M" in spec else ("W_in", "conv_w", "conv_b", "D", "gnorm_w", "W_out", "norm1_w")
        W = make_weights(cfg, seed, skip=("W_r", "W_dS") + attn + mamba, prefix=pre)
        if "M" not in spec:
            W.pop("dt_bias")
            W.pop("A_log")
        W["norm3_w"] = normal(pre + "norm3_w", (cfg.d_model,), 0.1, seed, "f32", 1.0)
        W["W_gate"] = normal(pre + "W_gate", (cfg.d_ff, cfg.d_model), cfg.d_model ** -0.5, seed, cfg.dtype)
        W["W_up"] = normal(pre + "W_up", (cfg.d_ff, cfg.d_model), cfg.d_model ** -0.5, seed, cfg.dtype)
        W["W_down"] = normal(pre + "W_down", (cfg.d_model, cfg.d_ff), cfg.d_ff ** -0.5, seed, cfg.dtype)
        W["cache"] = n_attn if "A" in spec else None
        n_attn += "A" in spec
        out.append(W)
    return shared, out


def make_drafter_inputs(cfg: StepConfig, seed: int = 0, n_caches: int = 3, extra_pages: int = 0) -> dict:
    """make_inputs plus the K/V caches of further target layers (``caches``: one dict per target
    layer an attention reads), all on the one page table."""
    x = make_inputs(cfg, seed, extra_pages)
    caches = [dict(k_cache=x.pop("k_cache"), v_cache=x.pop("v_cache"))]
    shape = caches[0]["k_cache"].shape
    for c in range(1, n_caches):
        caches.append(dict(k_cache=normal(f"k_cache{c}", shape, 1.0, seed, cfg.dtype),
                           v_cache=normal(f"v_cache{c}", shape, 1.0, seed, cfg.dtype)))
    x["caches"] = caches
    return x


def make_inject_weights(cfg: StepConfig, seed: int = 0, n_layers: int = 5) -> dict:
    """Weights of the drafter-side KV-injection stand-in: the fusion W_fc [d_model, |M| d_model]
    and, per drafter layer, W_k, W_v [Hkv D, d_model] and the key norm gain."""
    dm, kv = cfg.d_model, cfg.Hkv * cfg.D
    return {
        "W_fc": normal("inj.W_fc", (dm, cfg.d_h), cfg.d_h ** -0.5, seed, cfg.dtype),
        "layers": [{"W_k": normal(f"inj{l}.W_k", (kv, dm), dm ** -0.5, seed, cfg.dtype),
                    "W_v": normal(f"inj{l}.W_v", (kv, dm), dm ** -0.5, seed, cfg.dtype),
                    "k_norm_w": normal(f"inj{l}.k_norm_w", (cfg.D,), 0.1, seed, "f32", 1.0)}
                   for l in range(n_layers)],
    }


HEAD_VOCAB = 32000   # pruned drafter vocabulary (App. B.2)
HEAD_RANK = 256      # Markov rank (App. B.1)


def make_head_weights(cfg: StepConfig, seed: int = 0, vocab: int = HEAD_VOCAB, rank: int = HEAD_RANK) -> dict:
    """Draft-head weights: final norm gain, LM head [V, d_model] ~ N(0, 1/d_model), and the two
    rank-R Markov factors E_M, U_M [V, R] ~ N(0, 1/R) (bf16)."""
    return {
        "norm_f_w": normal("norm_f_w", (cfg.d_model,), 0.1, seed, "f32", 1.0),
        "W_lm": normal("W_lm", (vocab, cfg.d_model), cfg.d_model ** -0.5, seed, "bf16"),
        "E_M": normal("E_M", (vocab, rank), 1.0, seed, "bf16"),
        "U_M": normal("U_M", (vocab, rank), rank ** -0.5, seed, "bf16"),
    }


def make_head_inputs(cfg: StepConfig, seed: int = 0, vocab: int = HEAD_VOCAB, sample: bool = False) -> dict:
    """Hidden states [B, k, d_model] fp32 ~ N(0, 1), the last committed token of each request, and
    (sample=True) Gumbel noise -log(-log u), u ~ U(0, 1), for every (request, position, token)."""
    x = {
        "hidden": normal("head_hidden", (cfg.B, cfg.k, cfg.d_model), 1.0, seed, "f32"),
        "prev_tok": _stream(seed, "prev_tok").integers(0, vocab, size=cfg.B).astype(np.int32),
    }
    if sample:
        n = cfg.B * cfg.k * vocab
        u = np.empty(n, dtype=np.float64)
        nblk = (n + BLOCK - 1) // BLOCK
        for i in range(nblk):
            lo, hi = i * BLOCK, min(n, (i + 1) * BLOCK)
            u[lo:hi] = _stream(seed, "gumbel_u", i).random(hi - lo)
        u = np.clip(u, 1e-300, None)
        x["gumbel"] = (-np.log(-np.log(u))).astype(np.float32).reshape(cfg.B, cfg.k, vocab)
    return x
