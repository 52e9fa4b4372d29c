"""Plain float64 CPU oracle for the H-Spec block-drafting step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The HIP library never
calls it and shares no code with it.

Everything here is the plain definition of what the drafting step computes,
written for a reader to check against the paper by eye:

* cross-layer fusion and state projection, S_init = Proj_dS(Proj_r(Concat h)),
  reshaped to [n_heads, head_dim, d_state]  (Sec. 3.3.1, the fusion equation;
  App. B.1 "Mamba" for the reshape);
* the Mamba-2 mixer, with its selective recurrence S_i = A_i S_{i-1} + B_i x_i
  evaluated one token at a time from the injected state (Sec. 3.3.1);
* the attention module over the target's paged K/V cache plus the block's own
  K/V, with RoPE positions continuing the prefix (Sec. 3.3.2: KV dimension,
  attention mask, positional alignment; App. B.2 for Qwen3 attention and the
  sliding window);
* the drafting step, x1 = e + Mamba(RMSNorm(e)), out = x1 + Attn(RMSNorm(x1));
* the whole drafter (Sec. 3.3; App. B.1 "Number of drafter layers" and "Target-layer
  mapping"): one S_init shared by every layer's Mamba, then layers of Mamba, attention
  over that layer's own target cache (absent in the partial layer) and a SwiGLU MLP,
  each pre-normed with a residual;
* drafter-side KV injection (Sec. 2), the per-step cost of block-diffusion drafters that the
  method removes, as a comparison stand-in;
* the draft head: final RMSNorm, the LM head over the pruned vocabulary (App. B.2,
  "Pruned drafter vocabulary"), and the first-order Markov correction of each
  position's logits by the token chosen at the position before it (Sec. 3.3.3),
  then greedy or Gumbel-max sampled tokens.

Attention is the naive softmax over the full score row; the scan is the
sequential per-token recurrence.  ``ssd_chunked`` is a second float64
formulation (the SSD chunk algebra) kept only so that tests can pin the
sequential one against an independent derivation.

Pins: every primitive here (state projection layout, conv, pointwise functions,
RoPE, slot map, naive attention, the recurrence) is checked against textbook
special cases, closed forms and library routines.  The composed functions
``mamba_mixer``, ``attention_layer``, ``draft_step`` and ``drafter_forward`` are pinned
only through their parts and whole-function properties (zero input, causality, decay
rate, residual structure, dense-cache attention, the shared initial state, the
layer-to-cache mapping); the mixer's wiring (the order of the in_proj split, the SiLU after
the conv, the gated-norm gain) is pinned by one-channel and one-hot-selector cases with
closed forms; beyond those they are parity unpinned.  ``draft_head`` and
``kv_inject`` are pinned by special cases (no Markov term, a bigram chain, Gumbel-max
frequencies; slot placement and untouched slots).

Inputs are storage arrays: bf16 as uint16 bit patterns, or float32/float64.
They are widened to float64 here, block by block for the large state
projection.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "f64", "rmsnorm", "silu", "softplus", "state_init", "in_proj_split", "causal_conv1d",
    "ssd_sequential", "ssd_chunked", "gated_rmsnorm", "mamba_mixer", "gather_slots", "rope",
    "paged_attention", "attention_layer", "draft_step", "mlp", "drafter_forward", "kv_inject", "draft_head",
    "compare",
]


# ----------------------------------------------------------------------------- helpers

def _threads() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return 1


def f64(a, dtype: str | None = None) -> np.ndarray:
    """Widen a storage array to float64 (bf16 bit patterns are uint16)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def rmsnorm(x: np.ndarray, w, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softplus(x: np.ndarray) -> np.ndarray:
    """log(1 + e^x), evaluated without overflow."""
    return np.logaddexp(0.0, x)


# ------------------------------------------------- Sec. 3.3.1: fusion + state projection

def state_init(h_last, W_r, W_dS, H: int, P: int, N: int, block_rows: int = 1 << 15):
    """S_init = reshape(W_dS @ (W_r @ Concat h_n^{(m)})) per request.

    Sec. 3.3.1 (cross-layer fusion equation): F = Proj_r(Concat{h}), then
    S_init = Proj_dS(F); both projections are bias-free linear maps shared by
    every drafter layer.  ``h_last`` is the already concatenated
    [B, |M| d_h] last-position hidden state.  App. B.1: the d_S = H*P*N vector
    is reshaped to [n_heads, head_dim, d_state].
    Returns (S0 [B, H, P, N], F [B, r]).
    """
    h = f64(h_last)
    F = h @ f64(W_r).T
    d_S = H * P * N
    assert W_dS.shape[0] == d_S
    S = np.empty((h.shape[0], d_S))

    def rows(i0):                    # output rows are independent: blocks may run in any order
        i1 = min(d_S, i0 + block_rows)
        S[:, i0:i1] = F @ f64(W_dS[i0:i1]).T

    starts = range(0, d_S, block_rows)
    if len(starts) > 1:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(rows, starts))
    else:
        rows(0)
    return S.reshape(h.shape[0], H, P, N), F


# ------------------------------------------------------------ Sec. 3.3.1: Mamba-2 mixer

def in_proj_split(zxbcdt: np.ndarray, H: int, P: int, G: int, N: int):
    """Split the input projection into z, xBC and dt (Mamba-2 ordering)."""
    di = H * P
    z = zxbcdt[..., :di]
    xBC = zxbcdt[..., di:2 * di + 2 * G * N]
    dt = zxbcdt[..., 2 * di + 2 * G * N:]
    assert dt.shape[-1] == H
    return z, xBC, dt


def causal_conv1d(x: np.ndarray, w, b) -> np.ndarray:
    """Depthwise causal convolution over time with zero left state.

    out[t, c] = b[c] + sum_j w[c, j] * x[t - (K-1) + j, c], x[tau] = 0 for tau < 0.
    x: [..., T, C]; w: [C, K]; b: [C].
    """
    T = x.shape[-2]
    K = w.shape[1]
    out = np.broadcast_to(b, x.shape).copy()
    for t in range(T):
        for j in range(K):
            tau = t - (K - 1) + j
            if tau >= 0:
                out[..., t, :] += w[:, j] * x[..., tau, :]
    return out


def ssd_sequential(x, dt, A, Bm, Cm, Dskip, S0=None):
    """The selective recurrence, one draft position at a time (Sec. 3.3.1).

    Per head h (group g = h // (H / G)):
        S_t = exp(dt_t A_h) S_{t-1} + dt_t x_t (outer) B_t      [P, N]
        y_t = S_t C_t + D_h x_t
    starting from S_{-1} = S0 (the injected state).
    x: [B, T, H, P]; dt: [B, T, H]; A, Dskip: [H]; Bm, Cm: [B, T, G, N];
    S0: [B, H, P, N] or None (zeros).  Returns (y [B, T, H, P], S_final).
    """
    x, dt, A, Bm, Cm, Dskip = (f64(v) for v in (x, dt, A, Bm, Cm, Dskip))
    Bsz, T, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    assert H % G == 0
    grp = np.arange(H) // (H // G)
    S = np.zeros((Bsz, H, P, N)) if S0 is None else f64(S0).copy()
    y = np.empty((Bsz, T, H, P))
    for t in range(T):
        a = np.exp(dt[:, t, :] * A[None, :])                       # [B, H]
        Bt = Bm[:, t, grp, :]                                       # [B, H, N]
        Ct = Cm[:, t, grp, :]
        S = a[:, :, None, None] * S + (dt[:, t, :, None] * x[:, t])[:, :, :, None] * Bt[:, :, None, :]
        y[:, t] = (S @ Ct[:, :, :, None])[..., 0] + Dskip[None, :, None] * x[:, t]    # S_t C_t + D x_t
    return y, S


def ssd_chunked(x, dt, A, Bm, Cm, Dskip, S0=None, chunk: int = 16):
    """The same recurrence through the SSD chunk algebra (second formulation).

    Within a chunk, with l_t = sum_{u<=t} dt_u A (inclusive cumulative sum):
        y_t = exp(l_t) C_t S_in^T + sum_{s<=t} exp(l_t - l_s) dt_s (C_t . B_s) x_s + D x_t
        S_out = exp(l_end) S_in + sum_s exp(l_end - l_s) dt_s x_s (outer) B_s
    Used only to pin ``ssd_sequential`` in the tests.
    """
    x, dt, A, Bm, Cm, Dskip = (f64(v) for v in (x, dt, A, Bm, Cm, Dskip))
    Bsz, T, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    grp = np.arange(H) // (H // G)
    S = np.zeros((Bsz, H, P, N)) if S0 is None else f64(S0).copy()
    y = np.empty((Bsz, T, H, P))
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        dA = dt[:, c0:c1, :] * A[None, None, :]                     # [B, Q, H]
        l = np.cumsum(dA, axis=1)
        Bc = Bm[:, c0:c1][:, :, grp, :]                             # [B, Q, H, N]
        Cc = Cm[:, c0:c1][:, :, grp, :]
        xc = x[:, c0:c1]
        Q = c1 - c0
        # inter-chunk (state) contribution
        y_state = np.exp(l)[..., None] * np.einsum("bthn,bhpn->bthp", Cc, S)
        # intra-chunk contribution
        CB = np.einsum("bthn,bshn->bhts", Cc, Bc)
        lt = np.moveaxis(l, 1, 2)                                   # [B, H, Q]
        decay = np.exp(lt[:, :, :, None] - lt[:, :, None, :])
        mask = np.tril(np.ones((Q, Q), dtype=bool))
        Mx = np.where(mask, CB * decay, 0.0) * np.moveaxis(dt[:, c0:c1], 1, 2)[:, :, None, :]
        y_intra = np.einsum("bhts,bshp->bthp", Mx, xc)
        y[:, c0:c1] = y_state + y_intra + Dskip[None, None, :, None] * xc
        # state carry
        w_end = np.exp(lt[:, :, -1:] - lt) * np.moveaxis(dt[:, c0:c1], 1, 2)   # [B, H, Q]
        S = np.exp(lt[:, :, -1])[:, :, None, None] * S + np.einsum("bhs,bshp,bshn->bhpn", w_end, xc, Bc)
    return y, S


def gated_rmsnorm(y: np.ndarray, z: np.ndarray, w, G: int, eps: float) -> np.ndarray:
    """RMSNorm(y * SiLU(z)) * w, normalised within each of the G groups of channels."""
    g = y * silu(z)
    shp = g.shape
    gg = g.reshape(*shp[:-1], G, shp[-1] // G)
    gg = gg / np.sqrt(np.mean(gg * gg, axis=-1, keepdims=True) + eps)
    return gg.reshape(shp) * w


def mamba_mixer(u, S0, W, cfg, return_parts: bool = False):
    """One Mamba-2 mixer over the draft block, initialised from S0 (Sec. 3.3.1).

    u: [B, k, d_model] float64 (already normalised);  S0: [B, H, P, N].
    in_proj -> causal conv + SiLU on (x, B, C) -> dt = softplus(dt_raw + dt_bias),
    A = -exp(A_log) -> sequential recurrence from S0 -> y * SiLU(z) with grouped
    RMSNorm -> out_proj.  No biases on the projections.
    """
    H, P, N, G = cfg.H, cfg.P, cfg.N, cfg.G
    zxbcdt = u @ f64(W["W_in"]).T
    z, xBC, dt_raw = in_proj_split(zxbcdt, H, P, G, N)
    xBC = silu(causal_conv1d(xBC, f64(W["conv_w"]), f64(W["conv_b"])))
    Bsz, T = u.shape[0], u.shape[1]
    di = H * P
    x = xBC[..., :di].reshape(Bsz, T, H, P)
    Bm = xBC[..., di:di + G * N].reshape(Bsz, T, G, N)
    Cm = xBC[..., di + G * N:].reshape(Bsz, T, G, N)
    dt = softplus(dt_raw + f64(W["dt_bias"]))
    A = -np.exp(f64(W["A_log"]))
    y, S_fin = ssd_sequential(x, dt, A, Bm, Cm, f64(W["D"]), S0)
    yn = gated_rmsnorm(y.reshape(Bsz, T, di), z, f64(W["gnorm_w"]), G, cfg.eps)
    out = yn @ f64(W["W_out"]).T
    if return_parts:
        return out, dict(z=z, x=x, Bm=Bm, Cm=Cm, dt=dt, A=A, y=y, S_final=S_fin, yn=yn)
    return out


# ---------------------------------------------------------- Sec. 3.3.2: attention module

def gather_slots(page_table, ctx_lens, page_size: int, max_ctx_len: int) -> np.ndarray:
    """Physical slot of each logical cache position; -1 past the context length.

    slot(b, i) = page_table[b, i // page_size] * page_size + i % page_size.
    """
    pt = np.asarray(page_table)
    B = pt.shape[0]
    out = np.full((B, max_ctx_len), -1, dtype=np.int64)
    for b in range(B):
        for i in range(int(ctx_lens[b])):
            out[b, i] = int(pt[b, i // page_size]) * page_size + i % page_size
    return out.astype(np.int32)


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding at integer positions (angles in float64).

    For i < D/2: phi = pos * theta^(-2i/D);
    x'[i] = x[i] cos phi - x[i + D/2] sin phi; x'[i + D/2] = x[i + D/2] cos phi + x[i] sin phi.
    x: [..., T, heads, D]; pos: [..., T].
    """
    D = x.shape[-1]
    half = D // 2
    inv = theta ** (-(2.0 * np.arange(half)) / D)
    phi = np.asarray(pos, dtype=np.float64)[..., None] * inv            # [..., T, half]
    c = np.cos(phi)[..., None, :]
    s = np.sin(phi)[..., None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def paged_attention(q, k_blk, v_blk, k_cache, v_cache, page_table, ctx_lens, *,
                    page_size: int, window: int = 0, block_causal: bool = False,
                    scale: float | None = None, requests=None, kv_heads=None) -> np.ndarray:
    """Block queries over the target's paged K/V (in place) plus the block's K/V.

    Sec. 3.3.2: the reused target KVs are the prefix context of the block;
    block position j sits at position ctx_len + j.  Query j of request b sees
    cache keys i in [lo_j, L_b), lo_j = max(0, L_b + j - window + 1) when a
    sliding window is set, and block keys s in [0, k) (s <= j when
    ``block_causal``).  Query head hq reads KV head hq // (Hq / Hkv).
    Partial target-KV-head reuse (Sec. 3.3.2 "KV dimension"; future work in Sec. 5): the
    drafter's KV head h reads the target cache's head kv_heads[h] (default: head h).
    Naive softmax over the full score row (max subtracted).
    q: [B, k, Hq, D]; k_blk, v_blk: [B, k, Hkv, D]; caches [pages, ps, Hkv_target, D].
    Returns o [B, k, Hq, D] (only rows of ``requests`` filled if given).
    """
    q, kb, vb = f64(q), f64(k_blk), f64(v_blk)
    B, T, Hq, D = q.shape
    Hkv = kb.shape[2]
    g = Hq // Hkv
    scale = D ** -0.5 if scale is None else scale
    Hc = np.asarray(k_cache).shape[-2]                              # KV heads of the target cache
    kv_heads = list(range(Hkv)) if kv_heads is None or len(kv_heads) == 0 else list(kv_heads)
    assert len(kv_heads) == Hkv and all(0 <= t < Hc for t in kv_heads)
    kc = np.asarray(k_cache).reshape(-1, Hc, D)
    vc = np.asarray(v_cache).reshape(-1, Hc, D)
    o = np.zeros((B, T, Hq, D))
    for b in (range(B) if requests is None else requests):
        L = int(ctx_lens[b])
        slots = gather_slots(page_table[b:b + 1], [L], page_size, L)[0]
        Kc, Vc = f64(kc[slots]), f64(vc[slots])                     # [L, Hc, D]
        for h in range(Hkv):
            heads = np.arange(h * g, (h + 1) * g)                   # the query heads of KV head h
            Kh = np.ascontiguousarray(Kc[:, kv_heads[h], :])        # [L, D]: the target head it reuses
            Vh = np.ascontiguousarray(Vc[:, kv_heads[h], :])
            for j in range(T):
                pos = L + j
                lo = max(0, pos - window + 1) if window > 0 else 0
                nb = j + 1 if block_causal else T
                Q = q[b, j, heads]                                  # [g, D]
                # the full score row of each head: visible cache keys, then the block keys
                s = np.concatenate([Kh[lo:L] @ Q.T, kb[b, :nb, h] @ Q.T], axis=0) * scale   # [n, g]
                w = np.exp(s - s.max(axis=0))
                w = w / w.sum(axis=0)
                nc = L - lo
                o[b, j, heads] = w[:nc].T @ Vh[lo:L] + w[nc:].T @ vb[b, :nb, h]
    return o


def attention_layer(v, W, cache, cfg, return_parts: bool = False, requests=None):
    """Qwen3-style attention over target KV (Sec. 3.3.2, App. B.2).

    v: [B, k, d_model] float64 (already normalised).  Q/K/V projections,
    per-head RMSNorm of q and k, RoPE at positions ctx_len + j, attention over
    (target cache, block), output projection.  No residual here.
    """
    Bsz, T, _ = v.shape
    Hq, Hkv, D = cfg.Hq, cfg.Hkv, cfg.D
    q = (v @ f64(W["W_q"]).T).reshape(Bsz, T, Hq, D)
    kb = (v @ f64(W["W_k"]).T).reshape(Bsz, T, Hkv, D)
    vb = (v @ f64(W["W_v"]).T).reshape(Bsz, T, Hkv, D)
    q = rmsnorm(q, f64(W["q_norm_w"]), cfg.eps)
    kb = rmsnorm(kb, f64(W["k_norm_w"]), cfg.eps)
    L = np.asarray(cache["ctx_lens"], dtype=np.int64)
    pos = L[:, None] + np.arange(T)[None, :]
    q = rope(q, pos, cfg.rope_theta)
    kb = rope(kb, pos, cfg.rope_theta)
    o = paged_attention(q, kb, vb, cache["k_cache"], cache["v_cache"], cache["page_table"],
                        cache["ctx_lens"], page_size=cfg.page_size, window=cfg.window,
                        block_causal=cfg.block_causal, requests=requests,
                        kv_heads=getattr(cfg, "kv_heads", None))
    out = o.reshape(Bsz, T, Hq * D) @ f64(W["W_o"]).T
    if return_parts:
        return out, dict(q=q, k_blk=kb, v_blk=vb, o=o)
    return out


# ------------------------------------------------------------------- the drafting step

def draft_step(W, x, cfg, requests=None, return_parts: bool = False, progress=None):
    """x1 = e + Mamba(RMSNorm(e) g1; S_init);  out = x1 + Attn(RMSNorm(x1) g2).

    Sec. 3.3 (architecture: Mamba, then attention, in each drafter layer) with
    S_init from ``state_init`` (Sec. 3.3.1).  ``requests`` restricts the work
    to a subset of requests (rows of the batch); the outputs of the other rows
    are left as NaN.  ``progress``, if given, is called with the name of each
    finished stage (for long runs).
    """
    note = progress or (lambda stage: None)
    idx = np.arange(cfg.B) if requests is None else np.asarray(requests)
    S0, F = state_init(np.asarray(x["h_last"])[idx], W["W_r"], W["W_dS"], cfg.H, cfg.P, cfg.N)
    note("state projection")
    e = f64(np.asarray(x["block_emb"])[idx])
    u = rmsnorm(e, f64(W["norm1_w"]), cfg.eps)
    m_out, mparts = mamba_mixer(u, S0, W, cfg, return_parts=True)
    note("mamba")
    x1 = e + m_out
    v = rmsnorm(x1, f64(W["norm2_w"]), cfg.eps)
    cache = dict(k_cache=x["k_cache"], v_cache=x["v_cache"],
                 page_table=np.asarray(x["page_table"])[idx], ctx_lens=np.asarray(x["ctx_lens"])[idx])
    a_out, aparts = attention_layer(v, W, cache, cfg, return_parts=True)
    note("attention")
    out_sub = x1 + a_out
    out = np.full((cfg.B,) + out_sub.shape[1:], np.nan)
    out[idx] = out_sub
    if return_parts:
        return out, dict(S0=S0, F=F, x1=x1, **{"m_" + k: v for k, v in mparts.items()},
                         **{"a_" + k: v for k, v in aparts.items()})
    return out


# ---------------------------------------- Sec. 3.3 and App. B.1: the whole drafter

def mlp(x: np.ndarray, W) -> np.ndarray:
    """SwiGLU MLP of the drafter layers (hidden size = the target's, App. B.1 "MLP"):
    (SiLU(x W_gate^T) * (x W_up^T)) W_down^T."""
    return (silu(x @ f64(W["W_gate"]).T) * (x @ f64(W["W_up"]).T)) @ f64(W["W_down"]).T


def drafter_forward(layers, shared, x, caches, cfg, requests=None, progress=None):
    """The drafter's block forward (Sec. 3.3; App. B.1).

    S_init = state_init(h_last) is computed once, from the |M| fused target layers, and given
    to the Mamba module of every layer.  Then, from x = e (the block embeddings), for each
    layer W in ``layers``:
        x = x + Mamba(RMSNorm(x) norm1_w; S_init)
        x = x + Attn(RMSNorm(x) norm2_w) over caches[W["cache"]]   (layers with attention)
        x = x + MLP(RMSNorm(x) norm3_w)
    ``shared`` holds W_r and W_dS; ``caches`` is a list of dicts with k_cache and v_cache
    (one per target layer an attention reads); x holds h_last, block_emb, page_table and
    ctx_lens, the page table and lengths being shared by all target layers.  ``requests``
    restricts the work to some rows; the others are NaN.  ``progress``, if given, is called
    with the name of each finished stage.
    """
    note = progress or (lambda stage: None)
    idx = np.arange(cfg.B) if requests is None else np.asarray(requests)
    S0 = None
    if any(W.get("W_in") is not None for W in layers):
        S0, _ = state_init(np.asarray(x["h_last"])[idx], shared["W_r"], shared["W_dS"], cfg.H, cfg.P, cfg.N)
        note("state projection")
    h = f64(np.asarray(x["block_emb"])[idx])
    for li, W in enumerate(layers):
        if W.get("W_in") is not None:   # layers without a Mamba module skip it (block-diffusion backbone)
            h = h + mamba_mixer(rmsnorm(h, f64(W["norm1_w"]), cfg.eps), S0, W, cfg)
        if W.get("cache") is not None:
            c = caches[W["cache"]]
            cache = dict(k_cache=c["k_cache"], v_cache=c["v_cache"], page_table=np.asarray(x["page_table"])[idx],
                         ctx_lens=np.asarray(x["ctx_lens"])[idx])
            h = h + attention_layer(rmsnorm(h, f64(W["norm2_w"]), cfg.eps), W, cache, cfg)
        h = h + mlp(rmsnorm(h, f64(W["norm3_w"]), cfg.eps), W)
        note(f"layer {li}")
    out = np.full((cfg.B,) + h.shape[1:], np.nan)
    out[idx] = h
    return out


def kv_inject(h_new, W_fc, layers, caches, page_table, ctx_lens, cfg):
    """Drafter-side KV injection of a block-diffusion drafter (Sec. 2, "KV injection in block
    drafting"), the cost H-Spec removes: every new input position's fused target hidden state
    f = W_fc h_new (h_new: the |M| selected target layers, concatenated) is projected, for each
    drafter layer, into k = RoPE(RMSNorm_D(W_k f) k_norm_w) and v = W_v f at its position
    ctx_len + i, and appended to that layer's paged drafter cache.

    h_new [B, n, |M| d_model]; layers: dicts with W_k, W_v, k_norm_w; caches: one dict of
    k_cache/v_cache [num_pages, page_size, Hkv, D] per layer.  Returns the updated caches in
    float64 (copies); slots other than the appended ones keep their values.
    """
    f = f64(h_new) @ f64(W_fc).T
    Bsz, n = f.shape[0], f.shape[1]
    L = np.asarray(ctx_lens, dtype=np.int64)
    pos = L[:, None] + np.arange(n)[None, :]
    out = []
    for W, c in zip(layers, caches):
        k = (f @ f64(W["W_k"]).T).reshape(Bsz, n, cfg.Hkv, cfg.D)
        v = (f @ f64(W["W_v"]).T).reshape(Bsz, n, cfg.Hkv, cfg.D)
        k = rope(rmsnorm(k, f64(W["k_norm_w"]), cfg.eps), pos, cfg.rope_theta)
        kc, vc = f64(c["k_cache"]).copy(), f64(c["v_cache"]).copy()
        for b in range(Bsz):
            for i in range(n):
                p = int(pos[b, i])
                slot = int(page_table[b, p // cfg.page_size]) * cfg.page_size + p % cfg.page_size
                kc.reshape(-1, cfg.Hkv, cfg.D)[slot] = k[b, i]
                vc.reshape(-1, cfg.Hkv, cfg.D)[slot] = v[b, i]
        out.append(dict(k_cache=kc, v_cache=vc))
    return out


# ------------------------------------------- Sec. 3.3.3 and App. B.2: the draft head

def draft_head(hidden, W, prev_tok, eps: float, temperature: float = 1.0, gumbel=None, forced=None):
    """Draft tokens from the last hidden states of the block.

    logits_j = RMSNorm(hidden_j) g_f W_lm^T over the pruned vocabulary (App. B.2).
    The Markov head (Sec. 3.3.3; rank R = 256 in App. B.1) adds to position j a
    rank-R term selected by the token t_{j-1} chosen at the position before it:
        l'_j[v] = logits_j[v] + sum_r U_M[v, r] E_M[t_{j-1}, r],
    with t_{-1} = prev_tok, the request's last committed token.  Then
        t_j = argmax_v (l'_j[v] / temperature + gumbel_j[v])   (sampling), or
        t_j = argmax_v l'_j[v]                                  (greedy, gumbel None),
    the lowest index winning a tie.  Gumbel-max: with gumbel_j[v] = -log(-log u), u ~
    U(0, 1) drawn independently, t_j is a draw from softmax(l'_j / temperature).

    ``forced`` [B, k] replaces the chosen t_{j-1} by forced[:, j-1] in the Markov term
    (teacher forcing), so that a second implementation's chain can be checked step by
    step.  Returns (tokens [B, k] int64, corrected logits l' [B, k, V] float64).
    """
    h = f64(hidden)
    B, k = h.shape[0], h.shape[1]
    hn = rmsnorm(h, f64(W["norm_f_w"]), eps)
    logits = hn @ f64(W["W_lm"]).T
    E, U = f64(W["E_M"]), f64(W["U_M"])
    tokens = np.zeros((B, k), dtype=np.int64)
    out = np.empty_like(logits)
    prev = np.asarray(prev_tok, dtype=np.int64)
    for j in range(k):
        lj = logits[:, j, :] + E[prev] @ U.T
        out[:, j, :] = lj
        score = lj if gumbel is None else lj / temperature + f64(gumbel)[:, j, :]
        tokens[:, j] = np.argmax(score, axis=-1)
        prev = tokens[:, j] if forced is None else np.asarray(forced, dtype=np.int64)[:, j]
    return tokens, out


def compare(gpu, ref) -> dict:
    """max |gpu - ref| and ||gpu - ref||_2 / ||ref||_2 over all elements."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    d = g - r
    nr = np.linalg.norm(r)
    return dict(max_abs=float(np.max(np.abs(d))) if d.size else 0.0,
                rel_l2=float(np.linalg.norm(d) / nr) if nr > 0 else float(np.linalg.norm(d)),
                finite=bool(np.all(np.isfinite(g))))
