"""Algorithmic byte and flop counts of the drafting step (what the method must move).

Weights are read once per step, the target K/V once per step; nothing counts
re-reads.  Used by the benchmark to turn measured kernel times into achieved
GB/s and TFLOP/s.
"""
from __future__ import annotations

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak, TFLOP/s


def kv_bytes_per_token(Hkv: int, D: int, elem_bytes: int) -> int:
    """K plus V of one token in one layer (Table 1 accounting: bf16, all KV heads)."""
    return 2 * Hkv * D * elem_bytes


def visible_ctx(cfg, L: int) -> int:
    """Cache positions at least one block query sees: all L, or the last window - 1 under a
    sliding window (the query at L + j sees positions p > L + j - window)."""
    w = getattr(cfg, "window", 0)
    return min(int(L), w - 1) if w > 0 else int(L)


def sweep_bytes(cfg, ctx_lens, elem_bytes: int = 2) -> int:
    """Algorithmic bytes of the target-KV attention (sweep and split reduction together).

    Per visible context token: K and V rows of every KV head the drafter reads (the reused
    subset under partial target-KV-head reuse).  Per block position:
    its query heads, the block K/V, and the fp32 output row.  Split partials are not
    algorithmic bytes.
    """
    ctx = sum(visible_ctx(cfg, L) for L in ctx_lens)
    per_tok = kv_bytes_per_token(cfg.Hkv, cfg.D, elem_bytes)
    block = cfg.B * cfg.k * ((cfg.Hq + 2 * cfg.Hkv) * cfg.D * elem_bytes + cfg.Hq * cfg.D * 4)
    return ctx * per_tok + block


def sweep_flops(cfg, ctx_lens) -> int:
    """QK^T and PV over every key a query sees: 4 * D flops per (query head, key)."""
    w, causal = getattr(cfg, "window", 0), getattr(cfg, "block_causal", False)
    keys = 0
    for L in ctx_lens:
        for j in range(cfg.k):
            keys += (min(int(L), w - 1 - j) if w > 0 else int(L)) + (j + 1 if causal else cfg.k)
    return 4 * cfg.D * cfg.Hq * keys


def state_proj_bytes(cfg, elem_bytes: int = 2, s0_bytes: int = 2) -> int:
    """Proj_dS: W_dS once, F in, S0 out."""
    return cfg.d_S * cfg.rank * elem_bytes + cfg.B * cfg.rank * 4 + cfg.B * cfg.d_S * s0_bytes


def state_proj_flops(cfg) -> int:
    return 2 * cfg.B * cfg.d_S * cfg.rank


def scan_bytes(cfg, elem_bytes: int = 2) -> int:
    """SSD scan: S0, x, dt, B, C in; y out (fp32)."""
    B, T = cfg.B, cfg.k
    return (B * cfg.d_S * elem_bytes + B * T * cfg.d_inner * elem_bytes + B * T * cfg.H * 4
            + 2 * B * T * cfg.G * cfg.N * elem_bytes + B * T * cfg.d_inner * 4)


def weight_bytes(cfg, elem_bytes: int = 2) -> int:
    """All drafter weights read by one step."""
    dm = cfg.d_model
    n = (cfg.rank * cfg.d_h + cfg.d_S * cfg.rank + cfg.d_in_proj * dm + cfg.conv_dim * (cfg.conv_w + 1)
         + dm * cfg.d_inner + (cfg.Hq + 2 * cfg.Hkv) * cfg.D * dm + dm * cfg.Hq * cfg.D)
    return n * elem_bytes


def step_bytes(cfg, ctx_lens, elem_bytes: int = 2) -> int:
    """Whole step with S0 kept on chip: weights + target KV + block activations in and out."""
    act = cfg.B * cfg.d_h * elem_bytes + cfg.B * cfg.k * cfg.d_model * (elem_bytes + 4)
    ctx = sum(visible_ctx(cfg, L) for L in ctx_lens)
    return weight_bytes(cfg, elem_bytes) + ctx * kv_bytes_per_token(cfg.Hkv, cfg.D, elem_bytes) + act


def step_flops(cfg, ctx_lens) -> int:
    M = cfg.B * cfg.k
    dm = cfg.d_model
    gemm = 2 * (cfg.B * cfg.rank * cfg.d_h + M * cfg.d_in_proj * dm + M * dm * cfg.d_inner
                + M * (cfg.Hq + 2 * cfg.Hkv) * cfg.D * dm + M * dm * cfg.Hq * cfg.D)
    return gemm + state_proj_flops(cfg) + sweep_flops(cfg, ctx_lens)
