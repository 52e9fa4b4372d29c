"""ctypes binding of libhspec.so (the C ABI declared in include/hspec.h).

Argument marshalling only: torch tensors provide device memory and the current HIP stream;
every step of the drafting path runs in the library's kernels.  Importing this module does
not touch the GPU; ``lib()`` loads the shared library and raises if it is missing, so a
missing build can never fall back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import inputs as I

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhspec.so")
_lib = None

BF16, F32 = 0, 1
BLOCK_CAUSAL = 1
ATTN_PRECISE_IO = 2
W_DS_PACKED = 1
MAMBA_PRECISE_IO = 2
DEV_BAD_PAGE, DEV_BAD_CTX_LEN, DEV_BAD_TOKEN, DEV_NONFINITE = 1, 2, 4, 8
STATUS = {0: "HSPEC_OK", 1: "HSPEC_ERR_NULL", 2: "HSPEC_ERR_SHAPE", 3: "HSPEC_ERR_DTYPE",
          4: "HSPEC_ERR_UNSUPPORTED", 5: "HSPEC_ERR_WORKSPACE", 6: "HSPEC_ERR_LAUNCH"}


class MambaCfg(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("B", "k", "d_model", "d_h", "r", "H", "P", "N", "G", "chunk", "conv_w")] + [
        ("flags", C.c_uint), ("dtype", C.c_int), ("eps", C.c_float)]


class MambaW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("W_r", "W_dS", "W_in", "conv_w", "conv_b", "dt_bias", "A_log", "D",
                                           "gnorm_w", "W_out")]


class AttnCfg(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("B", "k", "d_model", "Hq", "Hkv", "D", "page_size", "max_pages",
                                        "num_pages", "window", "split_tokens")] + [
        ("flags", C.c_uint), ("dtype", C.c_int), ("eps", C.c_float), ("scale", C.c_float),
        ("rope_theta", C.c_double), ("Hkv_cache", C.c_int), ("kv_heads", C.POINTER(C.c_int32))]


class AttnW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("W_q", "W_k", "W_v", "W_o", "q_norm_w", "k_norm_w")]


class LayerW(C.Structure):
    _fields_ = [("mamba", C.POINTER(MambaW)), ("norm1_w", C.c_void_p), ("attn", C.POINTER(AttnW)),
                ("norm2_w", C.c_void_p), ("k_cache", C.c_void_p), ("v_cache", C.c_void_p), ("norm3_w", C.c_void_p),
                ("W_gate", C.c_void_p), ("W_up", C.c_void_p), ("W_down", C.c_void_p)]


class HeadCfg(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("B", "k", "d_model", "vocab", "rank")] + [
        ("eps", C.c_float), ("temperature", C.c_float)]


class HeadW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("norm_f_w", "W_lm", "E_M", "U_M")]


class HspecError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


EXPORTS = {
    "hspec_mamba_block_scan": (C.c_int, [C.POINTER(MambaCfg), C.POINTER(MambaW), C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "hspec_mamba_block_scan_workspace": (C.c_size_t, [C.POINTER(MambaCfg)]),
    "hspec_target_kv_block_attn": (C.c_int, [C.POINTER(AttnCfg), C.POINTER(AttnW), C.c_void_p, C.c_void_p,
                                             C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p,
                                             C.c_size_t, C.c_void_p]),
    "hspec_target_kv_block_attn_workspace": (C.c_size_t, [C.POINTER(AttnCfg), C.c_int]),
    "hspec_draft_step": (C.c_int, [C.POINTER(MambaCfg), C.POINTER(MambaW), C.c_void_p, C.POINTER(AttnCfg),
                                   C.POINTER(AttnW), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "hspec_draft_step_workspace": (C.c_size_t, [C.POINTER(MambaCfg), C.POINTER(AttnCfg), C.c_int]),
    "hspec_state_init": (C.c_int, [C.POINTER(MambaCfg), C.POINTER(MambaW), C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_size_t, C.c_void_p]),
    "hspec_state_init_workspace": (C.c_size_t, [C.POINTER(MambaCfg)]),
    "hspec_ssd_scan": (C.c_int, [C.c_int] * 7 + [C.c_int] + [C.c_void_p] * 9 + [C.c_void_p, C.c_size_t, C.c_void_p]),
    "hspec_ssd_scan_workspace": (C.c_size_t, [C.c_int] * 7),
    "hspec_paged_attn": (C.c_int, [C.POINTER(AttnCfg)] + [C.c_void_p] * 7 + [C.c_int, C.c_void_p, C.c_void_p,
                                                                          C.c_size_t, C.c_void_p]),
    "hspec_paged_attn_static": (C.c_int, [C.POINTER(AttnCfg), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                          C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p,
                                          C.c_void_p]),
    "hspec_paged_attn_workspace": (C.c_size_t, [C.POINTER(AttnCfg), C.c_int]),
    "hspec_paged_attn_phase": (C.c_int, [C.POINTER(AttnCfg)] + [C.c_void_p] * 7 + [C.c_int, C.c_void_p, C.c_void_p,
                                                                                C.c_size_t, C.c_uint, C.c_void_p]),
    "hspec_gather_slots": (C.c_int, [C.c_int] * 4 + [C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p,
                                                      C.c_void_p]),
    "hspec_linear": (C.c_int, [C.c_int] * 4 + [C.c_void_p] * 5 + [C.c_size_t, C.c_void_p]),
    "hspec_linear_workspace": (C.c_size_t, [C.c_int] * 4),
    "hspec_drafter_forward": (C.c_int, [C.POINTER(MambaCfg), C.POINTER(AttnCfg), C.c_int, C.c_int, C.c_void_p,
                                        C.c_void_p, C.POINTER(LayerW)] + [C.c_void_p] * 4 + [C.c_int, C.c_void_p,
                                                                                             C.c_void_p, C.c_size_t,
                                                                                             C.c_void_p]),
    "hspec_drafter_forward_workspace": (C.c_size_t, [C.POINTER(MambaCfg), C.POINTER(AttnCfg), C.c_int, C.c_int]),
    "hspec_kv_inject": (C.c_int, [C.POINTER(AttnCfg), C.c_int, C.c_int, C.c_void_p, C.c_void_p] +
                        [C.POINTER(C.c_void_p)] * 5 + [C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "hspec_kv_inject_workspace": (C.c_size_t, [C.POINTER(AttnCfg), C.c_int]),
    "hspec_draft_head": (C.c_int, [C.POINTER(HeadCfg), C.POINTER(HeadW)] + [C.c_void_p] * 7 + [C.c_size_t,
                                                                                          C.c_void_p]),
    "hspec_draft_head_workspace": (C.c_size_t, [C.POINTER(HeadCfg)]),
    "hspec_pack_w_ds_bytes": (C.c_size_t, [C.c_int, C.c_int]),
    "hspec_pack_w_ds": (C.c_int, [C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p]),
    "hspec_read_status": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_void_p]),
    "hspec_status_string": (C.c_char_p, [C.c_int]),
    "hspec_last_error": (C.c_char_p, []),
}


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libhspec.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with paper_2609_24197_amd.build")
        L = C.CDLL(_LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise HspecError(status, lib().hspec_last_error().decode())


# --------------------------------------------------------------------------- torch side

def _torch():
    import torch
    return torch


def stream_ptr():
    return C.c_void_p(_torch().cuda.current_stream().cuda_stream)


def ptr(t):
    """Device pointer of a contiguous CUDA tensor (None -> NULL)."""
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "expected a contiguous device tensor"
    return C.c_void_p(t.data_ptr())


def to_device(a: np.ndarray, dev="cuda"):
    """Storage array (uint16 bf16 bits, float32, int32) -> device tensor of the same bits."""
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


def workspace(nbytes: int, dev="cuda"):
    torch = _torch()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)


def dtype_code(cfg: I.StepConfig) -> int:
    return F32 if cfg.dtype == "f32" else BF16


def mamba_cfg(cfg: I.StepConfig, W: dict | None = None) -> MambaCfg:
    """The Mamba config; W_DS_PACKED is set when W carries "W_dS_packed" (see pack_w_ds), and
    MAMBA_PRECISE_IO with the config's precise_io."""
    flags = W_DS_PACKED if W is not None and W.get("W_dS_packed") is not None else 0
    flags |= MAMBA_PRECISE_IO if cfg.precise_io else 0
    return MambaCfg(cfg.B, cfg.k, cfg.d_model, cfg.d_h, cfg.rank, cfg.H, cfg.P, cfg.N, cfg.G, cfg.chunk,
                    cfg.conv_w, flags, dtype_code(cfg), cfg.eps)


def attn_cfg(cfg: I.StepConfig, max_pages: int, num_pages: int) -> AttnCfg:
    c = AttnCfg(cfg.B, cfg.k, cfg.d_model, cfg.Hq, cfg.Hkv, cfg.D, cfg.page_size, max_pages, num_pages,
                cfg.window, cfg.split_tokens,
                (BLOCK_CAUSAL if cfg.block_causal else 0) | (ATTN_PRECISE_IO if cfg.precise_io else 0), dtype_code(cfg),
                cfg.eps, 0.0, cfg.rope_theta, cfg.Hkv_target, None)
    if cfg.kv_heads:   # partial target-KV-head reuse: the array lives as long as the config
        c._kv_heads = (C.c_int32 * len(cfg.kv_heads))(*cfg.kv_heads)
        c.kv_heads = C.cast(c._kv_heads, C.POINTER(C.c_int32))
    return c


def mamba_w(W: dict) -> MambaW:
    """Weight pointers; a "W_dS_packed" entry replaces W_dS (pair it with mamba_cfg(cfg, W))."""
    names = ("W_r", "W_dS", "W_in", "conv_w", "conv_b", "dt_bias", "A_log", "D", "gnorm_w", "W_out")
    return MambaW(*(ptr(W.get("W_dS_packed", W.get("W_dS")) if n == "W_dS" else W.get(n)) for n in names))


def pack_w_ds(W_dS, d_S: int, r: int):
    """The packed copy of a bf16 W_dS [d_S, r] device tensor (hspec_pack_w_ds), as a new tensor."""
    import torch
    nbytes = lib().hspec_pack_w_ds_bytes(int(d_S), int(r))
    if nbytes == 0:
        raise HspecError(4, "W_dS shape cannot be packed")
    out = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=W_dS.device)
    _check(lib().hspec_pack_w_ds(int(d_S), int(r), ptr(W_dS), ptr(out), stream_ptr()))
    return out


def attn_w(W: dict) -> AttnW:
    return AttnW(*(ptr(W.get(n)) for n in ("W_q", "W_k", "W_v", "W_o", "q_norm_w", "k_norm_w")))


def read_status(ws) -> int:
    v = C.c_int32(0)
    _check(lib().hspec_read_status(ptr(ws), C.byref(v), stream_ptr()))
    return int(v.value)


# ------------------------------------------------------------------------ entry points

def draft_step_workspace(cfg, max_pages, num_pages, max_ctx_len) -> int:
    mc, ac = mamba_cfg(cfg), attn_cfg(cfg, max_pages, num_pages)
    return lib().hspec_draft_step_workspace(C.byref(mc), C.byref(ac), int(max_ctx_len))


def draft_step(cfg, W: dict, X: dict, out, ws, max_ctx_len: int):
    """out [B, k, d_model] fp32 = one drafting step (see hspec_draft_step)."""
    mc = mamba_cfg(cfg, W)
    ac = attn_cfg(cfg, X["page_table"].shape[1], X["k_cache"].shape[0])
    mw, aw = mamba_w(W), attn_w(W)
    _check(lib().hspec_draft_step(C.byref(mc), C.byref(mw), ptr(W["norm1_w"]), C.byref(ac), C.byref(aw),
                                  ptr(W["norm2_w"]), ptr(X["h_last"]), ptr(X["block_emb"]), ptr(X["k_cache"]),
                                  ptr(X["v_cache"]), ptr(X["page_table"]), ptr(X["ctx_lens"]), int(max_ctx_len),
                                  ptr(out), ptr(ws), ws.numel(), stream_ptr()))


def mamba_block_scan_workspace(cfg) -> int:
    mc = mamba_cfg(cfg)
    return lib().hspec_mamba_block_scan_workspace(C.byref(mc))


def mamba_block_scan(cfg, W, h_last, u, out, ws, S_final=None):
    mc, mw = mamba_cfg(cfg, W), mamba_w(W)
    _check(lib().hspec_mamba_block_scan(C.byref(mc), C.byref(mw), ptr(h_last), ptr(u), ptr(out), ptr(S_final),
                                        ptr(ws), ws.numel(), stream_ptr()))


def target_kv_block_attn_workspace(cfg, max_pages, num_pages, max_ctx_len) -> int:
    ac = attn_cfg(cfg, max_pages, num_pages)
    return lib().hspec_target_kv_block_attn_workspace(C.byref(ac), int(max_ctx_len))


def target_kv_block_attn(cfg, W, x, X, out, ws, max_ctx_len):
    ac = attn_cfg(cfg, X["page_table"].shape[1], X["k_cache"].shape[0])
    aw = attn_w(W)
    _check(lib().hspec_target_kv_block_attn(C.byref(ac), C.byref(aw), ptr(x), ptr(X["k_cache"]), ptr(X["v_cache"]),
                                            ptr(X["page_table"]), ptr(X["ctx_lens"]), int(max_ctx_len), ptr(out),
                                            ptr(ws), ws.numel(), stream_ptr()))


def state_init_workspace(cfg) -> int:
    mc = mamba_cfg(cfg)
    return lib().hspec_state_init_workspace(C.byref(mc))


def state_init(cfg, W, h_last, S0, ws):
    mc, mw = mamba_cfg(cfg, W), mamba_w(W)
    _check(lib().hspec_state_init(C.byref(mc), C.byref(mw), ptr(h_last), ptr(S0), ptr(ws), ws.numel(),
                                  stream_ptr()))


def ssd_scan_workspace(B, T, H, P, N, G, dtype) -> int:
    return lib().hspec_ssd_scan_workspace(B, T, H, P, N, G, dtype)


def ssd_scan(B, T, H, P, N, G, chunk, dtype, x, dt, A, Bm, Cm, Dskip, S0, y, S_final, ws):
    _check(lib().hspec_ssd_scan(B, T, H, P, N, G, chunk, dtype, ptr(x), ptr(dt), ptr(A), ptr(Bm), ptr(Cm),
                                ptr(Dskip), ptr(S0), ptr(y), ptr(S_final), ptr(ws), ws.numel(), stream_ptr()))


def paged_attn_workspace(cfg, max_pages, num_pages, max_ctx_len) -> int:
    ac = attn_cfg(cfg, max_pages, num_pages)
    return lib().hspec_paged_attn_workspace(C.byref(ac), int(max_ctx_len))


PHASE_WORKLIST, PHASE_SWEEP, PHASE_REDUCE = 1, 2, 4


def paged_attn(cfg, X, o, ws, max_ctx_len, acfg: AttnCfg | None = None, phases: int | None = None):
    """All of the attention core, or (phases: OR of PHASE_*) some of its launches in order."""
    ac = acfg or attn_cfg(cfg, X["page_table"].shape[1], X["k_cache"].shape[0])
    args = (C.byref(ac), ptr(X["q"]), ptr(X["k_blk"]), ptr(X["v_blk"]), ptr(X["k_cache"]), ptr(X["v_cache"]),
            ptr(X["page_table"]), ptr(X["ctx_lens"]), int(max_ctx_len), ptr(o), ptr(ws), ws.numel())
    if phases is None:
        _check(lib().hspec_paged_attn(*args, stream_ptr()))
    else:
        _check(lib().hspec_paged_attn_phase(*args, int(phases), stream_ptr()))


STATIC_WS_BYTES = 64 << 20   # HSPEC_STATIC_WS_BYTES


def paged_attn_static(cfg, X, o, max_ctx_len, status=None, acfg: AttnCfg | None = None):
    """The attention core on the library's fixed device array (no workspace argument)."""
    ac = acfg or attn_cfg(cfg, X["page_table"].shape[1], X["k_cache"].shape[0])
    _check(lib().hspec_paged_attn_static(C.byref(ac), ptr(X["q"]), ptr(X["k_blk"]), ptr(X["v_blk"]),
                                         ptr(X["k_cache"]), ptr(X["v_cache"]), ptr(X["page_table"]),
                                         ptr(X["ctx_lens"]), int(max_ctx_len), ptr(o), ptr(status), stream_ptr()))


def gather_slots(page_table, ctx_lens, page_size, num_pages, max_ctx_len, slots, status=None):
    B, max_pages = page_table.shape
    _check(lib().hspec_gather_slots(B, max_pages, page_size, num_pages, ptr(page_table), ptr(ctx_lens),
                                    int(max_ctx_len), ptr(slots), ptr(status), stream_ptr()))


def linear_workspace(dtype, M, N, K) -> int:
    return lib().hspec_linear_workspace(dtype, M, N, K)


def linear(dtype, A, W, C_out, ws, R=None):
    M, K = A.shape
    N = W.shape[0]
    _check(lib().hspec_linear(dtype, M, N, K, ptr(A), ptr(W), ptr(R), ptr(C_out), ptr(ws), ws.numel(),
                              stream_ptr()))


def head_cfg(cfg, vocab: int, rank: int, temperature: float = 1.0) -> HeadCfg:
    return HeadCfg(cfg.B, cfg.k, cfg.d_model, int(vocab), int(rank), cfg.eps, float(temperature))


def draft_head_workspace(hc: HeadCfg) -> int:
    return lib().hspec_draft_head_workspace(C.byref(hc))


def draft_head(hc: HeadCfg, W: dict, hidden, prev_tok, tokens, ws, logits=None, gumbel=None, forced=None):
    """tokens [B, k] int32 (and the corrected logits [B, k, V] if given) = hspec_draft_head."""
    hw = HeadW(*(ptr(W[n]) for n in ("norm_f_w", "W_lm", "E_M", "U_M")))
    _check(lib().hspec_draft_head(C.byref(hc), C.byref(hw), ptr(hidden), ptr(prev_tok), ptr(gumbel), ptr(forced),
                                  ptr(tokens), ptr(logits), ptr(ws), ws.numel(), stream_ptr()))


def drafter_forward_workspace(cfg, max_pages, num_pages, max_ctx_len) -> int:
    mc, ac = mamba_cfg(cfg), attn_cfg(cfg, max_pages, num_pages)
    return lib().hspec_drafter_forward_workspace(C.byref(mc), C.byref(ac), cfg.d_ff, int(max_ctx_len))


def drafter_forward(cfg, shared: dict, layers: list, X: dict, out, ws, max_ctx_len: int):
    """out [B, k, d_model] fp32 = the whole drafter over the block (hspec_drafter_forward).
    ``shared``: W_r, W_dS (or W_dS_packed); ``layers``: per-layer weight dicts of device tensors
    with "cache" = index into X["caches"] (None: no attention)."""
    mc = mamba_cfg(cfg, shared)
    ac = attn_cfg(cfg, X["page_table"].shape[1], X["caches"][0]["k_cache"].shape[0])
    keep = []
    arr = (LayerW * len(layers))()
    for i, W in enumerate(layers):
        mw = mamba_w(W) if W.get("W_in") is not None else None
        keep.append(mw)
        aw = None
        c = None
        if W.get("cache") is not None:
            aw = attn_w(W)
            keep.append(aw)
            c = X["caches"][W["cache"]]
        arr[i] = LayerW(C.pointer(mw) if mw is not None else None, ptr(W.get("norm1_w")),
                        C.pointer(aw) if aw is not None else None,
                        ptr(W.get("norm2_w")) if aw is not None else None, ptr(c["k_cache"]) if c else None,
                        ptr(c["v_cache"]) if c else None, ptr(W["norm3_w"]), ptr(W["W_gate"]), ptr(W["W_up"]),
                        ptr(W["W_down"]))
    W_dS = shared.get("W_dS_packed", shared.get("W_dS"))
    if "W_r" not in shared:
        shared = dict(shared, W_r=None)
    _check(lib().hspec_drafter_forward(C.byref(mc), C.byref(ac), cfg.d_ff, len(layers), ptr(shared["W_r"]), ptr(W_dS),
                                       arr, ptr(X.get("h_last")), ptr(X["block_emb"]), ptr(X["page_table"]),
                                       ptr(X["ctx_lens"]), int(max_ctx_len), ptr(out), ptr(ws), ws.numel(),
                                       stream_ptr()))


def kv_inject_workspace(cfg, max_pages, num_pages) -> int:
    ac = attn_cfg(cfg, max_pages, num_pages)
    return lib().hspec_kv_inject_workspace(C.byref(ac), cfg.d_h)


def kv_inject(cfg, IW: dict, h_new, caches: list, page_table, ctx_lens, ws):
    """Drafter-side KV injection (hspec_kv_inject): appends cfg.k new positions per request to
    each layer's cache in ``caches`` (dicts of k_cache/v_cache device tensors, in place)."""
    n = len(IW["layers"])
    ac = attn_cfg(cfg, page_table.shape[1], caches[0]["k_cache"].shape[0])
    arr = lambda xs: (C.c_void_p * n)(*[x.data_ptr() for x in xs])  # noqa: E731
    L = IW["layers"]
    _check(lib().hspec_kv_inject(C.byref(ac), cfg.d_h, n, ptr(h_new), ptr(IW["W_fc"]), arr([w["W_k"] for w in L]),
                                 arr([w["W_v"] for w in L]), arr([w["k_norm_w"] for w in L]),
                                 arr([c["k_cache"] for c in caches]), arr([c["v_cache"] for c in caches]),
                                 ptr(page_table), ptr(ctx_lens), ptr(ws), ws.numel(), stream_ptr()))
