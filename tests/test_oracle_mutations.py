"""Plant plausible mistakes in a copy of the oracle (on the CPU) and require a pin to catch each.

Every mutation is an exact source substitution; the test first checks that the
snippet exists so a mutation can never silently become a no-op.
"""
import os
import sys
import types

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from oracle_pins import PINS  # noqa: E402

SRC = open(O.__file__).read()

MUTATIONS = {
    "drop_skip_term": ("+ Dskip[None, :, None] * x[:, t]", ""),
    "A_sign": ('A = -np.exp(f64(W["A_log"]))', 'A = np.exp(f64(W["A_log"]))'),
    "dt_not_softplus": ('dt = softplus(dt_raw + f64(W["dt_bias"]))', 'dt = np.exp(dt_raw + f64(W["dt_bias"]))'),
    "no_dt_bias": ('dt = softplus(dt_raw + f64(W["dt_bias"]))', 'dt = softplus(dt_raw)'),
    "swap_B_C": ("Bt = Bm[:, t, grp, :]", "Bt = Cm[:, t, grp, :]"),
    "no_dt_on_input": ("(dt[:, t, :, None] * x[:, t])", "(x[:, t])"),
    "decay_before_not_after": ("a = np.exp(dt[:, t, :] * A[None, :])", "a = np.exp(A[None, :] + 0 * dt[:, t, :])"),
    "conv_off_by_one": ("tau = t - (K - 1) + j", "tau = t - K + j"),
    "conv_flipped_taps": ("out[..., t, :] += w[:, j] * x[..., tau, :]", "out[..., t, :] += w[:, K - 1 - j] * x[..., tau, :]"),
    "gate_without_silu": ("g = y * silu(z)", "g = y * z"),
    "gnorm_no_groups": ("gg = g.reshape(*shp[:-1], G, shp[-1] // G)", "gg = g.reshape(*shp[:-1], 1, shp[-1])"),
    "rmsnorm_sum_not_mean": ("np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)", "np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)"),
    "rmsnorm_no_eps": ("np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)", "np.sqrt(np.mean(x * x, axis=-1, keepdims=True))"),
    "state_reshape_order": ("return S.reshape(h.shape[0], H, P, N), F",
                            "return S.reshape(h.shape[0], H, N, P).transpose(0, 1, 3, 2), F"),
    "state_proj_transposed_Wr": ("F = h @ f64(W_r).T", "F = h @ f64(W_r)"),
    "slot_wrong_offset": ("out[b, i] = int(pt[b, i // page_size]) * page_size + i % page_size",
                          "out[b, i] = int(pt[b, i // page_size]) * page_size + i // page_size"),
    "rope_interleaved": ("x1, x2 = x[..., :half], x[..., half:]", "x1, x2 = x[..., 0::2], x[..., 1::2]"),
    "rope_sign": ("x1 * c - x2 * s, x2 * c + x1 * s", "x1 * c + x2 * s, x2 * c - x1 * s"),
    "rope_positions_from_zero": ("pos = L[:, None] + np.arange(T)[None, :]", "pos = 0 * L[:, None] + np.arange(T)[None, :]"),
    "qk_norm_missing": ('q = rmsnorm(q, f64(W["q_norm_w"]), cfg.eps)', "q = q"),
    "gqa_interleaved": ("heads = np.arange(h * g, (h + 1) * g)", "heads = np.arange(h, Hq, Hkv)"),
    "scale_by_D": ("scale = D ** -0.5 if scale is None else scale", "scale = 1.0 / D if scale is None else scale"),
    "window_off_by_one": ("lo = max(0, pos - window + 1) if window > 0 else 0", "lo = max(0, pos - window) if window > 0 else 0"),
    "causal_flipped": ("nb = j + 1 if block_causal else T", "nb = T if block_causal else j + 1"),
    "block_keys_dropped": ("s = np.concatenate([Kh[lo:L] @ Q.T, kb[b, :nb, h] @ Q.T], axis=0) * scale",
                           "s = np.concatenate([Kh[lo:L] @ Q.T, kb[b, :0, h] @ Q.T], axis=0) * scale"),
    "block_values_shifted": ("w[nc:].T @ vb[b, :nb, h]", "w[nc:].T @ np.roll(vb[b, :nb, h], 1, axis=0)"),
    "softmax_normalised_across_heads": ("w = w / w.sum(axis=0)", "w = w / w.sum()"),
    "missing_mamba_residual": ("x1 = e + m_out", "x1 = m_out"),
    "missing_attn_residual": ("out_sub = x1 + a_out", "out_sub = a_out"),
    "mlp_gate_up_swapped": ('return (silu(x @ f64(W["W_gate"]).T) * (x @ f64(W["W_up"]).T))',
                            'return (silu(x @ f64(W["W_up"]).T) * (x @ f64(W["W_gate"]).T))'),
    "drafter_mlp_no_residual": ("h = h + mlp(rmsnorm(h, f64(W[\"norm3_w\"]), cfg.eps), W)",
                                "h = mlp(rmsnorm(h, f64(W[\"norm3_w\"]), cfg.eps), W)"),
    "drafter_state_zeroed_after_first": ("h = h + mamba_mixer(rmsnorm(h, f64(W[\"norm1_w\"]), cfg.eps), S0, W, cfg)",
                                         "h = h + mamba_mixer(rmsnorm(h, f64(W[\"norm1_w\"]), cfg.eps), S0, W, cfg); S0 = 0 * S0"),
    "drafter_all_layers_cache0": ('c = caches[W["cache"]]', "c = caches[0]"),
    "inject_positions_from_zero": ("pos = L[:, None] + np.arange(n)[None, :]\n    out = []",
                                   "pos = 0 * L[:, None] + np.arange(n)[None, :]\n    out = []"),
    "inject_v_rotated": ("v = (f @ f64(W[\"W_v\"]).T).reshape(Bsz, n, cfg.Hkv, cfg.D)",
                         "v = rope((f @ f64(W[\"W_v\"]).T).reshape(Bsz, n, cfg.Hkv, cfg.D), pos, cfg.rope_theta)"),
    "inject_slot_wrong_page": ("slot = int(page_table[b, p // cfg.page_size]) * cfg.page_size + p % cfg.page_size",
                               "slot = int(page_table[b, p // cfg.page_size]) * cfg.page_size + (p + 1) % cfg.page_size"),
    "head_no_final_norm": ('hn = rmsnorm(h, f64(W["norm_f_w"]), eps)', "hn = h"),
    "markov_prev_never_advances": ("prev = tokens[:, j] if forced is None", "prev = prev if forced is None"),
    "markov_factors_swapped": ("lj = logits[:, j, :] + E[prev] @ U.T", "lj = logits[:, j, :] + U[prev] @ E.T"),
    "gumbel_sign": ("lj / temperature + f64(gumbel)[:, j, :]", "lj / temperature - f64(gumbel)[:, j, :]"),
    "temperature_multiplies": ("lj / temperature + f64(gumbel)[:, j, :]", "lj * temperature + f64(gumbel)[:, j, :]"),
    "conv_no_silu": ('xBC = silu(causal_conv1d(xBC, f64(W["conv_w"]), f64(W["conv_b"])))',
                     'xBC = causal_conv1d(xBC, f64(W["conv_w"]), f64(W["conv_b"]))'),
    "gnorm_no_gain": ("return gg.reshape(shp) * w", "return gg.reshape(shp)"),
    "in_proj_z_x_swapped": ("z = zxbcdt[..., :di]\n    xBC = zxbcdt[..., di:2 * di + 2 * G * N]",
                            "z = zxbcdt[..., di:2 * di]\n    xBC = np.concatenate([zxbcdt[..., :di], "
                            "zxbcdt[..., 2 * di:2 * di + 2 * G * N]], axis=-1)"),
    "xBC_B_C_swapped": ("Bm = xBC[..., di:di + G * N].reshape(Bsz, T, G, N)\n    Cm = xBC[..., di + G * N:].reshape(Bsz, T, G, N)",
                        "Cm = xBC[..., di:di + G * N].reshape(Bsz, T, G, N)\n    Bm = xBC[..., di + G * N:].reshape(Bsz, T, G, N)"),
    "dt_before_xBC": ("dt = zxbcdt[..., 2 * di + 2 * G * N:]", "dt = zxbcdt[..., di:di + H]"),
    "kv_subset_ignored": ("Kh = np.ascontiguousarray(Kc[:, kv_heads[h], :])", "Kh = np.ascontiguousarray(Kc[:, h, :])"),
    "chunk_decay_sign": ("decay = np.exp(lt[:, :, :, None] - lt[:, :, None, :])", "decay = np.exp(lt[:, :, None, :] - lt[:, :, :, None])"),
}


def _mutant(old, new):
    assert SRC.count(old) >= 1, old
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = O.__file__
    exec(compile(SRC.replace(old, new, 1), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_some_pin_catches(name):
    mod = _mutant(*MUTATIONS[name])
    caught = []
    for pin in PINS:
        try:
            pin(mod)
        except Exception:  # AssertionError or a crash both count as caught
            caught.append(pin.__name__)
    assert caught, f"mutation {name} passes every pin"
