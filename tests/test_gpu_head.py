"""Draft head on the GPU (hspec_draft_head) against the float64 oracle.

The logits must meet the floating-point bar.  Tokens are argmax decisions taken in fp32 on the GPU
and in fp64 by the oracle, and each position depends on the token chosen before it, so the oracle
is teacher-forced on the GPU's own chain (its Markov term at position j uses the GPU's token of
position j - 1).  Then, position by position: where the oracle's best score leads the runner-up by
more than twice the logit tolerance the tokens must be identical; elsewhere the GPU's token must
score within that margin of the best (several answers are correct inside it).
"""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from gpu_util import MAX_ABS, assert_close, dev, empty, host  # noqa: E402
from paper_2609_24197_amd import hspec, inputs as I  # noqa: E402

pytestmark = pytest.mark.gpu


def _cfg(B, k, d_model):
    return I.StepConfig(name="head", B=B, k=k, d_model=d_model, H=4, P=64, N=16, G=1, chunk=16, Hq=4, Hkv=1, D=64,
                        lengths="fixed:16")


def _run(cfg, V, R, W, x, T=1.0, sample=False, forced=None, with_logits=True):
    d = dev(dict(W, hidden=x["hidden"], prev_tok=x["prev_tok"]))
    g = hspec.to_device(x["gumbel"]) if sample else None
    f = hspec.to_device(forced) if forced is not None else None
    hc = hspec.head_cfg(cfg, V, R, T)
    ws = hspec.workspace(hspec.draft_head_workspace(hc))
    tok = empty((cfg.B, cfg.k), "i32")
    lg = empty((cfg.B, cfg.k, V)) if with_logits else None
    hspec.draft_head(hc, d, d["hidden"], d["prev_tok"], tok, ws, logits=lg, gumbel=g, forced=f)
    return host(tok), (host(lg) if with_logits else None), hspec.read_status(ws)


def _check_tokens(tok, ref_logits, T=1.0, gumbel=None, what=""):
    """Tokens against the teacher-forced oracle scores (see the module docstring)."""
    score = ref_logits / T + gumbel.astype(np.float64) if gumbel is not None else ref_logits
    tol = 2 * MAX_ABS / (T if gumbel is not None else 1.0)
    srt = np.sort(score, axis=-1)
    best, second = srt[..., -1], srt[..., -2]
    mine = np.take_along_axis(score, tok[..., None].astype(np.int64), axis=-1)[..., 0]
    decided = best - second > tol
    ref_tok = np.argmax(score, axis=-1)
    print(f"  {what}: {decided.sum()} of {decided.size} positions decided by more than {tol:.2g}", flush=True)
    assert np.array_equal(tok[decided], ref_tok[decided]), f"{what}: a clearly decided token differs"
    assert np.all(mine >= best - tol), f"{what}: a token scores more than {tol} below the best"


CASES = {
    # ragged vocabulary (1000 = 7 x 128 + 104), rank 64, two request tiles (70 = 64 + 6)
    "v1000_b3": (3, 5, 256, 1000, 64),
    "v1000_b70": (70, 4, 256, 1000, 64),
    "v4096_k16": (4, 16, 512, 4096, 256),
}


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("sample", [False, True], ids=["greedy", "gumbel"])
def test_draft_head(name, sample):
    B, k, dm, V, R = CASES[name]
    cfg = _cfg(B, k, dm)
    print(f"[draft_head] {name} sample={sample}", flush=True)
    W = I.make_head_weights(cfg, seed=11, vocab=V, rank=R)
    x = I.make_head_inputs(cfg, seed=11, vocab=V, sample=sample)
    T = 0.8 if sample else 1.0
    tok, lg, st = _run(cfg, V, R, W, x, T=T, sample=sample)
    assert st == 0
    assert tok.min() >= 0 and tok.max() < V
    _, ref = O.draft_head(x["hidden"], W, x["prev_tok"], cfg.eps, temperature=T,
                          gumbel=x.get("gumbel"), forced=tok)
    assert_close(lg, ref, f"{name} logits")
    _check_tokens(tok, ref, T=T, gumbel=x.get("gumbel"), what=f"{name} tokens")
    # without the logits output the tokens are the same (same kernels, same arithmetic)
    tok2, _, _ = _run(cfg, V, R, W, x, T=T, sample=sample, with_logits=False)
    assert np.array_equal(tok, tok2)


def test_draft_head_teacher_forced():
    """With forced tokens, position j's Markov term uses forced[j-1], not the chosen token."""
    cfg = _cfg(5, 6, 256)
    V, R = 700, 32
    W = I.make_head_weights(cfg, seed=12, vocab=V, rank=R)
    x = I.make_head_inputs(cfg, seed=12, vocab=V)
    forced = np.random.default_rng(5).integers(0, V, size=(cfg.B, cfg.k)).astype(np.int32)
    tok, lg, st = _run(cfg, V, R, W, x, forced=forced)
    assert st == 0
    _, ref = O.draft_head(x["hidden"], W, x["prev_tok"], cfg.eps, forced=forced)
    assert_close(lg, ref, "forced logits")
    _check_tokens(tok, ref, what="forced tokens")


def test_draft_head_bad_token_flagged():
    """A previous token outside [0, V) is read as 0 and raises HSPEC_DEV_BAD_TOKEN."""
    cfg = _cfg(2, 3, 256)
    V, R = 300, 32
    W = I.make_head_weights(cfg, seed=13, vocab=V, rank=R)
    x = I.make_head_inputs(cfg, seed=13, vocab=V)
    x["prev_tok"] = np.array([V + 5, 1], np.int32)
    tok, lg, st = _run(cfg, V, R, W, x)
    assert st & hspec.DEV_BAD_TOKEN
    _, ref = O.draft_head(x["hidden"], W, np.array([0, 1]), cfg.eps, forced=tok)
    assert_close(lg, ref, "bad-token logits")


@pytest.mark.parametrize("sample", [False, True], ids=["greedy", "gumbel"])
def test_draft_head_full_size(sample):
    """8b-serving-b64 shape (B 64, k 16, d_model 4096, V 32000, R 256), in the launch
    configuration the benchmark times; the oracle checks every request."""
    cfg = I.CONFIGS[3]
    V, R = I.HEAD_VOCAB, I.HEAD_RANK
    W = I.make_head_weights(cfg, seed=14)
    x = I.make_head_inputs(cfg, seed=14, sample=sample)
    T = 0.7 if sample else 1.0
    tok, lg, st = _run(cfg, V, R, W, x, T=T, sample=sample)
    assert st == 0
    g = x["gumbel"] if sample else None
    _, ref = O.draft_head(x["hidden"], W, x["prev_tok"], cfg.eps, temperature=T, gumbel=g, forced=tok)
    assert_close(lg, ref, "full-size logits")
    _check_tokens(tok, ref, T=T, gumbel=g, what="full-size tokens")
