"""The benchmark's algorithmic counts of the KV sweep against a brute-force count of the keys
each block query sees (Sec. 3.3.2: target prefix plus the block; App. B.2: sliding window)."""
import itertools

import pytest

from paper_2609_24197_amd import inputs as I
from paper_2609_24197_amd import roofline as RL


def _seen(L, k, window, causal):
    """(query j, key) pairs by the mask's definition: cache position p is visible to the query
    at position L + j unless the window hides it; block key s unless causality hides it."""
    pairs, cache_any = 0, set()
    for j in range(k):
        for p in range(L):
            if window <= 0 or (L + j) - p < window:
                pairs += 1
                cache_any.add(p)
        pairs += sum(1 for s in range(k) if not causal or s <= j)
    return pairs, len(cache_any)


@pytest.mark.parametrize("window,causal", list(itertools.product([0, 5, 16, 40], [False, True])))
def test_sweep_counts_match_brute_force(window, causal):
    cfg = I.StepConfig(name="t", B=5, k=5, d_model=64, H=2, P=16, N=16, G=1, chunk=4, Hq=4, Hkv=2, D=64,
                       lengths="list:0,1,4,37,90", window=window, block_causal=causal)
    lens = [0, 1, 4, 37, 90]
    pairs = sum(_seen(L, cfg.k, window, causal)[0] for L in lens)
    assert RL.sweep_flops(cfg, lens) == 4 * cfg.D * cfg.Hq * pairs
    ctx = sum(_seen(L, cfg.k, window, causal)[1] for L in lens)
    block = cfg.B * cfg.k * ((cfg.Hq + 2 * cfg.Hkv) * cfg.D * 2 + cfg.Hq * cfg.D * 4)
    assert RL.sweep_bytes(cfg, lens) == ctx * RL.kv_bytes_per_token(cfg.Hkv, cfg.D, 2) + block
