"""Helpers shared by the GPU parity tests: device upload, oracle comparison, tolerances."""
from __future__ import annotations

import numpy as np

from paper_2609_24197_amd import hspec, inputs as I

# Tolerance of every floating-point output against the float64 oracle (bf16 inputs, fp32
# accumulation): max |gpu - oracle| and relative L2 error.
MAX_ABS = 2e-2
REL_L2 = 5e-3


def dev(d: dict) -> dict:
    """Upload every numpy array of a dict (storage bits preserved); scalars pass through."""
    return {k: hspec.to_device(v) if isinstance(v, np.ndarray) else v for k, v in d.items()}


def host(t) -> np.ndarray:
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def assert_close(gpu, ref, what="", max_abs=MAX_ABS, rel_l2=REL_L2):
    import oracle.hspec_oracle as O
    c = O.compare(gpu, ref)
    print(f"  {what}: max_abs={c['max_abs']:.3e} rel_l2={c['rel_l2']:.3e}", flush=True)
    assert c["finite"], f"{what}: non-finite GPU output"
    assert c["max_abs"] <= max_abs, f"{what}: max_abs {c['max_abs']:.3e} > {max_abs}"
    assert c["rel_l2"] <= rel_l2, f"{what}: rel_l2 {c['rel_l2']:.3e} > {rel_l2}"
    return c


def empty(shape, dtype="f32"):
    import torch
    return torch.empty(shape, dtype=torch.float32 if dtype == "f32" else torch.int32, device="cuda")
