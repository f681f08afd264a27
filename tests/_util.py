"""Shared helpers of the test suite (no method arithmetic here)."""
import numpy as np
import torch

# Tolerances on the max-abs-normalised error max|gpu - oracle| / max|oracle|:
# fp32 path 1e-5; bf16 inputs with fp32 accumulation and a bf16 output 2e-2.
TOL = {"f32": 1e-5, "bf16": 2e-2}


def tdtype(dt):
    return torch.bfloat16 if dt == "bf16" else torch.float32


def to_np(t) -> np.ndarray:
    """Exact float64 copy of a (device or host) tensor."""
    return t.detach().float().cpu().double().numpy()


def dev(a, dt, device="cuda"):
    """numpy -> device tensor in the path dtype (bf16 rounding is torch's RNE)."""
    return torch.as_tensor(np.ascontiguousarray(a), dtype=torch.float32).to(tdtype(dt)).to(device)


def maxabs_err(g, o) -> float:
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    scale = np.abs(o).max() if o.size else 0.0
    if scale == 0.0:
        return float(np.abs(g).max()) if g.size else 0.0
    return float(np.abs(g - o).max() / scale)
