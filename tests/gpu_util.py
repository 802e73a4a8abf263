"""Helpers shared by the GPU tests: stored numpy arrays <-> torch tensors, the parity
metric, and running the oracle on the same stored inputs."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2208_05419_amd import synth

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray, dtype: str):
    import torch
    if dtype == "fp32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(
        torch.bfloat16).cuda()


def to_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def max_rel(g: np.ndarray, r: np.ndarray) -> float:
    """max_i |g_i - r_i| / max_i |r_i| (outputs cross zero, so no elementwise ratio)."""
    den = float(np.max(np.abs(r)))
    return float(np.max(np.abs(g - r))) / (den if den > 0 else 1.0)


def oracle_run(x_st, w_st, wl: synth.Workload, stages: bool = False):
    x = synth.widen(x_st, wl.dtype)
    w = {k: synth.widen(v, wl.dtype) for k, v in w_st.items()}
    return oracle.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam,
                                 wl.keep, stages=stages)


def dev_weights(w_st, dtype):
    return {k: to_dev(v, dtype) for k, v in w_st.items()}


def off_row0_rel(g: np.ndarray, r: np.ndarray) -> float:
    """max_rel over the rows h >= 1 of [B, H, W, C] arrays of the filter's delta.  The biases
    add the same value at every kept mode, and the inverse transform of that constant is a
    spike on row h = 0 which sets max |r| over the whole tensor (tens of times the rest), so
    max_rel over everything barely sees the other rows; this metric is normalised by those
    rows alone.  0 when H = 1."""
    if g.shape[1] < 2:
        return 0.0
    return max_rel(g[:, 1:], r[:, 1:])
