"""Seeded synthetic inputs for the AFNO filter workloads.

This module only draws random numbers and quantises them to the storage dtype; it
holds none of the filter's arithmetic, so both the HIP path's tests and the float64
oracle can take their inputs from it.

The workloads stand in for ERA5 fields (FourCastNet, section "Training and
Inference": 0.25 degree, 720 x 1440 pixels), which are not available: token grids
90 x 180 (8 x 8 patches) and 180 x 360 (4 x 4 patches, section "Model Innovations"),
embedding widths 768 and 1024 split into diagonal blocks.

Draw recipe (all from numpy's PCG64 ``default_rng``):
  * x: standard normal, float64, one stream seeded ``SeedSequence([seed, 1])``;
    the ensemble workload draws a shared base field from that stream and member m's
    perturbation 0.1 * N(0,1) from its own stream ``SeedSequence([seed, 2, m])``, so
    any subset of members can be generated on its own;
  * per-channel scale (heterogeneous-variable workload): U(0.5, 2.0) per channel,
    drawn from the x stream after x, shared over B, H, W;
  * weights: stream ``SeedSequence([seed, 3])``, in the order w1.re, w1.im, b1.re,
    b1.im, w2.re, w2.im, b2.re, b2.im, each N(0, 0.02^2).
Quantisation: float64 -> float32 with round-to-nearest-even; bf16 storage then
rounds that float32 to bf16 with round-to-nearest-even on the bit pattern.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    W: int
    C: int
    num_blocks: int
    dtype: str          # "fp32" or "bf16" storage for x, weights, biases and out
    lam: float
    keep: float
    x_kind: str = "normal"   # "normal" | "channel_scaled" | "ensemble"
    weight_std: float = 0.02
    hidden: int = 0          # hidden units per block; 0: the block size

    @property
    def hs(self) -> int:
        return self.hidden or self.C // self.num_blocks

    @property
    def bs(self) -> int:
        return self.C // self.num_blocks


WORKLOADS = {
    w.name: w for w in [
        Workload("afno16x32_c64_nb4_fp32", 1, 16, 32, 64, 4, "fp32", 0.01, 1.0),
        Workload("afno90x180_c768_nb8_fp32", 1, 90, 180, 768, 8, "fp32", 0.01, 1.0),
        Workload("afno90x180_c768_nb8_bf16_b4", 4, 90, 180, 768, 8, "bf16", 0.01, 1.0,
                 "channel_scaled"),
        Workload("afno180x360_c1024_nb8_bf16", 1, 180, 360, 1024, 8, "bf16", 0.01, 1.0),
        # the paper's own filter shape: 4x4 patches of the 0.25-degree grid, 32 blocks of 32
        Workload("afno180x360_c1024_nb32_bf16", 1, 180, 360, 1024, 32, "bf16", 0.01, 1.0),
        Workload("afno90x180_c768_nb8_bf16_ens100_keep0.5", 100, 90, 180, 768, 8, "bf16", 0.01,
                 0.5, "ensemble"),
        # hidden-size factor 2 (192 hidden units per block of 96)
        Workload("afno90x180_c768_nb8_hs192_bf16_b4", 4, 90, 180, 768, 8, "bf16", 0.01, 1.0,
                 "channel_scaled", hidden=192),
    ]
}

# The workload the headline throughput is quoted on (90 x 180 x 768, bf16, B=4).
HEADLINE = "afno90x180_c768_nb8_bf16_b4"


def f32_to_bf16_bits(a) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even; NaN -> quiet NaN."""
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = a.view(np.uint32)
    r = ((u + (((u >> 16) & 1) + np.uint32(0x7FFF))) >> 16).astype(np.uint16)
    r[np.isnan(a)] = 0x7FC0
    return r


def bf16_bits_to_f32(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def quantize(a, dtype: str) -> np.ndarray:
    """float64 -> stored form: float32 array ("fp32") or uint16 bf16 bit patterns ("bf16")."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    if dtype == "fp32":
        return f
    if dtype == "bf16":
        return f32_to_bf16_bits(f)
    raise ValueError(f"unknown dtype {dtype!r}")


def _x_rng(seed):
    return np.random.default_rng(np.random.SeedSequence([seed, 1]))


def make_x(wl: Workload, seed: int = 0, members=None) -> np.ndarray:
    """Token grid x [B', H, W, C] in stored form.  ``members`` selects batch entries
    (ensemble members) by index; None means all B."""
    H, W, C = wl.H, wl.W, wl.C
    idx = list(range(wl.B)) if members is None else [int(m) for m in members]
    rng = _x_rng(seed)
    if wl.x_kind == "ensemble":
        base = rng.standard_normal((H, W, C))
        out = np.empty((len(idx), H, W, C), dtype=np.float32 if wl.dtype == "fp32" else np.uint16)
        for n, m in enumerate(idx):
            prng = np.random.default_rng(np.random.SeedSequence([seed, 2, m]))
            out[n] = quantize(base + 0.1 * prng.standard_normal((H, W, C)), wl.dtype)
        return out
    x = rng.standard_normal((wl.B, H, W, C))
    if wl.x_kind == "channel_scaled":
        x *= rng.uniform(0.5, 2.0, size=C)
    elif wl.x_kind != "normal":
        raise ValueError(wl.x_kind)
    return quantize(x[idx], wl.dtype)


def make_weights(wl: Workload, seed: int = 0) -> dict:
    """Complex block weights and biases in stored form, (re, im) as the fastest index:
    w1 [nb][bs][hs][2], b1 [nb][hs][2], w2 [nb][hs][bs][2], b2 [nb][bs][2]; hs = wl.hs."""
    nb, bs = wl.num_blocks, wl.bs
    hs = wl.hs
    rng = np.random.default_rng(np.random.SeedSequence([seed, 3]))
    s = wl.weight_std

    def cplx(shape):
        re = s * rng.standard_normal(shape)
        im = s * rng.standard_normal(shape)
        return np.stack([re, im], axis=-1)

    w1 = cplx((nb, bs, hs))
    b1 = cplx((nb, hs))
    w2 = cplx((nb, hs, bs))
    b2 = cplx((nb, bs))
    return {k: quantize(v, wl.dtype) for k, v in (("w1", w1), ("b1", b1), ("w2", w2), ("b2", b2))}


def widen(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Stored form -> float64, exactly."""
    if dtype == "fp32":
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    return bf16_bits_to_f32(stored).astype(np.float64)


def make_block_params(wl: Workload, seed: int = 0, mlp_std: float = 0.02) -> dict:
    """Parameters of one AFNO block around the filter, stored form: LayerNorm gains 1 + 0.1 N,
    shifts 0.1 N over C; the channel MLP wa [C][4C], ba [4C], wb [4C][C], bb [C] with std
    mlp_std (biases 0.1 mlp_std); and the filter's weights (make_weights)."""
    C = wl.C
    rng = np.random.default_rng(np.random.SeedSequence([seed, 5]))
    p = dict(make_weights(wl, seed=seed))
    raw = {
        "ln1_g": 1.0 + 0.1 * rng.standard_normal(C), "ln1_b": 0.1 * rng.standard_normal(C),
        "ln2_g": 1.0 + 0.1 * rng.standard_normal(C), "ln2_b": 0.1 * rng.standard_normal(C),
        "wa": mlp_std * rng.standard_normal((C, 4 * C)), "ba": 0.1 * mlp_std * rng.standard_normal(4 * C),
        "wb": mlp_std * rng.standard_normal((4 * C, C)), "bb": 0.1 * mlp_std * rng.standard_normal(C),
    }
    p.update({k: quantize(v, wl.dtype) for k, v in raw.items()})
    return p
