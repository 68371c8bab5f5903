"""Seeded synthetic Fastmax inputs, shared by the tests, the bench and the smoke
check.  Holds no Fastmax arithmetic: only random draws and dtype casts.

Recipe (all draws float64 from ``numpy.random.default_rng([2402, 7901, key])``):
  q, k, v ~ i.i.d. N(0, 1), shape [B, H, N, D], drawn in that order;
  optionally a Bernoulli(frac) token mask [B, H, N] whose rows of q, k and v
  are multiplied by ``mask_scale`` (the long-sequence workload uses 5% and x4);
  optionally the upstream gradient dO ~ N(0, 1), drawn last.
Each tensor is then cast to the I/O dtype with round-to-nearest-even (float64
-> float32, and float32 -> bfloat16 for bf16).  The ``*64`` arrays returned
are the exact float64 values of the cast tensors, so a float64 reference
consumes exactly what the device consumes.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_PREFIX = (2402, 7901)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact float64 value of bfloat16 bit patterns."""
    u = np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


@dataclass
class Workload:
    """A named synthetic workload (shape, order, mask flag, dtype)."""
    name: str
    B: int
    H: int
    N: int
    D: int
    p: int
    causal: bool
    dtype: str               # "f32" or "bf16"
    key: int                 # third element of the seed
    mask_frac: float = 0.0
    mask_scale: float = 1.0
    with_dout: bool = False
    extra: dict = field(default_factory=dict)

    def tokens_heads(self) -> int:
        return self.B * self.H * self.N


# The five workloads the paper's claims are exercised on: a small non-causal
# head, the LRA-like D = 32 causal case (p = 1 and p = 2), a GPT-style causal
# layer, a long non-causal sequence with 5% of tokens scaled x4, and a causal
# forward+backward layer.
WORKLOADS = {
    "small_noncausal_f32": Workload("small_noncausal_f32", 1, 1, 256, 16, 2, False, "f32", 1),
    "lra_causal_f32_p1": Workload("lra_causal_f32_p1", 2, 4, 2048, 32, 1, True, "f32", 2),
    "lra_causal_f32_p2": Workload("lra_causal_f32_p2", 2, 4, 2048, 32, 2, True, "f32", 2),
    "gpt_causal_bf16": Workload("gpt_causal_bf16", 4, 16, 8192, 64, 2, True, "bf16", 3),
    "long_noncausal_bf16": Workload("long_noncausal_bf16", 1, 8, 131072, 64, 2, False, "bf16", 4,
                                    mask_frac=0.05, mask_scale=4.0),
    "fwdbwd_causal_bf16": Workload("fwdbwd_causal_bf16", 8, 12, 4096, 64, 2, True, "bf16", 5,
                                   with_dout=True),
    # the same layer shape and inputs without the causal mask (non-causal
    # forward and backward)
    "fwdbwd_noncausal_bf16": Workload("fwdbwd_noncausal_bf16", 8, 12, 4096, 64, 2, False, "bf16",
                                      5, with_dout=True),
    # head dimension 128 (the Llama-2 head size of Sec. 3.1's remark), causal,
    # p = 2: P = 8385 features, served by the float32 MFMA kernels
    "d128_causal_bf16": Workload("d128_causal_bf16", 1, 8, 4096, 128, 2, True, "bf16", 6,
                                 with_dout=True),
}


def _cast(x64: np.ndarray, dtype: str):
    """Returns (device_array, exact_float64_copy)."""
    x32 = x64.astype(np.float32)
    if dtype == "f32":
        return x32, x32.astype(np.float64)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x32)
        return bits, bf16_bits_to_f64(bits)
    raise ValueError(dtype)


def make_inputs(B: int, H: int, N: int, D: int, key: int, dtype: str,
                mask_frac: float = 0.0, mask_scale: float = 1.0,
                with_dout: bool = False, want64: bool = True) -> dict:
    """Draw one seeded input set.

    Returns a dict with q, k, v (and dout) in the device representation
    (float32 arrays, or uint16 bfloat16 bit patterns) and, if ``want64``,
    q64, k64, v64 (and dout64): their exact float64 values.
    """
    rng = np.random.default_rng([SEED_PREFIX[0], SEED_PREFIX[1], int(key)])
    shape = (B, H, N, D)
    raw = {}
    for name in ("q", "k", "v"):
        raw[name] = rng.standard_normal(shape)
    if mask_frac > 0.0:
        mask = rng.random((B, H, N)) < mask_frac
        for name in ("q", "k", "v"):
            raw[name][mask] *= mask_scale
        raw_mask = mask
    else:
        raw_mask = None
    if with_dout:
        raw["dout"] = rng.standard_normal(shape)
    out = {"mask": raw_mask}
    for name, x in raw.items():
        dev, x64 = _cast(x, dtype)
        out[name] = dev
        if want64:
            out[name + "64"] = x64
    return out


def workload_inputs(w: Workload, want64: bool = True, **override) -> dict:
    """Inputs of a named workload; ``override`` may change B, H, N (same recipe)."""
    B = override.get("B", w.B)
    H = override.get("H", w.H)
    N = override.get("N", w.N)
    return make_inputs(B, H, N, w.D, w.key, w.dtype, w.mask_frac, w.mask_scale,
                       w.with_dout, want64)
