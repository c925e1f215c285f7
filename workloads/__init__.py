"""Seeded synthetic inputs for the affine scan and the fused selective scan.

This module only draws random numbers and stores them in the dtypes the
kernels read.  It holds none of the method's arithmetic; both the oracle and
the HIP path consume exactly the arrays returned here.

Recipe (numpy ``Generator(PCG64(seed))``, every draw in fp64 and in the order
listed, then rounded to the storage dtype with round-to-nearest-even):

* bare affine scan, fp32: ``a ~ U[0.9, 1.0)`` (after rounding to fp32, values
  that reach 1.0 are clamped to the largest fp32 below 1), ``bx ~ N(0, 1)``,
  ``h0 = 0`` unless asked for (then ``h0 ~ N(0, 1)``).  Shape (B, D, L).
* bare affine scan, int32 wraparound: ``a, bx`` uniform over all int32 values;
  variant ``odd`` forces every ``a`` odd (every prefix product is then a unit of
  Z/2^32, so a lost carry anywhere changes the result); variant ``h0`` adds a
  uniform int32 initial state.
* fused selective scan ("Mamba-shaped"): ``x ~ N(0,1)`` (B,D,L);
  ``delta = softplus(s * N(0,1) + m)`` (B,D,L); ``A = -exp(U[ln lo, ln hi])``
  (D,N); ``Bm, Cm ~ N(0,1)`` (B,L,N); ``Dskip ~ N(0,1)`` (D,).  The standard
  recipe uses ``s=0.5, m=-4, lo=1, hi=16``; the stress recipe ``s=2, m=0,
  lo=0.01, hi=64``, which drives exp(delta A) from underflow to within a few
  fp32 ulps of one.  With ``dtype="bf16"`` the arrays x, delta, Bm, Cm are
  stored as bf16 (A and Dskip stay fp32); the fp32 values returned beside
  the bf16 bits are the exact widenings of those bits.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "WORKLOADS", "Workload", "affine_inputs", "affine_inputs_i32", "selective_inputs",
    "bf16_round", "bf16_widen", "sha256", "workload",
]


def sha256(arr) -> str:
    """Hex digest of an array's bytes (C order)."""
    return hashlib.sha256(np.ascontiguousarray(arr).tobytes()).hexdigest()


def bf16_round(v) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns the uint16 bits."""
    f = np.ascontiguousarray(v, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    rounded = (bits + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return rounded.astype(np.uint16)


def bf16_widen(bits) -> np.ndarray:
    """Exact fp32 value of bf16 bit patterns."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _softplus(v: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, v)


def affine_inputs(B: int, D: int, L: int, seed: int, with_h0: bool = False) -> dict:
    """fp32 inputs of the bare affine scan; see the module docstring."""
    rng = np.random.Generator(np.random.PCG64(seed))
    a = rng.uniform(0.9, 1.0, size=(B, D, L)).astype(np.float32)
    below_one = np.nextafter(np.float32(1.0), np.float32(0.0))
    np.minimum(a, below_one, out=a)
    bx = rng.standard_normal(size=(B, D, L)).astype(np.float32)
    h0 = rng.standard_normal(size=(B, D)).astype(np.float32) if with_h0 else None
    return {"a": a, "bx": bx, "h0": h0}


def affine_inputs_i32(B: int, D: int, L: int, seed: int, variant: str = "uniform") -> dict:
    """int32 wraparound inputs: variant in {"uniform", "odd", "h0"}."""
    if variant not in ("uniform", "odd", "h0"):
        raise ValueError(variant)
    rng = np.random.Generator(np.random.PCG64(seed))
    lo, hi = -(2 ** 31), 2 ** 31
    a = rng.integers(lo, hi, size=(B, D, L), dtype=np.int64).astype(np.int32)
    bx = rng.integers(lo, hi, size=(B, D, L), dtype=np.int64).astype(np.int32)
    if variant == "odd":
        a |= np.int32(1)
    h0 = None
    if variant == "h0":
        h0 = rng.integers(lo, hi, size=(B, D), dtype=np.int64).astype(np.int32)
    return {"a": a, "bx": bx, "h0": h0}


def selective_inputs(B: int, D: int, N: int, L: int, seed: int, dtype: str = "f32",
                     stress: bool = False, growth: bool = False) -> dict:
    """Inputs of the fused selective scan; see the module docstring.

    Returns fp32 arrays ``x, delta, A, Bm, Cm, Dskip`` (the values both sides
    use) and, for ``dtype="bf16"``, the bf16 bits ``x_bf16, delta_bf16,
    Bm_bf16, Cm_bf16`` the kernel reads.

    ``growth=True`` (with the stress recipe) draws A positive instead,
    ``A = +exp(U[ln 1e-5, ln 1e-3])``, so that exp(delta*A) is slightly above
    one and the states grow: the regime in which the exponential
    parameterisation amplifies rounding (reported only, not a gated workload).
    """
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    s, m, lo, hi = (2.0, 0.0, 0.01, 64.0) if stress else (0.5, -4.0, 1.0, 16.0)
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal(size=(B, D, L)).astype(np.float32)
    z = rng.standard_normal(size=(B, D, L))
    z *= s
    z += m
    delta = _softplus(z).astype(np.float32)
    del z
    if growth:
        lo, hi = 1e-5, 1e-3
    A = np.exp(rng.uniform(np.log(lo), np.log(hi), size=(D, N)))
    A = (A if growth else -A).astype(np.float32)
    Bm = rng.standard_normal(size=(B, L, N)).astype(np.float32)
    Cm = rng.standard_normal(size=(B, L, N)).astype(np.float32)
    Dskip = rng.standard_normal(size=(D,)).astype(np.float32)
    out = {"x": x, "delta": delta, "A": A, "Bm": Bm, "Cm": Cm, "Dskip": Dskip}
    if dtype == "bf16":
        for k in ("x", "delta", "Bm", "Cm"):
            bits = bf16_round(out[k])
            out[k + "_bf16"] = bits
            out[k] = bf16_widen(bits)
    return out


@dataclass(frozen=True)
class Workload:
    """One named synthetic workload: its path, shape, dtype and seed."""
    name: str
    path: str  # "affine" or "selective"
    B: int
    D: int
    L: int
    N: int = 1
    dtype: str = "f32"
    seed: int = 0
    stress: bool = False
    note: str = field(default="", compare=False)

    @property
    def elems(self) -> int:
        """B*L*D*N (N = 1 for the bare scan)."""
        return self.B * self.D * self.L * self.N

    def inputs(self) -> dict:
        if self.path == "affine":
            return affine_inputs(self.B, self.D, self.L, self.seed)
        return selective_inputs(self.B, self.D, self.N, self.L, self.seed, self.dtype,
                                self.stress)


WORKLOADS = {
    w.name: w for w in [
        Workload("affine_f32_b1_d64_l1024", "affine", 1, 64, 1024, 1, "f32", 1,
                 note="bare affine scan, fp32 (int32 variants use seeds 11, 12, 13)"),
        Workload("affine_f32_b1_d5120_l65536", "affine", 1, 5120, 65536, 1, "f32", 6,
                 note="bare affine scan at the long-sequence shape (bandwidth figure)"),
        Workload("affine_f32_b1_d64_l65536", "affine", 1, 64, 65536, 1, "f32", 7,
                 note="bare affine scan, few rows and a long sequence (schedule ablation)"),
        Workload("affine_f32_b8_d1536_l2048", "affine", 8, 1536, 2048, 1, "f32", 8,
                 note="bare affine scan at the Mamba-130M-like (b,d,t) shape (schedule ablation)"),
        Workload("selective_f32_b2_d256_n16_l512", "selective", 2, 256, 512, 16, "f32", 2,
                 note="Mamba-style selective scan, fp32"),
        Workload("selective_bf16_b8_d1536_n16_l2048", "selective", 8, 1536, 2048, 16, "bf16",
                 3, note="Mamba-130M-like shape, bf16 x/delta/B/C, fp32 state and y"),
        Workload("selective_f32_b1_d5120_n16_l65536", "selective", 1, 5120, 65536, 16, "f32",
                 4, note="long sequence, fp32"),
        Workload("selective_f32_b4_d2048_n16_l8192_stress", "selective", 4, 2048, 8192, 16,
                 "f32", 5, stress=True, note="numerical stress, fp32"),
    ]
}

INT_SEEDS = {"uniform": 11, "odd": 12, "h0": 13}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
