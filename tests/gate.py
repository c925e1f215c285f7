"""Acceptance gate for fp32 results against the fp64 oracle.

Reading of "relative tolerance 1e-4" (fp32 states vs the fp64 oracle): the
error of each element is measured against the magnitude of the terms that
make it up, ``mag`` (the sum of absolute values of the terms of the unrolled
form, Eq. (5), as carried by the oracle), not against |ref|, which can cancel
to zero:

    well-conditioned element  :  |got - ref| <= 1e-4 * mag
    ill-conditioned element   :  |got - ref| <= 1e-4 * mag + 4 * u32 * sens

where ``sens`` is the oracle's first-order sensitivity of the element to a
relative perturbation of every a_t, ``u32 = 2^-24``, and an element counts as
ill-conditioned when ``u32 * sens > 1e-5 * mag`` (storing exp(delta*A) in
fp32 alone can then move it by more than a tenth of the tolerance).  The
additive term admits a few ulps of error in each a_t (v_exp_f32 and the
rounding of delta*A*log2e) and nothing else; ill-conditioned elements are
reported separately, never folded into the 1e-4 figure.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24
REL = 1e-4


def fp_gate(got, ref, mag, sens=None, rel=REL):
    """Element-wise gate; returns a dict of statistics with key ``ok``."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    mag = np.asarray(mag, np.float64)
    err = np.abs(got - ref)
    if sens is None:
        ill = np.zeros(err.shape, bool)
        extra = 0.0
    else:
        sens = np.asarray(sens, np.float64)
        ill = U32 * sens > 1e-5 * mag
        extra = np.where(ill, 4 * U32 * sens, 0.0)
    bound = rel * mag + extra
    finite = np.isfinite(got)
    bad = ~finite | (err > bound)
    scaled = np.where(mag > 0, err / np.where(mag > 0, mag, 1.0), np.where(err > 0, np.inf, 0.0))
    well = ~ill
    return {
        "ok": not bool(bad.any()),
        "n": int(err.size),
        "n_bad": int(bad.sum()),
        "n_ill": int(ill.sum()),
        "max_err_over_mag_well": float(scaled[well].max()) if well.any() else 0.0,
        "max_err_over_mag_ill": float(scaled[ill].max()) if ill.any() else 0.0,
        "max_rel_naive": float((err / np.maximum(np.abs(ref), 1e-300)).max()) if err.size else 0.0,
        "first_bad": (tuple(int(i) for i in np.argwhere(bad)[0]) if bad.any() else None),
    }


def rownorm_rel(got, ref):
    """Max over rows (last axis) of ||got - ref||_2 / ||ref||_2 (rows with ref == 0 skipped)."""
    got = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    keep = den > 0
    return float((num[keep] / den[keep]).max()) if keep.any() else 0.0


def assert_gate(stats, what):
    assert stats["ok"], f"{what}: {stats}"
