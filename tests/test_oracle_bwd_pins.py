"""Pins of the backward oracle (CPU).

The paper gives the forward recurrence only; the backward is the chain rule
through it.  The oracle's gradients are pinned to things other than
themselves:
  * central finite differences of the (separately pinned) forward oracle, for
    every input element of a small problem with every option switched on;
  * reverse-mode automatic differentiation (torch, fp64, CPU) of a forward
    written independently here, term by term from Eq. (3) and the Mamba
    discretisation;
  * homogeneity: with a zero initial state y is linear in x, in B, in C and
    in Dskip separately, so sum(dx x), sum(dB B), sum(dC C) and dDskip Dskip
    recover the parts of sum(dy y) that scale with each;
  * the magnitude of every output bounds that output.
"""
import numpy as np
import pytest

import oracle


def _problem(seed, B=2, D=3, N=4, L=9, opts=("z", "bias", "softplus", "h0", "dhl", "D")):
    rng = np.random.Generator(np.random.PCG64(seed))
    f32 = lambda a: np.asarray(a, np.float32)
    p = {
        "x": f32(rng.standard_normal((B, D, L))),
        "delta": f32(rng.uniform(-1.0, 0.5, (B, D, L)) if "softplus" in opts
                     else rng.uniform(0.05, 0.6, (B, D, L))),
        "A": f32(-rng.uniform(0.3, 2.0, (D, N))),
        "Bm": f32(rng.standard_normal((B, L, N))),
        "Cm": f32(rng.standard_normal((B, L, N))),
        "Dskip": f32(rng.standard_normal(D)) if "D" in opts else None,
        "z": f32(rng.standard_normal((B, D, L))) if "z" in opts else None,
        "delta_bias": f32(rng.uniform(-0.5, 0.5, D)) if "bias" in opts else None,
        "h0": f32(rng.standard_normal((B, D, N))) if "h0" in opts else None,
    }
    dy = f32(rng.standard_normal((B, D, L)))
    dhl = f32(rng.standard_normal((B, D, N))) if "dhl" in opts else None
    return p, dy, dhl, "softplus" in opts


def _loss(p, dy, dhl, sp):
    o = oracle.selective_scan(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                              z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                              delta_softplus=sp)
    v = float(np.sum(dy.astype(np.float64) * o["y"]))
    if dhl is not None:
        v += float(np.sum(dhl.astype(np.float64) * o["h_last"]))
    return v


def _grads(p, dy, dhl, sp, bounds=False):
    return oracle.selective_scan_bwd(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                                     dy, dhl, z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                                     delta_softplus=sp, bounds=bounds)


_GRAD_OF = {"x": "dx", "delta": "ddelta", "A": "dA", "Bm": "dB", "Cm": "dC", "Dskip": "dDskip",
            "z": "dz", "delta_bias": "ddelta_bias", "h0": "dh0"}


@pytest.mark.parametrize("opts", [("z", "bias", "softplus", "h0", "dhl", "D"), ("D",), ()])
def test_bwd_matches_central_differences(opts):
    p, dy, dhl, sp = _problem(11 + len(opts), opts=opts)
    g = _grads(p, dy, dhl, sp, bounds=True)
    for name, gname in _GRAD_OF.items():
        if p[name] is None:
            continue
        arr = p[name]
        for idx in np.ndindex(arr.shape):
            v = float(arr[idx])
            eps = 2.0 ** -10 * max(1.0, abs(v))
            hi, lo = arr.copy(), arr.copy()
            hi[idx] = np.float32(v + eps)
            lo[idx] = np.float32(v - eps)
            q = dict(p)
            q[name] = hi
            fp = _loss(q, dy, dhl, sp)
            q[name] = lo
            fm = _loss(q, dy, dhl, sp)
            fd = (fp - fm) / (float(hi[idx]) - float(lo[idx]))
            got = float(g[gname][idx])
            mag = float(g["m_" + gname][idx])
            assert abs(fd - got) <= 2e-5 * mag + 1e-12, (name, idx, fd, got, mag)


def _torch_forward_loss(t, dy, dhl, sp):
    """Eq. (3) with the Mamba discretisation, written out step by step."""
    import torch
    x, dl = t["x"], t["delta"]
    if t["delta_bias"] is not None:
        dl = dl + t["delta_bias"][None, :, None]
    if sp:
        dl = torch.log1p(torch.exp(dl))
    Bsz, D, L = x.shape
    N = t["A"].shape[1]
    h = t["h0"] if t["h0"] is not None else torch.zeros((Bsz, D, N), dtype=torch.float64)
    ys = []
    for s in range(L):
        a = torch.exp(dl[:, :, s, None] * t["A"][None])
        u = (dl[:, :, s] * x[:, :, s])[:, :, None] * t["Bm"][:, None, s, :]
        h = a * h + u
        y = (t["Cm"][:, None, s, :] * h).sum(-1)
        if t["Dskip"] is not None:
            y = y + t["Dskip"][None, :] * x[:, :, s]
        if t["z"] is not None:
            zz = t["z"][:, :, s]
            y = y * (zz * torch.sigmoid(zz))
        ys.append(y)
    y = torch.stack(ys, dim=-1)
    loss = (torch.from_numpy(dy.astype(np.float64)) * y).sum()
    if dhl is not None:
        loss = loss + (torch.from_numpy(dhl.astype(np.float64)) * h).sum()
    return loss


@pytest.mark.parametrize("seed,opts", [(21, ("z", "bias", "softplus", "h0", "dhl", "D")),
                                       (22, ("softplus", "D")), (23, ("h0",))])
def test_bwd_matches_autodiff(seed, opts):
    torch = pytest.importorskip("torch")
    p, dy, dhl, sp = _problem(seed, B=2, D=5, N=3, L=17, opts=opts)
    t = {k: (None if v is None else torch.tensor(v.astype(np.float64), requires_grad=True))
         for k, v in p.items()}
    _torch_forward_loss(t, dy, dhl, sp).backward()
    g = _grads(p, dy, dhl, sp, bounds=True)
    for name, gname in _GRAD_OF.items():
        if t[name] is None:
            continue
        ref = t[name].grad.numpy()
        assert np.all(np.abs(g[gname] - ref) <= 1e-12 * g["m_" + gname] + 1e-300), name


def test_bwd_homogeneity():
    """With h0 = 0 and no gate, y is linear in x, in B, in C and in Dskip
    separately: sum(dx * x) = sum(dy * y), sum(dB * B) = sum(dC * C) =
    sum(dy * (y - Dskip x)) and dDskip . Dskip = sum(dy * Dskip x)."""
    p, dy, _, sp = _problem(31, B=2, D=4, N=5, L=23, opts=("D", "softplus", "bias"))
    o = oracle.selective_scan(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                              delta_bias=p["delta_bias"], delta_softplus=sp)
    g = _grads(p, dy, None, sp)
    dy64 = dy.astype(np.float64)
    total = np.sum(dy64 * o["y"])
    dpart = np.sum(dy64 * p["Dskip"][None, :, None].astype(np.float64) * p["x"])
    assert np.isclose(np.sum(g["dx"] * p["x"]), total, rtol=1e-12, atol=1e-12)
    assert np.isclose(np.sum(g["dB"] * p["Bm"]), total - dpart, rtol=1e-12, atol=1e-12)
    assert np.isclose(np.sum(g["dC"] * p["Cm"]), total - dpart, rtol=1e-12, atol=1e-12)
    assert np.isclose(np.sum(g["dDskip"] * p["Dskip"]), dpart, rtol=1e-12, atol=1e-12)


def test_bwd_magnitudes_bound_the_outputs():
    p, dy, dhl, sp = _problem(41, B=2, D=3, N=6, L=40)
    g = _grads(p, dy, dhl, sp, bounds=True)
    for gname in set(_GRAD_OF.values()):
        assert np.all(np.abs(g[gname]) <= g["m_" + gname] * (1 + 1e-12)), gname


def test_bwd_rows_subset_matches_full():
    p, dy, dhl, sp = _problem(51, B=2, D=4, N=3, L=12)
    full = _grads(p, dy, dhl, sp)
    rows = np.array([1, 4, 6])
    sub = oracle.selective_scan_bwd(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"], dy,
                                    dhl, z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                                    delta_softplus=sp, rows=rows)
    D = 4
    for k in ("dx", "ddelta", "dz", "dh0"):
        ref = full[k].reshape((-1,) + full[k].shape[2:])[rows]
        assert np.array_equal(sub[k], ref), k
    # the per-row shares of dA over all rows of d add up to dA[d]
    allrows = oracle.selective_scan_bwd(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                                        dy, dhl, z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                                        delta_softplus=sp, rows=np.arange(2 * D))
    assert np.allclose(allrows["dA_rows"].reshape(2, D, -1).sum(0), full["dA"], rtol=1e-14)
    assert np.allclose(allrows["dB"], full["dB"], rtol=1e-14, atol=1e-300)
