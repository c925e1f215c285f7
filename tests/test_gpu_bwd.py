"""GPU parity of the fused selective scan's backward pass (through the C ABI)
against the fp64 backward oracle.

Gate: every gradient element within 1e-4 of its magnitude (the oracle's sum
of the absolute values of the terms that make it up), the same rule as the
forward.  Cross-row sums (dA, dB, dC, dDskip, ddelta_bias) are added in a
fixed order, so repeated calls agree bit for bit.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from gate import assert_gate, fp_gate

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sw():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_00601_amd as pkg
    pkg.lib()
    return pkg


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def _bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda").view(
        torch.bfloat16)


def _inputs(B, D, N, L, seed, dtype, opts):
    inp = wl.selective_inputs(B, D, N, L, seed, dtype)
    rng = np.random.Generator(np.random.PCG64(seed + 5))
    ex = {"dy": rng.standard_normal((B, D, L)).astype(np.float32)}
    if "dybf16" in opts:
        ex["dy_bits"] = wl.bf16_round(ex["dy"])
        ex["dy"] = wl.bf16_widen(ex["dy_bits"])
    if "z" in opts:
        z = (rng.standard_normal((B, D, L)) * 2).astype(np.float32)
        if dtype == "bf16":
            ex["z_bits"] = wl.bf16_round(z)
            z = wl.bf16_widen(ex["z_bits"])
        ex["z"] = z
    if "bias" in opts:
        ex["delta_bias"] = rng.uniform(-2.0, 0.0, size=D).astype(np.float32)
    if "h0" in opts:
        ex["h0"] = rng.standard_normal((B, D, N)).astype(np.float32)
    if "dhl" in opts:
        ex["dh_last"] = rng.standard_normal((B, D, N)).astype(np.float32)
    return inp, ex


def _run(sw, inp, ex, dtype, opts, with_dskip=True):
    if dtype == "bf16":
        x, dl = _bf16_dev(inp["x_bf16"]), _bf16_dev(inp["delta_bf16"])
        Bm, Cm = _bf16_dev(inp["Bm_bf16"]), _bf16_dev(inp["Cm_bf16"])
        z = _bf16_dev(ex["z_bits"]) if "z" in ex else None
    else:
        x, dl, Bm, Cm = (_dev(inp[k]) for k in ("x", "delta", "Bm", "Cm"))
        z = _dev(ex["z"]) if "z" in ex else None
    dy = _bf16_dev(ex["dy_bits"]) if "dy_bits" in ex else _dev(ex["dy"])
    g = sw.selective_scan_bwd(
        x, dl, _dev(inp["A"]), Bm, Cm, _dev(inp["Dskip"]) if with_dskip else None, dy,
        _dev(ex["dh_last"]) if "dh_last" in ex else None, z=z,
        delta_bias=_dev(ex["delta_bias"]) if "delta_bias" in ex else None,
        h0=_dev(ex["h0"]) if "h0" in ex else None, delta_softplus="softplus" in opts)
    torch.cuda.synchronize()
    return g


def _ref(inp, ex, opts, rows=None, with_dskip=True):
    return oracle.selective_scan_bwd(
        inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
        inp["Dskip"] if with_dskip else None, ex["dy"], ex.get("dh_last"), z=ex.get("z"),
        delta_bias=ex.get("delta_bias"), h0=ex.get("h0"), delta_softplus="softplus" in opts,
        rows=rows, bounds=True)


def _check_all(g, o, what, keys):
    for k in keys:
        st = fp_gate(g[k].cpu().numpy(), o[k], o["m_" + k])
        assert_gate(st, f"{what} {k}")


# (B, D, N, L): D not a multiple of 16, ragged L, N below 16
_SHAPES = [(2, 37, 16, 203), (1, 16, 16, 64), (3, 5, 5, 17), (1, 20, 1, 9), (2, 33, 8, 1000)]
_OPTS = [(), ("z",), ("bias", "softplus"), ("h0", "dhl"), ("dybf16",),
         ("z", "bias", "softplus", "h0", "dhl")]


@pytest.mark.parametrize("shape", _SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", _OPTS)
def test_bwd_matches_oracle(sw, shape, dtype, opts):
    B, D, N, L = shape
    _say("case bwd", dtype, shape, opts)
    inp, ex = _inputs(B, D, N, L, 800 + B + D + N + L, dtype, opts)
    g = _run(sw, inp, ex, dtype, opts)
    o = _ref(inp, ex, opts)
    keys = ["dx", "ddelta", "dA", "dB", "dC", "dDskip", "dh0"]
    if "z" in opts:
        keys.append("dz")
    if "bias" in opts:
        keys.append("ddelta_bias")
    _check_all(g, o, f"{dtype} {shape} {opts}", keys)


def test_bwd_without_dskip_and_dh0(sw):
    inp, ex = _inputs(2, 19, 16, 77, 901, "f32", ())
    g = _run(sw, inp, ex, "f32", (), with_dskip=False)
    assert "dDskip" not in g
    o = _ref(inp, ex, (), with_dskip=False)
    _check_all(g, o, "no Dskip", ["dx", "ddelta", "dA", "dB", "dC", "dh0"])


def test_bwd_is_deterministic(sw):
    inp, ex = _inputs(2, 70, 16, 300, 902, "bf16", ("z", "bias", "softplus"))
    g1 = _run(sw, inp, ex, "bf16", ("z", "bias", "softplus"))
    g2 = _run(sw, inp, ex, "bf16", ("z", "bias", "softplus"))
    for k in g1:
        assert torch.equal(g1[k], g2[k]), k


def test_bwd_empty_sequence(sw):
    B, D, N = 2, 3, 16
    e = torch.empty((B, D, 0), device="cuda")
    A = torch.randn((D, N), device="cuda")
    Bm = torch.empty((B, 0, N), device="cuda")
    dhl = torch.randn((B, D, N), device="cuda")
    g = sw.selective_scan_bwd(e, e, A, Bm, Bm, torch.randn(D, device="cuda"), e, dhl)
    torch.cuda.synchronize()
    assert torch.equal(g["dh0"], dhl)
    assert torch.count_nonzero(g["dA"]) == 0 and torch.count_nonzero(g["dDskip"]) == 0


def test_bwd_rejects_N_above_64(sw):
    from paper_2606_00601_amd import ScanWeaverError
    x = torch.randn((1, 2, 8), device="cuda")
    with pytest.raises(ScanWeaverError):
        sw.selective_scan_bwd(x, x, torch.randn((2, 65), device="cuda"),
                              torch.randn((1, 8, 65), device="cuda"),
                              torch.randn((1, 8, 65), device="cuda"), None, x)


# N above 16: the states run as several passes of 16
@pytest.mark.parametrize("shape", [(2, 19, 17, 70), (1, 16, 32, 64), (2, 7, 64, 33), (1, 5, 40, 130)])
@pytest.mark.parametrize("opts", [(), ("z", "bias", "softplus", "h0", "dhl")])
def test_bwd_more_than_16_states(sw, shape, opts):
    B, D, N, L = shape
    _say("case bwd N>16", shape, opts)
    inp, ex = _inputs(B, D, N, L, 960 + N + L, "f32", opts)
    g = _run(sw, inp, ex, "f32", opts)
    o = _ref(inp, ex, opts)
    keys = ["dx", "ddelta", "dA", "dB", "dC", "dDskip", "dh0"]
    if "z" in opts:
        keys += ["dz", "ddelta_bias"]
    _check_all(g, o, f"N>16 {shape} {opts}", keys)


def test_bwd_full_size_sampled(sw):
    """The Mamba-130M-like shape (bf16, B=8, D=1536, N=16, L=2048) with the
    Mamba-block options: every row of one batch (its dB and dC are then
    complete), and every batch of a sample of channels (their dA, dDskip and
    ddelta_bias are then complete)."""
    w = wl.workload("selective_bf16_b8_d1536_n16_l2048")
    opts = ("z", "bias", "softplus", "dybf16")
    _say("case bwd full size", w.name, opts)
    inp, ex = _inputs(w.B, w.D, w.N, w.L, 8181, "bf16", opts)
    g = _run(sw, inp, ex, "bf16", opts)
    b0 = 5
    rng = np.random.Generator(np.random.PCG64(82))
    ds_ = np.sort(rng.choice(w.D, 24, replace=False))
    rows_b0 = b0 * w.D + np.arange(w.D)
    rows_d = (np.arange(w.B)[:, None] * w.D + ds_[None, :]).reshape(-1)
    o = _ref(inp, ex, opts, rows=rows_b0)
    for k in ("dx", "ddelta", "dz"):
        got = g[k].reshape(-1, w.L)[torch.as_tensor(rows_b0, device="cuda")].cpu().numpy()
        assert_gate(fp_gate(got, o[k], o["m_" + k]), f"full-size {k}")
    for k in ("dB", "dC"):
        assert_gate(fp_gate(g[k][b0].cpu().numpy(), o[k][b0], o["m_" + k][b0]), f"full-size {k}")
    o2 = _ref(inp, ex, opts, rows=rows_d)
    dA = o2["dA_rows"].reshape(w.B, len(ds_), w.N).sum(0)
    mA = o2["m_dA_rows"].reshape(w.B, len(ds_), w.N).sum(0)
    assert_gate(fp_gate(g["dA"][torch.as_tensor(ds_, device="cuda")].cpu().numpy(), dA, mA),
                "full-size dA")
    for k in ("dDskip", "ddelta_bias"):
        ref = o2[k + "_rows"].reshape(w.B, len(ds_)).sum(0)
        mag = o2["m_" + k + "_rows"].reshape(w.B, len(ds_)).sum(0)
        got = g[k][torch.as_tensor(ds_, device="cuda")].cpu().numpy()
        assert_gate(fp_gate(got, ref, mag), f"full-size {k}")


# ------------------------------------------- checkpoints handed over by the forward

@pytest.mark.parametrize("shape,layout", [((2, 37, 16, 203), "8"), ((2, 21, 16, 512), "16"),
                                          ((1, 9, 5, 96), "8")])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_checkpoints_and_backward_with_them(sw, monkeypatch, shape, layout, dtype):
    """The forward's training mode stores the state before every 8th step and
    the output before the gate; each slot matches the oracle's final state of
    the sequence cut there, the pre-gate output is the ungated forward's y bit
    for bit, and the backward fed with them gives the oracle's gradients,
    bit-identical to the backward that rebuilds them itself."""
    monkeypatch.setenv("SW_SS_LAYOUT", layout)
    # the training forward walks whole rows; so does the ungated forward it is
    # compared with bit for bit (narrow calls would otherwise be segmented)
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")
    B, D, N, L = shape
    opts = ("z", "bias", "softplus", "h0", "dhl")
    _say("case ckpt", dtype, shape, layout)
    inp, ex = _inputs(B, D, N, L, 930 + L, dtype, opts)
    if dtype == "bf16":
        x, dl = _bf16_dev(inp["x_bf16"]), _bf16_dev(inp["delta_bf16"])
        Bm, Cm = _bf16_dev(inp["Bm_bf16"]), _bf16_dev(inp["Cm_bf16"])
        z = _bf16_dev(ex["z_bits"])
    else:
        x, dl, Bm, Cm = (_dev(inp[k]) for k in ("x", "delta", "Bm", "Cm"))
        z = _dev(ex["z"])
    kw = dict(z=z, delta_bias=_dev(ex["delta_bias"]), h0=_dev(ex["h0"]), delta_softplus=True)
    ck = sw.new_ckpt(x, N)
    sp = torch.empty((B, D, L), dtype=torch.float32, device="cuda")
    y, hl = sw.selective_scan_fwd(x, dl, _dev(inp["A"]), Bm, Cm, _dev(inp["Dskip"]), ckpt=ck,
                                  s_pre=sp, **kw)
    ungated = {k: v for k, v in kw.items() if k != "z"}
    y_ungated, _ = sw.selective_scan_fwd(x, dl, _dev(inp["A"]), Bm, Cm, _dev(inp["Dskip"]),
                                         **ungated)
    torch.cuda.synchronize()
    assert torch.equal(sp, y_ungated)
    ckn = ck.cpu().numpy()
    nt8 = (L + 7) // 8
    for k in sorted({0, 1, nt8 // 2, nt8 - 1}):
        if k == 0:
            ref, mag, sens = ex["h0"], np.abs(ex["h0"]), np.zeros_like(ex["h0"])
        else:
            cut = lambda a: np.ascontiguousarray(a[..., :8 * k])  # noqa: E731
            o = oracle.selective_scan(cut(inp["x"]), cut(inp["delta"]), inp["A"],
                                      np.ascontiguousarray(inp["Bm"][:, :8 * k]),
                                      np.ascontiguousarray(inp["Cm"][:, :8 * k]), inp["Dskip"],
                                      bounds=True, z=cut(ex["z"]), delta_bias=ex["delta_bias"],
                                      h0=ex["h0"], delta_softplus=True)
            ref, mag, sens = o["h_last"], o["h_mag"], o["h_sens"]
        assert_gate(fp_gate(ckn[:, :, k, :N], ref, mag, sens), f"ckpt slot {k}")
    dy = _dev(ex["dy"])
    dhl = _dev(ex["dh_last"])
    args = (x, dl, _dev(inp["A"]), Bm, Cm, _dev(inp["Dskip"]), dy, dhl)
    g1 = sw.selective_scan_bwd(*args, ckpt=ck, **kw)
    g0 = sw.selective_scan_bwd(*args, **kw)
    g2 = sw.selective_scan_bwd(*args, ckpt=ck, s_pre=sp, **kw)
    g3 = sw.selective_scan_bwd(*args, s_pre=sp, **kw)
    torch.cuda.synchronize()
    o = _ref(inp, ex, opts)
    _check_all(g1, o, f"bwd with ckpt {dtype} {shape}",
               ["dx", "ddelta", "dA", "dB", "dC", "dDskip", "dz", "ddelta_bias", "dh0"])
    for k in g0:
        assert torch.equal(g0[k], g1[k]), k
        assert torch.equal(g0[k], g2[k]), k
        assert torch.equal(g0[k], g3[k]), k


def test_forward_checkpoints_reject_large_N(sw):
    from paper_2606_00601_amd import ScanWeaverError
    x = torch.randn((1, 2, 8), device="cuda")
    with pytest.raises(ScanWeaverError):
        sw.selective_scan_fwd(x, x, torch.randn((2, 17), device="cuda"),
                              torch.randn((1, 8, 17), device="cuda"),
                              torch.randn((1, 8, 17), device="cuda"), ckpt=sw.new_ckpt(x, 17))


def test_autograd_function_matches_oracle(sw):
    """selective_scan_fn under torch autograd: loss = sum(dy * y) gives the
    oracle's gradients for every differentiable input (fp32, all options)."""
    B, D, N, L = 2, 21, 16, 300
    opts = ("z", "bias", "softplus", "h0")
    inp, ex = _inputs(B, D, N, L, 990, "f32", opts)
    leaves = {k: _dev(inp[k]).requires_grad_() for k in ("x", "delta", "A", "Bm", "Cm", "Dskip")}
    z = _dev(ex["z"]).requires_grad_()
    bias = _dev(ex["delta_bias"]).requires_grad_()
    h0 = _dev(ex["h0"]).requires_grad_()
    y = sw.selective_scan_fn(leaves["x"], leaves["delta"], leaves["A"], leaves["Bm"],
                             leaves["Cm"], leaves["Dskip"], z=z, delta_bias=bias, h0=h0,
                             delta_softplus=True)
    (y * _dev(ex["dy"])).sum().backward()
    torch.cuda.synchronize()
    o = _ref(inp, ex, opts)
    got = {"dx": leaves["x"].grad, "ddelta": leaves["delta"].grad, "dA": leaves["A"].grad,
           "dB": leaves["Bm"].grad, "dC": leaves["Cm"].grad, "dDskip": leaves["Dskip"].grad,
           "dz": z.grad, "ddelta_bias": bias.grad, "dh0": h0.grad}
    for k, v in got.items():
        assert_gate(fp_gate(v.cpu().numpy(), o[k], o["m_" + k]), f"autograd {k}")


def test_autograd_chained_segments_match_one_call(sw):
    """Two segments chained through h0 = the first segment's h_last, under
    autograd with a loss on both y and the final state, give the gradients
    of one call over the whole sequence (the oracle's, with dh_last)."""
    B, D, N, L, L1 = 2, 19, 16, 260, 96
    opts = ("dhl",)
    inp, ex = _inputs(B, D, N, L, 4242, "f32", opts)
    leaves = {k: _dev(inp[k]).requires_grad_() for k in ("x", "delta", "A", "Bm", "Cm", "Dskip")}
    xs, ds = leaves["x"], leaves["delta"]
    y1, h1 = sw.selective_scan_fn(xs[:, :, :L1].contiguous(), ds[:, :, :L1].contiguous(),
                                  leaves["A"], leaves["Bm"][:, :L1].contiguous(),
                                  leaves["Cm"][:, :L1].contiguous(), leaves["Dskip"],
                                  return_last_state=True)
    y2, h2 = sw.selective_scan_fn(xs[:, :, L1:].contiguous(), ds[:, :, L1:].contiguous(),
                                  leaves["A"], leaves["Bm"][:, L1:].contiguous(),
                                  leaves["Cm"][:, L1:].contiguous(), leaves["Dskip"], h0=h1,
                                  return_last_state=True)
    dy = _dev(ex["dy"])
    loss = (y1 * dy[:, :, :L1]).sum() + (y2 * dy[:, :, L1:]).sum() + (h2 * _dev(ex["dh_last"])).sum()
    loss.backward()
    torch.cuda.synchronize()
    o = _ref(inp, ex, opts)
    got = {"dx": xs.grad, "ddelta": ds.grad, "dA": leaves["A"].grad, "dB": leaves["Bm"].grad,
           "dC": leaves["Cm"].grad, "dDskip": leaves["Dskip"].grad}
    for k, v in got.items():
        assert_gate(fp_gate(v.cpu().numpy(), o[k], o["m_" + k]), f"chained autograd {k}")


@pytest.mark.parametrize("shape", [(2, 21, 16, 512), (1, 16, 16, 64), (2, 37, 16, 203)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", [(), ("bias", "softplus", "h0", "dhl")])
def test_backward_without_checkpoints_takes_the_states_walk(sw, monkeypatch, shape, dtype, opts):
    """Without the forward's checkpoints and without a gate, a call the
    16-lane forward layout takes (N = 16, L a multiple of the vector width)
    gets its checkpoints from the forward's walk without y; other calls
    (L = 203) rebuild them in the backward kernel.  Either way the gradients
    are the oracle's and the same bits as with the training forward's
    checkpoints."""
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")  # the training forward walks whole rows
    B, D, N, L = shape
    _say("case bwd states walk", dtype, shape, opts)
    inp, ex = _inputs(B, D, N, L, 970 + L, dtype, opts)
    if dtype == "bf16":
        x, dl = _bf16_dev(inp["x_bf16"]), _bf16_dev(inp["delta_bf16"])
        Bm, Cm = _bf16_dev(inp["Bm_bf16"]), _bf16_dev(inp["Cm_bf16"])
    else:
        x, dl, Bm, Cm = (_dev(inp[k]) for k in ("x", "delta", "Bm", "Cm"))
    kw = {}
    if "bias" in opts:
        kw = dict(delta_bias=_dev(ex["delta_bias"]), h0=_dev(ex["h0"]), delta_softplus=True)
    A, Dk = _dev(inp["A"]), _dev(inp["Dskip"])
    dhl = _dev(ex["dh_last"]) if "dhl" in opts else None
    args = (x, dl, A, Bm, Cm, Dk, _dev(ex["dy"]), dhl)
    g0 = sw.selective_scan_bwd(*args, **kw)
    torch.cuda.synchronize()
    walked = "walk without y" in sw.last_launch()
    assert walked == (L % (8 if dtype == "bf16" else 4) == 0), sw.last_launch()
    ck = sw.new_ckpt(x, N)
    sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, ckpt=ck, **kw)
    g1 = sw.selective_scan_bwd(*args, ckpt=ck, **kw)
    torch.cuda.synchronize()
    assert sw.last_launch().endswith("checkpoints given"), sw.last_launch()
    for k in g0:
        assert torch.equal(g0[k], g1[k]), k
    keys = ["dx", "ddelta", "dA", "dB", "dC", "dDskip", "dh0"]
    if "bias" in opts:
        keys.append("ddelta_bias")
    _check_all(g0, _ref(inp, ex, opts), f"bwd states walk {dtype} {shape} {opts}", keys)
