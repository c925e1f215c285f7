"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Integer results must be bit-exact; fp32 results pass the gate of gate.py.
Small cases are compared element by element over whole outputs, at sizes that
span several workgroup tiles and a ragged tail; the full-size synthetic
workloads are run at their real shapes in the launch configuration the bench
uses and compared on seeded samples of rows that the oracle evaluates one by
one.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from gate import assert_gate, fp_gate, rownorm_rel

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
    pkg.lib()  # raises if the HIP library is missing: no fallback
    return pkg


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda").view(
        torch.bfloat16)


# ------------------------------------------------------------ bare affine scan

def _affine_check(sw, a, bx, h0=None):
    h = sw.affine_scan(dev(a), dev(bx), None if h0 is None else dev(h0)).cpu().numpy()
    ref, mag, sens = oracle.affine_scan(a, bx, h0, bounds=True)
    return fp_gate(h, ref, mag, sens), h, ref


def test_affine_f32_workload(sw):
    w = wl.workload("affine_f32_b1_d64_l1024")
    _say("case", w.name)
    inp = w.inputs()
    st, h, ref = _affine_check(sw, inp["a"], inp["bx"])
    assert_gate(st, w.name)
    assert st["n_ill"] == 0
    assert rownorm_rel(h, ref) <= 1e-4


@pytest.mark.parametrize("variant", ["uniform", "odd", "h0"])
def test_affine_i32_workload_bitexact(sw, variant):
    _say("case affine i32", variant)
    inp = wl.affine_inputs_i32(1, 64, 1024, wl.INT_SEEDS[variant], variant)
    h = sw.affine_scan_i32(dev(inp["a"]), dev(inp["bx"]),
                           None if inp["h0"] is None else dev(inp["h0"])).cpu().numpy()
    assert np.array_equal(h, oracle.affine_scan_i32(inp["a"], inp["bx"], inp["h0"]))


@pytest.mark.parametrize("L", [1, 2, 3, 63, 64, 65, 2047, 2048, 2049, 4097, 10007, 65536,
                               100003])
def test_affine_i32_ragged_and_multichunk_bitexact(sw, L):
    _say("case affine i32 L", L)
    inp = wl.affine_inputs_i32(2, 3, L, 1000 + L, "odd")
    h0 = wl.affine_inputs_i32(2, 3, 1, 2000 + L, "h0")["h0"]
    h = sw.affine_scan_i32(dev(inp["a"]), dev(inp["bx"]), dev(h0)).cpu().numpy()
    assert np.array_equal(h, oracle.affine_scan_i32(inp["a"], inp["bx"], h0))


def test_affine_i32_long_single_row_repeatable(sw):
    """One long row: every chunk carry crosses workgroups by look-back.  The
    ring is exact, so any lost or misordered carry shows as a bit difference;
    20 repeats must agree bit for bit."""
    _say("case affine i32 long row repeat")
    inp = wl.affine_inputs_i32(1, 1, 1 << 21, 77, "odd")
    a, bx = dev(inp["a"]), dev(inp["bx"])
    ref = oracle.affine_scan_i32(inp["a"], inp["bx"])
    first = sw.affine_scan_i32(a, bx)
    assert np.array_equal(first.cpu().numpy(), ref)
    for _ in range(20):
        assert torch.equal(sw.affine_scan_i32(a, bx), first)


@pytest.mark.parametrize("B,D,L", [(1, 1, 1), (2, 3, 5), (1, 4, 2049), (3, 5, 6151),
                                   (1, 2, 100001), (2, 2, 65536)])
def test_affine_f32_ragged(sw, B, D, L):
    _say("case affine f32", B, D, L)
    inp = wl.affine_inputs(B, D, L, 3000 + L, with_h0=True)
    st, _, _ = _affine_check(sw, inp["a"], inp["bx"], inp["h0"])
    assert_gate(st, f"affine f32 {B}x{D}x{L}")


# Shapes with at least 2048 rows and rows longer than one 2048-step chunk run
# the row-per-workgroup kernel (carry kept on chip); fewer rows run the
# chunk-parallel look-back kernel.  L % 4 == 0 takes the 16-byte path.
@pytest.mark.parametrize("L", [2 * 2048 + 4, 2 * 2048 + 37, 3 * 2048])
def test_affine_i32_many_rows_bitexact(sw, L):
    _say("case affine i32 many rows L", L)
    inp = wl.affine_inputs_i32(2, 1100, L, 4000 + L, "odd")
    h0 = wl.affine_inputs_i32(2, 1100, 1, 5000 + L, "h0")["h0"]
    h = sw.affine_scan_i32(dev(inp["a"]), dev(inp["bx"]), dev(h0)).cpu().numpy()
    assert np.array_equal(h, oracle.affine_scan_i32(inp["a"], inp["bx"], h0))
    h = sw.affine_scan_i32(dev(inp["a"]), dev(inp["bx"])).cpu().numpy()
    assert np.array_equal(h, oracle.affine_scan_i32(inp["a"], inp["bx"]))


@pytest.mark.parametrize("L", [3 * 2048 + 4, 2048 + 1])
def test_affine_f32_many_rows(sw, L):
    _say("case affine f32 many rows L", L)
    inp = wl.affine_inputs(3, 700, L, 6000 + L, with_h0=True)
    st, _, _ = _affine_check(sw, inp["a"], inp["bx"], inp["h0"])
    assert_gate(st, f"affine f32 3x700x{L}")


def test_affine_long_workload_sampled(sw):
    w = wl.workload("affine_f32_b1_d5120_l65536")
    _say("case", w.name)
    inp = w.inputs()
    h = sw.affine_scan(dev(inp["a"]), dev(inp["bx"]))
    rows = _sample_rows(w.B * w.D, 64, 98)
    a2 = inp["a"].reshape(-1, w.L)[rows]
    b2 = inp["bx"].reshape(-1, w.L)[rows]
    got = h.reshape(-1, w.L)[torch.from_numpy(rows).to("cuda")].cpu().numpy()
    ref, mag, sens = oracle.affine_scan(a2, b2, bounds=True)
    st = fp_gate(got, ref, mag, sens)
    _say("  h:", {k_: v for k_, v in st.items() if k_ != "first_bad"})
    assert_gate(st, w.name)
    assert bool(torch.isfinite(h).all())


def test_affine_weighted_prefix(sw):
    """Sec. 6.6, Eq. (10): h_t = alpha_t h_{t-1} + beta_t through the same scan
    (alpha -> a, beta -> b with x = 1)."""
    rng = np.random.Generator(np.random.PCG64(66))
    alpha = rng.uniform(0.0, 1.0, size=(2, 7, 3000)).astype(np.float32)
    beta = rng.uniform(0.0, 1.0, size=(2, 7, 3000)).astype(np.float32)
    st, _, _ = _affine_check(sw, alpha, beta)
    assert_gate(st, "weighted prefix")


def test_affine_empty(sw):
    e = torch.empty((2, 3, 0), device="cuda")
    assert sw.affine_scan(e, e).shape == (2, 3, 0)
    e = torch.empty((0, 3, 5), device="cuda")
    assert sw.affine_scan(e, e).shape == (0, 3, 5)


# ------------------------------------------------------------ fused selective scan

def _run_selective(sw, inp, dtype, with_dskip=True, want_h_last=True):
    if dtype == "bf16":
        x, dl = bf16_dev(inp["x_bf16"]), bf16_dev(inp["delta_bf16"])
        Bm, Cm = bf16_dev(inp["Bm_bf16"]), bf16_dev(inp["Cm_bf16"])
    else:
        x, dl, Bm, Cm = dev(inp["x"]), dev(inp["delta"]), dev(inp["Bm"]), dev(inp["Cm"])
    Dk = dev(inp["Dskip"]) if with_dskip else None
    y, hl = sw.selective_scan_fwd(x, dl, dev(inp["A"]), Bm, Cm, Dk, want_h_last=want_h_last)
    torch.cuda.synchronize()
    return y, hl


def _selective_check(sw, inp, dtype, rows=None, with_dskip=True):
    y, hl = _run_selective(sw, inp, dtype, with_dskip)
    Bsz, D, L = inp["x"].shape
    N = inp["A"].shape[1]
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"] if with_dskip else None, rows=rows, bounds=True)
    if rows is None:
        yg, hg = y.cpu().numpy(), hl.cpu().numpy()
    else:
        ridx = torch.as_tensor(np.asarray(rows), device="cuda")
        yg = y.reshape(Bsz * D, L).index_select(0, ridx).cpu().numpy()
        hg = hl.reshape(Bsz * D, N).index_select(0, ridx).cpu().numpy()
    sy = fp_gate(yg, o["y"], o["y_mag"], o["y_sens"])
    sh = fp_gate(hg, o["h_last"], o["h_mag"], o["h_sens"])
    return sy, sh, yg, o, y


@pytest.mark.parametrize("B,D,N,L", [(1, 1, 1, 1), (2, 70, 16, 200), (1, 33, 3, 37),
                                     (3, 31, 8, 64), (1, 40, 17, 33), (2, 9, 32, 129),
                                     (1, 5, 64, 100), (2, 64, 16, 31), (1, 3, 16, 5000),
                                     (2, 9, 5, 96), (1, 7, 12, 64), (1, 6, 40, 128)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_selective_small_full_compare(sw, B, D, N, L, dtype):
    _say("case selective", dtype, B, D, N, L)
    inp = wl.selective_inputs(B, D, N, L, 4000 + B * 7 + D * 13 + N * 17 + L, dtype)
    sy, sh, yg, o, _ = _selective_check(sw, inp, dtype)
    assert_gate(sy, f"y {dtype} {B}x{D}x{N}x{L}")
    assert_gate(sh, f"h_last {dtype} {B}x{D}x{N}x{L}")
    assert rownorm_rel(yg, o["y"]) <= 1e-4


def test_selective_no_dskip_no_hlast(sw):
    inp = wl.selective_inputs(2, 40, 16, 77, 4999, "f32")
    y, hl = _run_selective(sw, inp, "f32", with_dskip=False, want_h_last=False)
    assert hl is None
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"], None,
                              bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]), "no dskip")


def test_selective_L0_zeroes_h_last(sw):
    x = torch.empty((2, 3, 0), device="cuda")
    A = torch.randn((3, 16), device="cuda")
    Bm = torch.empty((2, 0, 16), device="cuda")
    hl = torch.full((2, 3, 16), 7.0, device="cuda")
    y, hl2 = sw.selective_scan_fwd(x, x, A, Bm, Bm, None, h_last=hl)
    torch.cuda.synchronize()
    assert y.shape == (2, 3, 0) and torch.all(hl2 == 0)


def test_selective_reduces_to_bare_scan(sw):
    """N=1, C=1, Dskip=0: y is the state itself, so the fused kernel must agree
    with the bare scan on a = exp(delta*A), bx = delta*B*x (oracle-checked)."""
    rng = np.random.Generator(np.random.PCG64(5150))
    B, D, L = 2, 37, 999
    inp = wl.selective_inputs(B, D, 1, L, 5151, "f32")
    inp["Cm"] = np.ones_like(inp["Cm"])
    inp["Dskip"] = np.zeros_like(inp["Dskip"])
    y, _ = _run_selective(sw, inp, "f32")
    a = np.exp(inp["delta"].astype(np.float64) * inp["A"][None, :, :1]).astype(np.float32)
    bx = (inp["delta"].astype(np.float64) * inp["x"] * inp["Bm"][:, None, :, 0]).astype(
        np.float32)
    h, mag, sens = oracle.affine_scan(a, bx, bounds=True)
    # a and bx are rounded to fp32 here, so allow the rounding of those inputs too
    st = fp_gate(y.cpu().numpy(), h, mag, sens, rel=2e-4)
    assert_gate(st, "fused vs bare")
    del rng


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_selective_chained_chunks_bitexact(sw, monkeypatch, dtype):
    """Several sequence chunks per row, chained through the published exact
    state, run the same per-step arithmetic as one chunk per row: the results
    must be bit-identical, and within the oracle gate."""
    _say("case selective chained chunks", dtype)
    inp = wl.selective_inputs(2, 21, 16, 3001, 6060, dtype)
    monkeypatch.setenv("SW_SS_TASKS_PER_WAVE", "1")
    y1, h1 = _run_selective(sw, inp, dtype)
    monkeypatch.setenv("SW_SS_TASKS_PER_WAVE", "16")  # 16 chunks of 192 steps per row
    y2, h2 = _run_selective(sw, inp, dtype)
    assert torch.equal(y1, y2) and torch.equal(h1, h2)
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], bounds=True)
    assert_gate(fp_gate(y2.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]), "chained y")
    assert_gate(fp_gate(h2.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                "chained h_last")


# ------------------------------------------------------------ full-size workloads

def _sample_rows(n_rows, k, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    pick = rng.choice(n_rows, size=min(k, n_rows), replace=False)
    # always include the first and last row (edges of the row tiling)
    return np.unique(np.concatenate([pick, [0, n_rows - 1]])).astype(np.int64)


@pytest.mark.parametrize("name,k", [("selective_f32_b2_d256_n16_l512", None),
                                    ("selective_bf16_b8_d1536_n16_l2048", 768),
                                    ("selective_f32_b1_d5120_n16_l65536", 48),
                                    ("selective_f32_b4_d2048_n16_l8192_stress", 384)])
def test_selective_workloads(sw, name, k):
    w = wl.workload(name)
    _say("case", name)
    inp = w.inputs()
    rows = None if k is None else _sample_rows(w.B * w.D, k, 99)
    sy, sh, yg, o, y = _selective_check(sw, inp, w.dtype, rows=rows)
    # the launches bench.py times at these shapes
    want = {"selective_f32_b2_d256_n16_l512": "selective_row16_kernel: 8 segments",
            "selective_bf16_b8_d1536_n16_l2048": "selective_row16_kernel: whole rows",
            "selective_f32_b1_d5120_n16_l65536": "selective_quad_kernel: ",
            "selective_f32_b4_d2048_n16_l8192_stress": "selective_row16_kernel: whole rows"}
    assert sw.last_launch().startswith(want[name]), sw.last_launch()
    _say("  launch:", sw.last_launch())
    _say("  y:", {k_: v for k_, v in sy.items() if k_ != "first_bad"})
    _say("  h_last:", {k_: v for k_, v in sh.items() if k_ != "first_bad"})
    assert_gate(sy, name + " y")
    assert_gate(sh, name + " h_last")
    assert bool(torch.isfinite(y).all())
    if not w.stress:
        assert sy["n_ill"] == 0
        assert rownorm_rel(yg, o["y"]) <= 1e-4


# ------------------------------------------------------------ ABI error paths on the GPU

def test_abi_rejects_bad_pointers(sw):
    lib = sw.lib()
    a = torch.zeros((1, 2, 8), device="cuda")
    h = torch.zeros((1, 2, 8), device="cuda")
    host = np.zeros(16, np.float32)
    rc = lib.sw_affine_scan(host.ctypes.data, a.data_ptr(), None, h.data_ptr(), 1, 2, 8)
    assert rc == 1 and "device memory" in sw.last_error()
    rc = lib.sw_affine_scan(a.data_ptr() + 2, a.data_ptr(), None, h.data_ptr(), 1, 2, 8)
    assert rc == 1 and "aligned" in sw.last_error()
    rc = lib.sw_affine_scan(a.data_ptr(), a.data_ptr(), None, a.data_ptr() + 16, 1, 2, 8)
    assert rc == 1 and "overlaps" in sw.last_error()
    rc = lib.sw_affine_scan(a.data_ptr(), a.data_ptr(), None, None, 1, 2, 8)
    assert rc == 1
    assert torch.all(h == 0)  # nothing was written
    x = torch.zeros((1, 2, 8), device="cuda")
    A = torch.zeros((2, 65), device="cuda")
    rc = lib.sw_selective_scan_fwd(x.data_ptr(), x.data_ptr(), A.data_ptr(), x.data_ptr(),
                                   x.data_ptr(), None, h.data_ptr(), None, 1, 2, 65, 8)
    assert rc == 2


# ------------------------------------------------------------ Mamba-block options

def _ex_inputs(B, D, N, L, seed, dtype, opts):
    inp = wl.selective_inputs(B, D, N, L, seed, dtype)
    rng = np.random.Generator(np.random.PCG64(seed + 77))
    ex = {}
    if "z" in opts:
        z = (rng.standard_normal(size=(B, D, L)) * 2).astype(np.float32)
        if dtype == "bf16":
            ex["z_bits"] = wl.bf16_round(z)
            z = wl.bf16_widen(ex["z_bits"])
        ex["z"] = z
    if "bias" in opts:
        # raw delta before softplus: the generator's softplus output is reused
        # as a raw value, shifted by a per-channel bias around -1
        ex["delta_bias"] = rng.uniform(-2.0, 0.0, size=D).astype(np.float32)
    if "h0" in opts:
        ex["h0"] = rng.standard_normal(size=(B, D, N)).astype(np.float32)
    return inp, ex


def _run_ex(sw, inp, ex, dtype, softplus, y_bf16):
    if dtype == "bf16":
        x, dl = bf16_dev(inp["x_bf16"]), bf16_dev(inp["delta_bf16"])
        Bm, Cm = bf16_dev(inp["Bm_bf16"]), bf16_dev(inp["Cm_bf16"])
        z = bf16_dev(ex["z_bits"]) if "z" in ex else None
    else:
        x, dl, Bm, Cm = dev(inp["x"]), dev(inp["delta"]), dev(inp["Bm"]), dev(inp["Cm"])
        z = dev(ex["z"]) if "z" in ex else None
    y, hl = sw.selective_scan_fwd(
        x, dl, dev(inp["A"]), Bm, Cm, dev(inp["Dskip"]), z=z,
        delta_bias=dev(ex["delta_bias"]) if "delta_bias" in ex else None,
        h0=dev(ex["h0"]) if "h0" in ex else None, delta_softplus=softplus,
        y_dtype=torch.bfloat16 if y_bf16 else torch.float32)
    torch.cuda.synchronize()
    return y, hl


def _ex_oracle(inp, ex, softplus, rows=None):
    return oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                                 inp["Dskip"], rows=rows, bounds=True, z=ex.get("z"),
                                 delta_bias=ex.get("delta_bias"), h0=ex.get("h0"),
                                 delta_softplus=softplus)


def _y_gate(yt, o, y_bf16, what, rows=None):
    yg = yt.float().cpu().numpy()
    if rows is not None:
        yg = yg.reshape(-1, yg.shape[-1])[rows]
    if y_bf16:
        # bf16 y: the fp32 result rounded once more, half an ulp of 8 bits
        err = np.abs(yg - o["y"])
        ok = err <= 2.0 ** -8 * np.abs(o["y"]) + 1.01e-4 * o["y_mag"] \
            + 4 * 2.0 ** -24 * o["y_sens"]
        assert ok.all(), f"{what}: bf16 y off at {np.argwhere(~ok)[:3]}"
    else:
        assert_gate(fp_gate(yg, o["y"], o["y_mag"], o["y_sens"]), what)


# (B, D, N, L): N = 16 with L % 8 == 0 takes the 16-lane kernel; the others the 8-lane one
_EX_SHAPES = [(2, 37, 16, 520), (1, 20, 16, 133), (2, 9, 5, 96)]
_EX_OPTS = [("h0",), ("bias", "softplus"), ("softplus",), ("z",), ("ybf16",),
            ("h0", "bias", "softplus", "z", "ybf16")]


@pytest.mark.parametrize("shape", _EX_SHAPES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", _EX_OPTS)
def test_selective_mamba_options(sw, shape, dtype, opts):
    B, D, N, L = shape
    _say("case selective options", dtype, shape, opts)
    inp, ex = _ex_inputs(B, D, N, L, 7000 + B + D + N + L, dtype, opts)
    softplus, y_bf16 = "softplus" in opts, "ybf16" in opts
    y, hl = _run_ex(sw, inp, ex, dtype, softplus, y_bf16)
    assert y.dtype == (torch.bfloat16 if y_bf16 else torch.float32)
    o = _ex_oracle(inp, ex, softplus)
    _y_gate(y, o, y_bf16, f"y {dtype} {shape} {opts}")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                f"h_last {dtype} {shape} {opts}")


@pytest.mark.parametrize("shape", _EX_SHAPES)
def test_selective_bf16_y_is_the_fp32_y_rounded(sw, shape):
    """bf16 y is the fp32 y of the same call rounded once to nearest even:
    bit-identical to torch's rounding of the fp32 output (both kernels)."""
    B, D, N, L = shape
    _say("case bf16 y rounding", shape)
    opts = ("h0", "bias", "softplus", "z")
    inp, ex = _ex_inputs(B, D, N, L, 8100 + B + D + N + L, "bf16", opts)
    y32, _ = _run_ex(sw, inp, ex, "bf16", True, False)
    y16, _ = _run_ex(sw, inp, ex, "bf16", True, True)
    assert torch.equal(y16, y32.to(torch.bfloat16))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["16", "8"])
def test_selective_continued_across_calls_bitexact(sw, monkeypatch, dtype, layout):
    """A sequence scanned in three calls, each starting from the previous
    call's h_last, runs the same per-step arithmetic as one call: y and the
    final state are bit-identical."""
    monkeypatch.setenv("SW_SS_LAYOUT", layout)
    # whole-row walks (this narrow shape would otherwise take the segmented
    # form, whose rounding depends on where the segments fall)
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")
    _say("case selective continued", dtype, layout)
    B, D, N, L = 2, 24, 16, 4096
    inp = wl.selective_inputs(B, D, N, L, 7777, dtype)
    k = "_bf16" if dtype == "bf16" else ""
    cv = (lambda a: bf16_dev(a)) if dtype == "bf16" else (lambda a: dev(a))
    x, dl, Bm, Cm = (inp[n + k] for n in ("x", "delta", "Bm", "Cm"))
    A, Dk = dev(inp["A"]), dev(inp["Dskip"])
    y_one, h_one = sw.selective_scan_fwd(cv(x), cv(dl), A, cv(Bm), cv(Cm), Dk)
    parts, h = [], None
    for t0, t1 in ((0, 1024), (1024, 1536), (1536, L)):
        yp, h = sw.selective_scan_fwd(cv(np.ascontiguousarray(x[:, :, t0:t1])),
                                      cv(np.ascontiguousarray(dl[:, :, t0:t1])), A,
                                      cv(np.ascontiguousarray(Bm[:, t0:t1])),
                                      cv(np.ascontiguousarray(Cm[:, t0:t1])), Dk, h0=h)
        parts.append(yp)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(parts, dim=2), y_one)
    assert torch.equal(h, h_one)


# Narrow calls split rows into segments (three launches composed with Eq. (7),
# carries kept in y's memory).  (B, D, L) and the forced count ("auto": the
# library's choice); D not a multiple of 16 leaves rows past D in the last
# workgroup; counts that do not divide L leave the last segment shorter
# (1000 / 3: 384, 384, 232), or, where the rest would be under a super-tile,
# add it to the last one (776 / 5 in fp32: 192 x 3 + 200); L below two
# super-tiles stays whole.
_SEG_CASES = [((1, 37, 1000), "3"), ((2, 16, 512), "16"), ((1, 5, 4096), "auto"),
              ((1, 48, 2048), "auto"), ((1, 20, 64), "16"), ((3, 7, 776), "5")]


@pytest.mark.parametrize("case", _SEG_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", [(), ("h0", "bias", "softplus", "z", "ybf16")])
def test_selective_segments(sw, monkeypatch, case, dtype, opts):
    (B, D, L), segs = case
    if segs != "auto":
        monkeypatch.setenv("SW_SS_SEGMENTS", segs)
    _say("case selective segments", dtype, (B, D, L), segs, opts)
    inp, ex = _ex_inputs(B, D, 16, L, 9100 + B + D + L, dtype, opts)
    softplus, y_bf16 = "softplus" in opts, "ybf16" in opts
    y, hl = _run_ex(sw, inp, ex, dtype, softplus, y_bf16)
    o = _ex_oracle(inp, ex, softplus)
    _y_gate(y, o, y_bf16, f"segments y {dtype} {(B, D, L)} {segs} {opts}")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                f"segments h_last {dtype} {(B, D, L)} {segs} {opts}")
    # the same call again gives the same bits (fixed segments, no atomics)
    y2, hl2 = _run_ex(sw, inp, ex, dtype, softplus, y_bf16)
    assert torch.equal(y, y2) and torch.equal(hl, hl2)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_selective_segments_no_dskip_no_hlast(sw, monkeypatch, dtype):
    """The segmented form with Dskip and h_last left out (h_last NULL: the last
    segment stores no state), against the oracle and the whole-row walk."""
    B, D, N, L = 1, 24, 16, 2048
    _say("case selective segments no dskip / h_last", dtype, (B, D, N, L))
    inp = wl.selective_inputs(B, D, N, L, 9321, dtype)
    monkeypatch.setenv("SW_SS_SEGMENTS", "6")
    y, hl = _run_selective(sw, inp, dtype, with_dskip=False, want_h_last=False)
    assert hl is None
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"], None,
                              bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]),
                f"segments no dskip {dtype}")
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")
    y1, _ = _run_selective(sw, inp, dtype, with_dskip=False, want_h_last=False)
    assert rownorm_rel(y.cpu().numpy(), y1.cpu().numpy()) <= 1e-5


# The correction form of the segmented walk (fp32 y): every segment walks from
# a zero state in one launch, a fold composes the carries, and a third launch
# walks each later segment again from its composed state until the carried
# part is negligible.  Short segments never reach that point (the walk covers
# the whole segment); the long ones stop early.  (B, D, L), forced count.
_CORR_CASES = [((1, 37, 1000), "3"), ((2, 16, 512), "4"), ((3, 7, 776), "5"),
               ((1, 20, 16384), "2"), ((1, 24, 8192), "auto")]


@pytest.mark.parametrize("case", _CORR_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", [(), ("h0", "bias", "softplus", "z")])
def test_selective_segments_correction(sw, monkeypatch, case, dtype, opts):
    (B, D, L), segs = case
    monkeypatch.setenv("SW_SS_SEGFORM", "2")
    if segs != "auto":
        monkeypatch.setenv("SW_SS_SEGMENTS", segs)
    _say("case selective segments correction", dtype, (B, D, L), segs, opts)
    inp, ex = _ex_inputs(B, D, 16, L, 9400 + B + D + L, dtype, opts)
    softplus = "softplus" in opts
    y, hl = _run_ex(sw, inp, ex, dtype, softplus, False)
    o = _ex_oracle(inp, ex, softplus)
    _y_gate(y, o, False, f"correction y {dtype} {(B, D, L)} {segs} {opts}")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                f"correction h_last {dtype} {(B, D, L)} {segs} {opts}")
    assert rownorm_rel(y.cpu().numpy(), o["y"]) <= 1e-5
    # the same call again gives the same bits (fixed segments, no atomics)
    y2, hl2 = _run_ex(sw, inp, ex, dtype, softplus, False)
    assert torch.equal(y, y2) and torch.equal(hl, hl2)


@pytest.mark.parametrize("kind", ["no_decay", "growth", "zero_carry", "stress"])
def test_selective_segments_correction_regimes(sw, monkeypatch, kind):
    """The correction walk where the carried part never fades (A = 0: the
    walk covers every segment whole), where it grows (A > 0), where there is
    none (x = 0 before the last segment: every composed state is zero and the
    walk stops after its first super-tile) and where it fades at very
    different rates per state (the stress recipe's delta and A)."""
    B, D, N, L = 1, 20, 16, 8192
    monkeypatch.setenv("SW_SS_SEGFORM", "2")
    monkeypatch.setenv("SW_SS_SEGMENTS", "4")
    _say("case selective segments correction regime", kind)
    inp = wl.selective_inputs(B, D, N, L, 9500, "f32", stress=(kind == "stress"))
    if kind == "no_decay":
        inp["A"] = np.zeros_like(inp["A"])
    elif kind == "growth":
        inp["A"] = np.abs(inp["A"]) * np.float32(1e-4)
    elif kind == "zero_carry":
        inp["x"] = inp["x"].copy()
        inp["x"][:, :, : 3 * L // 4] = 0.0
    y, hl = _run_selective(sw, inp, "f32")
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]), f"correction {kind} y")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                f"correction {kind} h_last")
    # against the whole-row walk of the same call
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")
    y1, hl1 = _run_selective(sw, inp, "f32")
    assert rownorm_rel(y.cpu().numpy(), y1.cpu().numpy()) <= 1e-5


# The planner's choices on a 256-CU part (section "Choosing the layout" of the
# design notes): few rows at L = 16384 take the correction form of the 16-lane
# layout, long rows the quad layout, rows that fill the GPU whole rows, and
# bf16 y keeps the records form.  Each call is also checked against the
# oracle on sampled rows.
_PLAN_CASES = [((1, 1280, 16384), "f32", False, "selective_row16_kernel: 6 segments of 2752 steps, correction"),
               ((1, 2560, 65536), "f32", False, "selective_quad_kernel: 16 segments"),
               ((1, 8192, 4096), "f32", False, "selective_row16_kernel: whole rows"),
               ((1, 1280, 4096), "f32", True, "selective_row16_kernel: 16 segments of 256 steps, records")]


@pytest.mark.parametrize("case", _PLAN_CASES)
def test_planner_choices(sw, case):
    (B, D, L), dtype, y_bf16, want = case
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the expected choices are those of a 256-CU part")
    _say("case planner", (B, D, L), dtype, "bf16 y" if y_bf16 else "")
    inp = wl.selective_inputs(B, D, 16, L, 9800 + D, dtype)
    x, dl = dev(inp["x"]), dev(inp["delta"])
    Bm, Cm = dev(inp["Bm"]), dev(inp["Cm"])
    y, hl = sw.selective_scan_fwd(x, dl, dev(inp["A"]), Bm, Cm, dev(inp["Dskip"]),
                                  y_dtype=torch.bfloat16 if y_bf16 else torch.float32)
    assert sw.last_launch().startswith(want), sw.last_launch()
    rows = _sample_rows(B * D, 24, 7)
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], rows=rows, bounds=True)
    ridx = torch.as_tensor(np.asarray(rows), device="cuda")
    _y_gate(y.reshape(B * D, L).index_select(0, ridx), o, y_bf16, f"planner y {(B, D, L)}")
    hg = hl.reshape(B * D, 16).index_select(0, ridx).cpu().numpy()
    assert_gate(fp_gate(hg, o["h_last"], o["h_mag"], o["h_sens"]), f"planner h_last {(B, D, L)}")


def _launch_plan(text):
    """(layout, segments, steps, form) from sw_last_launch()'s text."""
    import re
    if text.startswith("selective_fwd_kernel"):
        return (8, 1, None, "whole")
    layout = 4 if text.startswith("selective_quad_kernel") else 16
    m = re.search(r"(\d+) segments of (\d+) steps, (records|correction) form", text)
    if m:
        return (layout, int(m.group(1)), int(m.group(2)), m.group(3))
    assert text.endswith("whole rows"), text
    return (layout, 1, None, "whole")


# (B, D, N, L), input dtype, bf16 y: the benched shapes, a narrow long call of
# each layout, bf16 y (records form), an N the 16-lane layouts do not take
_PLAN_VS_LAUNCH = [((1, 5120, 16, 65536), "f32", False), ((8, 1536, 16, 2048), "bf16", False),
                   ((2, 256, 16, 512), "f32", False), ((1, 1280, 16, 16384), "f32", False),
                   ((1, 2560, 16, 32768), "bf16", False), ((1, 1280, 16, 4096), "f32", True),
                   ((1, 64, 8, 1000), "f32", False)]


@pytest.mark.parametrize("case", _PLAN_VS_LAUNCH)
def test_plan_query_matches_the_launch(sw, case):
    """sw_selective_scan_plan for this device names the kernels, segments and
    form the forward call then enqueues."""
    (B, D, N, L), dtype, y_bf16 = case
    _say("case plan vs launch", (B, D, N, L), dtype, "bf16 y" if y_bf16 else "")
    p = sw.selective_scan_plan(B, D, N, L, dtype, "bf16" if y_bf16 else "f32")
    inp = wl.selective_inputs(B, D, N, L, 9900 + D, dtype)
    if dtype == "bf16":
        x, dl = bf16_dev(inp["x_bf16"]), bf16_dev(inp["delta_bf16"])
        Bm, Cm = bf16_dev(inp["Bm_bf16"]), bf16_dev(inp["Cm_bf16"])
    else:
        x, dl, Bm, Cm = (dev(inp[k]) for k in ("x", "delta", "Bm", "Cm"))
    sw.selective_scan_fwd(x, dl, dev(inp["A"]), Bm, Cm, dev(inp["Dskip"]),
                          y_dtype=torch.bfloat16 if y_bf16 else torch.float32)
    torch.cuda.synchronize()
    got = _launch_plan(sw.last_launch())
    want = (p["layout"], p["segments"], p["segment_steps"] if p["segments"] > 1 else None,
            p["form"])
    assert got == want, (sw.last_launch(), p)


# The quad layout (four lanes per row, four states per lane, 16 rows per
# wavefront) taken by few-row, long calls; forced here on small shapes
# (SW_SS_QUAD=1) with the segment count given: D not a multiple of 64 leaves
# wavefronts with rows past D and wavefronts with none; L / k rounded up to 64
# steps leaves the last segment the shortest (2048 / 3: 704, 704, 640; 8192 /
# 7), and where that would leave it under 64 steps the length is rounded down
# and the last segment is the longest (160 / 2: 64 + 96; 1056 / 16: 15 x 64 +
# 96); one segment is the whole-row walk, down to rows of one tile (L = 32);
# L = 1040 (not whole 32-step tiles) falls back to the 16-lane layout.
# (B, D, L), segments.
_QUAD_CASES = [((1, 37, 1040), "2"), ((2, 100, 2048), "3"), ((1, 64, 4096), "4"),
                 ((1, 5, 16), "1"), ((3, 130, 512), "1"), ((1, 70, 8192), "7"),
                 ((1, 37, 160), "2"), ((1, 37, 1056), "16"), ((2, 70, 32), "1")]


@pytest.mark.parametrize("case", _QUAD_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("opts", [(), ("h0", "bias", "softplus", "z")])
def test_selective_quad(sw, monkeypatch, case, dtype, opts):
    (B, D, L), segs = case
    monkeypatch.setenv("SW_SS_QUAD", "1")
    monkeypatch.setenv("SW_SS_SEGMENTS", segs)
    _say("case selective quad", dtype, (B, D, L), segs, opts)
    inp, ex = _ex_inputs(B, D, 16, L, 9600 + B + D + L, dtype, opts)
    softplus = "softplus" in opts
    y, hl = _run_ex(sw, inp, ex, dtype, softplus, False)
    # the layout takes every call with whole 32-step tiles (L = 1040 is not one)
    assert ("selective_quad_kernel" in sw.last_launch()) == (L % 32 == 0), sw.last_launch()
    o = _ex_oracle(inp, ex, softplus)
    _y_gate(y, o, False, f"quad y {dtype} {(B, D, L)} {segs} {opts}")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                f"quad h_last {dtype} {(B, D, L)} {segs} {opts}")
    assert rownorm_rel(y.cpu().numpy(), o["y"]) <= 1e-5
    y2, hl2 = _run_ex(sw, inp, ex, dtype, softplus, False)
    assert torch.equal(y, y2) and torch.equal(hl, hl2)


@pytest.mark.parametrize("kind", ["no_decay", "growth", "zero_carry", "stress", "no_dskip"])
def test_selective_quad_regimes(sw, monkeypatch, kind):
    """The quad layout's correction walk where the carried part never fades,
    grows, is zero, or fades at very different rates (as for the 16-lane
    layout); and without Dskip and h_last."""
    B, D, N, L = 1, 90, 16, 8192
    monkeypatch.setenv("SW_SS_QUAD", "1")
    monkeypatch.setenv("SW_SS_SEGMENTS", "4")
    _say("case selective quad regime", kind)
    inp = wl.selective_inputs(B, D, N, L, 9700, "f32", stress=(kind == "stress"))
    if kind == "no_decay":
        inp["A"] = np.zeros_like(inp["A"])
    elif kind == "growth":
        inp["A"] = np.abs(inp["A"]) * np.float32(1e-4)
    elif kind == "zero_carry":
        inp["x"] = inp["x"].copy()
        inp["x"][:, :, : 3 * L // 4] = 0.0
    with_d = kind != "no_dskip"
    y, hl = _run_selective(sw, inp, "f32", with_dskip=with_d, want_h_last=with_d)
    assert sw.last_launch().startswith("selective_quad_kernel: 4 segments"), sw.last_launch()
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"] if with_d else None, bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]), f"quad {kind} y")
    if with_d:
        assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]),
                    f"quad {kind} h_last")
    else:
        assert hl is None
    # against the whole-row walk of the 16-lane layout
    monkeypatch.setenv("SW_SS_QUAD", "0")
    monkeypatch.setenv("SW_SS_SEGMENTS", "1")
    y1, _ = _run_selective(sw, inp, "f32", with_dskip=with_d, want_h_last=with_d)
    assert rownorm_rel(y.cpu().numpy(), y1.cpu().numpy()) <= 1e-5


def test_selective_L0_returns_h0(sw):
    x = torch.empty((2, 3, 0), device="cuda")
    A = torch.randn((3, 16), device="cuda")
    Bm = torch.empty((2, 0, 16), device="cuda")
    h0 = torch.randn((2, 3, 16), device="cuda")
    y, hl = sw.selective_scan_fwd(x, x, A, Bm, Bm, None, h0=h0)
    torch.cuda.synchronize()
    assert y.shape == (2, 3, 0) and torch.equal(hl, h0)


def test_selective_mamba_options_full_size(sw):
    """Every option at the Mamba-130M-like shape (bf16, B=8, D=1536, N=16,
    L=2048), in the bench's launch configuration, on sampled rows."""
    w = wl.workload("selective_bf16_b8_d1536_n16_l2048")
    _say("case options full size", w.name)
    opts = ("h0", "bias", "softplus", "z")
    inp, ex = _ex_inputs(w.B, w.D, w.N, w.L, 8080, "bf16", opts)
    for y_bf16 in (False, True):
        y, hl = _run_ex(sw, inp, ex, "bf16", True, y_bf16)
        rows = _sample_rows(w.B * w.D, 256, 81)
        o = _ex_oracle(inp, ex, True, rows=rows)
        _y_gate(y, o, y_bf16, f"full-size options y_bf16={y_bf16}", rows=rows)
        hg = hl.reshape(w.B * w.D, w.N).index_select(
            0, torch.as_tensor(rows, device="cuda")).cpu().numpy()
        assert_gate(fp_gate(hg, o["h_last"], o["h_mag"], o["h_sens"]), "full-size h_last")


# --------------------------------- Eq. (3)-(4): input and output projections

def _proj_inputs(B, D, L, seed, dtype="f32"):
    """a in [-1.05, 1.05] (growth and sign changes included), b, x, c ~ N(0,1),
    h0 ~ N(0,1); int32: full-range words with odd a."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if dtype == "i32":
        a, b, x, c = (rng.integers(-2**31, 2**31, size=(B, D, L), dtype=np.int64)
                      .astype(np.int32) for _ in range(4))
        a |= 1
        h0 = rng.integers(-2**31, 2**31, size=(B, D), dtype=np.int64).astype(np.int32)
        return a, b, x, c, h0
    a = rng.uniform(-1.05, 1.05, size=(B, D, L)).astype(np.float32)
    b, x, c = (rng.standard_normal(size=(B, D, L)).astype(np.float32) for _ in range(3))
    h0 = rng.standard_normal(size=(B, D)).astype(np.float32)
    return a, b, x, c, h0


# (B, D, L): element path (ragged L), one chunk, look-back chunks, and >= 2048
# rows longer than a chunk (the row-per-workgroup kernel), vector and ragged
_PROJ_SHAPES = [(2, 5, 37), (3, 7, 1024), (1, 3, 5003), (1, 2, 20480), (2, 1100, 4100),
                (1, 2100, 2049)]
_PROJ_OPTS = [("x", "c", "h0"), ("c",), ("x",), ()]


@pytest.mark.parametrize("shape", _PROJ_SHAPES)
@pytest.mark.parametrize("opts", _PROJ_OPTS)
def test_proj_f32(sw, shape, opts):
    B, D, L = shape
    _say("case proj f32", shape, opts)
    a, b, x, c, h0 = _proj_inputs(B, D, L, 9000 + L)
    x = x if "x" in opts else None
    c = c if "c" in opts else None
    h0 = h0 if "h0" in opts else None
    y, hl = sw.affine_scan_proj(dev(a), dev(b), None if x is None else dev(x),
                                None if c is None else dev(c), None if h0 is None else dev(h0))
    ref, href, ym, ys = oracle.affine_proj(a, b, x, c, h0, bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), ref, ym, ys), f"proj y {shape} {opts}")
    # h_last: the state before the output projection, gated by the state bounds
    _, hm, hs = oracle.affine_scan(a, b * (x if x is not None else 1.0),
                                   h0, bounds=True)
    assert_gate(fp_gate(hl.cpu().numpy(), href, hm[..., -1], hs[..., -1]),
                f"proj h_last {shape} {opts}")


@pytest.mark.parametrize("shape", _PROJ_SHAPES)
def test_proj_i32_bitexact(sw, shape):
    B, D, L = shape
    _say("case proj i32", shape)
    a, b, x, c, h0 = _proj_inputs(B, D, L, 9100 + L, "i32")
    for xx, cc, hh in ((x, c, h0), (None, c, None), (x, None, h0)):
        y, hl = sw.affine_scan_proj_i32(*(None if v is None else dev(v)
                                          for v in (a, b, xx, cc, hh)))
        ry, rh = oracle.affine_proj_i32(a, b, xx, cc, hh)
        assert np.array_equal(y.cpu().numpy(), ry)
        assert np.array_equal(hl.cpu().numpy(), rh)


def test_proj_weighted_prefix_is_the_bare_scan(sw):
    """Eq. (10) through the projection form (x = c = 1) runs the bare scan's
    arithmetic on the pairs (alpha, beta): bit-identical to sw_affine_scan,
    in both kernels, and within the gate of the oracle."""
    rng = np.random.Generator(np.random.PCG64(67))
    for B, D, L in ((2, 7, 3000), (2, 1100, 4100)):
        alpha = rng.uniform(0.0, 1.0, size=(B, D, L)).astype(np.float32)
        beta = rng.uniform(0.0, 1.0, size=(B, D, L)).astype(np.float32)
        y, hl = sw.affine_scan_proj(dev(alpha), dev(beta))
        h = sw.affine_scan(dev(alpha), dev(beta))
        assert torch.equal(y, h)
        assert torch.equal(hl, h[..., -1])
        ref, _, ym, ys = oracle.affine_proj(alpha, beta, bounds=True)
        assert_gate(fp_gate(y.cpu().numpy(), ref, ym, ys), f"weighted prefix {B}x{D}x{L}")


def test_proj_empty_and_L0(sw):
    e = torch.empty((2, 3, 0), device="cuda")
    h0 = torch.randn((2, 3), device="cuda")
    y, hl = sw.affine_scan_proj(e, e, h0=h0)
    torch.cuda.synchronize()
    assert y.shape == (2, 3, 0) and torch.equal(hl, h0)
    y, hl = sw.affine_scan_proj(e, e)
    torch.cuda.synchronize()
    assert torch.equal(hl, torch.zeros_like(h0))
    e = torch.empty((0, 3, 5), device="cuda")
    y, hl = sw.affine_scan_proj(e, e)
    assert y.shape == (0, 3, 5) and hl.shape == (0, 3)


# -------------------------------------- the paper's schedule (Blelloch tree)

# (B, D, L): one chunk, ragged tails, several chunks, many rows
_SCHED_SHAPES = [(1, 1, 1), (2, 3, 5), (1, 4, 2048), (1, 3, 2049), (2, 5, 6151), (1, 2, 100001),
                 (3, 700, 3 * 2048 + 4)]


@pytest.mark.parametrize("B,D,L", _SCHED_SHAPES)
def test_blelloch_schedule_i32_bitexact(sw, B, D, L):
    _say("case blelloch i32", B, D, L)
    inp = wl.affine_inputs_i32(B, D, L, 7000 + L, "odd")
    h0 = wl.affine_inputs_i32(B, D, 1, 7100 + L, "h0")["h0"]
    h = sw.affine_scan_schedule_i32(dev(inp["a"]), dev(inp["bx"]), dev(h0),
                                    schedule="blelloch").cpu().numpy()
    assert np.array_equal(h, oracle.affine_scan_i32(inp["a"], inp["bx"], h0))


@pytest.mark.parametrize("B,D,L", _SCHED_SHAPES)
def test_blelloch_schedule_f32(sw, B, D, L):
    _say("case blelloch f32", B, D, L)
    inp = wl.affine_inputs(B, D, L, 7200 + L, with_h0=True)
    h = sw.affine_scan_schedule(dev(inp["a"]), dev(inp["bx"]), dev(inp["h0"]),
                                schedule="blelloch").cpu().numpy()
    ref, mag, sens = oracle.affine_scan(inp["a"], inp["bx"], inp["h0"], bounds=True)
    assert_gate(fp_gate(h, ref, mag, sens), f"blelloch f32 {B}x{D}x{L}")


def test_blelloch_schedule_workloads(sw):
    """The paper's schedule on the bare-scan workloads: int32 bit-identical to
    the default schedule (the ring is exact), fp32 within the gate."""
    w = wl.workload("affine_f32_b1_d64_l1024")
    inp = w.inputs()
    h = sw.affine_scan_schedule(dev(inp["a"]), dev(inp["bx"]), schedule="blelloch").cpu().numpy()
    ref, mag, sens = oracle.affine_scan(inp["a"], inp["bx"], bounds=True)
    assert_gate(fp_gate(h, ref, mag, sens), w.name)
    for variant in ("uniform", "odd", "h0"):
        ii = wl.affine_inputs_i32(1, 64, 1024, wl.INT_SEEDS[variant], variant)
        args = (dev(ii["a"]), dev(ii["bx"]), None if ii["h0"] is None else dev(ii["h0"]))
        assert torch.equal(sw.affine_scan_schedule_i32(*args, schedule="blelloch"),
                           sw.affine_scan_i32(*args))
    w = wl.workload("affine_f32_b1_d5120_l65536")
    inp = w.inputs()
    h = sw.affine_scan_schedule(dev(inp["a"]), dev(inp["bx"]), schedule="blelloch")
    rows = _sample_rows(w.B * w.D, 32, 99)
    got = h.reshape(-1, w.L)[torch.from_numpy(rows).to("cuda")].cpu().numpy()
    ref, mag, sens = oracle.affine_scan(inp["a"].reshape(-1, w.L)[rows],
                                        inp["bx"].reshape(-1, w.L)[rows], bounds=True)
    assert_gate(fp_gate(got, ref, mag, sens), w.name + " blelloch")


@pytest.mark.parametrize("B,D,N,L", [(1, 3, 16, 37), (2, 5, 16, 2048), (1, 2, 5, 2049),
                                     (2, 3, 64, 100), (1, 2, 16, 5000)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_selective_blelloch_schedule(sw, B, D, N, L, dtype):
    """The fused form with the paper's schedule against the oracle."""
    _say("case selective blelloch", dtype, B, D, N, L)
    inp = wl.selective_inputs(B, D, N, L, 7300 + N + L, dtype)
    if dtype == "bf16":
        args = (bf16_dev(inp["x_bf16"]), bf16_dev(inp["delta_bf16"]), dev(inp["A"]),
                bf16_dev(inp["Bm_bf16"]), bf16_dev(inp["Cm_bf16"]), dev(inp["Dskip"]))
    else:
        args = tuple(dev(inp[k]) for k in ("x", "delta", "A", "Bm", "Cm", "Dskip"))
    y, hl = sw.selective_scan_fwd_schedule(*args, schedule="blelloch")
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], bounds=True)
    assert_gate(fp_gate(y.cpu().numpy(), o["y"], o["y_mag"], o["y_sens"]), "blelloch y")
    assert_gate(fp_gate(hl.cpu().numpy(), o["h_last"], o["h_mag"], o["h_sens"]), "blelloch h_last")


def test_selective_blelloch_schedule_full_size(sw):
    w = wl.workload("selective_bf16_b8_d1536_n16_l2048")
    _say("case selective blelloch full size")
    inp = w.inputs()
    y, _ = sw.selective_scan_fwd_schedule(
        bf16_dev(inp["x_bf16"]), bf16_dev(inp["delta_bf16"]), dev(inp["A"]),
        bf16_dev(inp["Bm_bf16"]), bf16_dev(inp["Cm_bf16"]), dev(inp["Dskip"]),
        schedule="blelloch", want_h_last=False)
    rows = _sample_rows(w.B * w.D, 96, 71)
    got = y.reshape(-1, w.L)[torch.as_tensor(rows, device="cuda")].cpu().numpy()
    o = oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], rows=rows, bounds=True)
    assert_gate(fp_gate(got, o["y"], o["y_mag"], o["y_sens"]), "blelloch full size")
