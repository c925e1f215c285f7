"""Maximum sizes: element counts and byte offsets past 2^31 (64-bit indexing),
through the C ABI.

Inputs are generated on the GPU with a seeded torch generator (the host would
need tens of GB for them); the oracle gets copies of the rows it checks.
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


def test_affine_i32_single_row_past_2_31_steps(sw):
    """One row of 2^31 + 37 steps with a = 1, bx = 1 and h0 = 5: the states
    are h_t = t + 6 modulo 2^32, whatever the schedule (every chunk carry
    crosses workgroups by look-back; t passes 2^31)."""
    L = (1 << 31) + 37
    _say("case affine i32 L =", L)
    a = torch.ones((1, 1, L), dtype=torch.int32, device="cuda")
    bx = torch.ones_like(a)
    h0 = torch.full((1, 1), 5, dtype=torch.int32, device="cuda")
    h = sw.affine_scan_i32(a, bx, h0)
    del a, bx
    torch.cuda.synchronize()
    t = torch.tensor([0, 1, (1 << 31) - 7, (1 << 31) - 6, 1 << 31, L - 2, L - 1], device="cuda")
    got = h.reshape(-1).index_select(0, t).cpu().numpy().view(np.uint32).astype(np.int64)
    want = (t.cpu().numpy().astype(np.int64) + 6) % (1 << 32)
    assert np.array_equal(got, want)
    # every state, on the GPU: h_t - t is 6 modulo 2^32 everywhere
    idx = torch.arange(L, device="cuda", dtype=torch.int64)
    diff = (h.reshape(-1).to(torch.int64) - idx) % (1 << 32)
    assert bool((diff == 6).all())


def test_selective_f32_past_2_31_elements(sw):
    """B*D*L = 1 * 16400 * 131072 > 2^31 elements of x, delta and y (8.6 GB
    each): the last rows (element offsets past 2^31) against the oracle."""
    B, D, N, L = 1, 16400, 16, 131072
    _say("case selective f32", B, D, N, L)
    g = torch.Generator(device="cuda").manual_seed(2026)
    x = torch.randn((B, D, L), device="cuda", generator=g)
    dl = torch.nn.functional.softplus(
        torch.randn((B, D, L), device="cuda", generator=g) * 0.5 - 4.0)
    A = -torch.exp(torch.rand((D, N), device="cuda", generator=g) * float(np.log(16.0)))
    Bm = torch.randn((B, L, N), device="cuda", generator=g)
    Cm = torch.randn((B, L, N), device="cuda", generator=g)
    Dk = torch.randn((D,), device="cuda", generator=g)
    y, hl = sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk)
    torch.cuda.synchronize()
    rows = np.array([0, D // 2, D - 17, D - 2, D - 1])
    assert rows[-1] * L > (1 << 31)
    ri = torch.as_tensor(rows, device="cuda")
    xs = x[0].index_select(0, ri).cpu().numpy()[None]
    ds = dl[0].index_select(0, ri).cpu().numpy()[None]
    o = oracle.selective_scan(xs, ds, A.index_select(0, ri).cpu().numpy(), Bm.cpu().numpy(),
                              Cm.cpu().numpy(), Dk.index_select(0, ri).cpu().numpy(), bounds=True)
    got = y[0].index_select(0, ri).cpu().numpy()[None]
    assert_gate(fp_gate(got, o["y"], o["y_mag"], o["y_sens"]), "large selective y")
    hg = hl[0].index_select(0, ri).cpu().numpy()[None]
    assert_gate(fp_gate(hg, o["h_last"], o["h_mag"], o["h_sens"]), "large selective h_last")


@pytest.mark.parametrize("L", [(1 << 24) - 200, (1 << 24) + 40])
def test_selective_bwd_long_row_both_addressing_paths(sw, L):
    """Backward over rows of about 2^24 steps: just below the length where a
    workgroup's 8-step checkpoints (16 rows x ceil(L/8) x 16 states x 4
    bytes, with the read-ahead) stop fitting 31-bit byte offsets, where the
    kernel reads through buffer resources, and just above it, where it falls
    back to 64-bit addresses.  Every gradient against the oracle."""
    B, D, N = 1, 3, 4
    _say("case selective bwd long row", B, D, N, L)
    inp = wl.selective_inputs(B, D, N, L, 31, "f32")
    rng = np.random.Generator(np.random.PCG64(36))
    dy = rng.standard_normal((B, D, L)).astype(np.float32)
    dev = lambda v: torch.from_numpy(np.ascontiguousarray(v)).to("cuda")
    g = sw.selective_scan_bwd(dev(inp["x"]), dev(inp["delta"]), dev(inp["A"]), dev(inp["Bm"]),
                              dev(inp["Cm"]), dev(inp["Dskip"]), dev(dy), None)
    torch.cuda.synchronize()
    o = oracle.selective_scan_bwd(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                                  inp["Dskip"], dy, None, bounds=True)
    for k in ("dx", "ddelta", "dA", "dB", "dC", "dDskip", "dh0"):
        if k not in o or g.get(k) is None:
            continue
        assert_gate(fp_gate(g[k].cpu().numpy(), o[k], o["m_" + k]), f"long-row bwd {k}")
