"""The entry point that allocates nothing, sw_affine_scan_noalloc, against the
bare scan it varies, sw_affine_scan, through the C ABI.

Both run the same look-back schedule; the only difference is where the
tickets and chunk carries live (a static array cleared by the call, against
the per-stream scratch).  Two calls in a row, the second smaller, must match
sw_affine_scan to the fp32 gate (and the fp64 oracle); on inputs whose every
composition is exact in fp32 (a in {0, 1}, small integer bx) the two must
agree bit for bit, which shows every carry crossed the static scratch
intact.  The largest call the array admits runs; one chunk more is refused
before anything is enqueued.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from gate import assert_gate, fp_gate

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CH = 2048          # steps per look-back chunk
MAX_CHUNKS = 65536  # SW_NOALLOC_MAX_CHUNKS


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


def _ptr(t):
    return None if t is None else t.data_ptr()


def _call(sw, name, a, bx, h0, out):
    B, D, L = a.shape
    with sw._on(a.device):
        st = getattr(sw.lib(), name)(_ptr(a), _ptr(bx), _ptr(h0), _ptr(out), B, D, L)
    return st


def _both(sw, a, bx, h0=None):
    ref = torch.empty_like(a)
    got = torch.full_like(a, float("nan"))
    assert _call(sw, "sw_affine_scan", a, bx, h0, ref) == 0, sw.lib().sw_last_error()
    assert _call(sw, "sw_affine_scan_noalloc", a, bx, h0, got) == 0, sw.lib().sw_last_error()
    torch.cuda.synchronize()
    return got, ref


def _exact_inputs(B, D, L, seed, bmax):
    """a in {0, 1} (mostly 1, so carries reach far), bx integers in [-bmax, bmax]:
    every partial composition is an integer below 2^24, exact in fp32 in any order."""
    g = np.random.default_rng(seed)
    a = (g.random((B, D, L)) < 0.9995).astype(np.float32)
    bx = g.integers(-bmax, bmax + 1, (B, D, L)).astype(np.float32)
    assert bmax * L < 2 ** 24
    return a, bx


def test_two_calls_second_smaller_against_sw_affine_scan(sw):
    # 2 x 3 rows of 147 chunks, then 1 x 2 rows of 49: both take the look-back kernel
    for (B, D, L) in [(2, 3, 300_007), (1, 2, 100_001)]:
        _say("case noalloc fp32", B, D, L)
        inp = wl.affine_inputs(B, D, L, 7000 + L, with_h0=True)
        a = torch.from_numpy(inp["a"]).cuda()
        bx = torch.from_numpy(inp["bx"]).cuda()
        h0 = torch.from_numpy(inp["h0"]).cuda()
        got, ref = _both(sw, a, bx, h0)
        want, mag, sens = oracle.affine_scan(inp["a"], inp["bx"], inp["h0"], bounds=True)
        g = got.cpu().numpy()
        assert_gate(fp_gate(g, ref.cpu().numpy(), mag), f"noalloc vs sw_affine_scan {B}x{D}x{L}")
        assert_gate(fp_gate(g, want, mag, sens), f"noalloc vs oracle {B}x{D}x{L}")


def test_two_calls_second_smaller_bit_exact(sw):
    for (B, D, L, seed) in [(1, 4, 1_000_003, 1), (1, 3, 70_000, 2)]:
        _say("case noalloc exact", B, D, L)
        a, bx = _exact_inputs(B, D, L, 8000 + seed, 8)
        got, ref = _both(sw, torch.from_numpy(a).cuda(), torch.from_numpy(bx).cuda())
        assert torch.equal(got, ref)
        h = got.cpu().numpy()
        assert np.array_equal(h[0, 0, :4096], oracle.affine_scan(a[:, :1, :4096],
                                                                 bx[:, :1, :4096])[0, 0])


@pytest.mark.parametrize("B,D,L", [(1, 5, 2048), (1, 1, 1), (2, 1100, 4100)])
def test_calls_without_scratch(sw, B, D, L):
    # one chunk per row, and enough rows for one workgroup each: no look-back
    _say("case noalloc no scratch", B, D, L)
    inp = wl.affine_inputs(B, D, L, 9000 + L, with_h0=False)
    got, ref = _both(sw, torch.from_numpy(inp["a"]).cuda(), torch.from_numpy(inp["bx"]).cuda())
    want, mag, _ = oracle.affine_scan(inp["a"], inp["bx"], None, bounds=True)
    assert_gate(fp_gate(got.cpu().numpy(), ref.cpu().numpy(), mag), f"no scratch {B}x{D}x{L}")


def test_largest_call_and_one_chunk_more(sw):
    D, L = 32, CH * CH  # 32 rows x 2048 chunks = 65536 chunks, the array's capacity
    assert D * (L // CH) == MAX_CHUNKS
    _say("case noalloc max", 1, D, L)
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    a = (torch.rand((1, D, L), generator=g, device="cuda") < 0.9999).float()
    bx = torch.randint(-1, 2, (1, D, L), generator=g, device="cuda").float()
    got, ref = _both(sw, a, bx)
    assert torch.equal(got, ref)
    # closed form of one row's last state: the sum of bx from the last zero of a on
    # (a_t = 0 gives h_t = bx_t)
    row_a, row_b = a[0, 5].cpu().numpy(), bx[0, 5].cpu().numpy()
    z = np.flatnonzero(row_a == 0)
    start = z[-1] if z.size else 0
    assert got[0, 5, -1].item() == float(row_b[start:].sum(dtype=np.float64))
    del a, bx, got, ref
    _say("case noalloc max + 1 chunk", 1, D, L + 1)
    a = torch.ones((1, D, L + 1), device="cuda")
    bx = torch.zeros_like(a)
    out = torch.full_like(a, 7.0)
    assert _call(sw, "sw_affine_scan_noalloc", a, bx, None, out) == 2
    msg = sw.lib().sw_last_error().decode()
    assert "65568" in msg and "65536" in msg, msg
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing was enqueued
