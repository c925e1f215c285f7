"""The fused forward captured into a HIP graph (through torch's graph capture)
and replayed: every replay, with eager calls and synchronizations between the
replays, gives the eager result bit for bit.

The N = 16 forward takes no scratch memory and allocates nothing, so it can be
captured; the entry points that use the per-stream scratch (the bare scan's
look-back, the chained chunks of the N != 16 kernel) or allocate (the
backward) are not graph-replay safe and are not captured here.
"""
import sys

import numpy as np
import pytest

import workloads as wl

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


def _bf(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda").view(
        torch.bfloat16)


@pytest.mark.parametrize("options", [False, True])
def test_forward_graph_replays_match_eager(sw, options):
    B, D, N, L = 2, 48, 16, 512
    _say("case graph replay", B, D, N, L, "options" if options else "plain")
    inp = wl.selective_inputs(B, D, N, L, 777, "bf16")
    x, dl = _bf(inp["x_bf16"]), _bf(inp["delta_bf16"])
    Bm, Cm = _bf(inp["Bm_bf16"]), _bf(inp["Cm_bf16"])
    A = torch.from_numpy(inp["A"]).to("cuda")
    Dk = torch.from_numpy(inp["Dskip"]).to("cuda")
    kw = {}
    if options:
        rng = np.random.Generator(np.random.PCG64(778))
        kw = dict(z=_bf(wl.bf16_round(rng.standard_normal((B, D, L)).astype(np.float32))),
                  delta_bias=torch.from_numpy(rng.uniform(-2, 0, D).astype(np.float32)).to("cuda"),
                  h0=torch.from_numpy(rng.standard_normal((B, D, N)).astype(np.float32)).to("cuda"),
                  delta_softplus=True)
    y_ref, h_ref = sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, **kw)
    torch.cuda.synchronize()
    y = torch.empty_like(y_ref)
    hl = torch.empty_like(h_ref)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, y=y, h_last=hl, **kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, y=y, h_last=hl, **kw)
    for i in range(4):
        y.fill_(float("nan"))
        hl.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), f"replay {i}: y differs"
        assert torch.equal(hl, h_ref), f"replay {i}: h_last differs"
        # eager work of the program between replays
        y2, h2 = sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, **kw)
        torch.cuda.synchronize()
        assert torch.equal(y2, y_ref) and torch.equal(h2, h_ref)
