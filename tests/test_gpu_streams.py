"""Concurrency: the look-back scratch (ticket counter and carry words) is kept
per (device, stream), and the stream setting is per host thread.  Calls on two
streams, interleaved without synchronisation, and calls from two host threads
each on its own stream, must give the oracle's results bit for bit (int32
ring, multi-chunk rows whose carries cross workgroups by look-back; fused scan
with its sequence chunks chained through carry words)."""
import sys
import threading

import numpy as np
import pytest

import oracle
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


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def test_two_streams_interleaved(sw):
    _say("case two streams")
    ins = [wl.affine_inputs_i32(1, 3, 300001 + 7 * i, 500 + i, "odd") for i in range(2)]
    refs = [oracle.affine_scan_i32(i["a"], i["bx"]) for i in ins]
    dev_in = [(_dev(i["a"]), _dev(i["bx"])) for i in ins]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    outs = [[], []]
    for rep in range(8):
        for k in range(2):
            with torch.cuda.stream(streams[k]):
                outs[k].append(sw.affine_scan_i32(*dev_in[k]))
    torch.cuda.synchronize()
    for k in range(2):
        for o in outs[k]:
            assert np.array_equal(o.cpu().numpy(), refs[k])


def test_two_host_threads_own_streams(sw, monkeypatch):
    """Each thread runs its own stream; the fused scan is cut into chained
    sequence chunks (8-lane kernel, several tasks per wavefront) so that its
    carry words are in use too."""
    _say("case two threads")
    monkeypatch.setenv("SW_SS_LAYOUT", "8")
    monkeypatch.setenv("SW_SS_TASKS_PER_WAVE", "16")
    ai = [wl.affine_inputs_i32(2, 2, 90001 + 5 * i, 600 + i, "odd") for i in range(2)]
    aref = [oracle.affine_scan_i32(i["a"], i["bx"]) for i in ai]
    si = wl.selective_inputs(1, 24, 16, 6000, 601, "f32")
    args = tuple(_dev(si[k]) for k in ("x", "delta", "A", "Bm", "Cm", "Dskip"))
    y_ref, h_ref = sw.selective_scan_fwd(*args)
    torch.cuda.synchronize()
    errors = []

    def worker(k):
        try:
            s = torch.cuda.Stream()
            a, bx = _dev(ai[k]["a"]), _dev(ai[k]["bx"])
            with torch.cuda.stream(s):
                for _ in range(10):
                    h = sw.affine_scan_i32(a, bx)
                    y, hl = sw.selective_scan_fwd(*args)
                    s.synchronize()
                    if not np.array_equal(h.cpu().numpy(), aref[k]):
                        errors.append(f"thread {k}: affine differs")
                    if not (torch.equal(y, y_ref) and torch.equal(hl, h_ref)):
                        errors.append(f"thread {k}: selective differs")
        except Exception as e:  # reported below
            errors.append(f"thread {k}: {e!r}")

    th = [threading.Thread(target=worker, args=(k,)) for k in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in th), "a worker thread did not finish"
    assert not errors, errors
