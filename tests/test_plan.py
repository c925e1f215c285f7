"""The fused forward's launch plan (sw_selective_scan_plan) checked on the
host: the segment geometry the kernels rely on, for every planned call over a
grid of sizes, and the choices of a 256-CU part on the shapes the GPU tests
run.  Priced for an explicit CU count, the query touches no device, so these
tests need no GPU.

What the kernels need of a segmented call (selective_scan16.hip,
selective_scan_quad.hip): segments of whole 64- / 128-step super-tiles
(16-lane layout, fp32 / bf16 inputs) or of a multiple of 64 steps (quad
layout); a last segment of at least one such unit, since its first words hold
the records of the segment before (48 words in the correction form); at most
16 segments; the quad layout only with fp32 y, whole 32-step tiles and no
checkpoints; checkpoints only from whole-row walks; the correction form only
with fp32 y.
"""
import itertools

import pytest

import paper_2606_00601_amd as sw

ENV = ("SW_SS_QUAD", "SW_SS_SEGMENTS", "SW_SS_SEGFORM", "SW_SS_LAYOUT")


@pytest.fixture(autouse=True)
def _clean_env(monkeypatch):
    for k in ENV:
        monkeypatch.delenv(k, raising=False)


def _check(p, B, D, N, L, dtype, ybf, train):
    where = (B, D, N, L, dtype, ybf, train, p)
    if B * D == 0 or L == 0:
        assert p == {"layout": 0, "segments": 0, "segment_steps": 0, "form": "whole"}, where
        return
    if N != 16 or L % 4:
        assert p["layout"] == 8 and p["segments"] == 1, where
    assert p["layout"] in (4, 8, 16), where
    k, ls = p["segments"], p["segment_steps"]
    assert 1 <= k <= 16, where
    if k == 1:
        assert ls == L and p["form"] == "whole", where
        return
    last = L - (k - 1) * ls
    assert not train, where  # checkpoints are written by whole-row walks
    assert p["form"] in ("records", "correction"), where
    if p["form"] == "correction":
        assert not ybf, where
    if p["layout"] == 4:
        assert not ybf and L % 32 == 0 and p["form"] == "correction", where
        assert ls % 64 == 0 and last >= 64, where
    else:
        unit = 64 if dtype == "f32" else 128
        assert p["layout"] == 16, where
        assert ls % unit == 0 and unit <= last < ls + unit, where


@pytest.mark.parametrize("dtype,ybf", [("f32", False), ("bf16", False), ("f32", True),
                                       ("bf16", True)])
def test_plan_geometry_over_a_grid_of_sizes(dtype, ybf):
    Ls = [1, 4, 64, 100, 160, 520, 1000, 1040, 1056, 2048, 4096, 6000, 8192, 16384, 32768,
          65536, 100000, 131072]
    Ds = [1, 5, 16, 37, 64, 256, 1280, 2560, 5120, 8192]
    n = 0
    for B, D, L in itertools.product((1, 2, 8), Ds, Ls):
        for train in (False, True):
            p = sw.selective_scan_plan(B, D, 16, L, dtype, "bf16" if ybf else "f32", train, 256)
            _check(p, B, D, 16, L, dtype, ybf, train)
            n += 1
    assert n == 3 * len(Ds) * len(Ls) * 2


def test_plan_forced_counts_keep_the_geometry(monkeypatch):
    """Every forced count of either layout and form gives a geometry the
    kernels accept (short rests joined or the length rounded down)."""
    for quad, form in (("0", "1"), ("0", "2"), ("1", None)):
        monkeypatch.setenv("SW_SS_QUAD", quad)
        if form:
            monkeypatch.setenv("SW_SS_SEGFORM", form)
        for k in range(1, 17):
            monkeypatch.setenv("SW_SS_SEGMENTS", str(k))
            for L in (64, 96, 160, 1000, 1056, 2080, 8192, 65504):
                for dtype in ("f32", "bf16"):
                    p = sw.selective_scan_plan(1, 37, 16, L, dtype, "f32", False, 256)
                    _check(p, 1, 37, 16, L, dtype, False, False)
                    assert p["segments"] <= k, (k, L, p)


# the choices of a 256-CU part (the same cases the GPU planner test runs)
_CHOICES = [((1, 1280, 16384), "f32", "f32", (16, 6, 2752, "correction")),
            ((1, 2560, 65536), "f32", "f32", (4, 16, 4096, "correction")),
            ((1, 8192, 4096), "f32", "f32", (16, 1, 4096, "whole")),
            ((1, 1280, 4096), "f32", "bf16", (16, 16, 256, "records")),
            ((1, 5120, 65536), "f32", "f32", (4, 9, 7296, "correction")),
            ((8, 1536, 2048), "bf16", "f32", (16, 1, 2048, "whole")),
            ((4, 2048, 8192), "f32", "f32", (16, 1, 8192, "whole")),
            ((2, 256, 512), "f32", "f32", (16, 8, 64, "records"))]


@pytest.mark.parametrize("case", _CHOICES)
def test_plan_choices_of_a_256_cu_part(case):
    (B, D, L), dt, yt, want = case
    p = sw.selective_scan_plan(B, D, 16, L, dt, yt, False, 256)
    assert (p["layout"], p["segments"], p["segment_steps"], p["form"]) == want, p


def test_plan_training_and_other_N_walk_whole_rows():
    p = sw.selective_scan_plan(1, 5120, 16, 65536, "f32", "f32", True, 256)
    assert (p["layout"], p["segments"]) == (16, 1)
    for N in (1, 8, 17, 64):
        p = sw.selective_scan_plan(1, 5120, N, 65536, "f32", "f32", False, 256)
        assert (p["layout"], p["segments"]) == (8, 1)


def test_plan_errors():
    from paper_2606_00601_amd import ScanWeaverError
    with pytest.raises(ScanWeaverError) as e:
        sw.selective_scan_plan(1, 16, 65, 64, cus=256)
    assert e.value.status == 2  # SW_ERR_UNSUPPORTED
    with pytest.raises(ScanWeaverError) as e:
        sw.selective_scan_plan(1, 16, 32, 64, train=True, cus=256)
    assert e.value.status == 2
    with pytest.raises(ScanWeaverError) as e:
        sw.selective_scan_plan(-1, 16, 16, 64, cus=256)
    assert e.value.status == 1  # SW_ERR_INVALID_ARG
    with pytest.raises(ScanWeaverError):
        sw.selective_scan_plan(1 << 20, 1 << 20, 16, 64, cus=256)
