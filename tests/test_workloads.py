"""The seeded generator: deterministic, the stated recipe, exact bf16 handling."""
import numpy as np

import workloads as wl


def test_deterministic():
    a = wl.selective_inputs(2, 8, 16, 33, 7, "bf16")
    b = wl.selective_inputs(2, 8, 16, 33, 7, "bf16")
    for k in a:
        assert wl.sha256(a[k]) == wl.sha256(b[k])
    c = wl.selective_inputs(2, 8, 16, 33, 8, "bf16")
    assert wl.sha256(a["x"]) != wl.sha256(c["x"])


def test_bf16_round_to_nearest_even():
    one = np.float32(1.0)
    cases = {
        float(one): 0x3F80,
        1.0 + 2.0 ** -8: 0x3F80,            # halfway between 1 and 1+2^-7: even is 1
        1.0 + 3 * 2.0 ** -8: 0x3F82,        # halfway, rounds up to even 1+2^-6
        1.0 + 2.0 ** -8 + 2.0 ** -20: 0x3F81,  # just above halfway
        -2.5: 0xC020,
    }
    vals = np.array(list(cases), np.float32)
    assert wl.bf16_round(vals).tolist() == list(cases.values())
    assert np.array_equal(wl.bf16_widen(wl.bf16_round(vals))[:1], vals[:1])


def test_bf16_values_are_the_widened_bits():
    inp = wl.selective_inputs(1, 4, 16, 50, 3, "bf16")
    for k in ("x", "delta", "Bm", "Cm"):
        assert np.array_equal(wl.bf16_widen(inp[k + "_bf16"]), inp[k])
    assert inp["A"].dtype == np.float32 and inp["Dskip"].dtype == np.float32


def test_affine_recipe():
    inp = wl.affine_inputs(1, 64, 1024, 1)
    a = inp["a"]
    assert a.dtype == np.float32 and a.min() >= 0.9 and a.max() < 1.0
    assert abs(float(inp["bx"].mean())) < 0.05 and abs(float(inp["bx"].std()) - 1) < 0.05
    odd = wl.affine_inputs_i32(1, 3, 500, 12, "odd")
    assert np.all(odd["a"] & 1)
    assert wl.affine_inputs_i32(1, 3, 5, 13, "h0")["h0"].shape == (1, 3)


def test_selective_recipe():
    inp = wl.selective_inputs(2, 64, 16, 512, 2)
    assert inp["x"].shape == (2, 64, 512) and inp["Bm"].shape == (2, 512, 16)
    assert inp["A"].shape == (64, 16) and inp["Dskip"].shape == (64,)
    assert np.all(inp["delta"] > 0) and float(np.median(inp["delta"])) < 0.05
    assert np.all(inp["A"] <= -1.0 + 1e-6) and np.all(inp["A"] >= -16.0 - 1e-4)
    st = wl.selective_inputs(1, 64, 16, 256, 5, stress=True)
    assert np.all(st["A"] < 0) and st["A"].max() > -0.02 and st["A"].min() < -50


def test_workload_table():
    w = wl.workload("selective_bf16_b8_d1536_n16_l2048")
    assert (w.B, w.D, w.N, w.L, w.dtype) == (8, 1536, 16, 2048, "bf16")
    assert w.elems == 8 * 1536 * 16 * 2048
    # six configurations of the target workload, two shapes of the schedule ablation
    assert len(wl.WORKLOADS) == 8
    assert {k for k in wl.WORKLOADS if "ablation" in wl.WORKLOADS[k].note} == {
        "affine_f32_b1_d64_l65536", "affine_f32_b8_d1536_l2048"}
