"""Pins of the oracle to facts that do not come from the oracle itself.

The paper prints no output values, so the oracle is pinned by:
  * brute force of the unrolled closed form, Sec. 3.2 Eq. (5), in exact
    rational arithmetic (fp inputs are exact binary fractions) and in exact
    integers modulo 2^32;
  * closed forms: constant a (geometric series), a = 1 (prefix sum), a = 0,
    and in Z/2^32 a = 2 and a = -1;
  * the algebra of Eq. (7): associativity, the identity pair, the
    non-commutativity that fixes the operand order, and split invariance
    (a segment's aggregate carries the state across a cut);
  * the hand-worked four-leaf tree of Fig. 2 (tests/golden);
  * for the fused form: exact rational brute force with a rounded to fp32,
    reduction to the bare recurrence, and the closed forms A = 0, a = 0
    (delta*A <= -800), B = 0 and a constant-parameter geometric series that
    fixes exp(delta*A) (base e, sign as given);
  * for the plain fp32 loop of the fused form: a float32 replica of its
    operation order (exact when a = 1), exactness on integer data, and the
    a-priori rounding bound of a sequential fp32 recurrence.
All of these run on the CPU.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
MASK = (1 << 32) - 1


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _frac(v):
    return Fraction(float(v))


def _brute_eq5(a_row, u_row, h0):
    """Eq. (5): h_t = (prod_{i<=t} a_i) h0 + sum_k (prod_{k<i<=t} a_i) u_k, exactly."""
    a = [_frac(v) for v in a_row]
    u = [_frac(v) for v in u_row]
    out = []
    for t in range(len(a)):
        p = Fraction(1)
        for i in range(t + 1):
            p *= a[i]
        s = p * _frac(h0)
        for k in range(t + 1):
            p = Fraction(1)
            for i in range(k + 1, t + 1):
                p *= a[i]
            s += p * u[k]
        out.append(s)
    return out


def _brute_eq5_int(a_row, u_row, h0):
    a = [int(v) & MASK for v in a_row]
    u = [int(v) & MASK for v in u_row]
    out = []
    for t in range(len(a)):
        p = 1
        for i in range(t + 1):
            p = (p * a[i]) & MASK
        s = (p * (int(h0) & MASK)) & MASK
        for k in range(t + 1):
            p = 1
            for i in range(k + 1, t + 1):
                p = (p * a[i]) & MASK
            s = (s + p * u[k]) & MASK
        out.append(s)
    return np.array(out, dtype=np.uint64).astype(np.uint32).view(np.int32)


# ---------------------------------------------------------------- bare, fp64

@pytest.mark.parametrize("seed,L", [(101, 1), (102, 7), (103, 24)])
def test_fp_matches_eq5_bruteforce(seed, L):
    rng = _rng(seed)
    rows = 3
    a = rng.uniform(-1.2, 1.2, size=(rows, L)).astype(np.float32)
    bx = rng.standard_normal(size=(rows, L)).astype(np.float32)
    h0 = rng.standard_normal(size=(rows,)).astype(np.float32)
    h, mag, sens = oracle.affine_scan(a, bx, h0, bounds=True)
    for r in range(rows):
        exact = _brute_eq5(a[r], bx[r], h0[r])
        for t in range(L):
            tol = 1e-14 * (mag[r, t] + sens[r, t]) + 1e-300
            assert abs(h[r, t] - float(exact[t])) <= tol


def test_bounds_match_their_definitions():
    """mag_t is the abs-sum of the Eq. (5) terms; sens_t = sum (t-k)|prod a||u_k|."""
    rng = _rng(7)
    L = 12
    a = rng.uniform(-1.1, 1.1, size=(1, L)).astype(np.float32)
    bx = rng.standard_normal(size=(1, L)).astype(np.float32)
    h0 = np.array([0.75], np.float32)
    h, mag, sens = oracle.affine_scan(a, bx, h0, bounds=True)
    av = [abs(_frac(v)) for v in a[0]]
    uv = [abs(_frac(v)) for v in bx[0]]
    for t in range(L):  # state index t is h_{t+1} in the 1-based notation
        m = abs(_frac(h0[0]))
        for i in range(t + 1):
            m *= av[i]
        s = m * (t + 1)
        for k in range(t + 1):
            p = Fraction(1)
            for i in range(k + 1, t + 1):
                p *= av[i]
            m += p * uv[k]
            s += p * uv[k] * (t - k)
        assert abs(mag[0, t] - float(m)) <= 1e-14 * float(m)
        assert abs(sens[0, t] - float(s)) <= 1e-14 * float(s) + 1e-300
        assert abs(h[0, t]) <= mag[0, t] * (1 + 1e-15)


def test_geometric_series_closed_form():
    """Constant a = c, constant u = v: h_t = c^t h0 + v (1 - c^t) / (1 - c)."""
    c, v, h0, L = np.float32(0.96875), np.float32(0.5), np.float32(2.0), 300
    a = np.full((1, L), c, np.float32)
    bx = np.full((1, L), v, np.float32)
    h = oracle.affine_scan(a, bx, np.array([h0]))[0]
    t = np.arange(1, L + 1, dtype=np.float64)
    ref = float(c) ** t * float(h0) + float(v) * (1 - float(c) ** t) / (1 - float(c))
    np.testing.assert_allclose(h, ref, rtol=1e-13, atol=0)


def test_unit_a_is_prefix_sum_exact():
    rng = _rng(8)
    L = 5000
    u = rng.integers(-1000, 1000, size=(2, L)).astype(np.float32)
    h0 = np.array([3.0, -7.0], np.float32)
    h = oracle.affine_scan(np.ones_like(u), u, h0)
    ref = np.cumsum(u.astype(np.float64), axis=1) + h0[:, None]
    assert np.array_equal(h, ref)


def test_zero_a_forgets_state():
    rng = _rng(9)
    u = rng.standard_normal(size=(3, 50)).astype(np.float32)
    h = oracle.affine_scan(np.zeros_like(u), u, np.array([5, 6, 7], np.float32))
    assert np.array_equal(h, u.astype(np.float64))


def test_empty_and_single_step():
    h = oracle.affine_scan(np.zeros((3, 0), np.float32), np.zeros((3, 0), np.float32))
    assert h.shape == (3, 0)
    h = oracle.affine_scan(np.array([[0.5]], np.float32), np.array([[2.0]], np.float32),
                           np.array([4.0], np.float32))
    assert h[0, 0] == 0.5 * 4.0 + 2.0


# ---------------------------------------------------------------- bare, int32

@pytest.mark.parametrize("seed,L,variant", [(111, 1, "u"), (112, 9, "u"), (113, 33, "odd"),
                                            (114, 40, "h0")])
def test_int_matches_eq5_bruteforce(seed, L, variant):
    rng = _rng(seed)
    rows = 3
    a = rng.integers(-2 ** 31, 2 ** 31, size=(rows, L), dtype=np.int64).astype(np.int32)
    if variant == "odd":
        a |= 1
    bx = rng.integers(-2 ** 31, 2 ** 31, size=(rows, L), dtype=np.int64).astype(np.int32)
    h0 = (rng.integers(-2 ** 31, 2 ** 31, size=(rows,), dtype=np.int64).astype(np.int32)
          if variant == "h0" else None)
    h = oracle.affine_scan_i32(a, bx, h0)
    for r in range(rows):
        ref = _brute_eq5_int(a[r], bx[r], 0 if h0 is None else h0[r])
        assert np.array_equal(h[r], ref)


def test_int_closed_forms():
    rng = _rng(12)
    L = 200
    u = rng.integers(-2 ** 31, 2 ** 31, size=(1, L), dtype=np.int64).astype(np.int32)
    uu = [int(v) & MASK for v in u[0]]
    h0 = 123456789
    # a = 1: prefix sum mod 2^32
    h = oracle.affine_scan_i32(np.ones_like(u), u, np.array([h0], np.int32))[0]
    acc, ref = h0, []
    for v in uu:
        acc = (acc + v) & MASK
        ref.append(acc)
    assert np.array_equal(h.view(np.uint32), np.array(ref, np.uint32))
    # a = 2: h_t = 2^t h0 + sum_k 2^(t-k) u_k mod 2^32 (only the last 32 terms survive)
    h = oracle.affine_scan_i32(np.full_like(u, 2), u, np.array([h0], np.int32))[0]
    for t in range(L):
        s = (pow(2, t + 1, 1 << 32) * h0) & MASK
        for k in range(max(0, t - 40), t + 1):
            s = (s + pow(2, t - k, 1 << 32) * uu[k]) & MASK
        assert int(h.view(np.uint32)[t]) == s
    # a = -1: alternating sum
    h = oracle.affine_scan_i32(np.full_like(u, -1), u, np.array([h0], np.int32))[0]
    for t in range(L):
        s = ((-1) ** (t + 1) * h0) & MASK
        for k in range(t + 1):
            s = (s + (-1) ** (t - k) * uu[k]) & MASK
        assert int(h.view(np.uint32)[t]) == s


# ---------------------------------------------------------------- Eq. (7)

def test_compose_associative_identity_noncommutative_u32():
    rng = _rng(21)
    p = rng.integers(0, 2 ** 32, size=(3000, 3, 2), dtype=np.uint64)
    ident = (1, 0)
    noncomm = 0
    for (p1, p2, p3) in p:
        left = oracle.compose_u32(oracle.compose_u32(p3, p2), p1)
        right = oracle.compose_u32(p3, oracle.compose_u32(p2, p1))
        assert left == right
        assert oracle.compose_u32(ident, p1) == (int(p1[0]), int(p1[1]))
        assert oracle.compose_u32(p1, ident) == (int(p1[0]), int(p1[1]))
        if oracle.compose_u32(p2, p1) != oracle.compose_u32(p1, p2):
            noncomm += 1
    assert noncomm > 2900  # the operand order matters almost always


def test_compose_associative_fp64():
    rng = _rng(22)
    for _ in range(2000):
        p1, p2, p3 = rng.uniform(-2, 2, size=(3, 2))
        l = oracle.compose(oracle.compose(p3, p2), p1)
        r = oracle.compose(p3, oracle.compose(p2, p1))
        scale = 1 + abs(p3[0] * p2[0] * p1[1]) + abs(p3[0] * p2[1]) + abs(p3[1])
        assert abs(l[0] - r[0]) <= 4 * 2 ** -53 * (1 + abs(p1[0] * p2[0] * p3[0]))
        assert abs(l[1] - r[1]) <= 8 * 2 ** -53 * scale
    # the later segment is the left operand: (a2,u2)(+)(a1,u1) applied to h is a2(a1 h+u1)+u2
    A, U = oracle.compose((3.0, 5.0), (2.0, 7.0))
    h = 11.0
    assert A * h + U == 3.0 * (2.0 * h + 7.0) + 5.0


def test_fig2_four_leaf_tree_golden():
    with open(os.path.join(GOLDEN, "fig2_four_leaf_tree.json")) as f:
        g = json.load(f)
    p1, p2, p3, p4 = [tuple(p) for p in g["pairs"]]
    assert oracle.compose(p2, p1) == tuple(map(float, g["p2_p1"]))
    assert oracle.compose(p4, p3) == tuple(map(float, g["p4_p3"]))
    root = oracle.compose(oracle.compose(p4, p3), oracle.compose(p2, p1))
    assert root == tuple(map(float, g["root"]))
    a = np.array([[p[0] for p in g["pairs"]]], np.int32)
    bx = np.array([[p[1] for p in g["pairs"]]], np.int32)
    h0 = np.array([g["h0"]], np.int32)
    A, U, h = oracle.affine_prefix_i32(a, bx, h0)
    assert A[0].tolist() == [p[0] for p in g["inclusive_prefixes"]]
    assert U[0].tolist() == [p[1] for p in g["inclusive_prefixes"]]
    assert h[0].tolist() == g["states"]
    assert oracle.affine_scan_i32(a, bx, h0)[0].tolist() == g["states"]
    assert oracle.affine_scan(a.astype(np.float32), bx.astype(np.float32),
                              h0.astype(np.float32))[0].tolist() == g["states"]


def test_prefix_route_equals_sequential_route():
    rng = _rng(23)
    a = rng.integers(-2 ** 31, 2 ** 31, size=(4, 777), dtype=np.int64).astype(np.int32)
    bx = rng.integers(-2 ** 31, 2 ** 31, size=(4, 777), dtype=np.int64).astype(np.int32)
    h0 = rng.integers(-2 ** 31, 2 ** 31, size=(4,), dtype=np.int64).astype(np.int32)
    _, _, h_pre = oracle.affine_prefix_i32(a, bx, h0)
    assert np.array_equal(h_pre, oracle.affine_scan_i32(a, bx, h0))
    af = rng.uniform(0.5, 1.0, size=(4, 777)).astype(np.float32)
    bf = rng.standard_normal(size=(4, 777)).astype(np.float32)
    h0f = rng.standard_normal(size=(4,)).astype(np.float32)
    _, _, hp = oracle.affine_prefix(af, bf, h0f)
    hs, mag, sens = oracle.affine_scan(af, bf, h0f, bounds=True)
    assert np.all(np.abs(hp - hs) <= 1e-13 * (mag + sens))


@pytest.mark.parametrize("cut", [1, 17, 500, 999])
def test_split_invariance_u32(cut):
    """h_L = A_{cut+1:L} h_cut + U_{cut+1:L}: the segment aggregate carries the state."""
    rng = _rng(24 + cut)
    L = 1000
    a = (rng.integers(-2 ** 31, 2 ** 31, size=(1, L), dtype=np.int64).astype(np.int32) | 1)
    bx = rng.integers(-2 ** 31, 2 ** 31, size=(1, L), dtype=np.int64).astype(np.int32)
    h0 = np.array([987654321], np.int32)
    h = oracle.affine_scan_i32(a, bx, h0)[0].view(np.uint32)
    Aseg, Useg, _ = oracle.affine_prefix_i32(a[:, cut:], bx[:, cut:])
    Aagg = int(Aseg[0, -1].view(np.uint32))
    Uagg = int(Useg[0, -1].view(np.uint32))
    assert (Aagg * int(h[cut - 1]) + Uagg) & MASK == int(h[-1])
    # and every intermediate state after the cut, from the segment's prefixes
    Ap = Aseg[0].view(np.uint32).astype(np.uint64)
    Up = Useg[0].view(np.uint32).astype(np.uint64)
    rebuilt = (Ap * np.uint64(int(h[cut - 1])) + Up) & np.uint64(MASK)
    assert np.array_equal(rebuilt.astype(np.uint32), h[cut:])


# ---------------------------------------------------------------- fused form

def _fused_inputs(rng, B, D, N, L, dyadic=False):
    if dyadic:  # small integers and powers of two: delta*x*B exact in fp32
        x = rng.integers(-4, 5, size=(B, D, L)).astype(np.float32)
        delta = (2.0 ** rng.integers(-6, -2, size=(B, D, L))).astype(np.float32)
        Bm = rng.integers(-4, 5, size=(B, L, N)).astype(np.float32)
        Cm = rng.integers(-4, 5, size=(B, L, N)).astype(np.float32)
    else:
        x = rng.standard_normal(size=(B, D, L)).astype(np.float32)
        delta = np.logaddexp(0, 0.5 * rng.standard_normal(size=(B, D, L)) - 2).astype(np.float32)
        Bm = rng.standard_normal(size=(B, L, N)).astype(np.float32)
        Cm = rng.standard_normal(size=(B, L, N)).astype(np.float32)
    A = -np.exp(rng.uniform(0, np.log(16), size=(D, N))).astype(np.float32)
    Dskip = rng.standard_normal(size=(D,)).astype(np.float32)
    return x, delta, A, Bm, Cm, Dskip


def test_fused_bruteforce_with_fp32_a():
    """a_mode=1 (a rounded to fp32) makes every quantity an exact binary
    fraction, so Eq. (5) per (b,d,n) plus the projection is checked exactly."""
    rng = _rng(31)
    B, D, N, L = 2, 3, 3, 10
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, a_mode=1, bounds=True)
    for b in range(B):
        for d in range(D):
            yref = [Fraction(float(Dskip[d])) * _frac(x[b, d, t]) for t in range(L)]
            for n in range(N):
                a32 = [np.float32(math.exp(float(delta[b, d, t]) * float(A[d, n])))
                       for t in range(L)]
                u = [_frac(delta[b, d, t]) * _frac(x[b, d, t]) * _frac(Bm[b, t, n])
                     for t in range(L)]
                h = Fraction(0)
                for t in range(L):
                    h = _frac(a32[t]) * h + u[t]
                    yref[t] += _frac(Cm[b, t, n]) * h
                tol = 1e-14 * o["h_mag"][b, d, n] + 1e-300
                assert abs(o["h_last"][b, d, n] - float(h)) <= tol
            for t in range(L):
                assert abs(o["y"][b, d, t] - float(yref[t])) <= 1e-14 * o["y_mag"][b, d, t] + 1e-300


def test_fused_reduces_to_bare_recurrence():
    rng = _rng(32)
    B, D, N, L = 2, 4, 5, 300
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, a_mode=1)
    for b in range(B):
        for d in range(D):
            y = Dskip[d].astype(np.float64) * x[b, d].astype(np.float64)
            for n in range(N):
                a32 = np.exp(delta[b, d].astype(np.float64) * float(A[d, n])).astype(np.float32)
                u = (delta[b, d] * x[b, d] * Bm[b, :, n]).astype(np.float32)  # exact: dyadic
                assert np.array_equal(u.astype(np.float64), delta[b, d].astype(np.float64)
                                      * x[b, d] * Bm[b, :, n])
                h = oracle.affine_scan(a32[None], u[None])[0]
                assert abs(o["h_last"][b, d, n] - h[-1]) <= 1e-12 * (1 + abs(h).max())
                y = y + Cm[b, :, n].astype(np.float64) * h
            np.testing.assert_allclose(o["y"][b, d], y, rtol=1e-12, atol=1e-12)


def test_fused_exp_parameterisation_geometric():
    """N=1, constant delta and A, x=B=C=1, Dskip=0: a = e^{delta A} and
    y_t = delta (1 - a^t) / (1 - a); fixes the base and sign of the exponent."""
    L, dl, Av = 400, 0.0625, -1.5
    x = np.ones((1, 1, L), np.float32)
    delta = np.full((1, 1, L), dl, np.float32)
    A = np.array([[Av]], np.float32)
    ones = np.ones((1, L, 1), np.float32)
    o = oracle.selective_scan(x, delta, A, ones, ones, np.zeros(1, np.float32))
    a = math.exp(dl * Av)
    t = np.arange(1, L + 1)
    ref = dl * (1 - a ** t) / (1 - a)
    np.testing.assert_allclose(o["y"][0, 0], ref, rtol=1e-12)
    np.testing.assert_allclose(o["h_last"][0, 0, 0], ref[-1], rtol=1e-12)


def test_fused_zero_A_is_prefix_sum():
    rng = _rng(33)
    B, D, N, L = 1, 2, 4, 1000
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    A[:] = 0.0
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip)
    for d in range(D):
        y = Dskip[d].astype(np.float64) * x[0, d]
        for n in range(N):
            h = np.cumsum(delta[0, d].astype(np.float64) * x[0, d] * Bm[0, :, n])
            y = y + Cm[0, :, n] * h
            assert o["h_last"][0, d, n] == h[-1]
        assert np.array_equal(o["y"][0, d], y)


def test_fused_underflowed_a_and_zero_B():
    rng = _rng(34)
    B, D, N, L = 2, 3, 4, 64
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    A2 = np.full_like(A, -1e6)  # delta*A <= -800 for every delta here: a == 0
    o = oracle.selective_scan(x, delta, A2, Bm, Cm, Dskip)
    for b in range(B):
        for d in range(D):
            u = delta[b, d, :, None].astype(np.float64) * x[b, d, :, None] * Bm[b]
            ref = (Cm[b] * u).sum(axis=1) + Dskip[d].astype(np.float64) * x[b, d]
            np.testing.assert_allclose(o["y"][b, d], ref, rtol=1e-15, atol=1e-15)
            assert np.array_equal(o["h_last"][b, d], u[-1])
    o = oracle.selective_scan(x, delta, A, np.zeros_like(Bm), Cm, Dskip)
    assert np.array_equal(o["y"], Dskip[None, :, None].astype(np.float64) * x)
    assert not np.any(o["h_last"])


def test_fused_row_subset_matches_full():
    rng = _rng(35)
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, 3, 5, 4, 37)
    full = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip)
    rows = np.array([14, 0, 7, 7, 3])
    sub = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, rows=rows)
    assert np.array_equal(sub["y"], full["y"].reshape(15, 37)[rows])
    assert np.array_equal(sub["h_last"], full["h_last"].reshape(15, 4)[rows])


def test_threads_do_not_change_results():
    rng = _rng(36)
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, 2, 33, 4, 50)
    one = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, threads=1)
    many = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, threads=8)
    assert np.array_equal(one["y"], many["y"])
    assert oracle.threads_used(3, 100) == 3
    assert oracle.threads_used(8, 2) == 2


# ------------------------------------------------------------ plain fp32 loop

def test_seq32_matches_float32_replica_when_a_is_one():
    """With A = 0 every a = expf(0) = 1 exactly, so the plain fp32 loop is fixed
    bit for bit by its order of operations: u = (delta*x)*B, h = a*h + u,
    y += C*h, then y += Dskip*x, each rounded to fp32, no FMA."""
    rng = _rng(41)
    B, D, N, L = 2, 3, 4, 40
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L)
    A[:] = 0.0
    got = oracle.selective_scan_seq32(x, delta, A, Bm, Cm, Dskip)
    f = np.float32
    for b in range(B):
        for d in range(D):
            y = [f(0.0)] * L
            for n in range(N):
                h = f(0.0)
                for t in range(L):
                    u = f(f(delta[b, d, t] * x[b, d, t]) * Bm[b, t, n])
                    h = f(f(f(1.0) * h) + u)
                    y[t] = f(y[t] + f(Cm[b, t, n] * h))
                assert got["h_last"][b, d, n] == h
            for t in range(L):
                assert got["y"][b, d, t] == f(y[t] + f(Dskip[d] * x[b, d, t]))


def test_seq32_exact_on_integer_data():
    """Small-integer data keep every fp32 intermediate exact: the fp32 loop then
    equals the fp64 loop exactly (A = 0)."""
    rng = _rng(42)
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, 2, 3, 4, 64, dyadic=True)
    A[:] = 0.0
    Dskip = rng.integers(-4, 5, size=Dskip.shape).astype(np.float32)
    s = oracle.selective_scan_seq32(x, delta, A, Bm, Cm, Dskip)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip)
    assert np.array_equal(s["y"].astype(np.float64), o["y"])
    assert np.array_equal(s["h_last"].astype(np.float64), o["h_last"])


def test_seq32_within_fp32_rounding_bound():
    """A direct fp32 evaluation stays within a few units of 2^-24 (mag + sens)
    of the fp64 loop: the a-priori bound of a sequential fp32 recurrence.  A
    dropped term, a wrong index or a transposed operand would exceed it."""
    rng = _rng(43)
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, 2, 5, 16, 700)
    s = oracle.selective_scan_seq32(x, delta, A, Bm, Cm, Dskip)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, bounds=True)
    u = 2.0 ** -24
    ey = np.abs(s["y"] - o["y"]) / (u * (o["y_mag"] + o["y_sens"]))
    eh = np.abs(s["h_last"] - o["h_last"]) / (u * (o["h_mag"] + o["h_sens"]))
    assert ey.max() <= 4.0 and eh.max() <= 4.0
    assert np.any(s["y"] != o["y"])  # it is an fp32 evaluation, not the fp64 one


# ------------------------------------------- optional inputs of a Mamba block

def test_fused_h0_split_invariance():
    """A scan of [0, L) equals a scan of [0, m) followed by a scan of [m, L)
    started from the first part's final state: the initial state carries the
    whole history (Sec. 3.2, the chunk-carry property).  Bit for bit on integer
    data (A = 0: every state is exact in fp32); within the fp32 rounding of the
    restart state on general data."""
    rng = _rng(51)
    B, D, N, L, m = 2, 3, 5, 120, 47

    def split(x, delta, A, Bm, Cm, Dskip):
        first = oracle.selective_scan(np.ascontiguousarray(x[:, :, :m]),
                                      np.ascontiguousarray(delta[:, :, :m]), A,
                                      np.ascontiguousarray(Bm[:, :m]),
                                      np.ascontiguousarray(Cm[:, :m]), Dskip)
        second = oracle.selective_scan(np.ascontiguousarray(x[:, :, m:]),
                                       np.ascontiguousarray(delta[:, :, m:]), A,
                                       np.ascontiguousarray(Bm[:, m:]),
                                       np.ascontiguousarray(Cm[:, m:]), Dskip,
                                       h0=first["h_last"].astype(np.float32))
        return first, second

    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    A[:] = 0.0
    Dskip = rng.integers(-3, 4, size=D).astype(np.float32)
    full = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip)
    first, second = split(x, delta, A, Bm, Cm, Dskip)
    assert np.array_equal(first["h_last"].astype(np.float32), first["h_last"])  # exact in fp32
    assert np.array_equal(np.concatenate([first["y"], second["y"]], axis=2), full["y"])
    assert np.array_equal(second["h_last"], full["h_last"])

    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, bounds=True)
    first, second = split(x, delta, A, Bm, Cm, Dskip)
    err = np.abs(second["y"] - o["y"][:, :, m:])
    assert np.all(err <= 2.0 ** -23 * o["y_mag"][:, :, m:] + 1e-300)
    # ignoring h0 would leave the restarted scan off by the decayed history
    cold = oracle.selective_scan(np.ascontiguousarray(x[:, :, m:]),
                                 np.ascontiguousarray(delta[:, :, m:]), A,
                                 np.ascontiguousarray(Bm[:, m:]), np.ascontiguousarray(Cm[:, m:]),
                                 Dskip)
    assert np.abs(cold["y"][:, :, 0] - o["y"][:, :, m]).max() > 1e3 * err[:, :, 0].max()


def test_fused_h0_closed_form():
    """A = 0 (a = 1) and B = 0 (u = 0): the state stays h0 and
    y_t = sum_n C_{t,n} h0_n + Dskip x_t exactly (integer data)."""
    rng = _rng(52)
    B, D, N, L = 2, 3, 4, 30
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    A[:] = 0.0
    Dskip = rng.integers(-3, 4, size=D).astype(np.float32)
    h0 = rng.integers(-5, 6, size=(B, D, N)).astype(np.float32)
    o = oracle.selective_scan(x, delta, A, np.zeros_like(Bm), Cm, Dskip, h0=h0, bounds=True)
    ref = np.einsum("bln,bdn->bdl", Cm.astype(np.float64), h0.astype(np.float64)) \
        + Dskip[None, :, None].astype(np.float64) * x
    assert np.array_equal(o["y"], ref)
    assert np.array_equal(o["h_last"], h0.astype(np.float64))
    assert np.array_equal(o["h_mag"], np.abs(h0).astype(np.float64))


def test_fused_delta_bias_is_an_addition():
    """Without softplus, delta_bias[d] is added to delta: with dyadic data the
    sum is exact in fp32, so it equals the plain loop on delta + bias."""
    rng = _rng(53)
    B, D, N, L = 2, 3, 4, 50
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L, dyadic=True)
    bias = (2.0 ** rng.integers(-6, -2, size=D)).astype(np.float32)
    o = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, delta_bias=bias)
    ref = oracle.selective_scan(x, delta + bias[None, :, None], A, Bm, Cm, Dskip)
    assert np.array_equal(o["y"], ref["y"]) and np.array_equal(o["h_last"], ref["h_last"])


def test_fused_softplus_closed_forms():
    """softplus(v) = log(1 + e^v): ln 2 at 0, v itself far above 0, e^v far
    below.  N = 1, A = 0, x = B = C = 1, Dskip = 0 make y_t the running sum of
    softplus(delta + bias), i.e. (t + 1) softplus(v) for constant v."""
    L = 64
    ones = np.ones((1, L, 1), np.float32)
    x = np.ones((1, 1, L), np.float32)
    A = np.zeros((1, 1), np.float32)
    t = np.arange(1, L + 1, dtype=np.float64)
    for v, sp in ((0.0, math.log(2.0)), (40.0, 40.0), (-40.0, math.exp(-40.0))):
        # split v into delta + bias to exercise both
        delta = np.full((1, 1, L), v / 2, np.float32)
        bias = np.array([v / 2], np.float32)
        o = oracle.selective_scan(x, delta, A, ones, ones, np.zeros(1, np.float32),
                                  delta_bias=bias, delta_softplus=True)
        np.testing.assert_allclose(o["y"][0, 0], t * sp, rtol=1e-14)


def test_fused_output_gate():
    """y <- y * silu(z), silu(z) = z / (1 + e^-z): zero at z = 0, z itself far
    above 0, and silu(z) + silu(-z) = z tanh(z/2) (which a sign error in the
    exponent turns into -z tanh(z/2))."""
    rng = _rng(54)
    B, D, N, L = 2, 3, 4, 40
    x, delta, A, Bm, Cm, Dskip = _fused_inputs(rng, B, D, N, L)
    plain = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, bounds=True)
    zero = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, z=np.zeros_like(x), bounds=True)
    assert not np.any(zero["y"]) and not np.any(zero["y_mag"])
    big = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, z=np.full_like(x, 100.0))
    assert np.array_equal(big["y"], 100.0 * plain["y"])
    z = rng.standard_normal(size=x.shape).astype(np.float32) * 3
    zp = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, z=z, bounds=True)
    zm = oracle.selective_scan(x, delta, A, Bm, Cm, Dskip, z=-z)
    z64 = z.astype(np.float64)
    np.testing.assert_allclose(zp["y"] + zm["y"], plain["y"] * z64 * np.tanh(z64 / 2),
                               rtol=1e-12, atol=1e-14 * plain["y_mag"].max())
    assert np.all(zp["y_mag"] <= plain["y_mag"] * np.abs(z64) * (1 + 1e-15))


# ------------------------------------ Eq. (3)-(4) with input/output projections

@pytest.mark.parametrize("seed,L", [(601, 1), (602, 9), (603, 20)])
def test_proj_matches_eq4_bruteforce(seed, L):
    """y_t = c_t h_t with h from Eq. (5) on u_k = b_k x_k, in exact rationals."""
    rng = _rng(seed)
    rows = 3
    a = rng.uniform(-1.2, 1.2, size=(rows, L)).astype(np.float32)
    b, x, c = (rng.standard_normal(size=(rows, L)).astype(np.float32) for _ in range(3))
    h0 = rng.standard_normal(size=(rows,)).astype(np.float32)
    y, h_last, ym, ys = oracle.affine_proj(a, b, x, c, h0, bounds=True)
    for r in range(rows):
        u = b[r].astype(np.float64) * x[r].astype(np.float64)  # exact: 24 + 24 bits
        exact = _brute_eq5(a[r], u, h0[r])
        for t in range(L):
            yt = _frac(c[r, t]) * exact[t]
            assert abs(y[r, t] - float(yt)) <= 1e-14 * (ym[r, t] + ys[r, t]) + 1e-300
        assert abs(h_last[r] - float(exact[-1])) <= 1e-14 * (abs(float(exact[-1])) + 1) * L


@pytest.mark.parametrize("seed,L", [(611, 1), (612, 40)])
def test_proj_int_matches_eq4_bruteforce(seed, L):
    rng = _rng(seed)
    rows = 2
    a, b, x, c = (rng.integers(-2**31, 2**31, size=(rows, L), dtype=np.int64).astype(np.int32)
                  for _ in range(4))
    a |= 1  # units: every prefix product keeps all bits, so no carry can hide
    h0 = rng.integers(-2**31, 2**31, size=(rows,), dtype=np.int64).astype(np.int32)
    y, h_last = oracle.affine_proj_i32(a, b, x, c, h0)
    for r in range(rows):
        u = ((b[r].astype(np.int64) & MASK) * (x[r].astype(np.int64) & MASK)) & MASK
        h = _brute_eq5_int(a[r], u, h0[r]).view(np.uint32).astype(np.uint64)
        yr = ((c[r].view(np.uint32).astype(np.uint64) * h) & MASK).astype(np.uint32)
        assert np.array_equal(y[r].view(np.uint32), yr)
        assert h_last[r] == h[-1].astype(np.uint32).view(np.int32)


def test_proj_closed_forms():
    """a = 1, b = 1: h is h0 plus the prefix sum of x (exact on integers), so
    y = c (h0 + cumsum x).  Weighted prefix of Eq. (10) with constant
    alpha = 1/2, beta = 1 (x = c = ones): h_t = 2 - (2 - h0) 2^-(t+1)."""
    rng = _rng(621)
    L = 300
    x = rng.integers(-50, 50, size=(2, L)).astype(np.float32)
    c = rng.integers(-4, 5, size=(2, L)).astype(np.float32)
    h0 = np.array([3.0, -7.0], np.float32)
    ones = np.ones((2, L), np.float32)
    y, hl = oracle.affine_proj(ones, ones, x, c, h0)
    expect = c.astype(np.float64) * (h0[:, None] + np.cumsum(x.astype(np.float64), axis=1))
    assert np.array_equal(y, expect)
    assert np.array_equal(hl, h0 + x.astype(np.float64).sum(axis=1))
    half = np.full((2, 40), 0.5, np.float32)
    y, hl = oracle.affine_proj(half, np.ones((2, 40), np.float32), None, None, h0)
    t = np.arange(40)
    expect = 2.0 - (2.0 - h0[:, None].astype(np.float64)) * 2.0 ** -(t + 1)
    assert np.array_equal(y, expect)  # dyadic with < 53 significant bits: exact in fp64
    assert np.array_equal(hl, expect[:, -1])


def test_proj_int_weighted_prefix_closed_form():
    """int32 ring, alpha = -1, beta = 1 (Eq. (10)): h_t alternates between
    1 - h0 and h0 modulo 2^32."""
    L = 7
    a = np.full((1, L), -1, np.int32)
    b = np.ones((1, L), np.int32)
    h0 = np.array([2**31 - 5], np.int32)
    y, hl = oracle.affine_proj_i32(a, b, None, None, h0)
    alt = [(1 - int(h0[0])) & MASK, int(h0[0]) & MASK]
    assert [int(v) & MASK for v in y[0]] == [alt[t % 2] for t in range(L)]
    assert (int(hl[0]) & MASK) == alt[(L - 1) % 2]


def test_proj_empty_sequence_keeps_h0():
    h0 = np.array([1.5, -2.0], np.float32)
    e = np.zeros((2, 0), np.float32)
    y, hl = oracle.affine_proj(e, e, None, None, h0)
    assert y.shape == (2, 0) and np.array_equal(hl, h0.astype(np.float64))
    y, hl = oracle.affine_proj(e, e)
    assert np.array_equal(hl, np.zeros(2))
