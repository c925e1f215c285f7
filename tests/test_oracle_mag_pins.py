"""Pins of the magnitude and sensitivity outputs of the fused and backward
oracles (CPU).

These outputs set the tolerance of every fused and backward parity gate, so
each is rebuilt here from its definition, term by term, in exact rational
arithmetic:

  * the state of Eq. (3) unrolled into the terms of Eq. (5),
        h_t = (prod_{i<=t} a_i) h0 + sum_{k<=t} (prod_{k<i<=t} a_i) u_k,
    with a_t = exp(delta'_t A_n), u_t = delta'_t x_t B_{t,n} and delta' the
    delta after the optional bias and softplus;
  * mag = the sum of the absolute values of those terms, and sens = the same
    sum with each term weighted by the number of a factors in it (the
    first-order change under a relative perturbation of every a);
  * for y = g (sum_n C h + Dskip x), g = silu(z) or 1: its terms are the
    products of g with every C-weighted state term and with Dskip x;
  * for the backward, every gradient written out as the sum of the products
    the chain rule makes of those terms (the adjoint of Eq. (3) unrolled the
    same way), and its magnitude as the sum of their absolute values.

The transcendental values (exp, softplus, sigmoid) are taken as the doubles
libm returns and then treated as exact rationals; the comparison tolerance
(1e-12 relative) is far below any plausible mistake.  Each test also checks
that the mistakes most likely to loosen the gates silently -- a magnitude
doubled, the Dskip x term dropped, the gate left out of y's magnitude, the
weight of a sensitivity term off by one -- would fail it.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle

REL = 1e-12


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _F(v):
    return Fraction(float(v))


def _softplus(v):
    return v + math.log1p(math.exp(-v)) if v > 0 else math.log1p(math.exp(v))


def _close(got, exact):
    """|got - exact| <= REL * |exact| elementwise (exact: Fractions)."""
    got = np.asarray(got, np.float64).ravel()
    ex = np.array([float(e) for e in np.asarray(exact, dtype=object).ravel()])
    return bool(np.all(np.abs(got - ex) <= REL * np.abs(ex) + 1e-300))


def _fails(got, exact):
    return not _close(got, exact)


def _problem(seed, B, D, N, L, opts):
    rng = _rng(seed)
    f32 = lambda a: np.asarray(a, np.float32)
    p = {
        "x": f32(rng.standard_normal((B, D, L))),
        "delta": f32(rng.uniform(-1.0, 0.5, (B, D, L)) if "softplus" in opts
                     else rng.uniform(0.05, 0.6, (B, D, L))),
        "A": f32(-rng.uniform(0.3, 2.0, (D, N))),
        "Bm": f32(rng.standard_normal((B, L, N))),
        "Cm": f32(rng.standard_normal((B, L, N))),
        "Dskip": f32(rng.standard_normal(D)) if "D" in opts else None,
        "z": f32(2 * rng.standard_normal((B, D, L))) if "z" in opts else None,
        "delta_bias": f32(rng.uniform(-0.5, 0.5, D)) if "bias" in opts else None,
        "h0": f32(rng.standard_normal((B, D, N))) if "h0" in opts else None,
        "softplus": "softplus" in opts,
    }
    dy = f32(rng.standard_normal((B, D, L)))
    dhl = f32(rng.standard_normal((B, D, N))) if "dhl" in opts else None
    return p, dy, dhl


class _Row:
    """Every term of Eq. (5) and of the output of one (b, d) row, exactly."""

    def __init__(self, p, b, d):
        L = p["x"].shape[2]
        N = p["A"].shape[1]
        self.L, self.N = L, N
        raw = [float(p["delta"][b, d, t]) + (float(p["delta_bias"][d])
                                             if p["delta_bias"] is not None else 0.0)
               for t in range(L)]
        dl = [_softplus(v) if p["softplus"] else v for v in raw]
        self.sg = [Fraction(1.0 / (1.0 + math.exp(-v))) if p["softplus"] else Fraction(1)
                   for v in raw]
        self.dl = [Fraction(v) for v in dl]
        self.x = [_F(p["x"][b, d, t]) for t in range(L)]
        self.Bv = [[_F(p["Bm"][b, t, n]) for n in range(N)] for t in range(L)]
        self.Cv = [[_F(p["Cm"][b, t, n]) for n in range(N)] for t in range(L)]
        self.An = [_F(p["A"][d, n]) for n in range(N)]
        self.a = [[Fraction(math.exp(dl[t] * float(p["A"][d, n]))) for n in range(N)]
                  for t in range(L)]
        self.Dx = [(_F(p["Dskip"][d]) if p["Dskip"] is not None else Fraction(0)) * self.x[t]
                   for t in range(L)]
        self.Dr = _F(p["Dskip"][d]) if p["Dskip"] is not None else Fraction(0)
        if p["z"] is not None:
            zs = [float(p["z"][b, d, t]) for t in range(L)]
            sig = [1.0 / (1.0 + math.exp(-z)) for z in zs]
            self.g = [Fraction(z * s) for z, s in zip(zs, sig)]
            # silu'(z) = sig + z sig (1 - sig): two terms
            self.gp_terms = [(Fraction(s), Fraction(z) * Fraction(s) * (1 - Fraction(s)))
                             for z, s in zip(zs, sig)]
        else:
            self.g = [Fraction(1)] * L
            self.gp_terms = [(Fraction(0), Fraction(0))] * L
        h0 = [_F(p["h0"][b, d, n]) if p["h0"] is not None else Fraction(0) for n in range(N)]
        # H[n][t + 1] = list of (term, number of a factors) for the state after step t;
        # H[n][0] = the initial state.
        self.H = []
        for n in range(N):
            rows = [[(h0[n], 0)]]
            for t in range(L):
                terms = []
                p0 = Fraction(1)
                for i in range(t + 1):
                    p0 *= self.a[i][n]
                terms.append((p0 * h0[n], t + 1))
                for k in range(t + 1):
                    pk = Fraction(1)
                    for i in range(k + 1, t + 1):
                        pk *= self.a[i][n]
                    terms.append((pk * self.dl[k] * self.x[k] * self.Bv[k][n], t - k))
                rows.append(terms)
            self.H.append(rows)

    def state_terms(self, n, t):
        """terms of h_t (t = -1: the initial state)."""
        return [v for v, _ in self.H[n][t + 1]]

    def mag(self, n, t):
        return sum(abs(v) for v, _ in self.H[n][t + 1])

    def sens(self, n, t):
        return sum(abs(v) * k for v, k in self.H[n][t + 1])

    def s_terms(self, t):
        """terms of the output before the gate, sum_n C h + Dskip x."""
        out = [self.Dx[t]]
        for n in range(self.N):
            out += [self.Cv[t][n] * v for v in self.state_terms(n, t)]
        return out


# ------------------------------------------------------------------ forward

FWD_OPTS = [("D",), ("D", "h0", "z", "bias", "softplus"), ()]


@pytest.mark.parametrize("opts", FWD_OPTS)
def test_fused_mag_and_sens_match_their_definitions(opts):
    B, D, N, L = 2, 2, 3, 9
    p, _, _ = _problem(701 + len(opts), B, D, N, L, opts)
    o = oracle.selective_scan(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                              z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                              delta_softplus=p["softplus"], bounds=True)
    for b in range(B):
        for d in range(D):
            r = _Row(p, b, d)
            y_mag, y_sens, y_val = [], [], []
            y_mag_nogate, y_mag_noD, y_sens_shift = [], [], []
            for t in range(L):
                g = abs(r.g[t])
                m = sum(abs(r.Cv[t][n]) * r.mag(n, t) for n in range(N)) + abs(r.Dx[t])
                s = sum(abs(r.Cv[t][n]) * r.sens(n, t) for n in range(N))
                y_mag.append(g * m)
                y_sens.append(g * s)
                y_val.append(r.g[t] * sum(r.s_terms(t)))
                y_mag_nogate.append(m)
                y_mag_noD.append(g * (m - abs(r.Dx[t])))
                # a sensitivity whose weights count one factor too many
                y_sens_shift.append(g * sum(abs(r.Cv[t][n]) * (r.sens(n, t) + r.mag(n, t))
                                            for n in range(N)))
            assert _close(o["y"][b, d], y_val)  # the value is the sum of the terms
            assert _close(o["y_mag"][b, d], y_mag)
            assert _close(o["y_sens"][b, d], y_sens)
            h_mag = [r.mag(n, L - 1) for n in range(N)]
            h_sens = [r.sens(n, L - 1) for n in range(N)]
            assert _close(o["h_mag"][b, d], h_mag)
            assert _close(o["h_sens"][b, d], h_sens)
            # the comparison above catches the mistakes that would loosen the gates
            assert _fails(2 * o["y_mag"][b, d], y_mag)
            assert _fails(2 * o["h_mag"][b, d], h_mag)
            assert _fails(0.5 * o["y_sens"][b, d], y_sens)
            assert _fails(o["y_sens"][b, d], y_sens_shift)
            if "D" in opts:
                assert _fails(o["y_mag"][b, d], y_mag_noD)
            if "z" in opts:
                assert _fails(o["y_mag"][b, d], y_mag_nogate)


def test_fused_mag_drops_nothing_with_cancelling_terms():
    """Terms of opposite sign: y sums to ~0 while its magnitude stays the sum
    of absolute values (C = (1, -1) on two equal states)."""
    L = 6
    x = np.ones((1, 1, L), np.float32)
    delta = np.full((1, 1, L), 0.25, np.float32)
    A = np.array([[-1.0, -1.0]], np.float32)
    Bm = np.ones((1, L, 2), np.float32)
    Cm = np.tile(np.array([1.0, -1.0], np.float32), (1, L, 1))
    o = oracle.selective_scan(x, delta, A, Bm, Cm, None, bounds=True)
    assert np.all(o["y"] == 0.0)
    # state magnitude of one lane, by Eq. (5): sum_k e^{-(t-k)/4} / 4
    a = Fraction(math.exp(-0.25))
    for t in range(L):
        m = sum(a ** (t - k) * Fraction(1, 4) for k in range(t + 1))
        assert abs(o["y_mag"][0, 0, t] - float(2 * m)) <= REL * float(2 * m)


# ------------------------------------------------------------------ backward

BWD_OPTS = [("z", "bias", "softplus", "h0", "dhl", "D"), ("D",), ("h0", "dhl")]


@pytest.mark.parametrize("opts", BWD_OPTS)
def test_bwd_values_and_magnitudes_match_their_definitions(opts):
    B, D, N, L = 2, 2, 3, 7
    p, dy, dhl = _problem(801 + len(opts), B, D, N, L, opts)
    g = oracle.selective_scan_bwd(p["x"], p["delta"], p["A"], p["Bm"], p["Cm"], p["Dskip"],
                                  dy, dhl, z=p["z"], delta_bias=p["delta_bias"], h0=p["h0"],
                                  delta_softplus=p["softplus"], bounds=True)
    # batch sums of dB, dC: lists of terms per (b, t, n)
    dB_terms = [[[[] for _ in range(N)] for _ in range(L)] for _ in range(B)]
    dC_terms = [[[[] for _ in range(N)] for _ in range(L)] for _ in range(B)]
    dA_terms = [[[] for _ in range(N)] for _ in range(D)]
    dD_terms = [[] for _ in range(D)]
    dbias_terms = [[] for _ in range(D)]
    for b in range(B):
        for d in range(D):
            r = _Row(p, b, d)
            ds = [_F(dy[b, d, t]) * r.g[t] for t in range(L)]
            dh_last = [_F(dhl[b, d, n]) if dhl is not None else Fraction(0) for n in range(N)]
            # lam_t: the adjoint of the state after step t, as a list of terms
            lam = []
            for n in range(N):
                ln = []
                for t in range(L):
                    terms = []
                    for s in range(t, L):
                        pr = Fraction(1)
                        for i in range(t + 1, s + 1):
                            pr *= r.a[i][n]
                        terms.append(pr * ds[s] * r.Cv[s][n])
                    pr = Fraction(1)
                    for i in range(t + 1, L):
                        pr *= r.a[i][n]
                    terms.append(pr * dh_last[n])
                    ln.append(terms)
                lam.append(ln)
            dx_t, ddl_t, dz_t = [], [], []
            for t in range(L):
                tx = [ds[t] * r.Dr]
                td = []
                for n in range(N):
                    prev = r.state_terms(n, t - 1)
                    for lv in lam[n][t]:
                        tx.append(lv * r.dl[t] * r.Bv[t][n])
                        td.append(lv * r.x[t] * r.Bv[t][n] * r.sg[t])
                        td += [lv * r.a[t][n] * r.An[n] * hv * r.sg[t] for hv in prev]
                        dA_terms[d][n] += [lv * r.a[t][n] * hv * r.dl[t] for hv in prev]
                        dB_terms[b][t][n].append(lv * r.dl[t] * r.x[t])
                    dC_terms[b][t][n] += [ds[t] * hv for hv in r.state_terms(n, t)]
                dx_t.append(tx)
                ddl_t.append(td)
                dbias_terms[d] += td
                dD_terms[d].append(ds[t] * r.x[t])
                if p["z"] is not None:
                    dz_t.append([_F(dy[b, d, t]) * sv * gv
                                 for sv in r.s_terms(t) for gv in r.gp_terms[t]])

            def chk(name, got, mgot, term_lists):
                val = [sum(ts) for ts in term_lists]
                mag = [sum(abs(v) for v in ts) for ts in term_lists]
                assert _close(got, val), name
                assert _close(mgot, mag), "m_" + name
                assert _fails(2 * np.asarray(mgot), mag), "m_" + name

            chk("dx", g["dx"][b, d], g["m_dx"][b, d], dx_t)
            chk("ddelta", g["ddelta"][b, d], g["m_ddelta"][b, d], ddl_t)
            if p["z"] is not None:
                chk("dz", g["dz"][b, d], g["m_dz"][b, d], dz_t)
            dh0 = [[r.a[0][n] * lv for lv in lam[n][0]] for n in range(N)]
            chk("dh0", g["dh0"][b, d], g["m_dh0"][b, d], dh0)
            if "D" in opts:  # the Dskip ds term of dx is visible in its magnitude
                mag_noD = [sum(abs(v) for v in ts[1:]) for ts in dx_t]
                assert _fails(g["m_dx"][b, d], mag_noD)
    for d in range(D):
        val = [sum(ts) for ts in dA_terms[d]]
        mag = [sum(abs(v) for v in ts) for ts in dA_terms[d]]
        assert _close(g["dA"][d], val) and _close(g["m_dA"][d], mag)
        assert _fails(2 * g["m_dA"][d], mag)
    for name, terms in (("dDskip", dD_terms), ("ddelta_bias", dbias_terms)):
        val = [sum(ts) for ts in terms]
        mag = [sum(abs(v) for v in ts) for ts in terms]
        assert _close(g[name], val), name
        assert _close(g["m_" + name], mag), "m_" + name
    for name, terms in (("dB", dB_terms), ("dC", dC_terms)):
        flat = [ts for bb in terms for tt in bb for ts in tt]
        val = [sum(ts) for ts in flat]
        mag = [sum(abs(v) for v in ts) for ts in flat]
        assert _close(g[name], val), name
        assert _close(g["m_" + name], mag), "m_" + name
        assert _fails(2 * g["m_" + name], mag), "m_" + name


# ------------------------------------------------------------------ softplus

@pytest.mark.parametrize("v,sp,sig", [(800.0, 800.0, 1.0), (-800.0, 0.0, 0.0),
                                      (30.0, 30.0 + math.exp(-30.0), 1.0 / (1.0 + math.exp(-30.0))),
                                      (0.0, math.log(2.0), 0.5)])
def test_softplus_far_from_zero(v, sp, sig):
    """softplus(v) = log(1 + e^v) is v itself far above zero (e^v overflows
    fp64 beyond v = 709) and e^v far below (e^-800 is below the smallest
    fp64, so 0).  N = 1, A = 0, x = B = C = 1 make y_t the running sum of
    softplus(delta + bias), i.e. (t + 1) softplus(v)."""
    L = 16
    ones = np.ones((1, L, 1), np.float32)
    x = np.ones((1, 1, L), np.float32)
    A = np.zeros((1, 1), np.float32)
    delta = np.full((1, 1, L), v / 2, np.float32)
    bias = np.array([v / 2], np.float32)
    o = oracle.selective_scan(x, delta, A, ones, ones, np.zeros(1, np.float32),
                              delta_bias=bias, delta_softplus=True)
    t = np.arange(1, L + 1, dtype=np.float64)
    assert np.all(np.isfinite(o["y"]))
    np.testing.assert_allclose(o["y"][0, 0], t * sp, rtol=1e-15, atol=0)
    dy = np.ones((1, 1, L), np.float32)
    g = oracle.selective_scan_bwd(x, delta, A, ones, ones, None, dy, None, delta_bias=bias,
                                  delta_softplus=True)
    # d y_s / d delta_t = sigmoid(v) for every s >= t; sigmoid(800) = 1, sigmoid(-800) = 0
    np.testing.assert_allclose(g["ddelta"][0, 0], (L - np.arange(L)) * sig, rtol=1e-15, atol=0)
