"""Pins of the oracle's gate producers (Sec. 3.1 step 2) and output epilogue
(Sec. 3.1 step 4, Fig. 2), CPU only.

Gates: alpha = exp(-A softplus(a + b_dt)), beta = sigma(b).  Closed forms at
points where softplus and sigma take exact values (softplus(0) = ln 2,
softplus(ln 2) = ln 3, softplus(ln(e - 1)) = 1, sigma(ln 3) = 3/4), the limits
A = 0 and z -> -inf (no decay), z -> +inf (softplus(z) -> z), the head of
stream s being s mod H, and central finite differences of the forward for
every gradient (dA and db_dt summed over a head's tokens).

Epilogue: o = y rstd gamma phi(g), rstd = 1 / sqrt(mean(y^2) + eps).  A
constant row normalises to its sign; at eps = 0 the norm is invariant to a
positive scale, odd, and has unit mean square; SiLU(ln 3) = (3/4) ln 3;
finite differences of every gradient; at eps = 0 each row's dy is orthogonal
to its y (the consequence of scale invariance)."""
import math

import numpy as np
import pytest

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


# ------------------------------------------------------------------ gates
def test_gates_closed_forms():
    A = np.array([1.0, 2.5, 0.0, 16.0])
    bdt = np.array([0.3, -1.2, 0.7, -0.05])
    H = 4
    # z = a + b_dt at ln(e - 1), 0, ln 2 for the three tokens of every head
    zs = np.array([math.log(math.e - 1.0), 0.0, math.log(2.0)])
    a = np.stack([zs - bdt[h] for h in range(H)])[None]          # [1, H, 3]
    b = np.tile(np.array([0.0, math.log(3.0), -math.log(3.0)]), (1, H, 1))
    al, be = oracle.gates(a, b, A, bdt)
    for h in range(H):
        want = [math.exp(-A[h]), 2.0 ** -A[h], 3.0 ** -A[h]]
        np.testing.assert_allclose(al[0, h], want, rtol=1e-13, atol=0)
    np.testing.assert_allclose(be[0, :, 0], 0.5, rtol=0, atol=1e-16)
    np.testing.assert_allclose(be[0, :, 1], 0.75, rtol=1e-14)
    np.testing.assert_allclose(be[0, :, 2], 0.25, rtol=1e-14)


def test_gates_limits_and_heads():
    H, B, T = 3, 2, 5
    A = np.array([0.0, 4.0, 9.0])
    bdt = np.zeros(H)
    a = np.zeros((B, H, T))
    a[:, :, 0] = -800.0          # softplus underflows to 0: no decay
    a[:, :, 1] = 40.0            # softplus(40) = 40 + 4e-18
    a[:, :, 2:] = _rng(1).standard_normal((B, H, T - 2))
    b = _rng(2).standard_normal((B, H, T)) * 5
    al, be = oracle.gates(a, b, A, bdt)
    assert np.all(al[:, 0] == 1.0), "A = 0 must not decay"
    assert np.all(al[:, :, 0] == 1.0), "z -> -inf must not decay"
    np.testing.assert_allclose(al[:, 1:, 1], np.exp(-40.0 * A[1:])[None].repeat(B, 0), rtol=1e-13)
    assert np.all((al > 0) & (al <= 1)) and np.all((be > 0) & (be < 1))
    # sigma(-b) = 1 - sigma(b)
    _, be_neg = oracle.gates(a, -b, A, bdt)
    np.testing.assert_allclose(be + be_neg, 1.0, rtol=1e-15)
    # the gate of stream (b, h) uses head h's parameters: decay grows with A
    assert np.all(al[:, 2, 2:] <= al[:, 1, 2:])


def test_gates_decrease_in_the_preactivation():
    a = np.linspace(-6, 6, 101)[None, None]
    al, _ = oracle.gates(a, a, np.array([2.0]), np.array([0.1]))
    assert np.all(np.diff(al[0, 0]) < 0)


def _fd(f, x, h=1e-6):
    g = np.empty_like(x)
    for i in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[i] += h
        xm[i] -= h
        g[i] = (f(xp) - f(xm)) / (2 * h)
    return g


def test_gates_bwd_finite_differences():
    rng = _rng(3)
    B, H, T = 2, 3, 4
    a = rng.standard_normal((B, H, T)) * 2
    b = rng.standard_normal((B, H, T)) * 2
    A = rng.uniform(0.0, 16.0, H)
    bdt = np.log(np.expm1(rng.uniform(0.001, 0.1, H)))      # inverse softplus, Sec. 4
    dal = rng.standard_normal((B, H, T))
    dbe = rng.standard_normal((B, H, T))
    da, db, dA, dbdt = oracle.gates_bwd(a, b, A, bdt, dal, dbe)

    def loss(a_, b_, A_, bd_):
        al, be = oracle.gates(a_, b_, A_, bd_)
        return float((al * dal).sum() + (be * dbe).sum())

    np.testing.assert_allclose(da, _fd(lambda x: loss(x, b, A, bdt), a), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(db, _fd(lambda x: loss(a, x, A, bdt), b), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dA, _fd(lambda x: loss(a, b, x, bdt), A), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(dbdt, _fd(lambda x: loss(a, b, A, x), bdt), rtol=1e-6, atol=1e-9)


def test_gates_bwd_closed_form_at_zero():
    # A = 1, z = 0: alpha = 1/2, d alpha/dz = -A alpha sigma(0) = -1/4; d beta/db at 0 = 1/4;
    # d alpha/dA = -softplus(0) alpha = -ln(2)/2
    one = np.ones((1, 1, 1))
    da, db, dA, dbdt = oracle.gates_bwd(0 * one, 0 * one, np.array([1.0]), np.array([0.0]), one, one)
    assert abs(da[0, 0, 0] + 0.25) < 1e-15 and abs(dbdt[0] + 0.25) < 1e-15
    assert abs(db[0, 0, 0] - 0.25) < 1e-15
    assert abs(dA[0] + math.log(2.0) / 2) < 1e-15


# ------------------------------------------------------------------ epilogue
@pytest.mark.parametrize("act", [0, 1])
def test_norm_gate_constant_rows(act):
    dv = 16
    c = np.array([3.0, -0.25, 1e-3])[:, None] * np.ones((3, dv))
    g = np.full((3, dv), math.log(3.0))
    o, rstd = oracle.norm_gate(c, g, np.ones(dv), 0.0, act)
    phi = 0.75 * math.log(3.0) if act else math.log(3.0)
    np.testing.assert_allclose(o, np.sign(c) * phi, rtol=1e-14)
    np.testing.assert_allclose(rstd, 1.0 / np.abs(c[:, 0]), rtol=1e-14)
    # eps enters under the root: rstd = 1 / sqrt(c^2 + eps)
    _, rs = oracle.norm_gate(c, g, np.ones(dv), 0.5, act)
    np.testing.assert_allclose(rs, 1.0 / np.sqrt(c[:, 0] ** 2 + 0.5), rtol=1e-14)


def test_norm_gate_scale_invariance_and_unit_mean_square():
    rng = _rng(5)
    y = rng.standard_normal((6, 24))
    gm = rng.uniform(0.5, 2.0, 24)
    g = rng.standard_normal((6, 24))
    o1, _ = oracle.norm_gate(y, g, gm, 0.0, 1)
    o2, _ = oracle.norm_gate(7.5 * y, g, gm, 0.0, 1)
    o3, _ = oracle.norm_gate(-y, g, gm, 0.0, 1)
    np.testing.assert_allclose(o2, o1, rtol=1e-13)
    np.testing.assert_allclose(o3, -o1, rtol=1e-15)
    on, _ = oracle.norm_gate(y, np.ones_like(y), np.ones(24), 0.0, 0)
    np.testing.assert_allclose((on ** 2).mean(-1), 1.0, rtol=1e-14)
    # gamma scales column c, the gate element c
    ogm, _ = oracle.norm_gate(y, np.ones_like(y), gm, 0.0, 0)
    np.testing.assert_allclose(ogm, on * gm, rtol=1e-14)
    og, _ = oracle.norm_gate(y, g, np.ones(24), 0.0, 0)
    np.testing.assert_allclose(og, on * g, rtol=1e-14)


@pytest.mark.parametrize("act", [0, 1])
@pytest.mark.parametrize("eps", [0.0, 1e-2])
def test_norm_gate_bwd_finite_differences(act, eps):
    rng = _rng(7 + act)
    rows, dv = 3, 8
    y = rng.standard_normal((rows, dv))
    g = rng.standard_normal((rows, dv)) * 2
    gm = rng.uniform(0.5, 2.0, dv)
    do = rng.standard_normal((rows, dv))
    dy, dg, dgm = oracle.norm_gate_bwd(y, g, gm, eps, act, do)

    def loss(y_, g_, gm_):
        return float((oracle.norm_gate(y_, g_, gm_, eps, act)[0] * do).sum())

    np.testing.assert_allclose(dy, _fd(lambda x: loss(x, g, gm), y), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dg, _fd(lambda x: loss(y, x, gm), g), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dgm, _fd(lambda x: loss(y, g, x), gm), rtol=1e-6, atol=1e-8)


def test_norm_gate_bwd_orthogonal_to_y_without_eps():
    rng = _rng(9)
    y = rng.standard_normal((5, 32))
    dy, _, _ = oracle.norm_gate_bwd(y, rng.standard_normal((5, 32)), rng.uniform(0.5, 2, 32), 0.0, 1,
                                    rng.standard_normal((5, 32)))
    assert np.abs((dy * y).sum(-1)).max() < 1e-12
