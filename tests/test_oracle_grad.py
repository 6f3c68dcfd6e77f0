"""Pins of the oracle's backward (CPU only).

* central finite differences (fp64, h = 1e-6) of the oracle's own forward,
  for every gradient the training path produces: v, alpha, beta, M_0, the
  write/read weights, and q, k through the addressing (selection held fixed);
* the dense special case: the oracle's gradients on the embedded Gated
  DeltaNet problem equal finite differences of the textbook dense recurrence
  Eq. (gdn-update);
* undoing the in-place writes (App. A.3) restores M_0 bit for bit.
"""
import numpy as np
import pytest

from tests.test_oracle_scan import dense_gdn, rand_problem

H_FD = 1e-6


def loss_scan(oracle_mod, p, dy, dmT):
    mem = np.array(p["m0"], dtype=np.float64, copy=True, order="C")
    y = oracle_mod.scan_fwd(p["w_idx"], p["w_val"], p["r_idx"], p["r_val"], p["v"], p["alpha"],
                            p["beta"], mem)
    return float((y * dy).sum() + (mem * dmT).sum())


def grads_scan(oracle_mod, p, dy, dmT):
    mem = np.array(p["m0"], dtype=np.float64, copy=True, order="C")
    y, saved = oracle_mod.scan_fwd(p["w_idx"], p["w_val"], p["r_idx"], p["r_val"], p["v"],
                                   p["alpha"], p["beta"], mem, save=True)
    g = oracle_mod.scan_bwd(p["w_idx"], p["w_val"], p["r_idx"], p["r_val"], p["v"], p["alpha"],
                            p["beta"], mem, saved, dy, dmem_T=dmT)
    g["mem_after"] = mem
    return g


def fd(fun, arr, sample, rng):
    """Central differences at `sample` random positions of arr (modified in place)."""
    flat = arr.reshape(-1)
    pos = rng.choice(flat.size, size=min(sample, flat.size), replace=False)
    out = []
    for i in pos:
        x0 = flat[i]
        flat[i] = x0 + H_FD
        fp = fun()
        flat[i] = x0 - H_FD
        fm = fun()
        flat[i] = x0
        out.append((fp - fm) / (2 * H_FD))
    return pos, np.array(out)


def check(an, pos, num, name):
    a = an.reshape(-1)[pos]
    scale = max(1.0, np.abs(num).max())
    err = np.abs(a - num).max() / scale
    assert err < 2e-7, f"{name}: max err {err:.3e}"


@pytest.mark.parametrize("seed", [0, 1])
def test_scan_gradients_finite_difference(oracle_mod, seed):
    p = rand_problem(100 + seed, S=2, T=14, N=10, W=3, R=4, dv=4)
    rng = np.random.default_rng(seed)
    dy = rng.standard_normal(p["v"].shape)
    dmT = rng.standard_normal(p["m0"].shape)
    g = grads_scan(oracle_mod, p, dy, dmT)
    f = lambda: loss_scan(oracle_mod, p, dy, dmT)
    for key, gk in [("v", "dv"), ("alpha", "dalpha"), ("beta", "dbeta"), ("m0", "dmem0"),
                    ("w_val", "dw_val"), ("r_val", "dr_val")]:
        pos, num = fd(f, p[key], 40, rng)
        check(g[gk], pos, num, key)


def test_undo_restores_initial_memory_bit_exact(oracle_mod):
    p = rand_problem(7, S=2, T=30, N=9, W=3, R=3, dv=5)
    dy = np.random.default_rng(0).standard_normal(p["v"].shape)
    g = grads_scan(oracle_mod, p, dy, np.zeros_like(p["m0"]))
    np.testing.assert_array_equal(g["mem_after"], p["m0"])


def test_gated_deltanet_gradients(oracle_mod):
    """Gradients of the dense special case equal finite differences of Eq. (gdn-update)."""
    rng = np.random.default_rng(3)
    T, dqk, dv = 9, 4, 3
    K = rng.standard_normal((T, dqk))
    Q = rng.standard_normal((T, dqk))
    V = rng.standard_normal((T, dv))
    al = rng.uniform(0.2, 1.0, T)
    be = rng.uniform(0.1, 0.9, T)
    S0 = rng.standard_normal((dqk, dv))
    dy = rng.standard_normal((T, dv))
    dST = rng.standard_normal((dqk, dv))
    ids = np.tile(np.arange(dqk, dtype=np.int32), (1, T, 1))
    p = dict(w_idx=ids, w_val=K[None], r_idx=ids, r_val=Q[None], v=V[None], alpha=al[None],
             beta=be[None], m0=S0[None])
    g = grads_scan(oracle_mod, p, dy[None], dST[None])

    def L():
        y, S = dense_gdn(S0, K, V, Q, al, be)
        return float((y * dy).sum() + (S * dST).sum())

    for arr, gk in [(K, "dw_val"), (Q, "dr_val"), (V, "dv"), (al, "dalpha"), (be, "dbeta"),
                    (S0, "dmem0")]:
        pos, num = fd(L, arr, arr.size, rng)
        check(g[gk][0] if gk != "dmem0" else g[gk][0], pos, num, gk)


@pytest.mark.parametrize("codebook", [True, False])
def test_layer_gradients_through_addressing(oracle_mod, codebook):
    """dq, dk through softmax -> outer sum -> sub-key scores, selection fixed."""
    rng = np.random.default_rng(21)
    S, T, s, k, dv = 1, 10, 5, 3, 4
    N = s * s
    dk = 6 if codebook else 2 * s
    xq = rng.standard_normal((S, 1, T, dk))
    xk = rng.standard_normal((S, 1, T, dk))
    cb = rng.standard_normal((1, 2, s, dk // 2)) if codebook else None
    v = rng.standard_normal((S, 1, T, dv))
    al = rng.uniform(0.2, 0.95, (S, 1, T))
    be = rng.uniform(0.1, 0.9, (S, 1, T))
    m0 = rng.standard_normal((S, 1, N, dv))
    dy = rng.standard_normal((S, 1, T, dv))

    def fwd(save=False):
        return oracle_mod.layer_forward(xq, xk, cb, v, al, be, m0, N, k, decide_f32=False, save=save)

    base = fwd(save=True)

    def L():
        o = fwd()
        assert np.array_equal(o["w_idx"], base["w_idx"]) and np.array_equal(o["r_idx"], base["r_idx"])
        return float((o["y"] * dy).sum())

    mem = base["mem"].copy()
    g = oracle_mod.scan_bwd(base["w_idx"], base["w_val"], base["r_idx"], base["r_val"], v, al, be,
                            mem, base["saved"], dy)
    dq = oracle_mod.address_bwd(cb, base["r_idx"], base["r_val"], g["dr_val"], N, dk)
    dkk = oracle_mod.address_bwd(cb, base["w_idx"], base["w_val"], g["dw_val"], N, dk)
    for arr, an, name in [(xq, dq, "q"), (xk, dkk, "k")]:
        pos, num = fd(L, arr, arr.size, rng)
        check(an, pos, num, name)
