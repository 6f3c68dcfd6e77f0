"""Pins of the oracle's forward recurrence (CPU only).

Each pin is fixed by the paper or by mathematics, not by the oracle's code:
* the dense special case (Sec. 3.1 "Connection to GDN"): with N = d_qk,
  every slot selected and the raw dense key/query as weights, the sparse
  recurrence is Gated DeltaNet, Eq. (gdn-update), written out here densely;
* single-slot closed form (W = R = 1 with unit weight);
* untouched rows stay bit-identical (Sec. 3.1 step 2, last sentence);
* linearity in (M_0, v) jointly, exact state carry across calls, and
  equivariance under a permutation of the value columns;
* the chunk-parallel form of App. A (segmented log-decay, gated sparse inner
  products Eq. (sparse-ip) via the two-pointer merge, triangular solve,
  retrieved / inter / delta-v correction) computed independently here must
  equal the eager recurrence.
"""
import numpy as np
import pytest


def rand_problem(seed, S=2, T=24, N=40, W=4, R=5, dv=6, m0_scale=1.0):
    rng = np.random.default_rng(seed)
    w_idx = np.stack([np.stack([np.sort(rng.choice(N, W, replace=False)) for _ in range(T)])
                      for _ in range(S)]).astype(np.int32)
    r_idx = np.stack([np.stack([np.sort(rng.choice(N, R, replace=False)) for _ in range(T)])
                      for _ in range(S)]).astype(np.int32)
    def sm(a):
        e = np.exp(a - a.max(-1, keepdims=True))
        return e / e.sum(-1, keepdims=True)
    w_val = sm(rng.standard_normal((S, T, W)))
    r_val = sm(rng.standard_normal((S, T, R)))
    v = rng.standard_normal((S, T, dv))
    alpha = rng.uniform(0.05, 0.99, (S, T))
    beta = rng.uniform(0.05, 0.99, (S, T))
    m0 = m0_scale * rng.standard_normal((S, N, dv))
    return dict(w_idx=w_idx, w_val=w_val, r_idx=r_idx, r_val=r_val, v=v, alpha=alpha,
                beta=beta, m0=m0)


def run(oracle_mod, p, save=False, m0=None):
    mem = np.array(p["m0"] if m0 is None else m0, dtype=np.float64, copy=True, order="C")
    out = oracle_mod.scan_fwd(p["w_idx"], p["w_val"], p["r_idx"], p["r_val"], p["v"], p["alpha"],
                              p["beta"], mem, save=save)
    return out, mem


# ------------------------------------------------------------------ GDN
def dense_gdn(S0, K, V, Q, alpha, beta):
    """Eq. (gdn-update): S <- a S + b k (v - a S^T k)^T ; output o_t = S_t^T q_t."""
    S = S0.copy()
    out = []
    for t in range(K.shape[0]):
        k, v, q = K[t], V[t], Q[t]
        S = alpha[t] * S + beta[t] * np.outer(k, v - alpha[t] * S.T @ k)
        out.append(S.T @ q)
    return np.array(out), S


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_reduces_to_gated_deltanet(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    T, dqk, dv = 20, 6, 5
    K = rng.standard_normal((T, dqk))
    Q = rng.standard_normal((T, dqk))
    V = rng.standard_normal((T, dv))
    al = rng.uniform(0.1, 1.0, T)
    be = rng.uniform(0.0, 1.0, T)
    S0 = rng.standard_normal((dqk, dv))
    ids = np.tile(np.arange(dqk, dtype=np.int32), (1, T, 1))
    mem = S0[None].copy()
    y = oracle_mod.scan_fwd(ids, K[None], ids, Q[None], V[None], al[None], be[None], mem)
    y_ref, S_ref = dense_gdn(S0, K, V, Q, al, be)
    np.testing.assert_allclose(y[0], y_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(mem[0], S_ref, rtol=0, atol=1e-12)


def test_single_slot_closed_form(oracle_mod):
    """W = R = 1, weight 1: M[i] <- (1 - b) a M[i] + b v and y = M[i] after the write;
    b = 1 overwrites the slot with v."""
    rng = np.random.default_rng(4)
    T, N, dv = 30, 5, 3
    wi = rng.integers(0, N, (1, T, 1)).astype(np.int32)
    ones = np.ones((1, T, 1))
    v = rng.standard_normal((1, T, dv))
    al = rng.uniform(0.1, 1.0, (1, T))
    be = rng.uniform(0.0, 1.0, (1, T))
    be[0, ::7] = 1.0
    m0 = rng.standard_normal((1, N, dv))
    mem = m0.copy()
    y = oracle_mod.scan_fwd(wi, ones, wi, ones, v, al, be, mem)
    M = m0[0].copy()
    for t in range(T):
        i = wi[0, t, 0]
        M[i] = (1 - be[0, t]) * al[0, t] * M[i] + be[0, t] * v[0, t]
        np.testing.assert_allclose(y[0, t], M[i], rtol=0, atol=1e-13)
        if be[0, t] == 1.0:
            np.testing.assert_allclose(y[0, t], v[0, t], rtol=0, atol=1e-15)
    np.testing.assert_allclose(mem[0], M, rtol=0, atol=1e-13)


def test_untouched_rows_bit_identical(oracle_mod):
    p = rand_problem(10, N=200, T=30)
    _, mem = run(oracle_mod, p)
    for s in range(mem.shape[0]):
        written = np.zeros(200, bool)
        written[p["w_idx"][s].ravel()] = True
        assert (~written).sum() > 50
        np.testing.assert_array_equal(mem[s][~written], p["m0"][s][~written])
        assert not np.array_equal(mem[s][written], p["m0"][s][written])


def test_linearity_in_memory_and_values(oracle_mod):
    p = rand_problem(11)
    q = rand_problem(12)
    c = -0.7
    y1, m1 = run(oracle_mod, p)
    p2 = dict(p, v=q["v"])
    y2, m2 = run(oracle_mod, p2, m0=q["m0"])
    p3 = dict(p, v=p["v"] + c * q["v"])
    y3, m3 = run(oracle_mod, p3, m0=p["m0"] + c * q["m0"])
    np.testing.assert_allclose(y3, y1 + c * y2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(m3, m1 + c * m2, rtol=0, atol=1e-12)


def test_state_carry_is_exact(oracle_mod):
    p = rand_problem(13, T=40)
    y, mem = run(oracle_mod, p)
    T1 = 17
    first = {k: (v[:, :T1] if k != "m0" else v) for k, v in p.items()}
    second = {k: (v[:, T1:] if k != "m0" else v) for k, v in p.items()}
    ya, mema = run(oracle_mod, first)
    yb, memb = run(oracle_mod, second, m0=mema)
    np.testing.assert_array_equal(np.concatenate([ya, yb], 1), y)
    np.testing.assert_array_equal(memb, mem)


def test_value_column_permutation(oracle_mod):
    p = rand_problem(14)
    perm = np.random.default_rng(0).permutation(p["v"].shape[-1])
    y, mem = run(oracle_mod, p)
    pp = dict(p, v=p["v"][..., perm])
    yp, memp = run(oracle_mod, pp, m0=p["m0"][..., perm])
    np.testing.assert_array_equal(yp, y[..., perm])
    np.testing.assert_array_equal(memp, mem[..., perm])


def test_read_sees_same_step_write(oracle_mod):
    """Eq. (sdm-read) reads M_t, after token t's write: reading exactly the slot
    just written with beta = 1 and weight 1 returns v_t."""
    N, dv, T = 8, 4, 3
    wi = np.array([[[2], [5], [2]]], np.int32)
    one = np.ones((1, T, 1))
    v = np.arange(T * dv, dtype=float).reshape(1, T, dv) + 1
    al = np.full((1, T), 0.5)
    be = np.ones((1, T))
    mem = np.full((1, N, dv), 9.0)
    y = oracle_mod.scan_fwd(wi, one, wi, one, v, al, be, mem)
    np.testing.assert_array_equal(y, v)


# ------------------------------------------------------------------ App. A
def two_pointer(Ia, va, la, Ib, vb, lb):
    """Gated sparse inner product of two slot-sorted lists (App. A.2):
    sum over matching slots of va * vb * exp(la - lb)."""
    a = b = 0
    acc = 0.0
    while a < len(Ia) and b < len(Ib):
        if Ia[a] == Ib[b]:
            acc += va[a] * vb[b] * np.exp(la[a] - lb[b])
            a += 1
            b += 1
        elif Ia[a] < Ib[b]:
            a += 1
        else:
            b += 1
    return acc


def chunked_forward(p, s, C):
    """One stream by the chunk-parallel form of App. A.1, chunks of C tokens."""
    wi, wv, ri, rv = p["w_idx"][s], p["w_val"][s], p["r_idx"][s], p["r_val"][s]
    V, al, be = p["v"][s], p["alpha"][s], p["beta"][s]
    M = p["m0"][s].copy()
    T = V.shape[0]
    ys = []
    for c0 in range(0, T, C):
        tok = range(c0, min(T, c0 + C))
        n = len(tok)
        # segmented cumulative log-decay: per slot, running sum of log alpha over
        # the chunk's tokens that write it; lam_w[t][n] after token t's own write,
        # lam_r[t][m] = the value for read slot j_m after token t
        acc = {}
        lam_w, lam_r = [], []
        for t in tok:
            for i in wi[t]:
                acc[i] = acc.get(i, 0.0) + np.log(al[t])
            lam_w.append(np.array([acc[i] for i in wi[t]]))
            lam_r.append(np.array([acc.get(j, 0.0) for j in ri[t]]))
        A = np.zeros((n, n))
        QK = np.zeros((n, n))
        for a, t in enumerate(tok):
            for b, u in enumerate(tok):
                if b < a:
                    A[a, b] = two_pointer(wi[t], wv[t], lam_w[a], wi[u], wv[u], lam_w[b])
                if b <= a:
                    QK[a, b] = two_pointer(ri[t], rv[t], lam_r[a], wi[u], wv[u], lam_w[b])
        Bt = be[c0:c0 + n]
        Msys = np.eye(n) + Bt[:, None] * np.tril(A, -1)
        dV_const = np.linalg.solve(Msys, Bt[:, None] * V[c0:c0 + n])
        Bcorr = np.linalg.solve(Msys, np.diag(-Bt))
        retrieved = np.stack([(wv[t] * np.exp(lam_w[a]))[:, None].T @ M[wi[t]] for a, t in enumerate(tok)])[:, 0]
        inter = np.stack([(rv[t] * np.exp(lam_r[a]))[:, None].T @ M[ri[t]] for a, t in enumerate(tok)])[:, 0]
        dv = dV_const + Bcorr @ retrieved
        ys.append(inter + np.tril(QK) @ dv)
        # write: per-slot decay to the chunk end, plus each token's decayed contribution
        newM = M.copy()
        touched = sorted(acc)
        for i in touched:
            newM[i] = np.exp(acc[i]) * M[i]
        for a, t in enumerate(tok):
            for nn, i in enumerate(wi[t]):
                newM[i] += np.exp(acc[i] - lam_w[a][nn]) * wv[t][nn] * dv[a]
        M = newM
    return np.concatenate(ys), M


@pytest.mark.parametrize("C", [1, 4, 16, 64])
def test_matches_chunk_parallel_form(oracle_mod, C):
    # a small table so that slots are re-used often inside a chunk
    p = rand_problem(20 + C, S=2, T=48, N=12, W=3, R=4, dv=5)
    y, mem = run(oracle_mod, p)
    for s in range(2):
        yc, Mc = chunked_forward(p, s, C)
        np.testing.assert_allclose(yc, y[s], rtol=0, atol=1e-10)
        np.testing.assert_allclose(Mc, mem[s], rtol=0, atol=1e-10)
