"""Pins of the oracle's addressing (CPU only).

What fixes the addressing independently of the oracle's own code:
* exhaustive numpy scoring of all N = s*s outer-sum slots, ranked by
  (score descending, slot id ascending), slot id = a*s + b (Sec. 2 outer sum,
  Sec. 3.1 step 1);
* the top-k-of-top-k identity of Sec. 2, checked as oracle two-stage ==
  oracle brute force;
* hand-derived tie cases and closed forms of the softmax (Sec. 4: read and
  write activations are softmax-normalised).
"""
import numpy as np
import pytest


def _numpy_scores(x, cb, s):
    """All N scores of every token, fp64: [B,H,T,s*s] with flat id a*s+b."""
    B, H, T, dk = x.shape
    if cb is None:
        s0, s1 = x[..., :s], x[..., s:]
    else:
        dh = dk // 2
        # cb [H,2,s,dh]: per head, sub-score j of half h = <x_h, cb[h][j]>
        s0 = np.einsum("bhtc,hjc->bhtj", x[..., :dh], cb[:, 0])
        s1 = np.einsum("bhtc,hjc->bhtj", x[..., dh:], cb[:, 1])
    return (s0[..., :, None] + s1[..., None, :]).reshape(B, H, T, s * s)


def _numpy_topk(scores, k):
    """Reference selection by exhaustive sort on (score desc, id asc)."""
    flat = scores.reshape(-1, scores.shape[-1])
    ids = np.arange(flat.shape[-1])
    out = np.empty((flat.shape[0], k), np.int64)
    for r in range(flat.shape[0]):
        order = np.lexsort((ids, -flat[r]))      # primary: -score, secondary: id
        out[r] = np.sort(order[:k])
    return out.reshape(scores.shape[:-1] + (k,))


def _rand_case(rng, B, H, T, s, dk=None, codebook=True):
    if codebook:
        dk = dk or 8
        x = rng.standard_normal((B, H, T, dk))
        cb = rng.standard_normal((H, 2, s, dk // 2))
    else:
        dk = 2 * s
        x = rng.standard_normal((B, H, T, dk))
        cb = None
    return x, cb


@pytest.mark.parametrize("codebook", [True, False])
@pytest.mark.parametrize("decide_f32", [False, True])
def test_selection_matches_exhaustive_numpy(oracle_mod, codebook, decide_f32):
    rng = np.random.default_rng(7)
    for s, k in [(4, 1), (4, 3), (5, 4), (6, 6), (8, 5), (8, 8), (16, 7)]:
        x, cb = _rand_case(rng, 2, 2, 6, s, codebook=codebook)
        N = s * s
        idx, val, score = oracle_mod.address(x, cb, N, k, decide_f32=decide_f32)
        sc = _numpy_scores(x, cb, s)
        ref = _numpy_topk(sc, k)
        np.testing.assert_array_equal(idx, ref)
        # the selected scores are the outer sums of the two sub-scores
        got = np.take_along_axis(sc, idx.astype(np.int64), axis=-1)
        tol = 1e-6 if decide_f32 else 1e-13
        np.testing.assert_allclose(score, got, rtol=0, atol=tol)
        assert np.all(np.diff(idx, axis=-1) > 0), "ids ascending and distinct"


@pytest.mark.parametrize("decide_f32", [False, True])
def test_two_stage_equals_brute_force(oracle_mod, decide_f32):
    """Sec. 2: top_k(s1 (+) s2) == top_k(top_k(s1) (+) top_k(s2)), many seeds."""
    for seed in range(40):
        rng = np.random.default_rng(1000 + seed)
        s = int(rng.integers(2, 12))
        k = int(rng.integers(1, s + 1))
        codebook = bool(seed % 2)
        x, cb = _rand_case(rng, 1, 2, 5, s, dk=6, codebook=codebook)
        a = oracle_mod.address(x, cb, s * s, k, decide_f32=decide_f32)
        b = oracle_mod.address(x, cb, s * s, k, decide_f32=decide_f32, brute=True)
        for u, w in zip(a, b):
            np.testing.assert_array_equal(u, w)


@pytest.mark.parametrize("s,k,codebook", [(40, 40, True), (72, 65, False), (128, 100, True), (128, 128, False)])
def test_large_k_matches_exhaustive_numpy_and_brute_force(oracle_mod, s, k, codebook):
    """k up to 128 (the largest k of the boundary), including k = sqrt(N): the
    two-stage selection against an exhaustive numpy sort of all N scores and
    against the oracle's own brute force."""
    rng = np.random.default_rng(11 + s + k)
    x, cb = _rand_case(rng, 1, 1, 3, s, codebook=codebook)
    idx, val, score = oracle_mod.address(x, cb, s * s, k)
    np.testing.assert_array_equal(idx, _numpy_topk(_numpy_scores(x, cb, s), k))
    b = oracle_mod.address(x, cb, s * s, k, brute=True)
    for u, w in zip((idx, val, score), b):
        np.testing.assert_array_equal(u, w)
    np.testing.assert_allclose(val.sum(-1), 1.0, rtol=0, atol=1e-12)


def test_exact_ties_take_lower_slot_id(oracle_mod):
    """Direct mode, s = 4.  Sub-scores s0 = [.5,.5,.1,.5], s1 = [.25,.25,0,.25]:
    nine slots tie at the maximum 0.75; the three with the lowest ids are
    (0,0)=0, (0,1)=1, (0,3)=3, each with weight 1/3."""
    x = np.array([0.5, 0.5, 0.1, 0.5, 0.25, 0.25, 0.0, 0.25]).reshape(1, 1, 1, 8)
    for f32 in (False, True):
        for brute in (False, True):
            idx, val, score = oracle_mod.address(x, None, 16, 3, decide_f32=f32, brute=brute)
            np.testing.assert_array_equal(idx[0, 0, 0], [0, 1, 3])
            np.testing.assert_allclose(val[0, 0, 0], [1 / 3] * 3, rtol=1e-15)
            np.testing.assert_allclose(score[0, 0, 0], [0.75] * 3, rtol=0)
    # k = 4 reaches into the second row of ties: ids 0,1,3 then 4
    for brute in (False, True):
        idx, _, _ = oracle_mod.address(x, None, 16, 4, brute=brute)
        np.testing.assert_array_equal(idx[0, 0, 0], [0, 1, 3, 4])


def test_duplicate_codebook_rows_tie(oracle_mod):
    """Codebook mode: duplicated sub-key rows give exactly equal sub-scores;
    the lower sub-key (hence lower slot id) must win."""
    rng = np.random.default_rng(3)
    s, dk = 6, 8
    cb = rng.standard_normal((1, 2, s, dk // 2))
    cb[0, 0, 4] = cb[0, 0, 1]          # half-0 rows 1 and 4 identical
    cb[0, 1, 5] = cb[0, 1, 2]          # half-1 rows 2 and 5 identical
    x = rng.standard_normal((1, 1, 20, dk))
    for f32 in (False, True):
        idx, _, _ = oracle_mod.address(x, cb, s * s, 4, decide_f32=f32)
        ref = _numpy_topk(_numpy_scores(x, cb, s), 4)
        np.testing.assert_array_equal(idx, ref)


def test_softmax_closed_forms(oracle_mod):
    rng = np.random.default_rng(11)
    x, cb = _rand_case(rng, 1, 2, 30, 8, codebook=True)
    # k = 1: the single weight is exactly 1
    _, val, _ = oracle_mod.address(x, cb, 64, 1)
    np.testing.assert_array_equal(val, 1.0)
    # weights sum to one and follow w_i / w_j = exp(s_i - s_j)
    _, val, score = oracle_mod.address(x, cb, 64, 5, decide_f32=False)
    np.testing.assert_allclose(val.sum(-1), 1.0, rtol=1e-14)
    ratio = val[..., :, None] / val[..., None, :]
    np.testing.assert_allclose(ratio, np.exp(score[..., :, None] - score[..., None, :]), rtol=1e-12)
    # equal scores -> uniform weights (all sub-scores zero)
    z = np.zeros((1, 1, 2, 16))
    idx, val, _ = oracle_mod.address(z, None, 64, 6)
    np.testing.assert_allclose(val, 1 / 6, rtol=1e-15)
    np.testing.assert_array_equal(idx[0, 0, 0], [0, 1, 2, 3, 4, 5])

