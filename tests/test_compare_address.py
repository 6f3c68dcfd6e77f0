"""The near-tie rule the GPU addressing parity uses (tests/gpu_util.py
compare_address), checked on the CPU against planted selections.

One direct-mode token with sqrt(N) = 8: sub-scores s0 = [3, 2, -5, ...] and
s1 = [3, 2 + u, -5, ...], u two fp32 ulps of 2 (one of 5, so the fp32 sum
keeps it).  Pair (a, b) scores s0[a] + s1[b] with flat id 8a + b (Sec. 3.1
step 1), so with k = 2 the oracle keeps slot 0 (score 6) and slot 1 (5 + u),
and slot 8 (score 5) is the runner-up, 4.8e-7 below the k-th place.  Choosing slot 8 instead of slot 1 is
a near-tie flip the rule must accept; dropping slot 0 for it, repeating or
misordering ids, an id out of range, a slot clear of the k-th place, or
weights that are not the softmax of the chosen slots' scores must fail."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import compare_address

S = 8
K = 2


def _token():
    s0 = np.full(S, -5.0, np.float32)
    s1 = np.full(S, -5.0, np.float32)
    s0[:2] = [3.0, 2.0]
    two_up = np.nextafter(np.nextafter(np.float32(2.0), np.float32(3.0)), np.float32(3.0))
    s1[:2] = [3.0, two_up]
    x = np.concatenate([s0, s1]).astype(np.float64)
    idx, val, _ = oracle.address(x[None, None, None], None, S * S, K, decide_f32=True)
    return x, idx[0, 0], val[0, 0]


def _softmax_of(x, ids):
    sc = np.array([np.float32(x[i // S]) + np.float32(x[S + i % S]) for i in ids], np.float64)
    e = np.exp(sc - sc.max())
    return e / e.sum()


def _check(x, oidx, oval, gidx, gval):
    return compare_address(np.asarray(gidx)[None], np.asarray(gval)[None], oidx, oval, x[None],
                           lambda r: None, S)


def test_oracle_selection_of_the_planted_token():
    x, oidx, _ = _token()
    assert oidx[0].tolist() == [0, 1]


def test_identical_selection_passes():
    x, oidx, oval = _token()
    st = _check(x, oidx, oval, oidx[0], oval[0])
    assert st["flips"] == 0 and st["rows_flipped"] == 0


def test_near_tie_flip_is_accepted_and_counted():
    x, oidx, oval = _token()
    ids = [0, 8]
    st = _check(x, oidx, oval, ids, _softmax_of(x, ids))
    assert st["rows_flipped"] == 1 and st["flips"] == 1
    assert 0 < st["max_gap"] < 1e-6


@pytest.mark.parametrize("ids,why", [
    ([1, 8], "best slot dropped for a near-tie"),
    ([8, 8], "repeated id"),
    ([8, 0], "ids not ascending"),
    ([0, 64], "id out of range"),
    ([0, 2], "slot far below the k-th place"),
])
def test_bad_selection_is_rejected(ids, why):
    x, oidx, oval = _token()
    ok_ids = [i for i in ids if 0 <= i < S * S]
    w = _softmax_of(x, ok_ids) if len(ok_ids) == K else np.full(K, 0.5)
    with pytest.raises(AssertionError):
        _check(x, oidx, oval, ids, w)


def test_flipped_row_with_wrong_weights_is_rejected():
    x, oidx, oval = _token()
    ids = [0, 8]
    with pytest.raises(AssertionError):
        _check(x, oidx, oval, ids, _softmax_of(x, ids)[::-1])


def test_equal_ids_with_wrong_weights_are_rejected():
    x, oidx, oval = _token()
    with pytest.raises(AssertionError):
        _check(x, oidx, oval, oidx[0], oval[0][::-1] + 0.0)
