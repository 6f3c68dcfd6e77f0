"""sdm_forward_noalloc (the allocation-free forward) against sdm_forward,
through the C ABI.  Both run the same kernels on the same inputs; the
allocation-free call keeps its records in the library's fixed device array and
runs one stage on the caller's stream, so ids, weights, y and the memory must
match sdm_forward bit for bit.  Two multi-token calls in a row, the second
smaller (the array keeps the first call's records), then single-token steps.
"""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_util import DEV, init_memory, to_dev
from paper_2607_07386_amd import sdm

pytestmark = pytest.mark.gpu

BIG = synth.Workload("t", B=2, H=4, T=300, d_k=128, d_v=128, N=4096, topk=32, seed=61)
SMALL = synth.Workload("t", B=1, H=2, T=70, d_k=64, d_v=64, N=1024, topk=16, seed=62, codebook=False)
DECODE = synth.Workload("t", B=4, H=4, T=1, d_k=64, d_v=32, N=1024, topk=8, seed=63)


def _inputs(w):
    inp = synth.Inputs(w)
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha), be=to_dev(inp.beta),
             cb=to_dev(inp.codebook))
    return inp, g


def _both(w, save=False):
    inp, g = _inputs(w)
    m_ref, m_na = init_memory(w, inp), init_memory(w, inp)
    Bx, Hx = inp.shape_bh
    s_ref = sdm.saved_buffer(Bx, Hx, w.T, w.topk, w.d_v, DEV) if save else None
    s_na = sdm.saved_buffer(Bx, Hx, w.T, w.topk, w.d_v, DEV) if save else None
    ref = sdm.forward(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], m_ref, w.N, w.topk, saved=s_ref)
    got = sdm.forward_noalloc(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], m_na, w.N, w.topk,
                              saved=s_na)
    torch.cuda.synchronize()
    ref["mem"], got["mem"] = m_ref, m_na
    if save:
        ref["saved"], got["saved"] = s_ref, s_na
    return ref, got


def _same(ref, got, keys, what):
    for key in keys:
        a, b = got[key].cpu().numpy(), ref[key].cpu().numpy()
        assert np.array_equal(a, b), (what, key)


def test_noalloc_matches_forward_twice_second_smaller():
    for w, save in ((BIG, True), (SMALL, False)):
        ref, got = _both(w, save)
        keys = ("r_idx", "r_val", "w_idx", "w_val", "y", "mem") + (("saved",) if save else ())
        _same(ref, got, keys, f"T={w.T}")


def test_noalloc_single_token_steps():
    w = DECODE
    inp, g = _inputs(w)
    m_ref, m_na = init_memory(w, inp), init_memory(w, inp)
    for _ in range(3):     # the same token three times: each step carries the state
        ref = sdm.forward(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], m_ref, w.N, w.topk)
        got = sdm.forward_noalloc(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], m_na, w.N, w.topk)
        torch.cuda.synchronize()
        ref["mem"], got["mem"] = m_ref, m_na
        _same(ref, got, ("r_idx", "r_val", "w_idx", "w_val", "y", "mem"), "decode")


def test_noalloc_rejects_sizes_past_the_array():
    w = SMALL
    inp, g = _inputs(w)
    cap = sdm.lib().sdm_forward_noalloc_max_bytes()
    need = sdm.lib().sdm_scan_fwd_workspace_bytes(w.B, w.H, w.T, w.topk, w.topk)
    assert need <= cap
    per_token_head = (need - 256) // (w.B * w.H * w.T)   # bytes of one token-head's record
    big_T = cap // per_token_head + 1    # one stream of this many tokens needs more than the array
    assert sdm.lib().sdm_scan_fwd_workspace_bytes(1, 1, big_T, w.topk, w.topk) > cap
    q = torch.zeros((1, 1, big_T, w.d_k), dtype=g["q"].dtype, device=DEV)
    v = torch.zeros((1, 1, big_T, w.d_v), dtype=g["v"].dtype, device=DEV)
    a = torch.zeros((1, 1, big_T), dtype=g["v"].dtype, device=DEV)
    m1 = torch.zeros((1, 1, w.N, w.d_v), device=DEV)
    with pytest.raises(sdm.SdmError) as e:
        sdm.forward_noalloc(q, q, None, None, v, a, a, m1, w.N, w.topk)
    assert e.value.status == -2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.count_nonzero(m1).item() == 0
