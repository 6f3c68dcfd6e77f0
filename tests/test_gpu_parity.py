"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bar: slot ids bit-exact except near-ties (a GPU-chosen slot outside the
oracle's set must score within 1e-6 of the oracle's k-th best score; such
flips are counted and reported); y, M_T and gradients within max relative
error 1e-4 (fp32 inputs) or 2e-2 (bf16 inputs, fp32 state).  The scan is
compared on the GPU's own slot ids and weights, so an addressing near-tie
never leaks into the scan comparison.  Rows no token writes must come back
bit-identical, and the backward must restore M_0 bit for bit.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2607_07386_amd import sdm
from tests.gpu_util import (DEV, REGRESSION_TOL, compare_address, gpu_forward, rel_err, to_dev, tol_for,
                            within)

pytestmark = pytest.mark.gpu

REPORT = os.environ.get("SDM_REPORT", "")


def report(name, **kw):
    line = json.dumps(dict(test=name, **kw), default=float)
    print(line, flush=True)
    if REPORT:
        with open(REPORT, "a") as f:
            f.write(line + "\n")


def np_(t):
    return t.detach().cpu().numpy()


def oracle_address_rows(w, inp, x_st, streams):
    """Oracle addressing of the given (flat) streams, decided in fp32 like the kernel."""
    x = x_st.f64.reshape((-1, w.T, w.d_k))[streams][:, None]
    if inp.codebook is not None:
        cbh = inp.codebook.f64
        heads = [inp.heads[s] for s in streams]
        out = [oracle.address(x[i:i + 1], cbh[heads[i]][None], w.N, w.topk, decide_f32=True)
               for i in range(len(streams))]
        return [np.concatenate([o[j] for o in out]) for j in range(3)], [cbh[h] for h in heads]
    return oracle.address(x, None, w.N, w.topk, decide_f32=True), [None] * len(streams)


def check_addressing(w, inp, g, streams):
    stats = {}
    for side, x_st, gi, gv in (("read", inp.q, g["r_idx"], g["r_val"]), ("write", inp.k, g["w_idx"], g["w_val"])):
        (oi, ov, _), cbs = oracle_address_rows(w, inp, x_st, streams)
        gidx = rows_of(gi, streams, (w.T, w.topk)).reshape(-1, w.topk)
        gval = rows_of(gv, streams, (w.T, w.topk)).reshape(-1, w.topk)
        x64 = x_st.f64.reshape(-1, w.T, w.d_k)[streams].reshape(-1, w.d_k)
        st = compare_address(gidx, gval, oi.reshape(-1, w.topk), ov.reshape(-1, w.topk),
                             x64, lambda r: cbs[r // w.T], w.sqrtN)
        stats[side] = st
    return stats


def oracle_scan_rows(w, inp, g, streams, m0_of_stream, save=False):
    """The oracle's scan of the given streams, fed the GPU's slot ids and weights."""
    S = len(streams)

    def take(t, last):
        return rows_of(t, streams, (w.T,) + last)

    wi, wv = take(g["w_idx"], (w.topk,)), take(g["w_val"], (w.topk,))
    ri, rv = take(g["r_idx"], (w.topk,)), take(g["r_val"], (w.topk,))
    v = inp.v.f64.reshape(-1, w.T, w.d_v)[streams]
    al = inp.alpha.f64.reshape(-1, w.T)[streams]
    be = inp.beta.f64.reshape(-1, w.T)[streams]
    mem = np.zeros((S, w.N, w.d_v), np.float64)
    for i, s in enumerate(streams):
        m0 = m0_of_stream(s)
        if m0 is not None:
            mem[i] = m0
    m_init = mem.copy()
    res = oracle.scan_fwd(wi, wv, ri, rv, v, al, be, mem, save=save)
    return dict(wi=wi, wv=wv, ri=ri, rv=rv, v=v, al=al, be=be, m_init=m_init, mem=mem,
                y=res[0] if save else res, saved=res[1] if save else None)


def rows_of(t, streams, last):
    """The sampled (b, h) streams of a device tensor, copied to the host alone."""
    return np_(t.reshape((-1,) + last)[torch.as_tensor(streams, device=t.device)])


def check_scan(w, g, o, streams, name):
    tol = tol_for(w)
    y = rows_of(g["y"], streams, (w.T, w.d_v))
    memg = rows_of(g["mem"], streams, (w.N, w.d_v))
    ey, em = rel_err(y, o["y"]), rel_err(memg, o["mem"])
    # rows no token writes: bit-identical to M_0
    untouched_ok = True
    for i in range(len(streams)):
        written = np.zeros(w.N, bool)
        written[o["wi"][i].ravel()] = True
        untouched_ok &= np.array_equal(memg[i][~written], o["m_init"][i][~written].astype(np.float32))
    report(name, y_rel_err=ey, mem_rel_err=em, tol=tol, regression_tol=REGRESSION_TOL,
           untouched_bit_exact=bool(untouched_ok))
    assert within(ey, w) and within(em, w), (ey, em)
    assert untouched_ok


def m0_fn(w, inp):
    if w.m0 == "zero":
        return lambda s: None
    return lambda s: inp.m0_head(inp.heads[s]).astype(np.float64)


# --------------------------------------------------------------- small cases
SMALL = {
    "c0-tiny-f32": synth.WORKLOADS[0],
    "bf16-mfma-ragged": synth.Workload("t", B=1, H=2, T=203, d_k=128, d_v=128, N=4096, topk=32, seed=11),
    "f32-direct-dv40": synth.Workload("t", B=2, H=1, T=97, d_k=32, d_v=40, N=256, topk=8, dtype="f32",
                                      seed=12, codebook=False),
    "bf16-direct": synth.Workload("t", B=1, H=3, T=70, d_k=64, d_v=32, N=1024, topk=16, seed=13, codebook=False),
    "bf16-s24-k24-dk48-dv36": synth.Workload("t", B=1, H=2, T=150, d_k=48, d_v=36, N=576, topk=24, seed=14),
    "bf16-fma-dk20": synth.Workload("t", B=1, H=1, T=90, d_k=20, d_v=16, N=400, topk=5, seed=15),
    "f32-k1": synth.Workload("t", B=1, H=2, T=65, d_k=16, d_v=8, N=100, topk=1, dtype="f32", seed=16),
    "bf16-k64-s128": synth.Workload("t", B=1, H=1, T=64, d_k=64, d_v=64, N=16384, topk=64, seed=17),
    # sqrt(N) = 512 and 1024: 8- and 4-token addressing workgroups (T not a multiple of either)
    "bf16-s512": synth.Workload("t", B=1, H=2, T=43, d_k=64, d_v=32, N=262144, topk=32, seed=24),
    "bf16-s1024": synth.Workload("t", B=1, H=1, T=26, d_k=128, d_v=16, N=1048576, topk=32, seed=25),
    # k in (64, 128]: two list entries per lane in addressing, 128-row scan plans
    "bf16-k128-s128": synth.Workload("t", B=1, H=2, T=70, d_k=64, d_v=40, N=16384, topk=128, seed=26),
    "f32-k100-s256-direct": synth.Workload("t", B=1, H=1, T=45, d_k=512, d_v=24, N=65536, topk=100,
                                           dtype="f32", seed=27, codebook=False),
    "bf16-k96-s512": synth.Workload("t", B=1, H=1, T=19, d_k=128, d_v=16, N=262144, topk=96, seed=28),
    "bf16-hazard-N64": synth.Workload("t", B=2, H=2, T=500, d_k=32, d_v=48, N=64, topk=8, seed=18),
    "f32-hazard-N16-k4": synth.Workload("t", B=1, H=1, T=333, d_k=8, d_v=4, N=16, topk=4, dtype="f32", seed=19),
    "bf16-T1": synth.Workload("t", B=2, H=2, T=1, d_k=32, d_v=32, N=256, topk=8, seed=20),
    "bf16-m0-shared": synth.Workload("t", B=3, H=2, T=120, d_k=32, d_v=32, N=1024, topk=8, seed=21, m0="shared"),
    "bf16-clustered": synth.Workload("t", B=1, H=2, T=400, d_k=64, d_v=32, N=4096, topk=16, seed=22,
                                     clustered_keys=True, n_clusters=8),
    # the paper's 1.4B layer (Table 1): H = 2, sqrt(N) = 240 (not a power of two), d_v = 960,
    # W = R = 64, direct-mode addressing (d_k = 2 sqrt(N))
    "paper-1.4b-layer": synth.Workload("t", B=1, H=2, T=130, d_k=480, d_v=960, N=57600, topk=64,
                                       seed=23, codebook=False),
    # the paper's 8B layer: sqrt(N) = 480, d_v = 1920, W = R = 64, direct mode (one stream; its
    # table is 1.8 GB)
    "paper-8b-layer": synth.Workload("t", B=1, H=1, T=24, d_k=960, d_v=1920, N=230400, topk=64,
                                     seed=29, codebook=False),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_forward_small(name, slice_width):
    w = SMALL[name]
    inp = synth.Inputs(w)
    g = gpu_forward(w, inp)
    S = w.B * w.H
    streams = list(range(S))
    st = check_addressing(w, inp, g, streams)
    report(name + "/address", **{f"{k}_{kk}": vv for k, v in st.items() for kk, vv in v.items()})
    o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp))
    check_scan(w, g, o, streams, f"{name}/sw{slice_width}/scan")


# Line-cooperative forward kernel (W = R = 32 or 64, d_v a multiple of 4 x slice width):
# against the oracle, and against the per-wave kernel (to 1e-5: the sums over rows
# are taken in another order), with and without the undo log.  N = 1024 with 32
# slots makes rows recur within the prefetch window and tokens read what they write.
FLINE = {
    "bf16-fline-ragged": synth.Workload("t", B=1, H=2, T=203, d_k=64, d_v=128, N=1024, topk=32, seed=51),
    "f32-fline-direct": synth.Workload("t", B=2, H=1, T=61, d_k=64, d_v=64, N=1024, topk=32, dtype="f32",
                                       seed=52, codebook=False),
    "bf16-fline-T5-m0": synth.Workload("t", B=2, H=1, T=5, d_k=32, d_v=64, N=1024, topk=32, seed=53,
                                       m0="shared"),
    # W = R = 64: each wave moves 16 of a token's 64 rows; two record chunks per lane
    "bf16-fline64-ragged": synth.Workload("t", B=1, H=2, T=150, d_k=64, d_v=128, N=4096, topk=64, seed=54),
    "f32-fline64-direct": synth.Workload("t", B=1, H=2, T=70, d_k=128, d_v=64, N=4096, topk=64, dtype="f32",
                                         seed=55, codebook=False, m0="shared"),
}


@pytest.mark.parametrize("save", [False, True])
@pytest.mark.parametrize("name", list(FLINE))
def test_forward_line_io(name, save, slice_width):
    w = FLINE[name]
    inp = synth.Inputs(w)
    streams = list(range(w.B * w.H))
    g = gpu_forward(w, inp, save=save)
    o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp))
    check_scan(w, g, o, streams, f"{name}/sw{slice_width}/save{int(save)}/fline")
    sdm.set_scan_line_io(False)
    try:
        gw = gpu_forward(w, inp, save=save)
    finally:
        sdm.set_scan_line_io(True)
    keys = ("y", "mem") + (("saved",) if save else ())
    for k in keys:
        assert rel_err(np_(g[k]), np_(gw[k]).astype(np.float64)) <= 1e-5, k


@pytest.mark.parametrize("name", ["bf16-fline-ragged", "f32-fline-direct", "bf16-fline64-ragged"])
def test_forward_prefetch_depths(name):
    """The line-cooperative forward at prefetch depths 4, 8 and 16 (how many
    tokens' rows are in flight; rows written inside the window come from the
    LDS ring): against the oracle, and bit for bit the same at every depth."""
    w = FLINE[name]
    inp = synth.Inputs(w)
    streams = list(range(w.B * w.H))
    outs = {}
    try:
        for pd in (4, 8, 16):
            sdm.set_scan_prefetch(pd)
            g = gpu_forward(w, inp, save=True, chunk=64)
            o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp))
            check_scan(w, g, o, streams, f"{name}/pd{pd}/fline")
            outs[pd] = {k: np_(g[k]) for k in ("y", "mem", "saved")}
    finally:
        sdm.set_scan_prefetch(0)
    for pd in (8, 16):
        for k in outs[4]:
            assert np.array_equal(outs[pd][k], outs[4][k]), (pd, k)


def test_empty_sequence_is_noop():
    w = synth.Workload("t", B=1, H=1, T=0, d_k=32, d_v=32, N=256, topk=8)
    dev = DEV
    z = torch.zeros((1, 1, 0, 32), dtype=torch.bfloat16, device=dev)
    idx, val = sdm.address(z, None, 256, 8)
    assert idx.numel() == 0
    mem = torch.randn((1, 1, 256, 32), device=dev)
    ref = mem.clone()
    e_i = torch.zeros((1, 1, 0, 8), dtype=torch.int32, device=dev)
    e_v = torch.zeros((1, 1, 0, 8), dtype=torch.float32, device=dev)
    g = torch.zeros((1, 1, 0), dtype=torch.bfloat16, device=dev)
    y = sdm.scan_fwd(e_i, e_v, e_i, e_v, z, g, g, mem)
    torch.cuda.synchronize()
    assert y.numel() == 0 and torch.equal(mem, ref)


# ------------------------------------------------- scan on hand-made index lists
def _scan_case(S, T, N, W, R, dv, idx_fn, seed, dtype=torch.float32, wscale=1.0):
    rng = np.random.default_rng(seed)
    wi = np.zeros((S, T, W), np.int32)
    ri = np.zeros((S, T, R), np.int32)
    for s in range(S):
        for t in range(T):
            wi[s, t], ri[s, t] = idx_fn(rng, s, t, wi[s])
    wv = (rng.random((S, T, W)) * wscale).astype(np.float32)
    rv = rng.standard_normal((S, T, R)).astype(np.float32)
    v = rng.standard_normal((S, T, dv)).astype(np.float32)
    al = rng.uniform(0.05, 1.0, (S, T)).astype(np.float32)
    be = rng.uniform(0.0, 1.0, (S, T)).astype(np.float32)
    m0 = rng.standard_normal((S, N, dv)).astype(np.float32)
    if dtype == torch.bfloat16:
        v, al, be = (synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(a)).reshape(a.shape) for a in (v, al, be))
    t_ = lambda a: torch.from_numpy(a).to(DEV)
    mem = t_(m0).reshape(S, 1, N, dv).contiguous()
    y = sdm.scan_fwd(t_(wi)[:, None], t_(wv)[:, None], t_(ri)[:, None], t_(rv)[:, None],
                     t_(v)[:, None].to(dtype), t_(al)[:, None].to(dtype), t_(be)[:, None].to(dtype), mem)
    torch.cuda.synchronize()
    memo = m0.astype(np.float64)
    yo = oracle.scan_fwd(wi, wv, ri, rv, v, al, be, memo)
    return np_(y)[:, 0], np_(mem)[:, 0], yo, memo


HAZARDS = {
    # every token writes slot 0 (plus random others) and reads it back
    "slot0-every-token": lambda rng, s, t, prev: (
        np.concatenate([[0], rng.choice(np.arange(1, 40), 5, replace=False)]).astype(np.int32),
        np.concatenate([[0], rng.choice(np.arange(1, 40), 3, replace=False)]).astype(np.int32)),
    # read set = previous token's write set (RAW across consecutive tokens)
    "read-prev-writes": lambda rng, s, t, prev: (
        rng.choice(24, 6, replace=False).astype(np.int32),
        (prev[t - 1] if t > 0 else rng.choice(24, 6, replace=False)).astype(np.int32)),
    # reads include this token's own writes, unsorted lists
    "read-own-writes-unsorted": lambda rng, s, t, prev: (
        (lambda a: (a, np.concatenate([a[:3], rng.choice(np.setdiff1d(np.arange(30), a), 3, replace=False)])))(
            rng.choice(30, 6, replace=False).astype(np.int32))),
    # write sets cycling with period 3 (re-touch at distance 3, inside the window)
    "period-3": lambda rng, s, t, prev: (
        (np.arange(6) + 6 * (t % 3)).astype(np.int32), (np.arange(6) + 6 * ((t + 1) % 3)).astype(np.int32)),
    # period 9: re-touch just beyond an 8-token prefetch window
    "period-9": lambda rng, s, t, prev: (
        (np.arange(4) + 4 * (t % 9)).astype(np.int32), (np.arange(6) + 4 * ((t + 5) % 9)).astype(np.int32)),
}


@pytest.mark.parametrize("name", list(HAZARDS))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_scan_hazards(name, dtype, slice_width):
    fn = HAZARDS[name]
    W = len(fn(np.random.default_rng(0), 0, 0, np.zeros((1, 8), np.int32))[0])
    R = len(fn(np.random.default_rng(0), 0, 0, np.zeros((1, 8), np.int32))[1])
    y, mem, yo, memo = _scan_case(3, 211, 48, W, R, 20, fn, seed=5, dtype=dtype)
    ey, em = rel_err(y, yo), rel_err(mem, memo)
    report(f"hazard/{name}/{dtype}/sw{slice_width}", y_rel_err=ey, mem_rel_err=em)
    assert ey < 1e-4 and em < 1e-4


# W != R with lists past 64 rows (the 8-column, four-pass plans): random sets
# over 300 slots, so rows recur within the prefetch window in most tokens.
# Write weights are scaled by 2 / sqrt(W): then beta kappa_n sum(kappa) <= 2 and
# a re-written row's factor alpha (1 - beta kappa_n sum(kappa)) stays in
# [-1, 1]; unscaled weights in [0, 1) grow rows past the fp32 range.
@pytest.mark.parametrize("W,R", [(128, 64), (40, 128), (128, 128)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_scan_wide_lists(W, R, dtype, slice_width):
    fn = lambda rng, s, t, prev: (rng.choice(300, W, replace=False).astype(np.int32),
                                  rng.choice(300, R, replace=False).astype(np.int32))
    y, mem, yo, memo = _scan_case(2, 150, 300, W, R, 24, fn, seed=9, dtype=dtype, wscale=2 / np.sqrt(W))
    ey, em = rel_err(y, yo), rel_err(mem, memo)
    report(f"wide/W{W}R{R}/{dtype}/sw{slice_width}", y_rel_err=ey, mem_rel_err=em)
    assert ey < 1e-4 and em < 1e-4


# Backward with lists of 64 and 128 rows (the per-wave kernel's four-pass
# shapes, which prefetch two tokens ahead instead of four): random sets over
# 150 slots, so most rows recur within the prefetch window.  Scan level, fp32,
# against the oracle's reverse pass; the memory must come back bit for bit.
@pytest.mark.parametrize("W,R", [(64, 64), (128, 96)])
def test_backward_wide_lists(W, R, slice_width):
    S, T, N, dv = 2, 70, 150, 24
    rng = np.random.default_rng(13 + W)
    wi = np.stack([np.stack([np.sort(rng.choice(N, W, replace=False)) for _ in range(T)]) for _ in range(S)])
    ri = np.stack([np.stack([np.sort(rng.choice(N, R, replace=False)) for _ in range(T)]) for _ in range(S)])
    wi, ri = wi.astype(np.int32), ri.astype(np.int32)
    wv = (rng.random((S, T, W)) * 2 / np.sqrt(W)).astype(np.float32)
    rv = rng.standard_normal((S, T, R)).astype(np.float32)
    v = rng.standard_normal((S, T, dv)).astype(np.float32)
    al = rng.uniform(0.05, 1.0, (S, T)).astype(np.float32)
    be = rng.uniform(0.0, 1.0, (S, T)).astype(np.float32)
    m0 = rng.standard_normal((S, N, dv)).astype(np.float32)
    dy = rng.standard_normal((S, T, dv)).astype(np.float32)
    t_ = lambda a: torch.from_numpy(a).to(DEV)[:, None].contiguous()
    mem = torch.from_numpy(m0).to(DEV)[:, None].contiguous()
    saved = sdm.saved_buffer(S, 1, T, W, dv, DEV)
    sdm.scan_fwd(t_(wi), t_(wv), t_(ri), t_(rv), t_(v), t_(al), t_(be), mem, saved=saved)
    g = sdm.scan_bwd(t_(wi), t_(wv), t_(ri), t_(rv), t_(v), t_(al), t_(be), mem, saved, t_(dy), want_dqk=False)
    torch.cuda.synchronize()
    memo = m0.astype(np.float64)
    _, P = oracle.scan_fwd(wi, wv, ri, rv, v, al, be, memo, save=True)
    og = oracle.scan_bwd(wi, wv, ri, rv, v, al, be, memo, P, dy.astype(np.float64))
    errs = {k: rel_err(np_(g[k])[:, 0], og[k]) for k in ("dv", "dalpha", "dbeta", "dw_val", "dr_val", "dmem0")}
    report(f"bwd-wide/W{W}R{R}/sw{slice_width}", **errs)
    for k, e in errs.items():
        assert e <= 1e-4, (k, e)
    assert np.array_equal(np_(mem)[:, 0], m0), "the undo did not restore M_0 bit for bit"


def test_gated_deltanet_reduction_on_gpu():
    """N = d_qk, every slot selected with the raw dense key/query as weights."""
    rng = np.random.default_rng(9)
    T, dqk, dv = 120, 16, 16
    K = rng.standard_normal((T, dqk)).astype(np.float32) * 0.25
    Q = rng.standard_normal((T, dqk)).astype(np.float32)
    V = rng.standard_normal((T, dv)).astype(np.float32)
    al = rng.uniform(0.5, 1.0, T).astype(np.float32)
    be = rng.uniform(0.0, 1.0, T).astype(np.float32)
    ids = np.tile(np.arange(dqk, dtype=np.int32), (T, 1))
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None].to(DEV)
    mem = torch.zeros((1, 1, dqk, dv), device=DEV)
    y = sdm.scan_fwd(t_(ids), t_(K), t_(ids), t_(Q), t_(V), t_(al), t_(be), mem)
    torch.cuda.synchronize()
    S = np.zeros((dqk, dv))
    ys = []
    for t in range(T):
        S = al[t] * S + be[t] * np.outer(K[t], V[t] - al[t] * S.T @ K[t])
        ys.append(S.T @ Q[t])
    assert rel_err(np_(y)[0, 0], np.array(ys)) < 1e-4
    assert rel_err(np_(mem)[0, 0], S) < 1e-4


def test_state_carry_bit_exact():
    w = SMALL["bf16-hazard-N64"]
    inp = synth.Inputs(w)
    g = gpu_forward(w, inp)
    T1 = 237
    mem = torch.zeros_like(g["mem"])
    ys = []
    for sl in (slice(0, T1), slice(T1, w.T)):
        part = lambda t: t[:, :, sl].contiguous()
        ys.append(sdm.scan_fwd(part(g["w_idx"]), part(g["w_val"]), part(g["r_idx"]), part(g["r_val"]),
                               part(g["v"]), part(g["alpha"]), part(g["beta"]), mem))
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(ys, 2), g["y"])
    assert torch.equal(mem, g["mem"])


def test_out_of_range_slot_is_clamped_and_reported():
    S, T, N, W, dv = 1, 20, 32, 4, 8
    wi = torch.randint(0, N, (S, 1, T, W), dtype=torch.int32, device=DEV)
    wi[0, 0, 5, 2] = N + 7          # out of range: clamped on the device, flagged
    wv = torch.rand((S, 1, T, W), device=DEV)
    v = torch.randn((S, 1, T, dv), device=DEV)
    g = torch.rand((S, 1, T), device=DEV)
    mem = torch.zeros((S, 1, N, dv), device=DEV)
    ws = sdm.fwd_workspace(S, 1, T, W, W, DEV)
    sdm.scan_fwd(wi, wv, wi.clamp(max=N - 1).contiguous(), wv, v, g, g, mem, workspace=ws)
    with pytest.raises(sdm.SdmError) as e:
        sdm.check_device_errors(ws)
    assert e.value.status == -5
    sdm.check_device_errors(ws)     # cleared


def test_debug_check_rejects_bad_slot_lists(monkeypatch):
    """SDM_DEBUG=1: a repeated id within a token's list, or an id outside
    [0, N), makes the scans return SDM_ERR_INVALID_ARG with their outputs
    untouched; valid lists give the same results as without the check."""
    S, T, N, W, R, dv = 2, 40, 64, 5, 4, 8
    rng = np.random.default_rng(3)
    wi = np.stack([np.stack([np.sort(rng.choice(N, W, replace=False)) for _ in range(T)]) for _ in range(S)])
    ri = np.stack([np.stack([np.sort(rng.choice(N, R, replace=False)) for _ in range(T)]) for _ in range(S)])
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a))[:, None].to(DEV)
    wi, ri = t_(wi.astype(np.int32)), t_(ri.astype(np.int32))
    wv, rv = t_(rng.random((S, T, W)).astype(np.float32)), t_(rng.random((S, T, R)).astype(np.float32))
    v = t_(rng.standard_normal((S, T, dv)).astype(np.float32))
    g = t_(rng.uniform(0.1, 1.0, (S, T)).astype(np.float32))
    m0 = torch.randn((S, 1, N, dv), device=DEV)
    mem_plain = m0.clone()
    y_plain = sdm.scan_fwd(wi, wv, ri, rv, v, g, g, mem_plain)
    monkeypatch.setenv("SDM_DEBUG", "1")
    mem = m0.clone()
    y = sdm.scan_fwd(wi, wv, ri, rv, v, g, g, mem)
    torch.cuda.synchronize()
    assert torch.equal(y, y_plain) and torch.equal(mem, mem_plain)
    dup = wi.clone()
    dup[1, 0, 17, 3] = dup[1, 0, 17, 1]
    oob = ri.clone()
    oob[0, 0, 5, 0] = N
    for wl, rl, what in ((dup, ri, "repeats"), (wi, oob, "outside")):
        for fn in (lambda m, yy: sdm.scan_fwd(wl, wv, rl, rv, v, g, g, m, y=yy),
                   lambda m, yy: sdm.scan_fwd_chunked(wl, wv, rl, rv, v, g, g, m, y=yy)):
            mem = m0.clone()
            yy = torch.full((S, 1, T, dv), 7.0, device=DEV)
            with pytest.raises(sdm.SdmError) as e:
                fn(mem, yy)
            assert e.value.status == -1 and what in str(e.value)
            torch.cuda.synchronize()
            assert torch.equal(mem, m0) and bool((yy == 7.0).all())
    saved = sdm.saved_buffer(S, 1, T, W, dv, DEV)
    mem = m0.clone()
    sdm.scan_fwd(wi, wv, ri, rv, v, g, g, mem, saved=saved)
    memT = mem.clone()
    with pytest.raises(sdm.SdmError) as e:
        sdm.scan_bwd(dup, wv, ri, rv, v, g, g, mem, saved, torch.ones((S, 1, T, dv), device=DEV), want_dqk=False)
    assert e.value.status == -1
    torch.cuda.synchronize()
    assert torch.equal(mem, memT)


# --------------------------------------------------------------- backward
BWD = {
    "bf16-small": synth.Workload("t", B=1, H=2, T=150, d_k=64, d_v=48, N=1024, topk=8, seed=31, train=True),
    "f32-direct-hazard": synth.Workload("t", B=2, H=1, T=120, d_k=16, d_v=8, N=64, topk=6, dtype="f32",
                                        seed=32, codebook=False, train=True),
    "bf16-m0-k32": synth.Workload("t", B=1, H=2, T=70, d_k=128, d_v=128, N=4096, topk=32, seed=33,
                                  m0="shared", train=True),
    "paper-1.4b-layer": synth.Workload("t", B=1, H=2, T=40, d_k=480, d_v=960, N=57600, topk=64,
                                       seed=34, codebook=False, m0="shared", train=True),
    "bf16-k128-m0": synth.Workload("t", B=1, H=2, T=70, d_k=64, d_v=40, N=16384, topk=128, seed=35,
                                   m0="shared", train=True),
    "paper-8b-layer": synth.Workload("t", B=1, H=1, T=12, d_k=960, d_v=1920, N=230400, topk=64,
                                     seed=37, codebook=False, train=True),
    "f32-k100-direct": synth.Workload("t", B=1, H=1, T=45, d_k=512, d_v=24, N=65536, topk=100, dtype="f32",
                                      seed=36, codebook=False, train=True),
}


def run_backward_case(w, inp, streams, chunk=64, fwd_chunk=None):
    """Forward with the undo log (separate calls, or sdm_forward with stage
    length fwd_chunk), then sdm_scan_bwd with the given chunk; oracle errors
    of the sampled streams."""
    g = gpu_forward(w, inp, save=True, chunk=fwd_chunk)
    dy = torch.from_numpy(inp.dy()).to(DEV)
    gr = sdm.scan_bwd(g["w_idx"], g["w_val"], g["r_idx"], g["r_val"], g["v"], g["alpha"], g["beta"],
                      g["mem"], g["saved"], dy, cb_q=g["cb"], cb_k=g["cb"], d_k=w.d_k, chunk=chunk)
    torch.cuda.synchronize()
    o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp), save=True)
    dy64 = rows_of(dy, streams, (w.T, w.d_v)).astype(np.float64)
    memT = o["mem"].copy()
    og = oracle.scan_bwd(o["wi"], o["wv"], o["ri"], o["rv"], o["v"], o["al"], o["be"], memT, o["saved"], dy64)
    assert np.array_equal(memT, o["m_init"])
    cb = inp.codebook.f64 if inp.codebook is not None else None
    out = {}
    for name, key, last in (("dv", "dv", (w.d_v,)), ("dalpha", "dalpha", ()), ("dbeta", "dbeta", ()),
                            ("dw_val", "dw_val", (w.topk,)), ("dr_val", "dr_val", (w.topk,))):
        gg = rows_of(gr[key], streams, (w.T,) + last)
        out[name] = rel_err(gg, og[name])
    gd = rows_of(gr["dmem0"], streams, (w.N, w.d_v))
    out["dmem0"] = rel_err(gd, og["dmem0"])
    # addressing gradients of the sampled streams, from the oracle's weight gradients
    for side, idx, val, dval, key in (("dq", o["ri"], o["rv"], og["dr_val"], "dq"),
                                      ("dk", o["wi"], o["wv"], og["dw_val"], "dk")):
        ref = np.concatenate([
            oracle.address_bwd(None if cb is None else cb[inp.heads[s]][None], idx[i:i + 1, None],
                               val[i:i + 1, None], dval[i:i + 1, None], w.N, w.d_k)
            for i, s in enumerate(streams)])[:, 0]
        gg = rows_of(gr[key], streams, (w.T, w.d_k))
        out[side] = rel_err(gg, ref)
    restored = rows_of(g["mem"], streams, (w.N, w.d_v))
    out["mem_restored_bit_exact"] = bool(np.array_equal(restored, o["m_init"].astype(np.float32)))
    return out, gr


@pytest.mark.parametrize("name", list(BWD))
def test_backward_small(name, slice_width):
    w = BWD[name]
    inp = synth.Inputs(w)
    streams = list(range(w.B * w.H))
    errs, _ = run_backward_case(w, inp, streams)
    report(f"{name}/sw{slice_width}/bwd", **errs)
    for k, e in errs.items():
        if k != "mem_restored_bit_exact":
            assert within(e, w), (k, e)
    assert errs["mem_restored_bit_exact"]


@pytest.mark.parametrize("name", ["bf16-small", "bf16-line-ragged", "bf16-line64-ragged"])
def test_backward_chunk_invariance(name):
    """chunk sets the backward's pipeline stages (chunk >= T: one stage); results
    are the same bit for bit (per-wave kernel, and the line-cooperative one)."""
    w = BWD.get(name) or LINE[name]
    inp = synth.Inputs(w)
    outs = []
    for chunk in (1, 16, 64, w.T):
        _, gr = run_backward_case(w, inp, [0], chunk=chunk)
        outs.append({k: np_(v) for k, v in gr.items()})
    for o in outs[1:]:
        for k in o:
            assert np.array_equal(o[k], outs[0][k]), k


# Line-cooperative backward kernel (8-column slices, W = R = 32 or 64, d_v a multiple of
# 32): against the oracle, and against the per-wave kernel (same arithmetic per slice; the
# compiler may contract a product into an fma differently, so to 1e-5, not bit for bit).  N = 1024 with 32
# slots per side (4096 with 64) makes a token's read and write sets share a slot in most
# tokens and rows recur within the prefetch window; T = 3 is shorter than the load lead.
LINE = {
    "bf16-line-ragged": synth.Workload("t", B=1, H=2, T=203, d_k=64, d_v=64, N=1024, topk=32, seed=41,
                                       train=True),
    "f32-line-direct": synth.Workload("t", B=2, H=1, T=66, d_k=64, d_v=32, N=1024, topk=32, dtype="f32",
                                      seed=42, codebook=False, train=True),
    "bf16-line-T3": synth.Workload("t", B=1, H=1, T=3, d_k=32, d_v=96, N=1024, topk=32, seed=43,
                                   m0="shared", train=True),
    "bf16-line64-ragged": synth.Workload("t", B=1, H=2, T=131, d_k=64, d_v=64, N=4096, topk=64, seed=44,
                                         train=True),
    "f32-line64-direct": synth.Workload("t", B=2, H=1, T=57, d_k=128, d_v=96, N=4096, topk=64, dtype="f32",
                                        seed=45, codebook=False, train=True),
    "bf16-line64-T3": synth.Workload("t", B=1, H=1, T=3, d_k=32, d_v=32, N=4096, topk=64, seed=46,
                                     m0="shared", train=True),
}


@pytest.mark.parametrize("name", list(LINE))
def test_backward_line_io(name):
    w = LINE[name]
    inp = synth.Inputs(w)
    streams = list(range(w.B * w.H))
    sdm.set_scan_slice_width(8)
    try:
        errs, g_line = run_backward_case(w, inp, streams)
        sdm.set_scan_line_io(False)
        g = gpu_forward(w, inp, save=True)
        dy = torch.from_numpy(inp.dy()).to(DEV)
        g_wave = sdm.scan_bwd(g["w_idx"], g["w_val"], g["r_idx"], g["r_val"], g["v"], g["alpha"], g["beta"],
                              g["mem"], g["saved"], dy, cb_q=g["cb"], cb_k=g["cb"], d_k=w.d_k, chunk=64)
        torch.cuda.synchronize()
    finally:
        sdm.set_scan_line_io(True)
        sdm.set_scan_slice_width(0)
    report(f"{name}/bwd-line", **errs)
    for k, e in errs.items():
        if k != "mem_restored_bit_exact":
            assert within(e, w), (k, e)
    assert errs["mem_restored_bit_exact"]
    for k in g_line:
        assert rel_err(np_(g_line[k]), np_(g_wave[k]).astype(np.float64)) <= 1e-5, k


@pytest.mark.parametrize("name", list(LINE))
def test_backward_line_prefetch_depths(name):
    """The line-cooperative backward at its default prefetch depth (4 tokens)
    and at 8: both against the oracle, and bit for bit the same (rows written
    inside the window come from the LDS rings at either depth)."""
    w = LINE[name]
    inp = synth.Inputs(w)
    streams = list(range(w.B * w.H))
    sdm.set_scan_slice_width(8)
    try:
        errs4, g4 = run_backward_case(w, inp, streams)
        sdm.set_scan_prefetch(8)
        errs8, g8 = run_backward_case(w, inp, streams)
    finally:
        sdm.set_scan_prefetch(0)
        sdm.set_scan_slice_width(0)
    for tag, errs in (("pd8", errs8), ("pd4", errs4)):
        report(f"{name}/bwd-line-{tag}", **errs)
        for k, e in errs.items():
            if k != "mem_restored_bit_exact":
                assert within(e, w), (tag, k, e)
        assert errs["mem_restored_bit_exact"], tag
    for k in g8:
        assert torch.equal(g8[k], g4[k]), k


# ------------------------------------------------- full-size workloads, sampled streams
# Each runs the calls bench.py times: the 1.4B-shaped forward as sdm_forward
# with 384-token stages, the training step as sdm_forward with the undo log
# (the library's stage choice) and then sdm_scan_bwd with chunk 64.  The
# learned-M0 workload runs sdm_forward with 1280-token stages, as bench.py
# does, and the long-context workload with the library's stages (a quarter
# of T).
def _full(cfg, streams_of, chunk):
    w = synth.WORKLOADS[cfg]
    inp = synth.Inputs(w)
    g = gpu_forward(w, inp, chunk=chunk)
    S = w.B * w.H
    streams = streams_of(S)
    st = check_addressing(w, inp, g, streams)
    report(f"c{cfg}/address", **{f"{k}_{kk}": vv for k, v in st.items() for kk, vv in v.items()})
    o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp))
    check_scan(w, g, o, streams, f"c{cfg}/scan")


@pytest.mark.slow
def test_full_c1():
    _full(1, lambda S: [0, S // 2 + 3, S - 1], chunk=384)


@pytest.mark.slow
def test_full_c2():
    _full(2, lambda S: [5], chunk=0)


@pytest.mark.slow
def test_full_c3():
    _full(3, lambda S: [0, S - 1], chunk=1280)


@pytest.mark.slow
def test_full_paper_1p4b_layer():
    """The paper's 1.4B layer shape as bench.py times it: 8 sequences of 4096
    tokens, sqrt(N) = 240, d_v = 960, top-64 reads and writes, direct mode,
    one sdm_forward call with the library's stages; two streams sampled."""
    w = synth.Workload("paper-1.4b-layer", B=8, H=2, T=4096, d_k=480, d_v=960, N=57600, topk=64, seed=6,
                       codebook=False)
    inp = synth.Inputs(w)
    g = gpu_forward(w, inp, chunk=0)
    streams = [1, 14]
    st = check_addressing(w, inp, g, streams)
    report("paper-1.4b/address", **{f"{k}_{kk}": vv for k, v in st.items() for kk, vv in v.items()})
    o = oracle_scan_rows(w, inp, g, streams, m0_fn(w, inp))
    check_scan(w, g, o, streams, "paper-1.4b/scan")


@pytest.mark.slow
def test_full_c4_training():
    w = synth.WORKLOADS[4]
    inp = synth.Inputs(w)
    S = w.B * w.H
    errs, _ = run_backward_case(w, inp, [1, S - 2], chunk=w.chunk, fwd_chunk=0)
    report("c4/bwd", **errs)
    for k, e in errs.items():
        if k != "mem_restored_bit_exact":
            assert within(e, w), (k, e)
    assert errs["mem_restored_bit_exact"]


def test_full_paper_1p4b_training():
    """The paper's 1.4B layer (W = R = 64, d_v = 960, direct addressing) at full size through
    the bench's training calls: sdm_forward with the undo log, then the staged backward
    (chunk 64), which runs the 64-row line-cooperative kernel; two sampled streams against
    the oracle's reverse pass on the GPU's own slot lists."""
    w = synth.Workload("paper-1.4b-layer", B=8, H=2, T=4096, d_k=480, d_v=960, N=57600, topk=64, seed=6,
                       codebook=False, train=True)
    inp = synth.Inputs(w)
    errs, _ = run_backward_case(w, inp, [3, 12], chunk=64, fwd_chunk=0)
    report("paper-1.4b/bwd", **errs)
    for k, e in errs.items():
        if k != "mem_restored_bit_exact":
            assert within(e, w), (k, e)
    assert errs["mem_restored_bit_exact"]


# ------------------------------------------------- prep records (read-after-write links)
FWD_PD, BWD_PD = 4, 4


def _rec_fwd(W, R):
    off_link = 8 * W + 8 * R
    off_ab = (off_link + 2 * (W + R) + 3) & ~3
    return off_link, off_ab, (off_ab + 8 + 15) & ~15


def _rec_bwd(W, R):
    off_lm = 8 * W + 8 * R
    off_ab = (off_lm + 2 * (2 * R + W) + 3) & ~3
    return off_lm, off_ab, (off_ab + 8 + 15) & ~15


def _links_fwd(wi, ri, PD):
    T, W = wi.shape
    R = ri.shape[1]
    out = np.full((T, W + R), -1, np.int64)
    for t in range(T):
        for r in range(W + R):
            slot = wi[t, r] if r < W else ri[t, r - W]
            for d in range(1, PD):   # earlier writers only, for both lists
                if t - d < 0:
                    break
                hit = np.nonzero(wi[t - d] == slot)[0]
                if hit.size:
                    out[t, r] = ((t - d) % PD) * W + hit[0]   # the writer's row in the scan's ring
                    break
    return out


def _links_bwd(wi, ri, PD, stage_end=None):
    """stage_end[t]: end (exclusive) of the backward stage holding token t; links
    never reach tokens at or past it (default: one stage)."""
    T, W = wi.shape
    R = ri.shape[1]
    if stage_end is None:
        stage_end = np.full(T, T)
    lm = np.full((T, R), -1, np.int64)
    lgr = np.full((T, R), -1, np.int64)
    lgw = np.full((T, W), -1, np.int64)

    def g_source(t, slot, allow_self):
        if allow_self:
            hit = np.nonzero(ri[t] == slot)[0]
            if hit.size:
                return int(hit[0])
        for d in range(1, PD):
            if t + d >= stage_end[t]:
                break
            hw = np.nonzero(wi[t + d] == slot)[0]
            if hw.size:
                return (d << 8) | (R + int(hw[0]))
            hr = np.nonzero(ri[t + d] == slot)[0]
            if hr.size:
                return (d << 8) | int(hr[0])
        return -1

    for t in range(T):
        for m in range(R):
            slot = ri[t, m]
            for d in range(1, PD):
                if t + d >= stage_end[t]:
                    break
                hw = np.nonzero(wi[t + d] == slot)[0]
                if hw.size:
                    lm[t, m] = (d << 8) | int(hw[0])
                    break
            lgr[t, m] = g_source(t, slot, False)
        for n in range(W):
            lgw[t, n] = g_source(t, wi[t, n], True)
    return np.concatenate([lm, lgr, lgw], 1)


@pytest.mark.parametrize("pd", [8, 16])
def test_prep_links_deep_window(pd):
    """Forward links over a window of 8 or 16 tokens (the line-cooperative
    kernel's deeper prefetch) equal a brute-force search; rows recur within
    the window (32 of 40 slots written per token)."""
    rng = np.random.default_rng(91 + pd)
    S, T, N, W, dv = 2, 150, 40, 32, 32
    wi = np.stack([np.stack([np.sort(rng.choice(N, W, replace=False)) for _ in range(T)]) for _ in range(S)])
    ri = np.stack([np.stack([np.sort(rng.choice(N, W, replace=False)) for _ in range(T)]) for _ in range(S)])
    wi, ri = wi.astype(np.int32), ri.astype(np.int32)
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a))[:, None].to(DEV)
    wv = t_((rng.random((S, T, W)) * 2 / np.sqrt(W)).astype(np.float32))
    rv = t_(rng.random((S, T, W)).astype(np.float32))
    v = t_(rng.standard_normal((S, T, dv)).astype(np.float32))
    g = t_(rng.uniform(0.1, 1.0, (S, T)).astype(np.float32))
    mem = torch.zeros((S, 1, N, dv), device=DEV)
    ws = sdm.fwd_workspace(S, 1, T, W, W, DEV)
    sdm.set_scan_prefetch(pd)
    try:
        y = sdm.scan_fwd(t_(wi), wv, t_(ri), rv, v, g, g, mem, workspace=ws)
        torch.cuda.synchronize()
    finally:
        sdm.set_scan_prefetch(0)
    off_link, _, rec = _rec_fwd(W, W)
    raw = np_(ws)[256:256 + S * T * rec].reshape(S, T, rec)
    got = raw[:, :, off_link:off_link + 2 * (2 * W)].copy().view(np.int16).astype(np.int64)
    for s_ in range(S):
        np.testing.assert_array_equal(got[s_], _links_fwd(wi[s_], ri[s_], pd))
    memo = np.zeros((S, N, dv))
    yo = oracle.scan_fwd(wi, np_(wv)[:, 0], ri, np_(rv)[:, 0], np_(v)[:, 0], np_(g)[:, 0], np_(g)[:, 0], memo)
    assert rel_err(np_(y)[:, 0], yo) <= 1e-5 and rel_err(np_(mem)[:, 0], memo) <= 1e-5


@pytest.mark.parametrize("sorted_lists", [True, False])
def test_prep_links_match_bruteforce(sorted_lists):
    """Links in the staged per-token records equal a brute-force search, for the
    forward and the backward window, across workgroup boundaries (T = 150 is
    64 + 64 + 22 tokens) and for unsorted slot lists.  The backward runs once as
    one stage (chunk = T) and once in its pipeline stages (chunk 64: tokens
    [86, 150), [64, 86), [0, 64)), whose links stop at the stage's end."""
    rng = np.random.default_rng(77)
    S, T, N, W, R, dv = 2, 150, 24, 5, 4, 8
    wi = np.stack([np.stack([rng.choice(N, W, replace=False) for _ in range(T)]) for _ in range(S)]).astype(np.int32)
    ri = np.stack([np.stack([rng.choice(N, R, replace=False) for _ in range(T)]) for _ in range(S)]).astype(np.int32)
    if sorted_lists:
        wi, ri = np.sort(wi, -1), np.sort(ri, -1)
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a))[:, None].to(DEV)
    wv = t_(rng.random((S, T, W)).astype(np.float32))
    rv = t_(rng.random((S, T, R)).astype(np.float32))
    v = t_(rng.standard_normal((S, T, dv)).astype(np.float32))
    g = t_(rng.random((S, T)).astype(np.float32))
    mem = torch.zeros((S, 1, N, dv), device=DEV)
    ws = sdm.fwd_workspace(S, 1, T, W, R, DEV)
    saved = sdm.saved_buffer(S, 1, T, W, dv, DEV)
    sdm.scan_fwd(t_(wi), wv, t_(ri), rv, v, g, g, mem, saved=saved, workspace=ws)
    torch.cuda.synchronize()
    off_link, _, rec = _rec_fwd(W, R)
    raw = np_(ws)[256:256 + S * T * rec].reshape(S, T, rec)
    got = raw[:, :, off_link:off_link + 2 * (W + R)].copy().view(np.int16).astype(np.int64)
    for s in range(S):
        np.testing.assert_array_equal(got[s], _links_fwd(wi[s], ri[s], FWD_PD))
    bws = sdm.bwd_workspace(S, 1, T, W, R, dv, DEV)
    off_lm, _, rec = _rec_bwd(W, R)
    staged_end = np.repeat([64, 86, 150], [64, 22, 64])
    for chunk, ends in ((T, None), (64, staged_end)):
        mem_c = mem.clone()
        sdm.scan_bwd(t_(wi), wv, t_(ri), rv, v, g, g, mem_c, saved, torch.zeros_like(v), workspace=bws,
                     want_dqk=False, chunk=chunk)
        torch.cuda.synchronize()
        raw = np_(bws)[256:256 + S * T * rec].reshape(S, T, rec)
        got = raw[:, :, off_lm:off_lm + 2 * (2 * R + W)].copy().view(np.int16).astype(np.int64)
        for s in range(S):
            np.testing.assert_array_equal(got[s], _links_bwd(wi[s], ri[s], BWD_PD, ends))
