"""The chunk-parallel forward scan (sdm_scan_fwd_chunked, App. A.1-A.2) against
the oracle's sequential scan in fp64.

Hand-made slot lists put re-used slots inside one 64-token chunk: every token
writing one slot, reads of the previous token's writes, reads of a token's own
writes, write sets with short periods, and a table of 16 rows where nearly every
slot is written by several tokens of each chunk.  Workloads through the GPU
addressing cover ragged chunks and slices, W != R, bf16 inputs and clustered
keys.  The chunked form reassociates the sums over a chunk and solves its
triangular system in fp32; the bar is the 1e-5 regression bound (the fp32
bar is 1e-4).  Every case runs at the three workgroup widths."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import DEV, init_memory, rel_err, to_dev
from paper_2607_07386_amd import sdm

pytestmark = pytest.mark.gpu
# The spec bar for fp32 is 1e-4; held here to the 1e-5 regression bound
# (measured errors are about 1e-7).
TOL = 1e-5


@pytest.fixture(autouse=True, params=[8, 16, 32], ids=["cols8", "cols16", "cols32"])
def chunk_cols(request):
    """Every case at each scan-workgroup width: the narrow kernel (8 columns,
    16 workgroups per 128-column stream) and the wide one at 16 and 32."""
    sdm.set_chunk_scan_cols(request.param)
    yield request.param
    sdm.set_chunk_scan_cols(0)


def np_(t):
    return t.detach().cpu().numpy()


def _lists_case(S, T, N, W, R, dv, idx_fn, seed, dtype=torch.float32, wsum=1.0):
    """Random weights on hand-made slot lists; write weights summing to about wsum per token."""
    rng = np.random.default_rng(seed)
    wi = np.zeros((S, T, W), np.int32)
    ri = np.zeros((S, T, R), np.int32)
    for s in range(S):
        for t in range(T):
            wi[s, t], ri[s, t] = idx_fn(rng, t, wi[s])
    wv = (rng.random((S, T, W)) * (2.0 * wsum / W)).astype(np.float32)
    rv = rng.standard_normal((S, T, R)).astype(np.float32)
    v = rng.standard_normal((S, T, dv)).astype(np.float32)
    al = rng.uniform(0.05, 1.0, (S, T)).astype(np.float32)
    be = rng.uniform(0.0, 1.0, (S, T)).astype(np.float32)
    m0 = rng.standard_normal((S, N, dv)).astype(np.float32)
    if dtype == torch.bfloat16:
        v, al, be = (synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(a)).reshape(a.shape) for a in (v, al, be))
    t_ = lambda a: torch.from_numpy(a).to(DEV)
    mem = t_(m0).reshape(S, 1, N, dv).contiguous()
    y = sdm.scan_fwd_chunked(t_(wi)[:, None], t_(wv)[:, None], t_(ri)[:, None], t_(rv)[:, None],
                             t_(v)[:, None].to(dtype), t_(al)[:, None].to(dtype), t_(be)[:, None].to(dtype), mem)
    torch.cuda.synchronize()
    memo = m0.astype(np.float64)
    yo = oracle.scan_fwd(wi, wv, ri, rv, v, al, be, memo)
    return np_(y)[:, 0], np_(mem)[:, 0], yo, memo


LISTS = {
    # every token writes slot 0 and reads it back
    "slot0-every-token": (6, 4, lambda rng, t, prev: (
        np.concatenate([[0], rng.choice(np.arange(1, 40), 5, replace=False)]).astype(np.int32),
        np.concatenate([[0], rng.choice(np.arange(1, 40), 3, replace=False)]).astype(np.int32))),
    # reads = the previous token's writes
    "read-prev-writes": (6, 6, lambda rng, t, prev: (
        rng.choice(24, 6, replace=False).astype(np.int32),
        (prev[t - 1] if t > 0 else rng.choice(24, 6, replace=False)).astype(np.int32))),
    # reads include the token's own writes; unsorted lists
    "read-own-writes-unsorted": (6, 6, lambda rng, t, prev: (
        (lambda a: (a, np.concatenate([a[:3], rng.choice(np.setdiff1d(np.arange(30), a), 3, replace=False)])))(
            rng.choice(30, 6, replace=False).astype(np.int32)))),
    # period-3 write sets
    "period-3": (6, 6, lambda rng, t, prev: (
        (np.arange(6) + 6 * (t % 3)).astype(np.int32), (np.arange(6) + 6 * ((t + 1) % 3)).astype(np.int32))),
    # 8 of 16 rows written per token: every slot has many writers in a chunk
    "dense-16-rows": (8, 5, lambda rng, t, prev: (
        np.sort(rng.choice(16, 8, replace=False)).astype(np.int32),
        rng.choice(16, 5, replace=False).astype(np.int32))),
}


@pytest.mark.parametrize("name", list(LISTS))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_chunked_hand_made_lists(name, dtype):
    W, R, fn = LISTS[name]
    # 211 tokens: three full chunks and a ragged one of 19
    y, mem, yo, memo = _lists_case(3, 211, 48, W, R, 20, fn, seed=7, dtype=dtype)
    ey, em = rel_err(y, yo), rel_err(mem, memo)
    print(f"chunked/{name}/{dtype}: y {ey:.2e} mem {em:.2e}", flush=True)
    assert ey < TOL and em < TOL


def test_chunked_unnormalised_weights():
    """Write weights summing to about 3 per token (beyond softmax outputs): the system is less
    benign, the bar the same."""
    W, R, fn = LISTS["read-prev-writes"]
    y, mem, yo, memo = _lists_case(2, 150, 48, W, R, 12, fn, seed=9, wsum=3.0)
    ey, em = rel_err(y, yo), rel_err(mem, memo)
    print(f"chunked/unnormalised: y {ey:.2e} mem {em:.2e}", flush=True)
    assert ey < TOL and em < TOL


WORKLOADS = {
    # ragged last chunk (T = 200) and slice (d_v = 36: one full 32-column slice and 4 columns)
    "f32-direct-dv36": synth.Workload("t", B=2, H=2, T=200, d_k=16, d_v=36, N=64, topk=8, dtype="f32",
                                      seed=71, codebook=False, m0="shared"),
    # codebook addressing, bf16, k = 32 (the 1.4B-shaped lists)
    "bf16-k32": synth.Workload("t", B=1, H=3, T=300, d_k=128, d_v=128, N=65536, topk=32, seed=72,
                               m0="shared"),
    # clustered keys (the long-context workload's key distribution), k = 32
    "bf16-clustered": synth.Workload("t", B=1, H=2, T=1024, d_k=128, d_v=128, N=262144, topk=32, seed=73,
                                     clustered_keys=True, m0="shared"),
    # k = 64, direct mode, d_v = 96
    "bf16-k64-direct": synth.Workload("t", B=1, H=2, T=130, d_k=128, d_v=96, N=4096, topk=64, seed=74,
                                      codebook=False, m0="shared"),
    # one token, k = 1
    "f32-T1-k1": synth.Workload("t", B=2, H=1, T=1, d_k=16, d_v=8, N=100, topk=1, dtype="f32", seed=75,
                                m0="shared"),
}


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_chunked_workloads(name):
    w = WORKLOADS[name]
    inp = synth.Inputs(w)
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
    r_idx, r_val = sdm.address(q, cb, w.N, w.topk)
    w_idx, w_val = sdm.address(k, cb, w.N, w.topk)
    mem = init_memory(w, inp)
    m0 = np_(mem).astype(np.float64)
    ws = sdm.chunked_workspace(*mem.shape[:2], w.T, w.topk, w.topk, DEV)
    y = sdm.scan_fwd_chunked(w_idx, w_val, r_idx, r_val, v, al, be, mem, workspace=ws)
    sdm.check_device_errors(ws)
    Bx, Hx = mem.shape[:2]
    S = Bx * Hx
    rs = lambda t, last: np_(t).reshape(S, w.T, last)
    memo = m0.reshape(S, w.N, w.d_v)
    yo = oracle.scan_fwd(rs(w_idx, w.topk), rs(w_val, w.topk).astype(np.float64), rs(r_idx, w.topk),
                         rs(r_val, w.topk).astype(np.float64), inp.v.f32.reshape(S, w.T, w.d_v).astype(np.float64),
                         inp.alpha.f32.reshape(S, w.T).astype(np.float64),
                         inp.beta.f32.reshape(S, w.T).astype(np.float64), memo)
    ey = rel_err(np_(y).reshape(S, w.T, w.d_v), yo)
    em = rel_err(np_(mem).reshape(S, w.N, w.d_v), memo)
    print(f"chunked/{name}: y {ey:.2e} mem {em:.2e}", flush=True)
    assert ey < TOL and em < TOL


def test_chunked_matches_sequential_kernel_closely():
    """Both GPU schedules on the same ids: they differ only by rounding."""
    w = WORKLOADS["bf16-k32"]
    inp = synth.Inputs(w)
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
    r_idx, r_val = sdm.address(q, cb, w.N, w.topk)
    w_idx, w_val = sdm.address(k, cb, w.N, w.topk)
    m1 = init_memory(w, inp)
    m2 = m1.clone()
    y1 = sdm.scan_fwd(w_idx, w_val, r_idx, r_val, v, al, be, m1)
    y2 = sdm.scan_fwd_chunked(w_idx, w_val, r_idx, r_val, v, al, be, m2)
    torch.cuda.synchronize()
    assert rel_err(np_(y2), np_(y1)) < TOL and rel_err(np_(m2), np_(m1)) < TOL


def test_chunked_flags_nonpositive_gate():
    S, T, N, W, dv = 1, 70, 32, 4, 8
    wi = torch.stack([torch.randperm(N, device=DEV)[:W] for _ in range(T)]).to(torch.int32).reshape(S, 1, T, W)
    wv = torch.rand((S, 1, T, W), device=DEV) / W
    v = torch.randn((S, 1, T, dv), device=DEV)
    al = torch.rand((S, 1, T), device=DEV) * 0.9 + 0.05
    al[0, 0, 66] = 0.0              # no log form: flagged (and taken as 1e-30)
    be = torch.rand((S, 1, T), device=DEV)
    mem = torch.zeros((S, 1, N, dv), device=DEV)
    ws = sdm.chunked_workspace(S, 1, T, W, W, DEV)
    sdm.scan_fwd_chunked(wi.contiguous(), wv, wi.contiguous(), wv, v, al, be, mem, workspace=ws)
    with pytest.raises(sdm.SdmError) as e:
        sdm.check_device_errors(ws)
    assert e.value.status == -5 and "alpha" in str(e.value)
    sdm.check_device_errors(ws)     # cleared


def test_chunked_empty_sequence_is_noop():
    mem = torch.randn((1, 1, 16, 8), device=DEV)
    ref = mem.clone()
    e_i = torch.zeros((1, 1, 0, 4), dtype=torch.int32, device=DEV)
    e_v = torch.zeros((1, 1, 0, 4), device=DEV)
    z = torch.zeros((1, 1, 0, 8), device=DEV)
    g = torch.zeros((1, 1, 0), device=DEV)
    y = sdm.scan_fwd_chunked(e_i, e_v, e_i, e_v, z, g, g, mem)
    torch.cuda.synchronize()
    assert y.numel() == 0 and torch.equal(mem, ref)


def test_chunked_ranges_overlap_coefficients():
    """33 chunks (2100 tokens, the last ragged): eight chunk ranges, the coefficients of each
    later range on the library's second stream beside the scan of the range before it."""
    W, R, fn = LISTS["read-own-writes-unsorted"]
    sdm.profile_enable(True)
    y, mem, yo, memo = _lists_case(2, 2100, 48, W, R, 20, fn, seed=11)
    n_coef, n_scan = sdm.profile_read("chunk_coef")[1], sdm.profile_read("chunk_scan")[1]
    sdm.profile_enable(False)
    ey, em = rel_err(y, yo), rel_err(mem, memo)
    print(f"chunked/ranges: y {ey:.2e} mem {em:.2e}", flush=True)
    assert n_coef == 8 and n_scan == 8
    assert ey < TOL and em < TOL


def test_chunked_repeat_spread():
    """The coefficient kernel adds the pair terms of A and QK with LDS atomics,
    so their rounding order, and the last bits of y and the table, may differ
    from run to run.  Two runs on the same inputs: the spread is measured and
    bounded (it stays at fp32 rounding)."""
    w = WORKLOADS["bf16-clustered"]
    inp = synth.Inputs(w)
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
    r_idx, r_val = sdm.address(q, cb, w.N, w.topk)
    w_idx, w_val = sdm.address(k, cb, w.N, w.topk)
    outs = []
    for _ in range(3):
        mem = init_memory(w, inp)
        y = sdm.scan_fwd_chunked(w_idx, w_val, r_idx, r_val, v, al, be, mem)
        torch.cuda.synchronize()
        outs.append((np_(y), np_(mem)))
    spread = max(max(rel_err(o[0], outs[0][0]), rel_err(o[1], outs[0][1])) for o in outs[1:])
    print(f"chunked/repeat spread: {spread:.2e}", flush=True)
    assert spread <= 1e-6


@pytest.mark.slow
def test_chunked_full_long_context(chunk_cols):
    """The long-context workload at full size (16 streams x 65536 tokens, clustered keys, 8 chunk
    ranges) at each workgroup width (the bench times the default, 32 columns); one sampled
    stream against the oracle fed the GPU's slot lists."""
    w = synth.WORKLOADS[2]
    inp = synth.Inputs(w)
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
    r_idx, r_val = sdm.address(q, cb, w.N, w.topk)
    w_idx, w_val = sdm.address(k, cb, w.N, w.topk)
    del q, k
    mem = torch.zeros((w.B, w.H, w.N, w.d_v), dtype=torch.float32, device=DEV)
    ws = sdm.chunked_workspace(w.B, w.H, w.T, w.topk, w.topk, DEV)
    y = sdm.scan_fwd_chunked(w_idx, w_val, r_idx, r_val, v, al, be, mem, workspace=ws)
    sdm.check_device_errors(ws)
    s = 5
    take = lambda t, last: np_(t).reshape(-1, w.T, last)[s:s + 1]
    memo = np.zeros((1, w.N, w.d_v), np.float64)
    yo = oracle.scan_fwd(take(w_idx, w.topk), take(w_val, w.topk).astype(np.float64), take(r_idx, w.topk),
                         take(r_val, w.topk).astype(np.float64), inp.v.f64.reshape(-1, w.T, w.d_v)[s:s + 1],
                         inp.alpha.f64.reshape(-1, w.T)[s:s + 1], inp.beta.f64.reshape(-1, w.T)[s:s + 1], memo)
    ey = rel_err(np_(y).reshape(-1, w.T, w.d_v)[s:s + 1], yo)
    em = rel_err(np_(mem).reshape(-1, w.N, w.d_v)[s:s + 1], memo)
    print(f"chunked/full-long-context stream {s}: y {ey:.2e} mem {em:.2e}", flush=True)
    assert ey < TOL and em < TOL
