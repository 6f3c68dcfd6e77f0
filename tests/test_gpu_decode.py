"""Single-token steps (decode): sdm_forward with T = 1 and no undo log runs the
addressing of both sides and the scan step in one launch.

Each case runs a few steps in a row on the carried memory, one token of a
T-token workload per step.  Every step is checked against the separate calls
(sdm_address twice, then sdm_scan_fwd) on a copy of the memory: the ids and
weights come from the same addressing code, bit for bit; y and the memory
agree to the rounding of the sums over rows, which the fused step takes in
another order.  The whole sequence is then checked against the oracle's scan
fed the GPU's ids and weights."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import DEV, init_memory, rel_err, to_dev
from paper_2607_07386_amd import sdm

pytestmark = pytest.mark.gpu

CASES = {
    # bf16 codebooks on the matrix cores, k = 32: the 1.4B-shaped addressing
    "bf16-mfma-k32": synth.Workload("t", B=3, H=4, T=5, d_k=128, d_v=128, N=65536, topk=32, seed=61,
                                    m0="shared"),
    # fp32 codebooks (FMA), d_v neither a multiple of 128 nor of the column chunk
    "f32-fma-dv200": synth.Workload("t", B=2, H=2, T=4, d_k=32, d_v=200, N=4096, topk=16, dtype="f32",
                                    seed=62, m0="shared"),
    # direct mode, N = 64 with 8 slots: reads and writes of a token share many rows
    "bf16-direct-N64": synth.Workload("t", B=4, H=2, T=6, d_k=16, d_v=36, N=64, topk=8, seed=63,
                                      codebook=False, m0="shared"),
    # the paper's 1.4B layer shape: sqrt(N) = 240, W = R = 64, d_v = 960, direct mode
    "paper-1.4b-layer": synth.Workload("t", B=2, H=2, T=3, d_k=480, d_v=960, N=57600, topk=64, seed=64,
                                       codebook=False, m0="shared"),
    # k in (64, 128]: two list entries per lane
    "bf16-k128": synth.Workload("t", B=1, H=3, T=3, d_k=64, d_v=40, N=16384, topk=128, seed=65, m0="shared"),
    # the smallest shapes: one slot per side, one column quad, sqrt(N) = 10
    "f32-k1-dv4": synth.Workload("t", B=3, H=1, T=4, d_k=16, d_v=4, N=100, topk=1, dtype="f32", seed=66,
                                 m0="shared"),
}


def _token(st, t):
    """Token t of a [B, H, T, ...] device tensor, contiguous, T = 1."""
    return st[:, :, t:t + 1].contiguous()


@pytest.mark.parametrize("name", list(CASES))
def test_decode_steps(name):
    w = CASES[name]
    inp = synth.Inputs(w)
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha), be=to_dev(inp.beta),
             cb=to_dev(inp.codebook))
    mem = init_memory(w, inp)
    m0 = mem.clone()
    Bx, Hx = inp.shape_bh
    ws = sdm.fwd_workspace(Bx, Hx, 1, w.topk, w.topk, DEV)
    sdm.profile_enable(True)
    steps = []
    for t in range(w.T):
        q, k, v, al, be = (_token(g[n], t) for n in ("q", "k", "v", "al", "be"))
        ref_mem = mem.clone()
        o = sdm.forward(q, k, g["cb"], g["cb"], v, al, be, mem, w.N, w.topk, workspace=ws)
        r_idx, r_val = sdm.address(q, g["cb"], w.N, w.topk)
        w_idx, w_val = sdm.address(k, g["cb"], w.N, w.topk)
        y_ref = sdm.scan_fwd(w_idx, w_val, r_idx, r_val, v, al, be, ref_mem)
        torch.cuda.synchronize()
        for key, ref in (("r_idx", r_idx), ("r_val", r_val), ("w_idx", w_idx), ("w_val", w_val)):
            assert torch.equal(o[key], ref), (name, t, key)
        ey, em = rel_err(o["y"].cpu().numpy(), y_ref.cpu().numpy()), rel_err(mem.cpu().numpy(),
                                                                                ref_mem.cpu().numpy())
        assert ey <= 1e-5 and em <= 1e-5, (name, t, ey, em)
        steps.append({kk: o[kk].cpu().numpy() for kk in ("r_idx", "r_val", "w_idx", "w_val", "y")})
    t_dec, n_dec = sdm.profile_read("decode")
    sdm.profile_enable(False)
    assert n_dec == w.T, "the single-token steps did not take the fused launch"

    # the oracle's scan over the whole sequence, fed the GPU's ids and weights
    S = Bx * Hx
    cat = lambda key, last: np.concatenate([s[key].reshape(S, 1, last) for s in steps], axis=1)
    wi, wv, ri, rv = cat("w_idx", w.topk), cat("w_val", w.topk), cat("r_idx", w.topk), cat("r_val", w.topk)
    memo = m0.cpu().numpy().reshape(S, w.N, w.d_v).astype(np.float64)
    yo = oracle.scan_fwd(wi, wv.astype(np.float64), ri, rv.astype(np.float64),
                         inp.v.f32.reshape(S, w.T, w.d_v).astype(np.float64),
                         inp.alpha.f32.reshape(S, w.T).astype(np.float64),
                         inp.beta.f32.reshape(S, w.T).astype(np.float64), memo)
    ey = rel_err(cat("y", w.d_v), yo)
    em = rel_err(mem.cpu().numpy().reshape(S, w.N, w.d_v), memo)
    assert ey <= 1e-4 and em <= 1e-4, (name, ey, em)


def test_decode_with_undo_log_takes_the_pipelined_path():
    """T = 1 with an undo log runs the usual kernels (the fused step saves nothing)."""
    w = CASES["bf16-direct-N64"]
    inp = synth.Inputs(w)
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha), be=to_dev(inp.beta))
    mem = init_memory(w, inp)
    Bx, Hx = inp.shape_bh
    saved = sdm.saved_buffer(Bx, Hx, 1, w.topk, w.d_v, DEV)
    sdm.profile_enable(True)
    q, k, v, al, be = (_token(g[n], 0) for n in ("q", "k", "v", "al", "be"))
    sdm.forward(q, k, None, None, v, al, be, mem, w.N, w.topk, saved=saved)
    torch.cuda.synchronize()
    n_dec, n_scan = sdm.profile_read("decode")[1], sdm.profile_read("fwd_scan")[1]
    sdm.profile_enable(False)
    assert n_dec == 0 and n_scan == 1


def test_decode_graph_replays_match_eager():
    """One decode step captured in a HIP graph (the fused single-token launch) and
    replayed token after token: each replay's ids, weights and y, and the memory at
    the end, equal the same steps run eagerly on a copy of the memory, bit for bit.
    Between replays the inputs of the next token are copied into the captured
    buffers and other eager work runs."""
    w = CASES["bf16-mfma-k32"]
    inp = synth.Inputs(w)
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha), be=to_dev(inp.beta))
    cb = to_dev(inp.codebook)
    mem0 = init_memory(w, inp)
    Bx, Hx = inp.shape_bh
    names = ("q", "k", "v", "al", "be")
    # eager steps on a copy
    mem_e = mem0.clone()
    ws_e = sdm.fwd_workspace(Bx, Hx, 1, w.topk, w.topk, DEV)
    eager = []
    for t in range(w.T):
        q, k, v, al, be = (_token(g[n], t) for n in names)
        o = sdm.forward(q, k, cb, cb, v, al, be, mem_e, w.N, w.topk, workspace=ws_e)
        torch.cuda.synchronize()
        eager.append({kk: o[kk].clone() for kk in ("r_idx", "r_val", "w_idx", "w_val", "y")})
    # the captured step: fixed input, output and state buffers
    buf = {n: _token(g[n], 0).clone() for n in names}
    mem_g = mem0.clone()
    ws_g = sdm.fwd_workspace(Bx, Hx, 1, w.topk, w.topk, DEV)
    y = torch.empty((Bx, Hx, 1, w.d_v), dtype=torch.float32, device=DEV)
    outs = {n: torch.empty((Bx, Hx, 1, w.topk), dtype=dt, device=DEV)
            for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32), ("w_idx", torch.int32),
                          ("w_val", torch.float32))}

    def step():
        sdm.forward(buf["q"], buf["k"], cb, cb, buf["v"], buf["al"], buf["be"], mem_g, w.N, w.topk,
                    workspace=ws_g, y=y, out=outs)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()   # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    mem_g.copy_(mem0)   # the warm-up step changed the state; the capture ran nothing
    scratch = torch.zeros(1 << 20, device=DEV)
    for t in range(w.T):
        for n in names:
            buf[n].copy_(_token(g[n], t))
        scratch.add_(1.0)   # other eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        for kk in ("r_idx", "r_val", "w_idx", "w_val"):
            assert torch.equal(outs[kk], eager[t][kk]), (t, kk)
        assert torch.equal(y, eager[t]["y"]), t
    assert torch.equal(mem_g, mem_e)
