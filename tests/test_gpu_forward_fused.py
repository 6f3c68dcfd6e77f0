"""The fused forward (sdm_forward: addressing pipelined with the scan over
chunks of tokens) against the three separate calls, whose parity with the
oracle the other GPU tests establish.  Chunking changes only where the scan
finds a row (HBM or the in-flight ring) and which stream runs the addressing,
never the arithmetic, so every output must match bit for bit."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_util import DEV, gpu_forward, init_memory, to_dev
from paper_2607_07386_amd import sdm

pytestmark = pytest.mark.gpu

CASES = {
    # T not a multiple of the chunk; clustered keys give frequent re-touches across chunk edges
    "bf16-codebook": synth.Workload("t", B=2, H=2, T=700, d_k=64, d_v=48, N=1024, topk=16, seed=41,
                                    clustered_keys=True, n_clusters=8),
    "f32-direct-N64": synth.Workload("t", B=1, H=3, T=333, d_k=16, d_v=8, N=64, topk=8, dtype="f32",
                                     seed=42, codebook=False),
    "bf16-k32": synth.Workload("t", B=1, H=2, T=520, d_k=128, d_v=128, N=4096, topk=32, seed=43),
    # 128 streams: an overlapped stage has more 16-token tiles than the capped addressing grid
    # has workgroups, so workgroups take several tiles
    "bf16-128-streams": synth.Workload("t", B=8, H=16, T=320, d_k=64, d_v=32, N=1024, topk=8, seed=44),
    # top-64 reads and writes, direct mode: the 64-row line-cooperative scan over token-range stages
    "bf16-direct-k64": synth.Workload("t", B=2, H=2, T=400, d_k=256, d_v=128, N=16384, topk=64, seed=45,
                                      codebook=False),
    # the paper's 1.4B layer (sqrt(N) = 240, d_v = 960, top-64, direct mode) at reduced T
    "paper-1.4b-layer": synth.Workload("t", B=1, H=2, T=300, d_k=480, d_v=960, N=57600, topk=64, seed=46,
                                       codebook=False),
}


def _fused(w, inp, chunk, save):
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha),
             be=to_dev(inp.beta), cb=to_dev(inp.codebook))
    mem = init_memory(w, inp)
    Bx, Hx = inp.shape_bh
    saved = sdm.saved_buffer(Bx, Hx, w.T, w.topk, w.d_v, DEV) if save else None
    o = sdm.forward(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], mem, w.N, w.topk,
                    saved=saved, chunk=chunk)
    torch.cuda.synchronize()
    o["mem"], o["saved"] = mem, saved
    return o


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("chunk", [0, 64, 100, 256, 384, 448, 4096])
def test_fused_forward_matches_separate_calls(name, chunk, slice_width):
    w = CASES[name]
    inp = synth.Inputs(w)
    ref = gpu_forward(w, inp, save=True)
    got = _fused(w, inp, chunk, save=True)
    for key in ("r_idx", "r_val", "w_idx", "w_val", "y", "mem", "saved"):
        a, b = got[key].cpu().numpy(), ref[key].cpu().numpy()
        assert np.array_equal(a, b), (name, chunk, key, np.abs(a.astype(np.float64) - b).max())


def test_fused_forward_inference_and_repeat():
    """No undo log; two calls in a row carry the state like two scan calls."""
    w = CASES["bf16-codebook"]
    inp = synth.Inputs(w)
    ref = gpu_forward(w, inp)
    g = dict(q=to_dev(inp.q), k=to_dev(inp.k), v=to_dev(inp.v), al=to_dev(inp.alpha),
             be=to_dev(inp.beta), cb=to_dev(inp.codebook))
    sdm.scan_fwd(ref["w_idx"], ref["w_val"], ref["r_idx"], ref["r_val"], ref["v"], ref["alpha"],
                 ref["beta"], ref["mem"])
    mem = init_memory(w, inp)
    ws = sdm.fwd_workspace(w.B, w.H, w.T, w.topk, w.topk, DEV)
    for _ in range(2):
        o = sdm.forward(g["q"], g["k"], g["cb"], g["cb"], g["v"], g["al"], g["be"], mem, w.N, w.topk,
                        workspace=ws, chunk=128)
    torch.cuda.synchronize()
    assert np.array_equal(mem.cpu().numpy(), ref["mem"].cpu().numpy())
