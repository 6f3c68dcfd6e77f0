"""Helpers shared by the GPU parity tests: upload of generated inputs, the HIP
path end to end, error metrics, and the near-tie accounting of addressing."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth
from paper_2607_07386_amd import sdm

DEV = "cuda:0"


def to_dev(st: synth.Stored | None, dev=DEV):
    if st is None:
        return None
    if st.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(st.bits).view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(np.ascontiguousarray(st.f32)).to(dev)


def rel_err(got, ref) -> float:
    """max |got - ref| / max |ref| (infinity-norm relative error of a tensor)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def tol_for(w: synth.Workload) -> float:
    return 1e-4 if w.dtype == "f32" else 2e-2


def init_memory(w: synth.Workload, inp: synth.Inputs, dev=DEV) -> torch.Tensor:
    Bx, Hx = inp.shape_bh
    mem = torch.empty((Bx, Hx, w.N, w.d_v), dtype=torch.float32, device=dev)
    if w.m0 == "zero":
        sdm.mem_init(mem, None)
    else:
        heads = inp.heads if Hx == 1 else list(range(w.H))
        if Hx == 1:
            for s, h in enumerate(heads):
                mem[s, 0].copy_(torch.from_numpy(inp.m0_head(h)).to(dev))
        else:
            m0 = torch.stack([torch.from_numpy(inp.m0_head(h)) for h in range(w.H)]).to(dev)
            sdm.mem_init(mem, m0)
            del m0
    return mem


def gpu_forward(w: synth.Workload, inp: synth.Inputs, save=False, dev=DEV):
    q, k, v = to_dev(inp.q, dev), to_dev(inp.k, dev), to_dev(inp.v, dev)
    al, be = to_dev(inp.alpha, dev), to_dev(inp.beta, dev)
    cb = to_dev(inp.codebook, dev)
    r_idx, r_val, r_sc = sdm.address(q, cb, w.N, w.topk, want_score=True)
    w_idx, w_val, w_sc = sdm.address(k, cb, w.N, w.topk, want_score=True)
    mem = init_memory(w, inp, dev)
    Bx, Hx = inp.shape_bh
    saved = sdm.saved_buffer(Bx, Hx, w.T, w.topk, w.d_v, dev) if save else None
    y = sdm.scan_fwd(w_idx, w_val, r_idx, r_val, v, al, be, mem, saved=saved)
    torch.cuda.synchronize()
    return dict(q=q, k=k, v=v, alpha=al, beta=be, cb=cb, r_idx=r_idx, r_val=r_val, r_score=r_sc,
                w_idx=w_idx, w_val=w_val, w_score=w_sc, mem=mem, y=y, saved=saved)


def sub_scores_f32(x64: np.ndarray, cb64: np.ndarray | None, s: int):
    """fp32-rounded sub-scores of one token (test-side, for measuring near-tie gaps)."""
    if cb64 is None:
        return x64[:s].astype(np.float32), x64[s:2 * s].astype(np.float32)
    dh = x64.shape[-1] // 2
    return ((cb64[0] @ x64[:dh]).astype(np.float32), (cb64[1] @ x64[dh:]).astype(np.float32))


def compare_address(gidx, gval, oidx, oval, oscore, x64, cb64_per_row, s, tie_gap=1e-6, val_tol=1e-4):
    """Ids must match exactly except near-ties: a GPU-chosen slot outside the
    oracle's set must score (in fp32, as both sides decide) within tie_gap of
    the oracle's k-th best score.  Returns stats; raises AssertionError on a
    real mismatch.  Arrays are [rows, k]; x64 [rows, d_k]; cb64_per_row(r) the
    row's codebook [2, s, d_k/2] or None."""
    gidx = np.asarray(gidx)
    oidx = np.asarray(oidx)
    rows_bad = np.nonzero((gidx != oidx).any(-1))[0]
    flips, gaps = 0, []
    for r in rows_bad:
        gs, os_ = set(gidx[r].tolist()), set(oidx[r].tolist())
        kth = float(np.min(oscore[r]))
        s0, s1 = sub_scores_f32(x64[r], cb64_per_row(r), s)
        for slot in gs - os_:
            sc = float(np.float32(s0[slot // s]) + np.float32(s1[slot % s]))
            gap = kth - sc
            gaps.append(gap)
            assert gap < tie_gap, f"row {r}: slot {slot} chosen with gap {gap:.3e} below the k-th score"
            flips += 1
    ok = np.ones(gidx.shape[0], bool)
    ok[rows_bad] = False
    verr = rel_err(np.asarray(gval)[ok], np.asarray(oval)[ok]) if ok.any() else 0.0
    assert verr <= val_tol, f"softmax weights rel err {verr:.3e}"
    return dict(rows=int(gidx.shape[0]), rows_flipped=int(len(rows_bad)), flips=flips,
                max_gap=float(max(gaps)) if gaps else 0.0, val_rel_err=verr)
