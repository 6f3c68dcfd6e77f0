#!/usr/bin/env python3
"""Throughput of the SDM hot path on one MI355X.

One step = one pass of the layer's sparse path over one batch of synthetic
input of the 1.4B-shaped workload (B=8, H=16, T=4096, d_k=d_v=128,
N=65536 slots per head, top-32 reads and writes, bf16 inputs, fp32 memory):
addressing of the read queries and of the write keys, then the forward scan,
as one sdm_forward call (addressing of the next chunk of tokens overlaps the
scan of the current one; steps do not overlap each other).  The same work as
three separate calls is timed too (`ms_per_step_sequential`).  The memory
table stays resident in HBM and carries from one step to the next (the
state-carry property: each step is a further 4096 tokens of every stream; the
work per step does not depend on the table's contents).

Further legs: the training step (forward with the undo log + backward with
addressing gradients) on the training workload (B=4, H=16, T=4096) under
"train"; the learned-M0 workload (B=4, H=8, T=8192, N=2^20): its M0
broadcast under "mem_init" and its forward steps under "learned_m0";
single-token decode steps under "decode"; the layer with its gate producers
and norm-gate epilogue fused (sdm_layer_fwd / sdm_layer_bwd) against the bare
path under "layer"; the paper's own 1.4B
and 8B layer shapes (H=2, sqrt(N)=240 and 480, d_v=960 and 1920, W=R=64,
direct-mode addressing; forward and training steps) under "paper_layer"; the
long-context scan (16 streams of 65536 tokens) by the sequential and the
chunk-parallel schedules under "long_context".

Printed: one JSON line.  `value` is forward tokens/s (B*T positions, all
heads) over the timed steps; `roofline` gives the forward scan kernel's
algorithmic HBM bytes per launch over its mean event-timed duration;
`cpu_baseline` is the CPU oracle timed on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SDM layer tokens/sec (fwd, fwd+bwd) at 1 GPU; achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix-core peak of the MI355X
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_fwd_scan_c1.json")
# sources of the forward scan kernel: the traffic file holds their hash
SCAN_SRCS = [os.path.join(ROOT, "paper_2607_07386_amd", "csrc", f)
             for f in ("scan_fwd.hip", "sdm_common.h", "sdm_internal.h", "sdm_reduce.h")]
# the forward scan kernel this workload runs (W = R = 32, d_v a multiple of 64:
# the line-cooperative kernel, the library's default)
SCAN_KERNEL = "scan_fwd_line_kernel"


def scan_src_hash():
    h = hashlib.sha256()
    for f in SCAN_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def fwd_scan_bytes_per_token_head(W, R, d_v, in_bytes):
    """Bytes the forward scan must move per (token, head), every row counted as
    the eager recurrence touches it: W rows gathered and W scattered, R rows
    gathered (fp32 rows of d_v), v, alpha and beta in, the slot ids and weights
    of both sides in, y out."""
    return (2 * W + R) * d_v * 4 + d_v * in_bytes + 2 * in_bytes + (W + R) * 8 + d_v * 4


def unique_row_bytes(w_idx, r_idx, d_v, in_bytes, window=64):
    """Stricter count: within each window of 64 tokens of a stream, every
    distinct slot is loaded once (read or written) and every distinct written
    slot stored once; the per-token vectors as above."""
    import numpy as np
    S, T, W = w_idx.shape
    R = r_idx.shape[2]
    nw = T // window
    wi = w_idx[:, :nw * window].reshape(S, nw, window * W)
    both = np.concatenate([wi, r_idx[:, :nw * window].reshape(S, nw, window * R)], axis=2)

    def distinct(a):
        a = np.sort(a, axis=2)
        return int((a[:, :, 1:] != a[:, :, :-1]).sum() + a.shape[0] * a.shape[1])
    rows = distinct(both) + distinct(wi)
    tokens = S * nw * window
    return rows * d_v * 4 + tokens * (d_v * in_bytes + 2 * in_bytes + (W + R) * 8 + d_v * 4), tokens


def bwd_scan_bytes_per_token_head(W, R, d_v, in_bytes):
    """Bytes the backward scan must move per (token, head): rows M_t[j_m],
    G[j_m] and G[i_n] read, P (the undo log) read, G[j_m], G[i_n] and the undo
    M[i_n] written, (4W + 3R) fp32 rows of d_v; plus dy and dv (fp32) and v."""
    return (4 * W + 3 * R) * d_v * 4 + d_v * (4 + 4 + in_bytes)


def scoring_mfma(w, call_ms):
    """The addressing's sub-key scoring against the bf16 matrix-core peak: per
    call (one side, every token-head) 2 sqrt(N) d_k flops per token-head (both
    halves, sqrt(N) sub-keys of d_k / 2), over the address kernel's time alone."""
    flops = 2 * w.sqrtN * w.d_k * w.B * w.H * w.T
    tf = flops / (call_ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": "address_kernel", "flops_per_call": flops, "call_ms": round(call_ms, 4),
            "achieved": round(tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 5),
            "note": "the kernel's time is mostly top-k selection on the vector ALUs; scoring alone is a "
                    "small part of it"}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(w, inp, n_streams, T_sample):
    """The oracle (fp64 C, OpenMP) on n_streams (b, h) streams x T_sample tokens:
    addressing of both sides + forward scan.  Returns tokens/s (positions across
    all H heads, i.e. token-heads / H)."""
    import numpy as np

    import oracle
    oracle.build(force=False)
    streams = list(range(n_streams))
    T = T_sample
    x_q = inp.q.f32.reshape(-1, w.T, w.d_k)[streams, :T][:, None].astype(np.float64)
    x_k = inp.k.f32.reshape(-1, w.T, w.d_k)[streams, :T][:, None].astype(np.float64)
    v = inp.v.f32.reshape(-1, w.T, w.d_v)[streams, :T].astype(np.float64)
    al = inp.alpha.f32.reshape(-1, w.T)[streams, :T].astype(np.float64)
    be = inp.beta.f32.reshape(-1, w.T)[streams, :T].astype(np.float64)
    cb = inp.codebook.f32.astype(np.float64)
    mem = np.zeros((n_streams, w.N, w.d_v))
    t0 = time.perf_counter()
    ri, rv, wi, wv = [], [], [], []
    for i, s in enumerate(streams):
        h = inp.heads[s]
        a = oracle.address(x_q[i:i + 1], cb[h][None], w.N, w.topk)
        b = oracle.address(x_k[i:i + 1], cb[h][None], w.N, w.topk)
        ri.append(a[0]); rv.append(a[1]); wi.append(b[0]); wv.append(b[1])
    cat = lambda xs: np.concatenate(xs)[:, 0]
    oracle.scan_fwd(cat(wi), cat(wv), cat(ri), cat(rv), v, al, be, mem)
    dt = time.perf_counter() - t0
    # one stream on one thread: the oracle's serial cost per stream
    cores = oracle.max_threads()
    oracle.set_threads(1)
    t1 = time.perf_counter()
    a = oracle.address(x_q[:1], cb[inp.heads[0]][None], w.N, w.topk)
    b = oracle.address(x_k[:1], cb[inp.heads[0]][None], w.N, w.topk)
    oracle.scan_fwd(b[0][:, 0], b[1][:, 0], a[0][:, 0], a[1][:, 0], v[:1], al[:1], be[:1], np.zeros((1, w.N, w.d_v)))
    dt1 = time.perf_counter() - t1
    oracle.set_threads(cores)
    return dict(value=n_streams * T / w.H / dt, unit="tokens/s", cores=cores,
                kind="oracle", wall_s=round(dt, 3), one_stream_one_thread_s=round(dt1, 3),
                sample=f"{n_streams} of {w.B * w.H} (b,h) streams x {T} tokens of the same workload; "
                       f"address(q)+address(k)+forward scan, fp64; tokens/s = streams*T/H/wall")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-train", action="store_true", help="skip the training-step measurement")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-streams", type=int, default=16)
    ap.add_argument("--cpu-tokens", type=int, default=4096)
    ap.add_argument("--only", choices=["fwd", "train", "learned", "decode", "paper", "address", "long", "layer"],
                    default=None,
                    help="run one leg only (profiling runs)")
    ap.add_argument("--no-sequential", action="store_true",
                    help="skip the reference timing of the forward step as three separate calls")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the memory-initialisation and decode legs")
    ap.add_argument("--chunk", type=int, default=384,
                    help="tokens per pipeline stage of the forward step (0: the library's choice, a "
                         "quarter of T; 384, measured best for this workload, by default)")
    ap.add_argument("--learned-chunk", type=int, default=1280,
                    help="tokens per pipeline stage of the learned-M0 forward step (0: the library's "
                         "choice, a quarter of T; 1280, measured best there, by default)")
    ap.add_argument("--train-chunk", type=int, default=0,
                    help="tokens per pipeline stage of the training step's forward (0: the library's "
                         "choice, measured best there)")
    ap.add_argument("--paper-shapes", default="1.4b,8b",
                    help="the paper's layer shapes the paper leg times (comma-separated: 1.4b, 8b)")
    ap.add_argument("--calib", action="store_true",
                    help="first run one plain 512 MiB copy (sdm_mem_init from a [16, 65536, 128] fp32 "
                         "source): the reference dispatch for scaling HBM counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the SDM path is measured on one GPU only (the streams shard with no exchange "
                                   "in the forward; no multi-GPU path is built); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2607_07386_amd import sdm

    def to_dev(st):
        if st.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(st.bits).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(st.f32)).to(dev)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    out = {"metric": METRIC}
    w = synth.WORKLOADS[1]

    if args.calib:
        src = torch.ones((16, 65536, 128), dtype=torch.float32, device=dev)
        dst = torch.empty((1, 16, 65536, 128), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        sdm.mem_init(dst, src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = src.numel() * 4
        del src, dst

    # ------------------------------------------------------------ forward
    if args.only in (None, "fwd"):
        log("generating forward workload inputs")
        inp = synth.Inputs(w)
        q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
        al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
        B, H, T = w.B, w.H, w.T
        mem = torch.empty((B, H, w.N, w.d_v), dtype=torch.float32, device=dev)
        sdm.mem_init(mem, None)
        ws = sdm.fwd_workspace(B, H, T, w.topk, w.topk, dev)
        y = torch.empty((B, H, T, w.d_v), dtype=torch.float32, device=dev)
        outs = {n: torch.empty((B, H, T, w.topk), dtype=dt, device=dev)
                for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32),
                              ("w_idx", torch.int32), ("w_val", torch.float32))}

        def step():
            # addressing of both sides and the scan in one call, pipelined over chunks of tokens
            sdm.forward(q, k, cb, cb, v, al, be, mem, w.N, w.topk, workspace=ws, y=y, out=outs,
                        chunk=args.chunk)

        def step_sequential():
            r_idx, r_val = sdm.address(q, cb, w.N, w.topk)
            w_idx, w_val = sdm.address(k, cb, w.N, w.topk)
            sdm.scan_fwd(w_idx, w_val, r_idx, r_val, v, al, be, mem, workspace=ws, y=y)

        log("warmup")
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        # events inside the timed steps bracket the scan kernel only (the roofline's
        # kernel); the other kernels are timed in extra steps afterwards
        sdm.profile_select(["fwd_scan"])
        sdm.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        log(f"timing {args.steps} steps")
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        e0.record(stream)
        evs[0].record(stream)
        for i in range(args.steps):
            step()
            evs[i + 1].record(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        per_step = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
        kern = {"fwd_scan": sdm.profile_read("fwd_scan")}
        sdm.profile_enable(False)
        sdm.profile_select(None)
        sdm.profile_enable(True)
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        kern_all = {name: sdm.profile_read(name) for name in ("address", "fwd_prep", "fwd_scan")}
        sdm.profile_enable(False)
        # reference: the same work as three separate calls on one stream (not the reported value)
        ms_seq = seq_scan_ms = None
        if not args.no_sequential:
            sdm.profile_enable(True)
            e0.record(stream)
            for _ in range(3):
                step_sequential()
            e1.record(stream)
            torch.cuda.synchronize()
            ms_seq = round(e0.elapsed_time(e1) / 3, 4)
            t_scan, n_scan = sdm.profile_read("fwd_scan")
            t_addr, n_addr = sdm.profile_read("address")
            sdm.profile_enable(False)
            seq_scan_ms = t_scan / max(n_scan, 1)
            out["scoring"] = scoring_mfma(w, t_addr / max(n_addr, 1))
        tokens = B * T
        scan_launches = max(kern["fwd_scan"][1], 1)
        scan_ms = kern["fwd_scan"][0] / scan_launches
        unit_bytes = fwd_scan_bytes_per_token_head(w.topk, w.topk, w.d_v, 2)
        tokens_per_launch = B * H * T * args.steps / scan_launches
        launch_bytes = round(unit_bytes * tokens_per_launch)
        achieved = launch_bytes / (scan_ms * 1e-3) / 1e9
        # stricter count from the ids of the last step (host copy, outside the timed region)
        r_last, w_last = outs["r_idx"], outs["w_idx"]
        uniq_bytes, uniq_tokens = unique_row_bytes(
            w_last.reshape(B * H, T, -1).cpu().numpy(), r_last.reshape(B * H, T, -1).cpu().numpy(), w.d_v, 2)
        uniq_launch = uniq_bytes * tokens_per_launch / uniq_tokens
        traffic = None
        if os.path.exists(TRAFFIC_FILE):
            tr = json.load(open(TRAFFIC_FILE))
            if tr.get("scan_sources_sha256") == scan_src_hash():
                traffic = tr.get("hbm_bytes_per_launch")
        out.update({
            "value": round(tokens / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
            "data": "synthetic",
            "config": {"workload": "1.4B-shaped SDM layer forward: B=8 H=16 T=4096 d_k=d_v=128 "
                                   "N=65536 top-32 reads/writes, bf16 q/k/v/gates, fp32 memory",
                       "global_batch": B, "seq_len": T, "heads": H, "slots_per_head": w.N,
                       "topk": w.topk, "inputs": "bf16", "state": "f32", "parallelism": "none (1 GPU)",
                       "pipeline": f"sdm_forward(chunk={args.chunk}): addressing of stage c+1 overlaps the "
                                   f"scan of stage c; {round(scan_launches / args.steps)} stages per step, "
                                   f"{round(args.steps * T / scan_launches)} tokens on average"},
            "ms_per_step_median": round(per_step[len(per_step) // 2], 4),
            "ms_per_step_min": round(per_step[0], 4),
            "ms_per_step_sequential": ms_seq,
            "kernels_ms": {n: round(v[0] / max(v[1], 1), 4) for n, v in kern_all.items()},
            "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                         "kernel": SCAN_KERNEL, "algorithmic_bytes_per_token_head": unit_bytes,
                         "algorithmic_bytes_per_launch": launch_bytes, "kernel_ms": round(scan_ms, 4),
                         "unique_row_bytes_per_launch": round(uniq_launch),
                         "frac_unique_rows": round(uniq_launch / (scan_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         # the same kernel over all 4096 tokens with nothing running beside it
                         # (the sequential reference above)
                         "standalone_kernel_ms": None if seq_scan_ms is None else round(seq_scan_ms, 4),
                         "frac_standalone": None if seq_scan_ms is None else round(
                             unit_bytes * B * H * T / (seq_scan_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        })
        if not args.no_cpu_baseline:
            log("cpu baseline (oracle)")
            out["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_streams, min(args.cpu_tokens, w.T))
        del q, k, v, al, be, cb, mem, ws, y, outs
        torch.cuda.empty_cache()

    # ------------------------------------------------------------ training step
    if not args.no_train and args.only in (None, "train"):
        wt = synth.WORKLOADS[4]
        log("generating training workload inputs")
        inp = synth.Inputs(wt)
        q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
        al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
        dy = torch.from_numpy(inp.dy()).to(dev)
        B, H, T = wt.B, wt.H, wt.T
        mem = torch.zeros((B, H, wt.N, wt.d_v), dtype=torch.float32, device=dev)
        saved = sdm.saved_buffer(B, H, T, wt.topk, wt.d_v, dev)
        fws = sdm.fwd_workspace(B, H, T, wt.topk, wt.topk, dev)
        bws = sdm.bwd_workspace(B, H, T, wt.topk, wt.topk, wt.d_v, dev)
        dmem0 = torch.empty_like(mem)
        y = torch.empty((B, H, T, wt.d_v), dtype=torch.float32, device=dev)

        touts = {n: torch.empty((B, H, T, wt.topk), dtype=dt, device=dev)
                 for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32),
                               ("w_idx", torch.int32), ("w_val", torch.float32))}

        def tstep():
            # forward with the undo log (addressing pipelined with the scan), then the backward
            o = sdm.forward(q, k, cb, cb, v, al, be, mem, wt.N, wt.topk, saved=saved, workspace=fws,
                            y=y, out=touts, chunk=args.train_chunk)
            sdm.scan_bwd(o["w_idx"], o["w_val"], o["r_idx"], o["r_val"], v, al, be, mem, saved, dy,
                         cb_q=cb, cb_k=cb, d_k=wt.d_k, chunk=wt.chunk, workspace=bws, dmem0=dmem0)

        for _ in range(args.warmup):
            tstep()
        torch.cuda.synchronize()
        sdm.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        log(f"timing {args.steps} training steps")
        e0.record(stream)
        for _ in range(args.steps):
            tstep()
        e1.record(stream)
        torch.cuda.synchronize()
        tms = e0.elapsed_time(e1) / args.steps
        kern = {n: sdm.profile_read(n) for n in ("address", "fwd_prep", "fwd_scan", "bwd_prep",
                                                   "bwd_scan", "bwd_reduce", "address_bwd", "mem_init")}
        sdm.profile_enable(False)
        # the backward scan's roofline: its algorithmic bytes per launch (every row the
        # reverse step touches, plus dy, dv and v) over its mean event-timed duration
        b_unit = bwd_scan_bytes_per_token_head(wt.topk, wt.topk, wt.d_v, 2)
        b_launches = max(kern["bwd_scan"][1], 1)
        b_ms = kern["bwd_scan"][0] / b_launches
        b_tokens = B * H * T * args.steps / b_launches
        b_bytes = round(b_unit * b_tokens)
        b_ach = b_bytes / (b_ms * 1e-3) / 1e9
        out["train"] = {
            "value": round(B * T / (tms * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(tms, 4),
            "workload": "training step: B=4 H=16 T=4096 d_k=d_v=128 N=65536 top-32, chunk 64; "
                        "address(q,k) + forward with undo log (one sdm_forward call) + backward "
                        "(dq, dk, dv, dalpha, dbeta, dM0)",
            "kernels_ms": {n: round(v[0] / max(v[1], 1), 4) for n, v in kern.items()},
            "roofline": {"bound": "hbm", "kernel": "bwd_scan", "achieved": round(b_ach, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(b_ach / HBM_PEAK_GBS, 4), "traffic": None,
                         "algorithmic_bytes_per_token_head": b_unit, "algorithmic_bytes_per_launch": b_bytes,
                         "kernel_ms": round(b_ms, 4), "launches_per_step": round(b_launches / args.steps, 2)},
        }
    extra = not args.no_extra
    # ------------------------------------------------------------ learned M0 (a9 + forward)
    if (extra and args.only is None) or args.only == "learned":
        out.update(learned_m0_leg(sdm, to_dev, stream, dev, args))

    # ------------------------------------------------------------ decode steps (T = 1)
    if (extra and args.only is None) or args.only == "decode":
        wd = synth.Workload("decode", B=16, H=16, T=1, d_k=128, d_v=128, N=65536, topk=32, seed=5)
        log("timing single-token decode steps")
        ind = synth.Inputs(wd)
        q, k, v = to_dev(ind.q), to_dev(ind.k), to_dev(ind.v)
        al, be, cb = to_dev(ind.alpha), to_dev(ind.beta), to_dev(ind.codebook)
        mem = torch.zeros((wd.B, wd.H, wd.N, wd.d_v), dtype=torch.float32, device=dev)
        ws = sdm.fwd_workspace(wd.B, wd.H, 1, wd.topk, wd.topk, dev)
        y = torch.empty((wd.B, wd.H, 1, wd.d_v), dtype=torch.float32, device=dev)
        douts = {n: torch.empty((wd.B, wd.H, 1, wd.topk), dtype=dt, device=dev)
                 for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32),
                               ("w_idx", torch.int32), ("w_val", torch.float32))}

        def dstep():
            sdm.forward(q, k, cb, cb, v, al, be, mem, wd.N, wd.topk, workspace=ws, y=y, out=douts)

        for _ in range(5):
            dstep()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        nd = 100
        e0.record(stream)
        for _ in range(nd):
            dstep()
        e1.record(stream)
        torch.cuda.synchronize()
        dms = e0.elapsed_time(e1) / nd
        # the same steps replayed from a HIP graph of 20 captured calls: the device's
        # time per step, without the per-call host work (argument checks, launch)
        gsteps = 20
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            dstep()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(gsteps):
                dstep()
        graph.replay()
        torch.cuda.synchronize()
        nrep = 10
        e0.record(stream)
        for _ in range(nrep):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        gms = e0.elapsed_time(e1) / (nrep * gsteps)
        del graph
        out["decode"] = {
            "workload": f"one token per step for B={wd.B} sequences, H={wd.H}, N={wd.N}, d={wd.d_v}, "
                        f"top-{wd.topk}; memory resident; one sdm_forward call per step (T = 1: one fused launch)",
            "us_per_step": round(dms * 1e3, 2), "tokens_per_s": round(wd.B / (dms * 1e-3), 1),
            "us_per_step_graph": round(gms * 1e3, 2), "tokens_per_s_graph": round(wd.B / (gms * 1e-3), 1)}
        del q, k, v, al, be, cb, mem, ws, y, douts
        torch.cuda.empty_cache()

    # ------------------------------------------------------------ addressing alone
    if args.only == "address":
        # both sides' addressing of the forward workload, one call after the other
        log("addressing: generating inputs")
        ia = synth.Inputs(w)
        q, k, cb = to_dev(ia.q), to_dev(ia.k), to_dev(ia.codebook)
        for _ in range(args.warmup):
            sdm.address(q, cb, w.N, w.topk)
            sdm.address(k, cb, w.N, w.topk)
        torch.cuda.synchronize()
        sdm.profile_enable(True)
        for _ in range(args.steps):
            sdm.address(q, cb, w.N, w.topk)
            sdm.address(k, cb, w.N, w.topk)
        torch.cuda.synchronize()
        t_addr, n_addr = sdm.profile_read("address")
        sdm.profile_enable(False)
        out["scoring"] = scoring_mfma(w, t_addr / max(n_addr, 1))
        del q, k, cb

    # ------------------------------------------------------------ long context: both scan schedules
    if (extra and args.only is None) or args.only == "long":
        wl = synth.WORKLOADS[2]
        log("long context: generating inputs and addressing")
        il = synth.Inputs(wl)
        q, k, v = to_dev(il.q), to_dev(il.k), to_dev(il.v)
        al, be, cb = to_dev(il.alpha), to_dev(il.beta), to_dev(il.codebook)
        ri, rv = sdm.address(q, cb, wl.N, wl.topk)
        wi, wv = sdm.address(k, cb, wl.N, wl.topk)
        del q, k
        mem = torch.zeros((wl.B, wl.H, wl.N, wl.d_v), dtype=torch.float32, device=dev)
        yl = torch.empty((wl.B, wl.H, wl.T, wl.d_v), dtype=torch.float32, device=dev)
        wsf = sdm.fwd_workspace(wl.B, wl.H, wl.T, wl.topk, wl.topk, dev)
        wsc = sdm.chunked_workspace(wl.B, wl.H, wl.T, wl.topk, wl.topk, dev)
        units = wl.B * wl.H * wl.T
        lbytes = fwd_scan_bytes_per_token_head(wl.topk, wl.topk, wl.d_v, 2) * units
        res = {"workload": f"long context: B={wl.B} H={wl.H} T={wl.T} N={wl.N} d_v={wl.d_v} top-{wl.topk}, "
                           f"clustered keys; the scan alone on the workload's own slot lists",
               "scan_algorithmic_bytes": lbytes}
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for name, fn, kinds in (
                ("sequential", lambda: sdm.scan_fwd(wi, wv, ri, rv, v, al, be, mem, workspace=wsf, y=yl),
                 ("fwd_prep", "fwd_scan")),
                ("chunked", lambda: sdm.scan_fwd_chunked(wi, wv, ri, rv, v, al, be, mem, workspace=wsc, y=yl),
                 ("chunk_coef", "chunk_scan"))):
            log(f"long context: timing the {name} scan")
            fn()
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(3):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 3
            sdm.profile_enable(True)
            fn()
            torch.cuda.synchronize()
            kms = {kk: round(sdm.profile_read(kk)[0], 3) for kk in kinds}
            sdm.profile_enable(False)
            gbs = lbytes / (ms * 1e-3) / 1e9
            res[name] = {"ms": round(ms, 3), "tokens_per_s": round(wl.B * wl.T / (ms * 1e-3), 1),
                         "GB_s": round(gbs, 1), "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                         "kernels_ms": kms}
        res["chunked_speedup"] = round(res["sequential"]["ms"] / res["chunked"]["ms"], 3)
        out["long_context"] = res
        del v, al, be, cb, ri, rv, wi, wv, mem, yl, wsf, wsc
        torch.cuda.empty_cache()

    # ------------------------------------------------------------ the steps either side (gates, epilogue)
    if (extra and args.only is None) or args.only == "layer":
        out["layer"] = layer_leg(sdm, to_dev, stream, dev, args)

    # ------------------------------------------------------------ the paper's 1.4B and 8B layers
    if (extra and args.only is None) or args.only == "paper":
        # Table 1's layers, direct-mode addressing (d_k = 2 sqrt(N)), top-64 reads and writes,
        # H = 2: the 1.4B layer has N = 240^2 slots of d_v = 960 (8 sequences of 4096 tokens),
        # the 8B layer N = 480^2 slots of d_v = 1920 (4 sequences of 4096 tokens)
        shapes = (("1.4b", 240, synth.Workload("paper-1.4b-layer", B=8, H=2, T=4096, d_k=480, d_v=960,
                                               N=57600, topk=64, seed=6, codebook=False)),
                  ("8b", 480, synth.Workload("paper-8b-layer", B=4, H=2, T=4096, d_k=960, d_v=1920,
                                             N=230400, topk=64, seed=8, codebook=False)))
        out["paper_layer"] = {}
        want = set(args.paper_shapes.split(","))
        for tag, root, wp in shapes:
            if tag in want:
                out["paper_layer"][tag] = paper_layer(sdm, to_dev, wp, tag, root, stream, dev)

    print(json.dumps(out), flush=True)


def layer_leg(sdm, to_dev, stream, dev, args):
    """The cost of the steps either side of the recurrence: forward steps of the
    1.4B-shaped workload through sdm_layer_fwd (gates formed in the scan's
    records from their pre-activations, norm-gate epilogue per stage) against
    sdm_forward on precomputed gates; training steps of the training workload
    through sdm_layer_fwd + sdm_layer_bwd against sdm_forward + sdm_scan_bwd."""
    import torch

    import synth

    res = {}
    for tag, wl, train in (("fwd", synth.WORKLOADS[1], False), ("train", synth.WORKLOADS[4], True)):
        log(f"layer: {tag} inputs")
        inp = synth.Inputs(wl)
        li = synth.LayerInputs(wl)
        q, k, v, cb = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.codebook)
        a, b, g = to_dev(li.a_pre), to_dev(li.b_pre), to_dev(li.g)
        A, bdt, gm = (torch.from_numpy(x).to(dev) for x in (li.A, li.b_dt, li.gamma))
        al, be = sdm.gates(a, b, A, bdt)
        al16, be16 = al.to(torch.bfloat16), be.to(torch.bfloat16)   # the plain path's gates, in the input dtype
        B, H, T = wl.B, wl.H, wl.T
        mem = torch.zeros((B, H, wl.N, wl.d_v), dtype=torch.float32, device=dev)
        ws = sdm.fwd_workspace(B, H, T, wl.topk, wl.topk, dev)
        saved = sdm.saved_buffer(B, H, T, wl.topk, wl.d_v, dev) if train else None
        chunk = args.chunk if not train else args.train_chunk
        dout = torch.from_numpy(li.dout).to(dev) if train else None
        dy = torch.from_numpy(inp.dy()).to(dev) if train else None
        bws = sdm.bwd_workspace(B, H, T, wl.topk, wl.topk, wl.d_v, dev) if train else None
        lws = (torch.empty(sdm.lib().sdm_layer_bwd_workspace_bytes(B, H, T, wl.topk, wl.topk, wl.d_v),
                           dtype=torch.uint8, device=dev) if train else None)

        def plain():
            o = sdm.forward(q, k, cb, cb, v, al16, be16, mem, wl.N, wl.topk, saved=saved, workspace=ws, chunk=chunk)
            if train:
                sdm.scan_bwd(o["w_idx"], o["w_val"], o["r_idx"], o["r_val"], v, al16, be16, mem, saved, dy,
                             cb_q=cb, cb_k=cb, d_k=wl.d_k, chunk=wl.chunk, workspace=bws)

        def layer():
            o = sdm.layer_fwd(q, k, cb, cb, v, a, b, g, A, bdt, gm, 1e-6, 1, mem, wl.N, wl.topk, wl.topk,
                              saved=saved, workspace=ws, chunk=chunk)
            if train:
                sdm.layer_bwd(o, v, a, b, g, A, bdt, gm, 1e-6, 1, mem, saved, dout, cb_q=cb, cb_k=cb, d_k=wl.d_k,
                              chunk=wl.chunk, workspace=lws)

        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        times = {}
        for name, fn in (("plain", plain), ("layer", layer)):
            for _ in range(2):
                fn()
            torch.cuda.synchronize()
            n = max(3, args.steps // 2)
            e0.record(stream)
            for _ in range(n):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            times[name] = e0.elapsed_time(e1) / n
        sdm.profile_select(["norm_gate", "gates"])
        sdm.profile_enable(True)
        layer()
        torch.cuda.synchronize()
        kms = {kk: round(sdm.profile_read(kk)[0], 4) for kk in ("norm_gate", "gates")}
        sdm.profile_enable(False)
        sdm.profile_select(None)
        res[tag] = {"workload": f"{wl.name}: B={B} H={H} T={T} d_v={wl.d_v} top-{wl.topk}; gates from bf16 "
                                f"pre-activations (A, b_dt per head), epilogue RMS norm x SiLU gate, eps 1e-6",
                    "ms_per_step_layer": round(times["layer"], 4), "ms_per_step_plain": round(times["plain"], 4),
                    "added_ms": round(times["layer"] - times["plain"], 4),
                    "tokens_per_s_layer": round(B * T / (times["layer"] * 1e-3), 1),
                    "kernels_ms_per_step": kms}
        del q, k, v, cb, a, b, g, A, bdt, gm, al, be, al16, be16, mem, ws, saved, dout, dy, bws, lws
        torch.cuda.empty_cache()
    return res


def learned_m0_leg(sdm, to_dev, stream, dev, args):
    """The learned-M0 workload (B=4 H=8 T=8192 N=2^20 d=128 top-32): the shared
    M0 broadcast to every sequence, timed alone (excluded from the step), and
    forward steps (one sdm_forward call each, pipeline stages of args.learned_chunk) on the
    resident table, with the scan's roofline."""
    import torch

    import synth

    w3 = synth.WORKLOADS[3]
    log("learned M0: generating inputs")
    inp = synth.Inputs(w3)
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    al, be, cb = to_dev(inp.alpha), to_dev(inp.beta), to_dev(inp.codebook)
    B, H, T = w3.B, w3.H, w3.T
    # M0 ~ N(0, 0.02^2), drawn on the device: the bytes moved do not depend on the values
    # (the parity tests use the seeded host generator)
    g = torch.Generator(device=dev)
    g.manual_seed(w3.seed)
    m0 = torch.randn((H, w3.N, w3.d_v), dtype=torch.float32, device=dev, generator=g).mul_(0.02)
    mem = torch.empty((B, H, w3.N, w3.d_v), dtype=torch.float32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sdm.mem_init(mem, m0)
    torch.cuda.synchronize()
    log("learned M0: timing the broadcast")
    e0.record(stream)
    for _ in range(3):
        sdm.mem_init(mem, m0)
    e1.record(stream)
    torch.cuda.synchronize()
    ims = e0.elapsed_time(e1) / 3
    moved = mem.numel() * 4 + m0.numel() * 4
    res = {"mem_init": {
        "workload": f"M0 [H={H}, N={w3.N}, d_v={w3.d_v}] fp32 broadcast to B={B} sequences",
        "ms": round(ims, 4), "bytes_written": mem.numel() * 4, "bytes_read_unique": m0.numel() * 4,
        "GB_s": round(moved / (ims * 1e-3) / 1e9, 1)}}
    ws = sdm.fwd_workspace(B, H, T, w3.topk, w3.topk, dev)
    y = torch.empty((B, H, T, w3.d_v), dtype=torch.float32, device=dev)
    outs = {n: torch.empty((B, H, T, w3.topk), dtype=dt, device=dev)
            for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32),
                          ("w_idx", torch.int32), ("w_val", torch.float32))}

    chunk = getattr(args, "learned_chunk", 0)

    def step():
        sdm.forward(q, k, cb, cb, v, al, be, mem, w3.N, w3.topk, workspace=ws, y=y, out=outs, chunk=chunk)

    sdm.mem_init(mem, m0)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"learned M0: timing {args.steps} forward steps")
    sdm.profile_select(["fwd_scan"])
    sdm.profile_enable(True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    t_scan, n_scan = sdm.profile_read("fwd_scan")
    sdm.profile_enable(False)
    sdm.profile_select(None)
    sdm.profile_enable(True)
    for _ in range(2):
        step()
    torch.cuda.synchronize()
    kms = {n: round(sdm.profile_read(n)[0] / 2, 4) for n in ("address", "fwd_prep", "fwd_scan")}
    sdm.profile_enable(False)
    n_scan = max(n_scan, 1)
    scan_ms = t_scan / n_scan
    unit = fwd_scan_bytes_per_token_head(w3.topk, w3.topk, w3.d_v, 2)
    launch_bytes = round(unit * B * H * T * args.steps / n_scan)
    ach = launch_bytes / (scan_ms * 1e-3) / 1e9
    res["learned_m0"] = {
        "workload": f"learned initial memory: B={B} H={H} T={T} d_k=d_v={w3.d_v} N={w3.N} top-{w3.topk}, "
                    f"bf16 inputs, fp32 memory (16 GiB); one sdm_forward call per step (stages of "
                    f"{chunk or 'T/4'} tokens), the M0 broadcast excluded (under mem_init)",
        "value": round(B * T / (ms * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(ms, 4),
        "kernels_ms_per_step": kms,
        "roofline": {"bound": "hbm", "kernel": "fwd_scan", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes_per_token_head": unit, "algorithmic_bytes_per_launch": launch_bytes,
                     "kernel_ms": round(scan_ms, 4), "launches_per_step": round(n_scan / args.steps, 2)}}
    del q, k, v, al, be, cb, m0, mem, ws, y, outs
    torch.cuda.empty_cache()
    return res


def paper_layer(sdm, to_dev, wp, tag, root, stream, dev):
    """Forward and training steps of one of the paper's layer shapes; returns the timings."""
    import torch

    import synth

    log(f"paper {tag} layer: generating inputs")
    ip = synth.Inputs(wp)
    q, k, v = to_dev(ip.q), to_dev(ip.k), to_dev(ip.v)
    al, be = to_dev(ip.alpha), to_dev(ip.beta)
    B, H, T = wp.B, wp.H, wp.T
    mem = torch.empty((B, H, wp.N, wp.d_v), dtype=torch.float32, device=dev)
    sdm.mem_init(mem, None)
    ws = sdm.fwd_workspace(B, H, T, wp.topk, wp.topk, dev)
    y = torch.empty((B, H, T, wp.d_v), dtype=torch.float32, device=dev)
    pouts = {n: torch.empty((B, H, T, wp.topk), dtype=dt, device=dev)
             for n, dt in (("r_idx", torch.int32), ("r_val", torch.float32),
                           ("w_idx", torch.int32), ("w_val", torch.float32))}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        sdm.profile_enable(True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        kms = {name: round(sdm.profile_read(name)[0] / n, 4)
               for name in ("address", "fwd_prep", "fwd_scan", "bwd_prep", "bwd_scan", "bwd_reduce",
                            "address_bwd", "mem_init")}
        sdm.profile_enable(False)
        return e0.elapsed_time(e1) / n, {kk: vv for kk, vv in kms.items() if vv > 0}

    log(f"paper {tag} layer: timing forward steps")
    pms, pk = timed(lambda: sdm.forward(q, k, None, None, v, al, be, mem, wp.N, wp.topk, workspace=ws,
                                        y=y, out=pouts), 5)
    # both sides' addressing alone: inside the pipelined step the address launches share the
    # device with the scan, and their event times measure that overlap, not their cost
    sdm.address(q, None, wp.N, wp.topk)
    torch.cuda.synchronize()
    sdm.profile_enable(True)
    for _ in range(3):
        sdm.address(q, None, wp.N, wp.topk)
        sdm.address(k, None, wp.N, wp.topk)
    torch.cuda.synchronize()
    addr_alone = sdm.profile_read("address")[0] / 3
    sdm.profile_enable(False)
    fbytes = fwd_scan_bytes_per_token_head(wp.topk, wp.topk, wp.d_v, 2) * B * H * T
    res = {"workload": f"the paper's {tag.upper()} layer shape: B={B} H={H} T={T} N={wp.N} (sqrt {root}) "
                       f"d_v={wp.d_v} top-{wp.topk} reads/writes, direct-mode addressing d_k={wp.d_k}, "
                       f"bf16 inputs, fp32 memory",
           "fwd": {"ms_per_step": round(pms, 3), "tokens_per_s": round(B * T / (pms * 1e-3), 1),
                   "kernels_ms": pk, "address_both_sides_alone_ms": round(addr_alone, 4),
                   "scan_algorithmic_bytes": fbytes,
                   "scan_GB_s": round(fbytes / (pk["fwd_scan"] * 1e-3) / 1e9, 1),
                   "scan_frac_of_hbm_peak": round(fbytes / (pk["fwd_scan"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}}
    log(f"paper {tag} layer: timing training steps")
    saved = sdm.saved_buffer(B, H, T, wp.topk, wp.d_v, dev)
    bws = sdm.bwd_workspace(B, H, T, wp.topk, wp.topk, wp.d_v, dev)
    dmem0 = torch.empty((B, H, wp.N, wp.d_v), dtype=torch.float32, device=dev)
    dy = torch.from_numpy(ip.dy()).to(dev)

    def pstep_train():
        o = sdm.forward(q, k, None, None, v, al, be, mem, wp.N, wp.topk, saved=saved, workspace=ws, y=y,
                        out=pouts)
        sdm.scan_bwd(o["w_idx"], o["w_val"], o["r_idx"], o["r_val"], v, al, be, mem, saved, dy,
                     d_k=wp.d_k, chunk=64, workspace=bws, dmem0=dmem0)

    tms, tk = timed(pstep_train, 3)
    # backward rows: (4W + 3R) d_v fp32 (M_t and G reads, G and undo writes, saved P), plus
    # dy and dv (fp32) and v (bf16) per token-head
    bbytes = ((4 * wp.topk + 3 * wp.topk) * wp.d_v * 4 + wp.d_v * (4 + 4 + 2)) * B * H * T
    res["train"] = {"ms_per_step": round(tms, 3), "tokens_per_s": round(B * T / (tms * 1e-3), 1),
                    "kernels_ms": tk, "bwd_scan_algorithmic_bytes": bbytes,
                    "bwd_scan_GB_s": round(bbytes / (tk["bwd_scan"] * 1e-3) / 1e9, 1),
                    "bwd_scan_frac_of_hbm_peak": round(bbytes / (tk["bwd_scan"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del q, k, v, al, be, mem, ws, y, pouts, saved, bws, dmem0, dy
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
