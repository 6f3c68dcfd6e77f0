"""CPU oracle for the SDM recurrence: test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library and its Python binding
never import it.  All arithmetic is in ``sdm_oracle.c`` (plain C, fp64); this
file only compiles it and marshals numpy arrays.

Function map (paper passages in the C source):
  address        top-k-of-top-k addressing (Sec. 2, Sec. 3.1 step 1, Sec. 4, App. A.2)
  address_brute  the same by exhaustive scoring of all N slots
  scan_fwd       Sec. 3.1 steps 2-3, Eqs. (sdm-decay), (sdm-write), (sdm-read)
  scan_bwd       reverse mode with undo of the in-place writes (App. A.3)
  address_bwd    gradient of the softmax weights w.r.t. the projected vectors
  gates          forget / input gates from their pre-activations (Sec. 3.1 step 2)
  gates_bwd      their reverse mode, with the per-head sums for A and b_dt
  norm_gate      RMS norm of each head's read vector times the output gate (Sec. 3.1 step 4)
  norm_gate_bwd  its reverse mode
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sdm_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, no fast-math, no FMA contraction)."""
    if not force and os.path.exists(_LIB_PATH) and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC",
           "-std=c11", "-Wall", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
                build()
            lib = ctypes.CDLL(_LIB_PATH)
            P = ctypes.c_void_p
            I = ctypes.c_int
            L = ctypes.c_int64
            lib.orc_address.argtypes = [P, P, I, I, I, I, L, I, I, P, P, P]
            lib.orc_address_brute.argtypes = [P, P, I, I, I, I, L, I, I, P, P, P]
            lib.orc_scan_fwd.argtypes = [I, I, I, L, I, I, P, P, P, P, P, P, P, P, P, P]
            lib.orc_scan_bwd.argtypes = [I, I, I, L, I, I, P, P, P, P, P, P, P, P, P, P, P,
                                         P, P, P, P, P]
            lib.orc_address_bwd.argtypes = [P, I, I, I, I, L, I, P, P, P, P]
            lib.orc_gates.argtypes = [I, I, I, P, P, P, P, P, P]
            lib.orc_gates_bwd.argtypes = [I, I, I, P, P, P, P, P, P, P, P, P, P]
            D = ctypes.c_double
            lib.orc_norm_gate.argtypes = [L, I, P, P, P, D, I, P, P]
            lib.orc_norm_gate_bwd.argtypes = [L, I, P, P, P, D, I, P, P, P, P]
            lib.orc_set_threads.argtypes = [I]
            lib.orc_set_threads.restype = None
            for f in ("orc_address", "orc_address_brute", "orc_scan_fwd", "orc_scan_bwd",
                      "orc_address_bwd", "orc_gates", "orc_gates_bwd", "orc_norm_gate", "orc_norm_gate_bwd",
                      "orc_max_threads"):
                getattr(lib, f).restype = ctypes.c_int
            _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def max_threads() -> int:
    return _load().orc_max_threads()


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (for timing)."""
    _load().orc_set_threads(int(n))


def address(x, codebook, N: int, topk: int, decide_f32: bool = True, brute: bool = False):
    """x [B,H,T,dk]; codebook [H,2,sqrtN,dk/2] or None.  Returns idx, val, score."""
    x = _f64(x)
    cb = _f64(codebook)
    B, H, T, dk = x.shape
    idx = np.empty((B, H, T, topk), np.int32)
    val = np.empty((B, H, T, topk), np.float64)
    score = np.empty((B, H, T, topk), np.float64)
    fn = _load().orc_address_brute if brute else _load().orc_address
    rc = fn(_p(x), _p(cb), B, H, T, dk, N, topk, int(decide_f32), _p(idx), _p(val), _p(score))
    if rc != 0:
        raise ValueError("oracle address: invalid arguments")
    return idx, val, score


def scan_fwd(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, save: bool = False):
    """Arrays [S,T,...] (any leading batch dims flattened into S); mem [S,N,dv] fp64 is
    updated in place to M_T.  Returns y [S,T,dv] and (if save) P [S,T,W,dv]."""
    lead = v.shape[:-2]
    T, dv = v.shape[-2:]
    S = int(np.prod(lead)) if lead else 1
    W = w_idx.shape[-1]
    R = r_idx.shape[-1]
    assert mem.dtype == np.float64 and mem.flags.c_contiguous
    N = mem.shape[-2]
    wi, ri = _i32(w_idx), _i32(r_idx)
    wv, rv, vv, al, be = _f64(w_val), _f64(r_val), _f64(v), _f64(alpha), _f64(beta)
    y = np.empty(lead + (T, dv), np.float64)
    saved = np.empty(lead + (T, W, dv), np.float64) if save else None
    _load().orc_scan_fwd(S, T, dv, N, W, R, _p(wi), _p(wv), _p(ri), _p(rv), _p(vv), _p(al), _p(be),
                         _p(mem), _p(y), _p(saved))
    return (y, saved) if save else y


def scan_bwd(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, saved, dy, dmem_T=None):
    """mem [S,N,dv] = M_T on entry, M_0 on return.  Returns dict of gradients."""
    lead = v.shape[:-2]
    T, dv = v.shape[-2:]
    S = int(np.prod(lead)) if lead else 1
    W = w_idx.shape[-1]
    R = r_idx.shape[-1]
    N = mem.shape[-2]
    assert mem.dtype == np.float64 and mem.flags.c_contiguous
    G = np.zeros(mem.shape, np.float64) if dmem_T is None else np.array(dmem_T, dtype=np.float64)
    out = dict(dv=np.empty(lead + (T, dv)), dalpha=np.empty(lead + (T,)), dbeta=np.empty(lead + (T,)),
               dw_val=np.empty(lead + (T, W)), dr_val=np.empty(lead + (T, R)))
    wi, ri = _i32(w_idx), _i32(r_idx)
    wv, rv, vv, al, be = _f64(w_val), _f64(r_val), _f64(v), _f64(alpha), _f64(beta)
    sv, yb = _f64(saved), _f64(dy)
    _load().orc_scan_bwd(S, T, dv, N, W, R, _p(wi), _p(wv), _p(ri), _p(rv), _p(vv), _p(al), _p(be),
                         _p(mem), _p(sv), _p(yb), _p(G), _p(out["dv"]), _p(out["dalpha"]),
                         _p(out["dbeta"]), _p(out["dw_val"]), _p(out["dr_val"]))
    out["dmem0"] = G
    return out


def address_bwd(codebook, idx, val, dval, N: int, d_k: int):
    """dL/dx [B,H,T,dk] from dL/dval through the softmax and the sub-key scores."""
    idx = _i32(idx)
    val, dval, cb = _f64(val), _f64(dval), _f64(codebook)
    B, H, T, k = idx.shape
    dx = np.empty((B, H, T, d_k), np.float64)
    rc = _load().orc_address_bwd(_p(cb), B, H, T, d_k, N, k, _p(idx), _p(val), _p(dval), _p(dx))
    if rc != 0:
        raise ValueError("oracle address_bwd: invalid arguments")
    return dx


def gates(a, b, A, b_dt):
    """a, b [B,H,T] pre-activations; A, b_dt [H].  Returns alpha, beta [B,H,T]."""
    a, b, A, bd = _f64(a), _f64(b), _f64(A), _f64(b_dt)
    H = A.shape[0]
    T = a.shape[-1]
    S = a.size // T if T else int(np.prod(a.shape[:-1]))
    al, be = np.empty(a.shape), np.empty(a.shape)
    if _load().orc_gates(S, H, T, _p(a), _p(b), _p(A), _p(bd), _p(al), _p(be)) != 0:
        raise ValueError("oracle gates: invalid arguments")
    return al, be


def gates_bwd(a, b, A, b_dt, dalpha, dbeta):
    """Gradients of the gates: returns da, db [B,H,T] and dA, db_dt [H]."""
    a, b, A, bd = _f64(a), _f64(b), _f64(A), _f64(b_dt)
    dal, dbe = _f64(dalpha), _f64(dbeta)
    H = A.shape[0]
    T = a.shape[-1]
    S = a.size // T if T else int(np.prod(a.shape[:-1]))
    da, db = np.empty(a.shape), np.empty(a.shape)
    dA, dbd = np.empty(H), np.empty(H)
    if _load().orc_gates_bwd(S, H, T, _p(a), _p(b), _p(A), _p(bd), _p(dal), _p(dbe), _p(da), _p(db), _p(dA),
                             _p(dbd)) != 0:
        raise ValueError("oracle gates_bwd: invalid arguments")
    return da, db, dA, dbd


def norm_gate(y, g, gamma, eps: float, act: int):
    """y, g [..., d_v]; gamma [d_v].  Returns o [..., d_v] and rstd [...]."""
    y, g, gm = _f64(y), _f64(g), _f64(gamma)
    dv = y.shape[-1]
    rows = y.size // dv
    o = np.empty(y.shape)
    rstd = np.empty(y.shape[:-1])
    if _load().orc_norm_gate(rows, dv, _p(y), _p(g), _p(gm), float(eps), int(act), _p(o), _p(rstd)) != 0:
        raise ValueError("oracle norm_gate: invalid arguments")
    return o, rstd


def norm_gate_bwd(y, g, gamma, eps: float, act: int, dout):
    """Returns dy, dg [..., d_v] and dgamma [d_v]."""
    y, g, gm, do = _f64(y), _f64(g), _f64(gamma), _f64(dout)
    dv = y.shape[-1]
    rows = y.size // dv
    dy, dg, dgm = np.empty(y.shape), np.empty(y.shape), np.empty(dv)
    if _load().orc_norm_gate_bwd(rows, dv, _p(y), _p(g), _p(gm), float(eps), int(act), _p(do), _p(dy), _p(dg),
                                 _p(dgm)) != 0:
        raise ValueError("oracle norm_gate_bwd: invalid arguments")
    return dy, dg, dgm


def layer_forward(x_q, x_k, cb, v, alpha, beta, m0, N, topk, decide_f32=True, save=False):
    """Convenience: address both sides, then run the forward scan.  m0 [S,N,dv] fp64 (copied)."""
    ri, rv, rs = address(x_q, cb, N, topk, decide_f32)
    wi, wv, ws = address(x_k, cb, N, topk, decide_f32)
    mem = np.array(m0, dtype=np.float64, copy=True)
    res = scan_fwd(wi, wv, ri, rv, v, alpha, beta, mem, save=save)
    return dict(w_idx=wi, w_val=wv, r_idx=ri, r_val=rv, mem=mem,
                y=res[0] if save else res, saved=res[1] if save else None)
