"""Python binding of libsdm.so: argument marshalling only.

Every step of the SDM path runs in the HIP kernels behind the C ABI declared
in ``include/sdm.h``; this module checks every tensor's shape, dtype and
placement against the sizes it passes (before any launch), allocates
outputs and workspaces with torch (device memory), and passes raw pointers and
the current HIP stream.  There is no fallback: if the library is missing or a
call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsdm.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "sdm.h")

SDM_F32, SDM_BF16 = 0, 1
_STATUS = {0: "SDM_OK", -1: "SDM_ERR_INVALID_ARG", -2: "SDM_ERR_UNSUPPORTED",
           -3: "SDM_ERR_WORKSPACE", -4: "SDM_ERR_HIP", -5: "SDM_ERR_DEVICE_CHECK"}


class SdmError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed: {_STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libsdm.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} not found: build it with "
                              "`python -m paper_2607_07386_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P, I, I64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
        L.sdm_address.argtypes = [P, I, P, I, I, I, I, I64, I, P, P, P, P]
        L.sdm_scan_fwd.argtypes = [P, P, I, P, P, I, P, P, P, I, P, I, I, I, I, I64, P, P, SZ, P, SZ, P]
        L.sdm_scan_bwd.argtypes = [P, P, I, I, P, P, I, P, P, I, P, P, P, I, P, P, SZ, P, P, I,
                                   I, I, I, I, I64, P, P, P, P, P, P, P, P, P, SZ, P]
        L.sdm_mem_init.argtypes = [P, P, I, I, I64, I, P]
        L.sdm_forward.argtypes = [P, P, I, P, P, I, I, P, P, P, I, P, I, I, I, I, I64, P, P, P, P, P, P,
                                  SZ, I, P, SZ, P]
        L.sdm_scan_fwd_chunked.argtypes = [P, P, I, P, P, I, P, P, P, I, P, I, I, I, I, I64, P, P, SZ, P]
        F = ctypes.c_float
        L.sdm_gates.argtypes = [P, P, I, P, P, I, I, I, P, P, P]
        L.sdm_gates_bwd.argtypes = [P, P, I, P, P, P, P, I, I, I, P, P, P, P, P]
        L.sdm_norm_gate.argtypes = [P, P, I, P, F, I, I, I, I, I, P, P, P]
        L.sdm_norm_gate_bwd_workspace_bytes.argtypes = [I, I, I, I]
        L.sdm_norm_gate_bwd_workspace_bytes.restype = SZ
        L.sdm_norm_gate_bwd.argtypes = [P, P, I, P, F, I, P, I, I, I, I, P, P, P, P, SZ, P]
        L.sdm_layer_fwd.argtypes = [P, P, I, P, P, I, I, I, P, P, P, P, I, P, P, P, F, I, P, I, I, I, I, I64,
                                    P, P, P, P, P, P, P, P, SZ, I, P, SZ, P]
        L.sdm_layer_bwd_workspace_bytes.argtypes = [I, I, I, I, I, I]
        L.sdm_layer_bwd_workspace_bytes.restype = SZ
        L.sdm_layer_bwd.argtypes = [P, P, I, I, P, P, I, P, P, I, P, P, P, P, I, P, P, P, F, I, P, P, SZ, P, P,
                                    P, I, I, I, I, I, I64, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
        L.sdm_forward_noalloc.argtypes = [P, P, I, P, P, I, I, P, P, P, I, P, I, I, I, I, I64, P, P, P, P, P,
                                          P, SZ, P]
        L.sdm_forward_noalloc_max_bytes.argtypes = []
        L.sdm_forward_noalloc_max_bytes.restype = SZ
        L.sdm_scan_fwd_workspace_bytes.argtypes = [I, I, I, I, I]
        L.sdm_scan_fwd_chunked_workspace_bytes.argtypes = [I, I, I, I, I]
        L.sdm_scan_saved_bytes.argtypes = [I, I, I, I, I]
        L.sdm_scan_bwd_workspace_bytes.argtypes = [I, I, I, I, I, I]
        for f in ("sdm_scan_fwd_workspace_bytes", "sdm_scan_saved_bytes", "sdm_scan_bwd_workspace_bytes",
                  "sdm_scan_fwd_chunked_workspace_bytes"):
            getattr(L, f).restype = SZ
        L.sdm_check_device_errors.argtypes = [P, P]
        L.sdm_profile_enable.argtypes = [I]
        L.sdm_profile_select.argtypes = [ctypes.c_uint]
        L.sdm_set_scan_slice_width.argtypes = [I]
        L.sdm_set_scan_line_io.argtypes = [I]
        L.sdm_set_chunk_scan_cols.argtypes = [I]
        L.sdm_set_scan_prefetch.argtypes = [I]
        L.sdm_profile_read.argtypes = [I, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
        L.sdm_status_string.argtypes = [I]
        L.sdm_status_string.restype = ctypes.c_char_p
        L.sdm_last_error.restype = ctypes.c_char_p
        L.sdm_version.restype = ctypes.c_char_p
        for f in ("sdm_address", "sdm_scan_fwd", "sdm_scan_fwd_chunked", "sdm_scan_bwd", "sdm_mem_init",
                  "sdm_forward_noalloc", "sdm_gates", "sdm_gates_bwd", "sdm_norm_gate", "sdm_norm_gate_bwd",
                  "sdm_layer_fwd", "sdm_layer_bwd",
                  "sdm_check_device_errors",
                  "sdm_profile_enable", "sdm_profile_select", "sdm_profile_read"):
            getattr(L, f).restype = I
        _lib = L
    return _lib


def header_symbols() -> list[str]:
    """Names of the functions include/sdm.h declares."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(sdm_[a-z_0-9]+)\s*\(", txt)))


def _check(fn: str, rc: int):
    if rc != 0:
        raise SdmError(fn, rc, lib().sdm_last_error().decode())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SDM_F32
    if t.dtype == torch.bfloat16:
        return SDM_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dev(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("all tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("all tensors must be contiguous")
        dev = dev or t.device
        if t.device != dev:
            raise ValueError("all tensors must be on the same device")
    return dev


def _expect(t, name: str, shape, dtypes):
    """Raise unless t is a tensor of exactly this shape and one of these dtypes.
    The C ABI sees only pointers and the sizes derived from one tensor, so
    every other tensor must agree with them before anything is launched."""
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {[str(d) for d in dtypes]}")


_IN = (torch.float32, torch.bfloat16)
_F32 = (torch.float32,)
_I32 = (torch.int32,)


def _expect_dims(t, name: str, nd: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dim() != nd:
        raise ValueError(f"{name} must have {nd} dimensions, got shape {tuple(t.shape)}")


def _check_scan_args(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem):
    """Shapes and dtypes of a scan's inputs; returns (B, H, T, d_v, W, R, N)."""
    _expect_dims(v, "v", 4)
    _expect_dims(mem, "mem", 4)
    _expect_dims(w_idx, "w_idx", 4)
    _expect_dims(r_idx, "r_idx", 4)
    B, H, T, dv = v.shape
    W, R = w_idx.shape[-1], r_idx.shape[-1]
    N = mem.shape[-2]
    if v.dtype not in _IN:
        raise TypeError(f"v has dtype {v.dtype}, expected float32 or bfloat16")
    _expect(alpha, "alpha", (B, H, T), (v.dtype,))
    _expect(beta, "beta", (B, H, T), (v.dtype,))
    _expect(w_idx, "w_idx", (B, H, T, W), _I32)
    _expect(w_val, "w_val", (B, H, T, W), _F32)
    _expect(r_idx, "r_idx", (B, H, T, R), _I32)
    _expect(r_val, "r_val", (B, H, T, R), _F32)
    _expect(mem, "mem", (B, H, N, dv), _F32)
    return B, H, T, dv, W, R, N


def _check_codebook(cb, name, x, N):
    if cb is None:
        return
    s = int(round(N ** 0.5))
    dk = x.shape[-1]
    _expect(cb, name, (x.shape[1], 2, s, dk // 2), (x.dtype,))


def _check_ws(ws, need: int, name="workspace"):
    if ws is None:
        return
    if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or ws.dim() != 1:
        raise TypeError(f"{name} must be a 1-D uint8 tensor")
    if ws.numel() < need:
        raise ValueError(f"{name} holds {ws.numel()} bytes, {need} needed")


def _ws(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 256-byte (or better) aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def address(x: torch.Tensor, codebook: torch.Tensor | None, N: int, topk: int,
            want_score: bool = False):
    """Product-key addressing of one side.  x [B,H,T,d_k]; codebook [H,2,sqrtN,d_k/2]
    (same dtype) or None for direct mode.  Returns (idx int32, val fp32[, score])."""
    _expect_dims(x, "x", 4)
    if x.dtype not in _IN:
        raise TypeError(f"x has dtype {x.dtype}, expected float32 or bfloat16")
    _check_codebook(codebook, "codebook", x, N)
    dev = _dev(x, codebook)
    B, H, T, dk = x.shape
    idx = torch.empty((B, H, T, topk), dtype=torch.int32, device=dev)
    val = torch.empty((B, H, T, topk), dtype=torch.float32, device=dev)
    score = torch.empty_like(val) if want_score else None
    rc = lib().sdm_address(_ptr(x), _dtype_code(x), _ptr(codebook), B, H, T, dk, N, topk,
                           _ptr(idx), _ptr(val), _ptr(score), _stream(dev))
    _check("sdm_address", rc)
    return (idx, val, score) if want_score else (idx, val)


def fwd_workspace(B, H, T, W, R, device) -> torch.Tensor:
    return _ws(lib().sdm_scan_fwd_workspace_bytes(B, H, T, W, R), device)


def saved_buffer(B, H, T, W, d_v, device) -> torch.Tensor:
    return torch.empty((B, H, T, W, d_v), dtype=torch.float32, device=device)


def scan_fwd(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, saved=None, workspace=None, y=None):
    """Sparse gated-delta scan, in place on mem (M_0 -> M_T).  Returns y [B,H,T,d_v] fp32."""
    B, H, T, dv, W, R, N = _check_scan_args(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem)
    if saved is not None:
        _expect(saved, "saved", (B, H, T, W, dv), _F32)
    if y is not None:
        _expect(y, "y", (B, H, T, dv), _F32)
    _check_ws(workspace, lib().sdm_scan_fwd_workspace_bytes(B, H, T, W, R) if workspace is not None else 0)
    dev = _dev(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, saved, y)
    if y is None:
        y = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = fwd_workspace(B, H, T, W, R, dev)
    sb = saved.numel() * 4 if saved is not None else 0
    rc = lib().sdm_scan_fwd(_ptr(w_idx), _ptr(w_val), W, _ptr(r_idx), _ptr(r_val), R, _ptr(v),
                            _ptr(alpha), _ptr(beta), _dtype_code(v), _ptr(mem), B, H, T, dv, N,
                            _ptr(y), _ptr(saved), sb, _ptr(workspace), workspace.numel(),
                            _stream(dev))
    _check("sdm_scan_fwd", rc)
    return y


def chunked_workspace(B, H, T, W, R, device) -> torch.Tensor:
    return _ws(lib().sdm_scan_fwd_chunked_workspace_bytes(B, H, T, W, R), device)


def scan_fwd_chunked(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, workspace=None, y=None):
    """The same recurrence as scan_fwd by the chunk-parallel form (64-token chunks), in place on
    mem.  Inference only (no undo log); W, R <= 64.  Returns y [B,H,T,d_v] fp32."""
    B, H, T, dv, W, R, N = _check_scan_args(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem)
    if y is not None:
        _expect(y, "y", (B, H, T, dv), _F32)
    _check_ws(workspace, lib().sdm_scan_fwd_chunked_workspace_bytes(B, H, T, W, R) if workspace is not None else 0)
    dev = _dev(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, y)
    if y is None:
        y = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = chunked_workspace(B, H, T, W, R, dev)
    rc = lib().sdm_scan_fwd_chunked(_ptr(w_idx), _ptr(w_val), W, _ptr(r_idx), _ptr(r_val), R, _ptr(v),
                                    _ptr(alpha), _ptr(beta), _dtype_code(v), _ptr(mem), B, H, T, dv, N,
                                    _ptr(y), _ptr(workspace), workspace.numel(), _stream(dev))
    _check("sdm_scan_fwd_chunked", rc)
    return y


def _forward_args(q, k, cb_q, cb_k, v, alpha, beta, mem, N, topk, saved, y, out, workspace):
    """Checks of sdm_forward's arguments; returns (B, H, T, d_k, d_v, device, outputs)."""
    _expect_dims(q, "q", 4)
    _expect_dims(v, "v", 4)
    _expect_dims(mem, "mem", 4)
    B, H, T, dk = q.shape
    dv = v.shape[-1]
    if q.dtype not in _IN:
        raise TypeError(f"q has dtype {q.dtype}, expected float32 or bfloat16")
    _expect(k, "k", (B, H, T, dk), (q.dtype,))
    _check_codebook(cb_q, "cb_q", q, N)
    _check_codebook(cb_k, "cb_k", q, N)
    if v.dtype not in _IN:
        raise TypeError(f"v has dtype {v.dtype}, expected float32 or bfloat16")
    _expect(v, "v", (B, H, T, dv), (v.dtype,))
    _expect(alpha, "alpha", (B, H, T), (v.dtype,))
    _expect(beta, "beta", (B, H, T), (v.dtype,))
    _expect(mem, "mem", (B, H, N, dv), _F32)
    if saved is not None:
        _expect(saved, "saved", (B, H, T, topk, dv), _F32)
    o = dict(out or {})
    if y is not None:
        o["y"] = y
    shp = (B, H, T, topk)
    for name, dt in (("r_idx", _I32), ("w_idx", _I32), ("r_val", _F32), ("w_val", _F32)):
        if name in o:
            _expect(o[name], f"out['{name}']", shp, dt)
    if "y" in o:
        _expect(o["y"], "y", (B, H, T, dv), _F32)
    _check_ws(workspace, lib().sdm_scan_fwd_workspace_bytes(B, H, T, topk, topk) if workspace is not None else 0)
    dev = _dev(q, k, cb_q, cb_k, v, alpha, beta, mem, saved, *o.values())
    for name, dt in (("r_idx", torch.int32), ("w_idx", torch.int32), ("r_val", torch.float32),
                     ("w_val", torch.float32)):
        if name not in o:
            o[name] = torch.empty(shp, dtype=dt, device=dev)
    if "y" not in o:
        o["y"] = torch.empty((B, H, T, dv), dtype=torch.float32, device=dev)
    return B, H, T, dk, dv, dev, o


def forward(q, k, cb_q, cb_k, v, alpha, beta, mem, N: int, topk: int, saved=None, workspace=None,
            y=None, out=None, chunk: int = 0):
    """The layer's memory forward in one call: addressing of q (read side) and k (write side)
    pipelined with the scan over chunks of tokens; in place on mem.  Returns a dict with y,
    r_idx, r_val, w_idx, w_val.  out: optional dict of preallocated outputs of those names."""
    B, H, T, dk, dv, dev, o = _forward_args(q, k, cb_q, cb_k, v, alpha, beta, mem, N, topk, saved, y, out,
                                            workspace)
    if workspace is None:
        workspace = fwd_workspace(B, H, T, topk, topk, dev)
    sb = saved.numel() * 4 if saved is not None else 0
    rc = lib().sdm_forward(_ptr(q), _ptr(k), _dtype_code(q), _ptr(cb_q), _ptr(cb_k), dk, topk, _ptr(v),
                           _ptr(alpha), _ptr(beta), _dtype_code(v), _ptr(mem), B, H, T, dv, N,
                           _ptr(o["r_idx"]), _ptr(o["r_val"]), _ptr(o["w_idx"]), _ptr(o["w_val"]),
                           _ptr(o["y"]), _ptr(saved), sb, int(chunk), _ptr(workspace), workspace.numel(),
                           _stream(dev))
    _check("sdm_forward", rc)
    return o


def forward_noalloc(q, k, cb_q, cb_k, v, alpha, beta, mem, N: int, topk: int, saved=None, y=None, out=None):
    """sdm_forward_noalloc: the same forward with no workspace (the library's fixed device
    array holds its records), every step on the current stream.  Outputs not given in
    out / y are allocated here by torch; the C entry point itself allocates nothing."""
    B, H, T, dk, dv, dev, o = _forward_args(q, k, cb_q, cb_k, v, alpha, beta, mem, N, topk, saved, y, out,
                                            None)
    sb = saved.numel() * 4 if saved is not None else 0
    rc = lib().sdm_forward_noalloc(_ptr(q), _ptr(k), _dtype_code(q), _ptr(cb_q), _ptr(cb_k), dk, topk, _ptr(v),
                                   _ptr(alpha), _ptr(beta), _dtype_code(v), _ptr(mem), B, H, T, dv, N,
                                   _ptr(o["r_idx"]), _ptr(o["r_val"]), _ptr(o["w_idx"]), _ptr(o["w_val"]),
                                   _ptr(o["y"]), _ptr(saved), sb, _stream(dev))
    _check("sdm_forward_noalloc", rc)
    return o


def _check_gate_params(A, b_dt, H):
    _expect(A, "A", (H,), _F32)
    _expect(b_dt, "b_dt", (H,), _F32)


def gates(a_pre, b_pre, A, b_dt):
    """Forget and input gates from their pre-activations (Sec. 3.1 step 2):
    alpha = exp(-A softplus(a + b_dt)), beta = sigma(b).  a_pre, b_pre [B,H,T];
    A, b_dt [H] fp32.  Returns (alpha, beta) fp32 [B,H,T]."""
    _expect_dims(a_pre, "a_pre", 3)
    B, H, T = a_pre.shape
    if a_pre.dtype not in _IN:
        raise TypeError(f"a_pre has dtype {a_pre.dtype}, expected float32 or bfloat16")
    _expect(b_pre, "b_pre", (B, H, T), (a_pre.dtype,))
    _check_gate_params(A, b_dt, H)
    dev = _dev(a_pre, b_pre, A, b_dt)
    al = torch.empty((B, H, T), dtype=torch.float32, device=dev)
    be = torch.empty_like(al)
    _check("sdm_gates", lib().sdm_gates(_ptr(a_pre), _ptr(b_pre), _dtype_code(a_pre), _ptr(A), _ptr(b_dt), B, H, T,
                                         _ptr(al), _ptr(be), _stream(dev)))
    return al, be


def gates_bwd(a_pre, b_pre, A, b_dt, dalpha, dbeta):
    """Reverse mode of gates: returns (da, db [B,H,T], dA, db_dt [H]), fp32."""
    _expect_dims(a_pre, "a_pre", 3)
    B, H, T = a_pre.shape
    if a_pre.dtype not in _IN:
        raise TypeError(f"a_pre has dtype {a_pre.dtype}, expected float32 or bfloat16")
    _expect(b_pre, "b_pre", (B, H, T), (a_pre.dtype,))
    _check_gate_params(A, b_dt, H)
    _expect(dalpha, "dalpha", (B, H, T), _F32)
    _expect(dbeta, "dbeta", (B, H, T), _F32)
    dev = _dev(a_pre, b_pre, A, b_dt, dalpha, dbeta)
    da = torch.empty((B, H, T), dtype=torch.float32, device=dev)
    db = torch.empty_like(da)
    dA = torch.empty((H,), dtype=torch.float32, device=dev)
    dbd = torch.empty_like(dA)
    _check("sdm_gates_bwd", lib().sdm_gates_bwd(_ptr(a_pre), _ptr(b_pre), _dtype_code(a_pre), _ptr(A), _ptr(b_dt),
                                                 _ptr(dalpha), _ptr(dbeta), B, H, T, _ptr(da), _ptr(db), _ptr(dA),
                                                 _ptr(dbd), _stream(dev)))
    return da, db, dA, dbd


def _check_norm_gate(y, g, gamma):
    _expect_dims(y, "y", 4)
    B, H, T, dv = y.shape
    _expect(y, "y", (B, H, T, dv), _F32)
    _expect(g, "g", (B, H, T, dv), _IN)
    if gamma is not None:
        _expect(gamma, "gamma", (dv,), _F32)
    return B, H, T, dv


def norm_gate(y, g, gamma, eps: float, act: int, want_rstd: bool = False):
    """Output epilogue (Sec. 3.1 step 4): o = y rstd gamma phi(g) per (b,h,t) row,
    rstd = 1/sqrt(mean(y^2) + eps), phi identity (act 0) or SiLU (act 1).
    Returns o (and rstd)."""
    B, H, T, dv = _check_norm_gate(y, g, gamma)
    dev = _dev(y, g, gamma)
    o = torch.empty_like(y)
    rstd = torch.empty((B, H, T), dtype=torch.float32, device=dev) if want_rstd else None
    _check("sdm_norm_gate", lib().sdm_norm_gate(_ptr(y), _ptr(g), _dtype_code(g), _ptr(gamma), float(eps), int(act),
                                                 B, H, T, dv, _ptr(o), _ptr(rstd), _stream(dev)))
    return (o, rstd) if want_rstd else o


def norm_gate_bwd(y, g, gamma, eps: float, act: int, dout, want_dgamma: bool = True):
    """Reverse mode of norm_gate: returns dy, dg and dgamma (None if not wanted)."""
    B, H, T, dv = _check_norm_gate(y, g, gamma)
    _expect(dout, "dout", (B, H, T, dv), _F32)
    dev = _dev(y, g, gamma, dout)
    dy = torch.empty_like(y)
    dg = torch.empty_like(y)
    dgamma = torch.empty((dv,), dtype=torch.float32, device=dev) if want_dgamma else None
    ws = _ws(lib().sdm_norm_gate_bwd_workspace_bytes(B, H, T, dv), dev)
    _check("sdm_norm_gate_bwd", lib().sdm_norm_gate_bwd(_ptr(y), _ptr(g), _dtype_code(g), _ptr(gamma), float(eps),
                                                         int(act), _ptr(dout), B, H, T, dv, _ptr(dy), _ptr(dg),
                                                         _ptr(dgamma), _ptr(ws), ws.numel(), _stream(dev)))
    return dy, dg, dgamma


def layer_fwd(q, k, cb_q, cb_k, v, a_pre, b_pre, g, A, b_dt, gamma, eps: float, act: int, mem, N: int, W: int,
              R: int, saved=None, workspace=None, chunk: int = 0, want_rstd: bool = False):
    """The layer from its projections to W_o's input (Sec. 3.1 steps 1-4): addressing (top-R
    reads of q, top-W writes of k), gates formed inside the scan's records, the recurrence in
    place on mem, and the norm-gate epilogue per pipeline stage.  Returns a dict with o, y,
    r_idx, r_val, w_idx, w_val (and rstd)."""
    _expect_dims(q, "q", 4)
    _expect_dims(v, "v", 4)
    _expect_dims(mem, "mem", 4)
    B, H, T, dk = q.shape
    dv = v.shape[-1]
    if q.dtype not in _IN or v.dtype not in _IN:
        raise TypeError("q and v must be float32 or bfloat16")
    _expect(k, "k", (B, H, T, dk), (q.dtype,))
    _check_codebook(cb_q, "cb_q", q, N)
    _check_codebook(cb_k, "cb_k", q, N)
    _expect(v, "v", (B, H, T, dv), (v.dtype,))
    _expect(a_pre, "a_pre", (B, H, T), (v.dtype,))
    _expect(b_pre, "b_pre", (B, H, T), (v.dtype,))
    _expect(g, "g", (B, H, T, dv), (v.dtype,))
    _check_gate_params(A, b_dt, H)
    if gamma is not None:
        _expect(gamma, "gamma", (dv,), _F32)
    _expect(mem, "mem", (B, H, N, dv), _F32)
    if saved is not None:
        _expect(saved, "saved", (B, H, T, W, dv), _F32)
    _check_ws(workspace, lib().sdm_scan_fwd_workspace_bytes(B, H, T, W, R) if workspace is not None else 0)
    dev = _dev(q, k, cb_q, cb_k, v, a_pre, b_pre, g, A, b_dt, gamma, mem, saved)
    f32 = dict(dtype=torch.float32, device=dev)
    o = dict(r_idx=torch.empty((B, H, T, R), dtype=torch.int32, device=dev), r_val=torch.empty((B, H, T, R), **f32),
             w_idx=torch.empty((B, H, T, W), dtype=torch.int32, device=dev), w_val=torch.empty((B, H, T, W), **f32),
             y=torch.empty((B, H, T, dv), **f32), o=torch.empty((B, H, T, dv), **f32))
    o["rstd"] = torch.empty((B, H, T), **f32) if want_rstd else None
    if workspace is None:
        workspace = fwd_workspace(B, H, T, W, R, dev)
    sb = saved.numel() * 4 if saved is not None else 0
    rc = lib().sdm_layer_fwd(_ptr(q), _ptr(k), _dtype_code(q), _ptr(cb_q), _ptr(cb_k), dk, W, R, _ptr(v),
                             _ptr(a_pre), _ptr(b_pre), _ptr(g), _dtype_code(v), _ptr(A), _ptr(b_dt), _ptr(gamma),
                             float(eps), int(act), _ptr(mem), B, H, T, dv, N, _ptr(o["r_idx"]), _ptr(o["r_val"]),
                             _ptr(o["w_idx"]), _ptr(o["w_val"]), _ptr(o["y"]), _ptr(o["o"]), _ptr(o["rstd"]),
                             _ptr(saved), sb, int(chunk), _ptr(workspace), workspace.numel(), _stream(dev))
    _check("sdm_layer_fwd", rc)
    return o


def layer_bwd(fwd, v, a_pre, b_pre, g, A, b_dt, gamma, eps: float, act: int, mem, saved, dout, dmem_T=None,
              cb_q=None, cb_k=None, d_k: int | None = None, chunk: int = 64, want_dqk: bool = True,
              want_dgamma: bool = True, workspace=None):
    """Reverse mode of layer_fwd (fwd: its returned dict).  mem: M_T in, M_0 out.  Returns a dict
    with dv, da, db, dA, db_dt, dg, dgamma, dmem0 and (if want_dqk) dq, dk."""
    w_idx, w_val, r_idx, r_val, y = fwd["w_idx"], fwd["w_val"], fwd["r_idx"], fwd["r_val"], fwd["y"]
    B, H, T, dv_, W, R, N = _check_scan_args(w_idx, w_val, r_idx, r_val, v, a_pre, b_pre, mem)
    _expect(g, "g", (B, H, T, dv_), (v.dtype,))
    _check_gate_params(A, b_dt, H)
    if gamma is not None:
        _expect(gamma, "gamma", (dv_,), _F32)
    _expect(saved, "saved", (B, H, T, W, dv_), _F32)
    _expect(y, "y", (B, H, T, dv_), _F32)
    _expect(dout, "dout", (B, H, T, dv_), _F32)
    if dmem_T is not None:
        _expect(dmem_T, "dmem_T", (B, H, N, dv_), _F32)
    if want_dqk:
        if d_k is None:
            raise ValueError("d_k is required for addressing gradients")
        for cb, nm in ((cb_q, "cb_q"), (cb_k, "cb_k")):
            if cb is not None:
                _expect(cb, nm, (H, 2, int(round(N ** 0.5)), d_k // 2), _IN)
    _check_ws(workspace, lib().sdm_layer_bwd_workspace_bytes(B, H, T, W, R, dv_) if workspace is not None else 0)
    dev = _dev(w_idx, w_val, r_idx, r_val, v, a_pre, b_pre, g, A, b_dt, gamma, mem, saved, y, dout, dmem_T, cb_q,
               cb_k)
    f32 = dict(dtype=torch.float32, device=dev)
    out = dict(dv=torch.empty((B, H, T, dv_), **f32), da=torch.empty((B, H, T), **f32),
               db=torch.empty((B, H, T), **f32), dA=torch.empty((H,), **f32), db_dt=torch.empty((H,), **f32),
               dg=torch.empty((B, H, T, dv_), **f32), dmem0=torch.empty((B, H, N, dv_), **f32),
               dgamma=torch.empty((dv_,), **f32) if want_dgamma else None)
    dq = dk = None
    cb_dtype = SDM_F32
    if want_dqk:
        dq = torch.empty((B, H, T, d_k), **f32)
        dk = torch.empty((B, H, T, d_k), **f32)
        cb = cb_q if cb_q is not None else cb_k
        cb_dtype = _dtype_code(cb) if cb is not None else SDM_F32
    if workspace is None:
        workspace = _ws(lib().sdm_layer_bwd_workspace_bytes(B, H, T, W, R, dv_), dev)
    rc = lib().sdm_layer_bwd(_ptr(cb_q), _ptr(cb_k), cb_dtype, int(d_k or 0), _ptr(w_idx), _ptr(w_val), W,
                             _ptr(r_idx), _ptr(r_val), R, _ptr(v), _ptr(a_pre), _ptr(b_pre), _ptr(g), _dtype_code(v),
                             _ptr(A), _ptr(b_dt), _ptr(gamma), float(eps), int(act), _ptr(mem), _ptr(saved),
                             saved.numel() * 4, _ptr(y), _ptr(dout), _ptr(dmem_T), int(chunk), B, H, T, dv_, N,
                             _ptr(dq), _ptr(dk), _ptr(out["dv"]), _ptr(out["da"]), _ptr(out["db"]), _ptr(out["dA"]),
                             _ptr(out["db_dt"]), _ptr(out["dg"]), _ptr(out["dgamma"]), _ptr(out["dmem0"]),
                             _ptr(workspace), workspace.numel(), _stream(dev))
    _check("sdm_layer_bwd", rc)
    if want_dqk:
        out["dq"], out["dk"] = dq, dk
    return out


def bwd_workspace(B, H, T, W, R, d_v, device) -> torch.Tensor:
    return _ws(lib().sdm_scan_bwd_workspace_bytes(B, H, T, W, R, d_v), device)


def scan_bwd(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, saved, dy, dmem_T=None,
             cb_q=None, cb_k=None, d_k: int | None = None, chunk: int = 64, want_dqk: bool = True,
             workspace=None, dmem0=None):
    """Backward of scan_fwd (+ addressing).  mem: M_T in, M_0 out.  Returns a dict of
    gradients: dv, dalpha, dbeta, dmem0, dw_val, dr_val and (if want_dqk) dq, dk."""
    B, H, T, dv_, W, R, N = _check_scan_args(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem)
    _expect(saved, "saved", (B, H, T, W, dv_), _F32)
    _expect(dy, "dy", (B, H, T, dv_), _F32)
    if dmem_T is not None:
        _expect(dmem_T, "dmem_T", (B, H, N, dv_), _F32)
    if dmem0 is not None:
        _expect(dmem0, "dmem0", (B, H, N, dv_), _F32)
    if want_dqk:
        if d_k is None:
            raise ValueError("d_k is required for addressing gradients")
        for cb, nm in ((cb_q, "cb_q"), (cb_k, "cb_k")):
            if cb is not None:
                _expect(cb, nm, (H, 2, int(round(N ** 0.5)), d_k // 2), _IN)
        if cb_q is not None and cb_k is not None and cb_q.dtype != cb_k.dtype:
            raise TypeError("cb_q and cb_k must share a dtype")
    _check_ws(workspace, lib().sdm_scan_bwd_workspace_bytes(B, H, T, W, R, dv_) if workspace is not None else 0)
    dev = _dev(w_idx, w_val, r_idx, r_val, v, alpha, beta, mem, saved, dy, dmem_T, cb_q, cb_k, dmem0)
    f32 = dict(dtype=torch.float32, device=dev)
    out = dict(dv=torch.empty((B, H, T, dv_), **f32), dalpha=torch.empty((B, H, T), **f32),
               dbeta=torch.empty((B, H, T), **f32),
               dmem0=dmem0 if dmem0 is not None else torch.empty((B, H, N, dv_), **f32),
               dw_val=torch.empty((B, H, T, W), **f32), dr_val=torch.empty((B, H, T, R), **f32))
    dq = dk = None
    cb_dtype = SDM_F32
    if want_dqk:
        dq = torch.empty((B, H, T, d_k), **f32)
        dk = torch.empty((B, H, T, d_k), **f32)
        cb = cb_q if cb_q is not None else cb_k
        cb_dtype = _dtype_code(cb) if cb is not None else SDM_F32
    if workspace is None:
        workspace = bwd_workspace(B, H, T, W, R, dv_, dev)
    rc = lib().sdm_scan_bwd(_ptr(cb_q), _ptr(cb_k), cb_dtype, int(d_k or 0), _ptr(w_idx),
                            _ptr(w_val), W, _ptr(r_idx), _ptr(r_val), R, _ptr(v), _ptr(alpha),
                            _ptr(beta), _dtype_code(v), _ptr(mem), _ptr(saved), saved.numel() * 4,
                            _ptr(dy), _ptr(dmem_T), chunk, B, H, T, dv_, N, _ptr(dq), _ptr(dk),
                            _ptr(out["dv"]), _ptr(out["dalpha"]), _ptr(out["dbeta"]),
                            _ptr(out["dmem0"]), _ptr(out["dw_val"]), _ptr(out["dr_val"]),
                            _ptr(workspace), workspace.numel(), _stream(dev))
    _check("sdm_scan_bwd", rc)
    if want_dqk:
        out["dq"], out["dk"] = dq, dk
    return out


def mem_init(dst: torch.Tensor, m0: torch.Tensor | None):
    """dst [B,H,N,d_v] = m0 [H,N,d_v] broadcast over B (or zero when m0 is None)."""
    _expect_dims(dst, "dst", 4)
    B, H, N, dv = dst.shape
    _expect(dst, "dst", (B, H, N, dv), _F32)
    if m0 is not None:
        _expect(m0, "m0", (H, N, dv), _F32)
    dev = _dev(dst, m0)
    rc = lib().sdm_mem_init(_ptr(dst), _ptr(m0), B, H, N, dv, _stream(dev))
    _check("sdm_mem_init", rc)
    return dst


def check_device_errors(workspace: torch.Tensor):
    rc = lib().sdm_check_device_errors(_ptr(workspace), _stream(workspace.device))
    _check("sdm_check_device_errors", rc)


KERNELS = {"address": 0, "fwd_prep": 1, "fwd_scan": 2, "bwd_prep": 3, "bwd_scan": 4, "bwd_reduce": 5,
           "address_bwd": 6, "mem_init": 7, "decode": 8, "chunk_coef": 9, "chunk_scan": 10, "norm_gate": 11,
           "gates": 12}


def set_chunk_scan_cols(cols: int):
    """Columns per workgroup of the chunked scan: 8 (narrow kernel), 16, 32, or 0 for the default (32)."""
    _check("sdm_set_chunk_scan_cols", lib().sdm_set_chunk_scan_cols(int(cols)))


def set_scan_slice_width(sw: int):
    """Columns per scan wave: 0 automatic, or force 8 / 16 (process-wide)."""
    _check("sdm_set_scan_slice_width", lib().sdm_set_scan_slice_width(int(sw)))


def set_scan_prefetch(pd: int):
    """Forward scan prefetch depth: 0 automatic, or force 4 / 8 / 16 (process-wide)."""
    _check("sdm_set_scan_prefetch", lib().sdm_set_scan_prefetch(int(pd)))


def set_scan_line_io(on: bool):
    """Scans: line-cooperative table I/O where the shape allows (default) or per-wave pieces (process-wide)."""
    _check("sdm_set_scan_line_io", lib().sdm_set_scan_line_io(int(bool(on))))


def profile_enable(on: bool = True):
    """Start (or stop) HIP-event timing of every kernel the library launches; clears totals."""
    _check("sdm_profile_enable", lib().sdm_profile_enable(int(on)))


def profile_select(kernels=None):
    """Time only these kernel kinds (names of KERNELS) while profiling is on; None: all."""
    mask = (1 << len(KERNELS)) - 1 if kernels is None else sum(1 << KERNELS[k] for k in kernels)
    _check("sdm_profile_select", lib().sdm_profile_select(mask))


def profile_read(kernel: str):
    """(total_ms, launches) of one kernel kind since profile_enable(True)."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check("sdm_profile_read", lib().sdm_profile_read(KERNELS[kernel], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
