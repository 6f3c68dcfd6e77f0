"""Host-side checks of the C ABI (CPU only: no call here reaches a kernel).

* libsdm.so loads and exports every function include/sdm.h declares;
* every rule the header states is enforced on the host: a bad call returns
  the documented negative status with a message and launches nothing;
* sizing helpers: the undo log is T*W*d_v elements per stream, which
  reproduces the in-place + undo memory figures of App. A.3 (fixture in
  tests/golden/undo_log_sizes.json).
"""
import ctypes
import json
import os

import pytest

from paper_2607_07386_amd import sdm

L = sdm.lib()
P = ctypes.c_void_p
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "undo_log_sizes.json")

# Fake, 256-byte aligned, never dereferenced addresses: validation rejects the
# call before any launch, so these are only compared, never used.
A = 0x10000000
B_ = 0x20000000


def test_exports_every_declared_symbol():
    names = sdm.header_symbols()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), f"{n} declared in sdm.h but not exported"
    for n in ("sdm_address", "sdm_scan_fwd", "sdm_scan_bwd"):
        assert n in names


def test_status_strings_and_version():
    for code in (0, -1, -2, -3, -4, -5):
        assert L.sdm_status_string(code)
    assert b"gfx950" in L.sdm_version()


def addr(**kw):
    a = dict(x=A, x_dtype=1, cb=B_, B=1, H=1, T=4, d_k=128, N=65536, topk=32, idx=A, val=A, score=None)
    a.update(kw)
    return L.sdm_address(a["x"], a["x_dtype"], a["cb"], a["B"], a["H"], a["T"], a["d_k"], a["N"],
                         a["topk"], a["idx"], a["val"], a["score"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(N=65535), -1), (dict(N=0), -1), (dict(topk=0), -1), (dict(topk=257), -1),
    (dict(N=100 * 100, topk=101), -1), (dict(N=256 * 256, topk=129), -2), (dict(d_k=127), -1), (dict(d_k=1024), -2),
    (dict(cb=None, d_k=100), -1), (dict(x=None), -1), (dict(idx=None), -1), (dict(x=A + 4), -1),
    (dict(x_dtype=7), -1), (dict(T=-1), -1), (dict(B=70000), -2), (dict(N=2048 * 2048), -2),
])
def test_address_validation(kw, code):
    assert addr(**kw) == code
    assert L.sdm_last_error()


def test_address_empty_is_noop():
    assert addr(T=0) == 0
    assert addr(B=0) == 0


def fwd(**kw):
    a = dict(wi=A, wv=A, W=32, ri=A, rv=A, R=32, v=A, al=A, be=A, dt=1, mem=A, B=1, H=1, T=8, dv=128,
             N=65536, y=A, saved=None, sb=0, ws=A, wsb=1 << 30)
    a.update(kw)
    return L.sdm_scan_fwd(a["wi"], a["wv"], a["W"], a["ri"], a["rv"], a["R"], a["v"], a["al"],
                          a["be"], a["dt"], a["mem"], a["B"], a["H"], a["T"], a["dv"], a["N"], a["y"],
                          a["saved"], a["sb"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(W=0), -1), (dict(R=0), -1), (dict(W=129), -2), (dict(R=129), -2), (dict(dv=6), -1), (dict(dv=8192), -2),
    (dict(N=0), -1), (dict(dt=2), -1), (dict(mem=None), -1), (dict(y=None), -1), (dict(v=A + 2), -1),
    (dict(ws=None), -1), (dict(ws=A + 16), -1), (dict(wsb=100), -3),
    (dict(saved=A, sb=10), -3), (dict(saved=A + 8, sb=1 << 40), -1), (dict(B=-1), -1),
])
def test_scan_fwd_validation(kw, code):
    assert fwd(**kw) == code
    assert L.sdm_last_error()


def fwd_chunked(**kw):
    a = dict(wi=A, wv=A, W=32, ri=A, rv=A, R=32, v=A, al=A, be=A, dt=1, mem=A, B=1, H=1, T=8, dv=128,
             N=65536, y=A, ws=A, wsb=1 << 30)
    a.update(kw)
    return L.sdm_scan_fwd_chunked(a["wi"], a["wv"], a["W"], a["ri"], a["rv"], a["R"], a["v"], a["al"],
                                  a["be"], a["dt"], a["mem"], a["B"], a["H"], a["T"], a["dv"], a["N"], a["y"],
                                  a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(W=0), -1), (dict(R=0), -1), (dict(W=65), -2), (dict(R=65), -2), (dict(W=129), -2), (dict(dv=6), -1),
    (dict(N=0), -1), (dict(dt=2), -1), (dict(mem=None), -1), (dict(y=None), -1), (dict(y=A + 4), -1),
    (dict(ws=None), -1), (dict(ws=A + 16), -1), (dict(wsb=100), -3), (dict(B=-1), -1),
])
def test_scan_fwd_chunked_validation(kw, code):
    assert fwd_chunked(**kw) == code
    assert L.sdm_last_error()


def test_scan_fwd_chunked_empty_is_noop():
    assert fwd_chunked(T=0, ws=None, y=None) == 0
    assert fwd_chunked(B=0, ws=None, y=None) == 0


def test_chunked_workspace_size():
    # one record per (stream, 64-token chunk) after a 256-byte header
    one = L.sdm_scan_fwd_chunked_workspace_bytes(1, 1, 64, 32, 32)
    assert one > 256 and (one - 256) % 256 == 0
    assert L.sdm_scan_fwd_chunked_workspace_bytes(2, 3, 65, 32, 32) == 256 + 12 * (one - 256)
    assert L.sdm_scan_fwd_chunked_workspace_bytes(1, 1, 64, 0, 32) == 0


def bwd(**kw):
    a = dict(cbq=A, cbk=A, cbdt=1, dk=128, wi=A, wv=A, W=32, ri=A, rv=A, R=32, v=A, al=A, be=A, dt=1,
             mem=A, saved=A, sb=1 << 40, dy=A, dmT=None, chunk=64, B=1, H=1, T=8, dv=128, N=65536,
             dq=A, dkk=A, dvo=A, da=A, db=A, dm0=A, dwv=None, drv=None, ws=A, wsb=1 << 40)
    a.update(kw)
    return L.sdm_scan_bwd(a["cbq"], a["cbk"], a["cbdt"], a["dk"], a["wi"], a["wv"], a["W"], a["ri"],
                          a["rv"], a["R"], a["v"], a["al"], a["be"], a["dt"], a["mem"], a["saved"],
                          a["sb"], a["dy"], a["dmT"], a["chunk"], a["B"], a["H"], a["T"], a["dv"],
                          a["N"], a["dq"], a["dkk"], a["dvo"], a["da"], a["db"], a["dm0"], a["dwv"],
                          a["drv"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(chunk=0), -1), (dict(saved=None), -1), (dict(dy=None), -1), (dict(dm0=None), -1),
    (dict(sb=16), -3), (dict(wsb=16), -3), (dict(N=1000), -1), (dict(cbq=None, dk=100), -1),
    (dict(W=300), -2), (dict(dvo=A + 4), -1), (dict(cbdt=5), -1),
])
def test_scan_bwd_validation(kw, code):
    assert bwd(**kw) == code
    assert L.sdm_last_error()


def test_slice_width_setting():
    for sw in (8, 16, 0):
        assert L.sdm_set_scan_slice_width(sw) == 0
    for sw in (-1, 4, 12, 32):
        assert L.sdm_set_scan_slice_width(sw) == -1
        assert b"width" in L.sdm_last_error()


def test_scan_prefetch_setting():
    for pd in (4, 8, 16, 0):
        assert L.sdm_set_scan_prefetch(pd) == 0
    for pd in (-1, 2, 12, 32):
        assert L.sdm_set_scan_prefetch(pd) == -1
        assert b"depth" in L.sdm_last_error()


def test_chunk_scan_cols_setting():
    for c in (8, 16, 32, 0):
        assert L.sdm_set_chunk_scan_cols(c) == 0
    for c in (-1, 4, 24, 64):
        assert L.sdm_set_chunk_scan_cols(c) == -1
        assert b"expected 0" in L.sdm_last_error()


def test_scan_line_io_setting():
    for on in (0, 1):
        assert L.sdm_set_scan_line_io(on) == 0
    for on in (-1, 2, 8):
        assert L.sdm_set_scan_line_io(on) == -1
        assert b"expected 0 or 1" in L.sdm_last_error()
    assert L.sdm_set_scan_line_io(1) == 0


def test_profile_select():
    n = len(sdm.KERNELS)
    assert L.sdm_profile_select(1 << 2) == 0
    assert L.sdm_profile_select((1 << n) - 1) == 0
    assert L.sdm_profile_select(1 << n) == -1
    assert b"unknown kernel kinds" in L.sdm_last_error()
    assert L.sdm_profile_select((1 << n) - 1) == 0


def test_mem_init_validation():
    assert L.sdm_mem_init(None, None, 1, 1, 16, 4, None) == -1
    assert L.sdm_mem_init(A, None, 1, 1, 16, 6, None) == -1
    assert L.sdm_mem_init(A + 4, None, 1, 1, 16, 4, None) == -1
    assert L.sdm_mem_init(A, None, 65536, 2, 16, 4, None) == -2


def test_sizes():
    assert L.sdm_scan_saved_bytes(4, 16, 4096, 32, 128) == 4 * 16 * 4096 * 32 * 128 * 4
    ws = L.sdm_scan_fwd_workspace_bytes(8, 16, 4096, 32, 32)
    assert ws > 8 * 16 * 4096 * (32 + 32) * 8       # slots + weights of every token
    assert L.sdm_scan_bwd_workspace_bytes(4, 16, 4096, 32, 32, 128) > ws // 2
    assert L.sdm_scan_fwd_workspace_bytes(1, 1, 0, 32, 32) >= 256


def test_undo_log_matches_paper_memory_figures():
    """App. A.3: state checkpoints vs in-place + undo, 8B layer, T=16384, C=128, W=64."""
    g = json.load(open(GOLDEN))
    H, N, dv, T, C, W = (g["layer"][k] for k in ("H", "N", "d_v", "T", "C", "W"))
    elem = g["bytes_per_element"]
    per_chunk_states = (T // C) * H * N * dv * elem
    undo = L.sdm_scan_saved_bytes(1, H, T, W, dv) // 4 * elem   # library counts fp32 elements
    assert abs(per_chunk_states / 1e9 - g["paper_gb"]["checkpoints"]) < 0.5
    assert abs(undo / 1e9 - g["paper_gb"]["undo"]) < 0.1
    assert round(per_chunk_states / 1e9, 2) == g["derived_gb"]["checkpoints"]
    assert round(undo / 1e9, 2) == g["derived_gb"]["undo"]


def test_every_supported_shape_has_a_launch_plan():
    """Every W, R <= 128 and d_v the header allows gets a scan plan whose staged
    per-token records fit the staging registers and LDS: validation gets past
    the plan and stops at the (deliberately) too-small workspace."""
    for W in range(1, 129):
        for R in (1, 7, 16, 17, 31, 32, 33, 48, 63, 64, 65, 96, 127, 128):
            for dv, dt in ((4, 0), (36, 1), (128, 1), (960, 0), (4096, 1)):
                assert fwd(W=W, R=R, dv=dv, dt=dt, wsb=0) == -3, (W, R, dv, dt)
                assert bwd(W=W, R=R, dv=dv, dt=dt, wsb=0, cbq=None, cbk=None, dq=None, dkk=None) == -3, \
                    (W, R, dv, dt)


def test_forward_validation():
    """sdm_forward validates like the three calls it fuses, plus its chunk argument."""
    def fw(**kw):
        a = dict(q=A, k=A, xdt=1, cbq=B_, cbk=B_, dk=128, topk=32, v=A, al=A, be=A, dt=1, mem=A, B=1,
                 H=1, T=8, dv=128, N=65536, ri=A, rv=A, wi=A, wv=A, y=A, saved=None, sb=0, chunk=0, ws=A,
                 wsb=1 << 30)
        a.update(kw)
        return L.sdm_forward(a["q"], a["k"], a["xdt"], a["cbq"], a["cbk"], a["dk"], a["topk"], a["v"],
                             a["al"], a["be"], a["dt"], a["mem"], a["B"], a["H"], a["T"], a["dv"], a["N"],
                             a["ri"], a["rv"], a["wi"], a["wv"], a["y"], a["saved"], a["sb"], a["chunk"],
                             a["ws"], a["wsb"], None)
    for kw, code in ((dict(chunk=-1), -1), (dict(N=65535), -1), (dict(topk=129, N=256 * 256), -2), (dict(k=None), -1),
                     (dict(ri=A + 4), -1), (dict(dv=6), -1), (dict(wsb=100), -3), (dict(y=None), -1),
                     (dict(cbk=A + 2), -1), (dict(xdt=5), -1)):
        assert fw(**kw) == code, kw
        assert L.sdm_last_error()
    assert fw(T=0) == 0


def test_noalloc_refuses_sizes_past_its_array_on_the_host():
    """sdm_forward_noalloc's size check comes before any device call (CPU only)."""
    cap = L.sdm_forward_noalloc_max_bytes()
    assert cap == 64 << 20
    B, H, T, k = 16, 16, 100000, 32
    assert L.sdm_scan_fwd_workspace_bytes(B, H, T, k, k) > cap
    rc = L.sdm_forward_noalloc(A, A, 1, B_, B_, 128, k, A, A, A, 1, A, B, H, T, 128, 65536,
                               A, A, A, A, A, None, 0, None)
    assert rc == -2 and b"scratch" in L.sdm_last_error()
    # an empty call needs nothing and returns at once
    assert L.sdm_forward_noalloc(A, A, 1, B_, B_, 128, k, A, A, A, 1, A, B, H, 0, 128, 65536,
                                 A, A, A, A, A, None, 0, None) == 0


def test_gates_and_epilogue_validation():
    """Host checks of the gate and epilogue entry points (CPU only)."""
    F = ctypes.c_float
    # sdm_gates(a, b, dtype, A, b_dt, B, H, T, alpha, beta, stream)
    assert L.sdm_gates(A, A, 5, A, A, 1, 2, 8, A, A, None) == -1            # dtype
    assert L.sdm_gates(A, A, 1, None, A, 1, 2, 8, A, A, None) == -1         # A
    assert L.sdm_gates(None, A, 1, A, A, 1, 2, 8, A, A, None) == -1         # pre-activation
    assert L.sdm_gates(A, A, 1, A, A, 1, 2, 8, None, A, None) == -1         # output
    assert L.sdm_gates(A, A, 1, A, A, 1, 2, 0, None, None, None) == 0       # empty
    # sdm_norm_gate(y, g, g_dtype, gamma, eps, act, B, H, T, d_v, o, rstd, stream)
    ng = L.sdm_norm_gate
    assert ng(A, A, 1, None, F(1e-5), 2, 1, 1, 4, 64, A, None, None) == -1  # act
    assert ng(A, A, 1, None, F(-1.0), 0, 1, 1, 4, 64, A, None, None) == -1  # eps
    assert ng(A, A, 1, None, F(1e-5), 0, 1, 1, 4, 66, A, None, None) == -1  # d_v
    assert ng(A, A, 1, None, F(1e-5), 0, 1, 1, 4, 8192, A, None, None) == -2
    assert ng(A, A + 4, 1, None, F(1e-5), 0, 1, 1, 4, 64, A, None, None) == -1   # alignment
    assert ng(A, A, 1, None, F(1e-5), 0, 1, 1, 4, 64, None, None, None) == -1    # o
    assert ng(A, A, 1, None, F(1e-5), 0, 1, 1, 0, 64, None, None, None) == 0     # empty
    need = L.sdm_norm_gate_bwd_workspace_bytes(2, 3, 100, 128)
    assert need >= 128 * 4 and need % 256 == 0
    assert L.sdm_norm_gate_bwd(A, A, 1, None, F(1e-5), 0, A, 2, 3, 100, 128, A, A, A, A, need - 1, None) == -3
    assert L.sdm_layer_bwd_workspace_bytes(2, 3, 100, 32, 32, 128) > L.sdm_scan_bwd_workspace_bytes(2, 3, 100, 32, 32, 128)
