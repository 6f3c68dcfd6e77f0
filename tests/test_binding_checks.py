"""The Python binding checks every tensor's shape and dtype against the sizes
it hands to the C ABI, before anything is launched: the library sees only
pointers, so a mismatched tensor would otherwise be read or written out of
bounds.  CPU tensors are used, so a call that passes the shape checks stops at
the placement check ("must be on the GPU") and nothing reaches the device."""
import pytest
import torch

from paper_2607_07386_amd import sdm

B, H, T, DV, W, R, N, DK = 2, 3, 5, 8, 4, 6, 64, 16


def _scan_args():
    f32, bf = torch.float32, torch.bfloat16
    return dict(w_idx=torch.zeros((B, H, T, W), dtype=torch.int32), w_val=torch.zeros((B, H, T, W), dtype=f32),
                r_idx=torch.zeros((B, H, T, R), dtype=torch.int32), r_val=torch.zeros((B, H, T, R), dtype=f32),
                v=torch.zeros((B, H, T, DV), dtype=bf), alpha=torch.zeros((B, H, T), dtype=bf),
                beta=torch.zeros((B, H, T), dtype=bf), mem=torch.zeros((B, H, N, DV), dtype=f32))


BAD_SCAN = {
    "w_val short": ("w_val", torch.zeros((B, H, T, W - 1))),
    "w_idx int64": ("w_idx", torch.zeros((B, H, T, W), dtype=torch.int64)),
    "r_val fp64": ("r_val", torch.zeros((B, H, T, R), dtype=torch.float64)),
    "r_idx other T": ("r_idx", torch.zeros((B, H, T + 1, R), dtype=torch.int32)),
    "alpha fp32 beside bf16 v": ("alpha", torch.zeros((B, H, T))),
    "beta wrong heads": ("beta", torch.zeros((B, H - 1, T), dtype=torch.bfloat16)),
    "mem other d_v": ("mem", torch.zeros((B, H, N, DV + 4))),
    "mem fewer heads": ("mem", torch.zeros((B, H - 1, N, DV))),
    "mem bf16": ("mem", torch.zeros((B, H, N, DV), dtype=torch.bfloat16)),
    "mem 3-d": ("mem", torch.zeros((H, N, DV))),
}


def _raises_before_device(fn, what):
    with pytest.raises((ValueError, TypeError)) as e:
        fn()
    assert "GPU" not in str(e.value), f"{what}: reached the placement check: {e.value}"
    return str(e.value)


def _reaches_device(fn):
    with pytest.raises(ValueError, match="on the GPU"):
        fn()


def test_scan_fwd_good_args_reach_the_placement_check():
    _reaches_device(lambda: sdm.scan_fwd(**_scan_args()))
    a = _scan_args()
    _reaches_device(lambda: sdm.scan_fwd(**a, saved=torch.zeros((B, H, T, W, DV)), y=torch.zeros((B, H, T, DV))))


@pytest.mark.parametrize("case", list(BAD_SCAN))
def test_scan_fwd_rejects(case):
    name, t = BAD_SCAN[case]
    a = _scan_args()
    a[name] = t
    msg = _raises_before_device(lambda: sdm.scan_fwd(**a), case)
    assert name in msg


@pytest.mark.parametrize("case", list(BAD_SCAN))
def test_scan_fwd_chunked_rejects(case):
    name, t = BAD_SCAN[case]
    a = _scan_args()
    a[name] = t
    _raises_before_device(lambda: sdm.scan_fwd_chunked(**a), case)


@pytest.mark.parametrize("kw,t", [("saved", torch.zeros((B, H, T, W, DV - 4))),
                                  ("saved", torch.zeros((B, H, T, R, DV))),
                                  ("y", torch.zeros((B, H, T, DV - 4))),
                                  ("y", torch.zeros((B, H, T, DV), dtype=torch.bfloat16)),
                                  ("workspace", torch.zeros(16, dtype=torch.uint8)),
                                  ("workspace", torch.zeros(1 << 20, dtype=torch.float32))])
def test_scan_fwd_rejects_outputs(kw, t):
    a = _scan_args()
    _raises_before_device(lambda: sdm.scan_fwd(**a, **{kw: t}), kw)


def _bwd_extra():
    return dict(saved=torch.zeros((B, H, T, W, DV)), dy=torch.zeros((B, H, T, DV)))


@pytest.mark.parametrize("case", list(BAD_SCAN))
def test_scan_bwd_rejects(case):
    name, t = BAD_SCAN[case]
    a = _scan_args()
    a[name] = t
    _raises_before_device(lambda: sdm.scan_bwd(**a, **_bwd_extra(), want_dqk=False), case)


@pytest.mark.parametrize("kw,t", [("saved", torch.zeros((B, H, T - 1, W, DV))),
                                  ("dy", torch.zeros((B, H, T, DV), dtype=torch.bfloat16)),
                                  ("dy", torch.zeros((B, H, T, DV + 4))),
                                  ("dmem_T", torch.zeros((B, H, N + 1, DV))),
                                  ("dmem0", torch.zeros((B, H, N, DV - 4))),
                                  ("cb_q", torch.zeros((H, 2, 8, DK // 2 + 1))),
                                  ("cb_k", torch.zeros((H + 1, 2, 8, DK // 2)))])
def test_scan_bwd_rejects_extras(kw, t):
    a = _scan_args()
    ex = _bwd_extra()
    args = dict(a, **ex)
    args[kw] = t
    _raises_before_device(lambda: sdm.scan_bwd(**args, d_k=DK), kw)


def test_scan_bwd_good_args_reach_the_placement_check():
    a = _scan_args()
    cb = torch.zeros((H, 2, 8, DK // 2), dtype=torch.bfloat16)
    _reaches_device(lambda: sdm.scan_bwd(**a, **_bwd_extra(), cb_q=cb, cb_k=cb, d_k=DK,
                                         dmem0=torch.zeros((B, H, N, DV))))


def _fwd_args():
    a = _scan_args()
    return dict(q=torch.zeros((B, H, T, DK), dtype=torch.bfloat16), k=torch.zeros((B, H, T, DK), dtype=torch.bfloat16),
                cb_q=torch.zeros((H, 2, 8, DK // 2), dtype=torch.bfloat16),
                cb_k=torch.zeros((H, 2, 8, DK // 2), dtype=torch.bfloat16),
                v=a["v"], alpha=a["alpha"], beta=a["beta"], mem=a["mem"], N=N, topk=W)


@pytest.mark.parametrize("kw,t", [("k", torch.zeros((B, H, T, DK + 2), dtype=torch.bfloat16)),
                                  ("k", torch.zeros((B, H, T, DK))),
                                  ("cb_q", torch.zeros((H, 2, 8, DK // 2))),
                                  ("cb_k", torch.zeros((H, 2, 7, DK // 2), dtype=torch.bfloat16)),
                                  ("alpha", torch.zeros((B, H, T + 1), dtype=torch.bfloat16)),
                                  ("mem", torch.zeros((B, H, N, DV + 4))),
                                  ("saved", torch.zeros((B, H, T, W + 1, DV))),
                                  ("y", torch.zeros((B, H, T, DV + 4)))])
def test_forward_rejects(kw, t):
    a = _fwd_args()
    a[kw] = t
    _raises_before_device(lambda: sdm.forward(**a), kw)


@pytest.mark.parametrize("name,t", [("r_idx", torch.zeros((B, H, T, W + 1), dtype=torch.int32)),
                                    ("w_idx", torch.zeros((B, H, T, W), dtype=torch.int64)),
                                    ("r_val", torch.zeros((B, H, T, W), dtype=torch.bfloat16)),
                                    ("w_val", torch.zeros((B, H, T - 1, W)))])
def test_forward_rejects_preallocated_outputs(name, t):
    _raises_before_device(lambda: sdm.forward(**_fwd_args(), out={name: t}), name)


def test_forward_good_args_reach_the_placement_check():
    _reaches_device(lambda: sdm.forward(**_fwd_args(), saved=torch.zeros((B, H, T, W, DV)),
                                        out={"r_idx": torch.zeros((B, H, T, W), dtype=torch.int32)}))


def test_address_and_mem_init_reject():
    x = torch.zeros((B, H, T, DK), dtype=torch.bfloat16)
    _raises_before_device(lambda: sdm.address(x, torch.zeros((H, 2, 8, DK // 2)), N, W), "codebook dtype")
    _raises_before_device(lambda: sdm.address(x, torch.zeros((H, 2, 8, DK), dtype=torch.bfloat16), N, W),
                          "codebook width")
    _raises_before_device(lambda: sdm.address(x[0], None, N, W), "x 3-d")
    _reaches_device(lambda: sdm.address(x, torch.zeros((H, 2, 8, DK // 2), dtype=torch.bfloat16), N, W))
    dst = torch.zeros((B, H, N, DV))
    _raises_before_device(lambda: sdm.mem_init(dst, torch.zeros((H, N, DV + 4))), "m0 width")
    _raises_before_device(lambda: sdm.mem_init(dst, torch.zeros((H + 1, N, DV))), "m0 heads")
    _raises_before_device(lambda: sdm.mem_init(dst.to(torch.bfloat16), None), "dst dtype")
    _reaches_device(lambda: sdm.mem_init(dst, torch.zeros((H, N, DV))))
