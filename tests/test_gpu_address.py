"""Addressing edge cases on the GPU against the oracle (Sec. 2 product keys,
Sec. 4 softmax over the selected scores).

Rows whose scores tie exactly (a zero query scores 0 against every sub-key)
must take the lowest ids (score descending, id ascending), so the selection's
candidate bound overflows and the general path decides; rows equal to a
codebook entry, and ordinary rows, are mixed in.  Each sub-key count runs one
of the addressing kernels: sqrt(N) = 256 the tile with every score in LDS,
512 and 1024 the kernel that keeps scores in registers (d_k / 2 = 32 and 64).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_07386_amd import sdm
from tests.gpu_util import DEV, compare_address

pytestmark = pytest.mark.gpu


def _bf16_round(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


@pytest.mark.parametrize("s,dk,k,T", [(256, 128, 32, 37), (512, 64, 32, 41), (1024, 128, 32, 29),
                                      (1024, 128, 7, 18), (600, 128, 16, 23)])
def test_address_ties_zero_rows_and_codebook_rows(s, dk, k, T):
    rng = np.random.default_rng(s + dk + k)
    H = 2
    dh = dk // 2
    cb = _bf16_round(rng.standard_normal((H, 2, s, dh)) / np.sqrt(dh))
    x = rng.standard_normal((1, H, T, dk))
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    x[0, :, 0] = 0.0                                   # every score 0: a complete tie
    x[0, :, T // 2] = 0.0
    for h in range(H):                                 # rows made of codebook entries
        x[0, h, 1, :dh] = cb[h, 0, 5].float().numpy()
        x[0, h, 1, dh:] = cb[h, 1, s - 1].float().numpy()
    xb = _bf16_round(x)
    gi, gv = sdm.address(xb.to(DEV), cb.to(DEV), s * s, k)
    torch.cuda.synchronize()
    x64, cb64 = xb.double().numpy(), cb.double().numpy()
    oi, ov, _ = oracle.address(x64, cb64, s * s, k, decide_f32=True)
    gi, gv = gi.cpu().numpy(), gv.cpu().numpy()
    for h in range(H):
        # exact ties: the k lowest ids, equal weights
        for t in (0, T // 2):
            assert np.array_equal(gi[0, h, t], oi[0, h, t]), (h, t, gi[0, h, t], oi[0, h, t])
            np.testing.assert_allclose(gv[0, h, t], 1.0 / k, rtol=1e-6)
        compare_address(gi[0, h], gv[0, h], oi[0, h], ov[0, h], x64[0, h], lambda r: cb64[h], s)
