"""GPU parity of the fused decode-GEMV with tiled activations: larger batches
on larger matrices read x from a tiled copy in the workspace (the 16 batch
rows of each 8-column chunk contiguous), on the matrix-core kernel and on the
persistent one. Every output against a float64 product of the exact bf16
values, sampled outputs against the oracle's exactly rounded sums
(|y - y_ref| <= 1e-3 * sum_k |w x|); the untiled path (the same call without
a workspace reads x directly, and sums over column blocks in one block, so its
rounding can differ) meets the same bound.
"""
import numpy as np
import pytest

from gen import random_bf16, random_x
from oracle import gemv as ogemv
from oracle.gemv import bf16_to_f64

pytestmark = pytest.mark.gpu
TOL = 1e-3

hl = pytest.importorskip("paper_2502_00922_amd.hufflm")


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    hl.lib()
    return t


# (rows, cols): 2048 x 16384 runs the matrix-core kernel, 4100 x 8192 the
# persistent one (a ragged last row block); both exceed 32M weights, where
# batches of 8 and more take the tiled path.
@pytest.mark.parametrize("shape,batch", [((2048, 16384), 8), ((2048, 16384), 16), ((4100, 8192), 12),
                                         ((4100, 8192), 16)])
def test_tiled_activations(torch, shape, batch):
    print(f"xtile {shape} batch {batch}", flush=True)
    w = random_bf16(shape, seed=batch)
    dt = hl.DeviceTensor(hl.encode(w))
    x = random_x(batch, shape[1], seed=batch + 1, dtype="bf16")
    xd = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    y = dt.gemv(xd).cpu().numpy()
    y_direct = dt.gemv(xd, workspace=False).cpu().numpy()
    torch.cuda.synchronize()
    Wf, Xf = bf16_to_f64(w), bf16_to_f64(x)
    ref, den = Xf @ Wf.T, np.abs(Xf) @ np.abs(Wf).T + 1e-30
    for out in (y, y_direct):
        err = np.abs(out - ref) / den
        assert err.max() <= TOL, float(err.max())
    rows = [0, shape[0] - 1, shape[0] // 2]
    yo, do = ogemv.gemv_rows(w, x, rows=rows)
    assert np.max(np.abs(y[:, rows] - yo) / (do + 1e-30)) <= TOL
