"""GPU parity of the non-persistent fused kernels on matrices with few column
blocks or few row blocks: blocks launched with fewer than four waves (one
group column per wave), and matrices split over columns so that every CU gets
a block (k-part partial sums through the workspace), on both the matrix-core
kernel (bf16 x) and the vector kernel (fp32 x), with and without a workspace.
Same bar as the other GEMV tests: |y - y_ref| / (sum |w x| + 1e-30) <= 1e-3
per output against the oracle's fp64 product.
"""
import numpy as np
import pytest

from gen import random_bf16, random_x
from oracle import gemv as ogemv

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


def _to_dev_x(torch, x):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(x).cuda()


# (rows, cols) at S = 64 with 16-row groups of 4 segments: column blocks =
# cols / 256, row blocks = ceil(rows / 16).
#   (48, 256):   1 column block  -> one-wave blocks
#   (40, 512):   2 column blocks -> two-wave blocks, a ragged last row block
#   (100, 768):  3 column blocks -> three-wave blocks
#   (512, 2048): 32 row blocks, 8 column blocks -> split over columns into
#                one-wave blocks with 8 k-parts
#   (1000, 4096): 63 row blocks (ragged), 16 column blocks -> 4 k-parts of
#                four-wave blocks
SHAPES = [(48, 256), (40, 512), (100, 768), (512, 2048), (1000, 4096)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("xdt", ["bf16", "f32"])
def test_narrow_and_split_blocks(torch, shape, xdt):
    w = random_bf16(shape, seed=shape[0] + 3 * shape[1])
    dt = hl.DeviceTensor(hl.encode(w, seg_len=64, grp_rows=16))
    for batch in (1, 5, 16):
        x = random_x(batch, shape[1], seed=batch * 11 + shape[0], dtype=xdt)
        y_ref, den = ogemv.gemv_rows(w, x)
        for ws in (None, False):
            print(f"narrow {shape} x={xdt} batch={batch} workspace={'no' if ws is False else 'yes'}", flush=True)
            y = dt.gemv(_to_dev_x(torch, x), workspace=ws)
            torch.cuda.synchronize()
            err = ogemv.rel_err(y.cpu().numpy(), y_ref, den)
            assert np.max(err) <= TOL, (shape, xdt, batch, ws, float(np.max(err)))


def test_split_blocks_repeatable(torch):
    # the k-part partial sums are added in k order by the last block to
    # arrive, and the arrival counters are reset: repeated calls agree bit
    # for bit
    w = random_bf16((512, 2048), seed=17)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=64, grp_rows=16))
    x = _to_dev_x(torch, random_x(4, 2048, seed=5, dtype="bf16"))
    first = dt.gemv(x).cpu().numpy()
    for _ in range(3):
        assert np.array_equal(dt.gemv(x).cpu().numpy(), first)
