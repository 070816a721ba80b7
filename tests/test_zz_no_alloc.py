"""GPU test of the allocation-free product (hl_decode_gemv_noalloc): its
outputs equal hl_decode_gemv's bit for bit (the same kernels, the library's
per-GPU scratch in place of the caller's workspace), on two calls in a row,
the second with a smaller input, and for shapes that split the product over
k-parts (counters and partial sums in the scratch) or tile the activations."""
import ctypes

import numpy as np
import pytest

from gen import random_bf16, random_fp16, random_x

pytestmark = pytest.mark.gpu

hl = pytest.importorskip("paper_2502_00922_amd.hufflm")


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    hl.lib()
    return t


def _dev_x(torch, x):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    if x.dtype == np.float16:
        return torch.from_numpy(x).cuda()
    return torch.from_numpy(x).cuda()


def _pair(torch, blob, x):
    dt = hl.DeviceTensor(blob)
    xd = _dev_x(torch, x)
    R = dt.shape[0]
    y_ref = torch.full((x.shape[0], R), float("nan"), dtype=torch.float32, device="cuda")
    y_na = torch.full_like(y_ref, float("nan"))
    dt.gemv(xd, y_ref)
    dt.gemv_noalloc(xd, y_na)
    torch.cuda.synchronize()
    return y_ref.cpu().numpy(), y_na.cpu().numpy()


# (matrix, batch, x dtype, encoder keywords): the first of each pair is the
# larger call; 1024x4096 splits over k-parts (few row blocks), batch 16 tiles
# the activations, 4352x8192 runs the persistent kernel
CASES = [
    (((1024, 4096), 16, "bf16", {}), ((512, 2048), 5, "bf16", {})),
    (((4352, 8192), 16, "bf16", {}), ((1000, 4096), 3, "f32", {})),
    (((1024, 4096), 12, "bf16", {"whole_exponent": True}), ((256, 1024), 1, "bf16", {})),
    (((1024, 2048), 16, "f16", {"fp16": True}), ((512, 1024), 2, "f16", {"fp16": True})),
]


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_equals_workspace_product(torch, first, second):
    for k, (shape, batch, xdt, kw) in enumerate((first, second)):
        print(f"noalloc call {k}: {shape} batch {batch} x {xdt} {kw}", flush=True)
        w = (random_fp16 if kw.get("fp16") else random_bf16)(shape, seed=shape[0] + batch)
        blob = hl.encode(w, **kw)
        x = random_x(batch, shape[1], seed=batch, dtype=xdt)
        y_ref, y_na = _pair(torch, blob, x)
        assert not np.isnan(y_ref).any()
        assert np.array_equal(y_ref, y_na), f"call {k}: noalloc differs from the workspace product"


def test_noalloc_reports_oversized_scratch(torch):
    # the scratch limit: a product whose tiled activations alone exceed it
    w = random_bf16((16, 1 << 17), seed=5)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=64))
    need = int(hl.lib().hl_gemv_workspace_bytes(ctypes.byref(dt.view), 16))
    assert need > (4 << 20)
    x = _dev_x(torch, random_x(16, 1 << 17, seed=1, dtype="bf16"))
    y = torch.empty((16, 16), dtype=torch.float32, device="cuda")
    with pytest.raises(hl.HLError) as e:
        dt.gemv_noalloc(x, y)
    assert e.value.status == hl.HL_EUNSUPPORTED
