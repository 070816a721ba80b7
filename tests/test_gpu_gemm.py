"""GPU parity of the prefill decode-GEMM (many activation rows, each weight
tile decoded once per chunk of up to 128 tokens and multiplied with all of
them on the matrix cores).

Every output against a float64 product of the exact bf16 values and sampled
outputs against the oracle's exactly rounded sums, |y - y_ref| <= 1e-3 *
sum_k |w x|: token counts 1 .. 300 (one and several chunks, ragged last
tile), ragged row sets and row blocks, S = 32 and 64, both bf16 formats,
repeated calls on one workspace; up to 64 tokens on the persistent kernel
(one, two or four 16-token tiles); unsupported requests are reported.
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


def _xdev(torch, x):
    return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()


def _check(torch, dt, w, T, seed):
    x = random_x(T, w.shape[1], seed=seed, dtype="bf16")
    y = dt.gemm(_xdev(torch, x)).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    Wf, Xf = bf16_to_f64(w), bf16_to_f64(x)
    err = np.abs(y - Xf @ Wf.T) / (np.abs(Xf) @ np.abs(Wf).T + 1e-30)
    assert err.max() <= TOL, (T, float(err.max()))
    rng = np.random.default_rng(seed)
    rows = sorted({0, w.shape[0] - 1} | set(int(r) for r in rng.integers(0, w.shape[0], 4)))
    toks = sorted({0, T - 1, int(rng.integers(0, T))})
    yo, do = ogemv.gemv_rows(w, x[toks], rows=rows)
    assert np.max(np.abs(y[np.ix_(toks, rows)] - yo) / (do + 1e-30)) <= TOL


@pytest.mark.parametrize("T", [1, 5, 16, 17, 64, 100, 128, 129, 300])
def test_token_counts(torch, T):
    print(f"gemm T={T}", flush=True)
    w = random_bf16((300, 2048), seed=T)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=64))
    _check(torch, dt, w, T, seed=T)


@pytest.mark.parametrize("shape,S,whole", [((4100, 1024), 64, False), ((256, 4096), 32, False),
                                           ((513, 4096), 64, True), ((16, 256), 64, False),
                                           ((1, 512), 32, True)])
def test_shapes_and_formats(torch, shape, S, whole):
    print(f"gemm {shape} S={S} whole={whole}", flush=True)
    w = random_bf16(shape, seed=shape[0] + S)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=S, whole_exponent=whole))
    assert dt.view.grp_rows == 16
    for T in (33, 128):
        _check(torch, dt, w, T, seed=T + S)


def _persistent_shape(torch, rows, cols, S):
    """Whether a product of this shape runs on the persistent kernel: at least
    one 16-row block per compute unit and two 256-column groups per wave of a
    block of eight."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    RB, CB = -(-rows // 16), cols // (4 * S)
    return RB >= cus and CB >= 8 and RB * CB >= 2 * cus * 8


@pytest.mark.parametrize("shape,S,fmt", [((4100, 4096), 64, "split"), ((4100, 4096), 64, "whole"),
                                         ((4096, 4096), 32, "split"), ((4112, 8192), 64, "split_unbounded")])
def test_persistent_up_to_64_tokens(torch, shape, S, fmt):
    """Up to 64 tokens on matrices the persistent kernel takes: one 16-token
    tile per decode step, two (17..32 tokens) or four (33..64, columns of 16
    words or more; else the chunked kernel), sums per row block in one block;
    ragged last row block (4100 rows), bounded-pair and joint tables."""
    print(f"gemm persistent {shape} S={S} {fmt}", flush=True)
    assert _persistent_shape(torch, shape[0], shape[1], S)
    kw = {"whole": {"whole_exponent": True}, "split_unbounded": {"pair_max": 0}}.get(fmt, {})
    w = random_bf16(shape, seed=shape[0] + S + len(fmt))
    dt = hl.DeviceTensor(hl.encode(w, seg_len=S, **kw))
    for T in (1, 7, 16, 17, 23, 32, 33, 50, 64):
        print(f"  T={T}", flush=True)
        _check(torch, dt, w, T, seed=T + S)


def test_persistent_tiles_70b_gate(torch):
    """The 70B gate matrix (28672x8192, drawn from its own seed) at 24, 32 and
    64 tokens on the two- and four-tile forms: sampled rows against the oracle's exactly
    rounded sums, every output against a float32 product of the original
    weights (torch, on the GPU), within 1e-3 of sum_k |w x|."""
    from gen import workload_matrices, gen_matrix
    spec = workload_matrices(5)[4]
    print(f"gemm persistent tiles {spec.rows}x{spec.cols}", flush=True)
    w = gen_matrix(spec)
    dt = hl.DeviceTensor(hl.encode(w))
    assert _persistent_shape(torch, spec.rows, spec.cols, 64)
    wf = torch.from_numpy(w.view(np.int16)).cuda().view(torch.bfloat16).float()
    rng = np.random.default_rng(5)
    rows = sorted({0, spec.rows - 1} | set(int(r) for r in rng.integers(0, spec.rows, 6)))
    for T in (24, 32, 64):
        print(f"  T={T}", flush=True)
        x = random_x(T, spec.cols, seed=T, dtype="bf16")
        xd = _xdev(torch, x)
        y = dt.gemm(xd)
        xf = xd.float()
        ref = xf @ wf.T
        den = xf.abs() @ wf.abs().T
        err = ((y - ref).abs() / (den + 1e-30)).max().item()
        assert err <= TOL, (T, err)
        yo, do = ogemv.gemv_rows(w, x, rows=rows)
        yh = y.cpu().numpy().astype(np.float64)
        assert np.max(np.abs(yh[:, rows] - yo) / (do + 1e-30)) <= TOL
    del wf


def test_persistent_tiles_repeat(torch):
    print("gemm persistent tiles repeated", flush=True)
    w = random_bf16((4100, 4096), seed=11)
    dt = hl.DeviceTensor(hl.encode(w))
    for T in (29, 61):
        x = _xdev(torch, random_x(T, 4096, seed=12, dtype="bf16"))
        y1 = dt.gemm(x).cpu().numpy()
        for _ in range(3):
            assert np.array_equal(y1, dt.gemm(x).cpu().numpy())   # fixed summation order


def test_repeated_calls_share_the_workspace(torch):
    print("gemm repeated", flush=True)
    w = random_bf16((600, 1024), seed=3)
    dt = hl.DeviceTensor(hl.encode(w))
    x = random_x(70, 1024, seed=4, dtype="bf16")
    y1 = dt.gemm(_xdev(torch, x)).cpu().numpy()
    for _ in range(3):
        y2 = dt.gemm(_xdev(torch, x)).cpu().numpy()
        assert np.array_equal(y1, y2)           # fixed summation order
    _check(torch, dt, w, 20, seed=9)            # smaller call after a larger one


def test_unsupported_requests(torch):
    w = random_bf16((64, 512), seed=1)
    dt32 = hl.DeviceTensor(hl.encode(w, seg_len=64, grp_rows=32))
    with pytest.raises(hl.HLError) as ei:
        dt32.gemm(torch.zeros((4, 512), dtype=torch.bfloat16, device="cuda"))
    assert ei.value.status == hl.HL_EUNSUPPORTED
    dt128 = hl.DeviceTensor(hl.encode(w, seg_len=128))
    with pytest.raises(hl.HLError):
        dt128.gemm(torch.zeros((4, 512), dtype=torch.bfloat16, device="cuda"))
    dt = hl.DeviceTensor(hl.encode(w))
    with pytest.raises(ValueError):
        dt.gemm(torch.zeros((4, 512), dtype=torch.float32, device="cuda"))
