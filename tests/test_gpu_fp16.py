"""GPU parity of the float16 {1,5,5,5} format (three 32-symbol codes and a
raw sign plane): its decode kernel and its matrix-core decode-GEMV.

* decode equals the encoder's input bit for bit (every shape and group shape);
* decode-GEMV (16-row groups, float16 x) against the oracle's exactly rounded
  fp64 sums, |y - y_ref| <= 1e-3 * sum_k |w x|, at batch 1..16, with one and
  several blocks per row block;
* code shapes: every float16 pattern (decode only: infinities and NaNs),
  one-symbol fields, long exponent and low-mantissa codes together, and pairs
  of weights whose six codes overflow the decoder's 64-bit window (the
  bit-serial path);
* the format's limits: other activation types and other group shapes are
  reported as unsupported.
"""
import numpy as np
import pytest

from gen import random_fp16, random_x
from oracle import codec, gemv as ogemv

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


def _decode(torch, dt):
    out = dt.decode()
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint16)


def _x(torch, x):
    return torch.from_numpy(x).cuda()


def _check_gemv(torch, dt, w, batches, seed=0, rows=None):
    for batch in batches:
        x = random_x(batch, w.shape[1], seed=seed + batch, dtype="f16")
        y = dt.gemv(_x(torch, x))
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        y_ref, den = ogemv.gemv_rows(w, x, rows=rows, weights="fp16")
        got = y if rows is None else y[:, rows]
        assert np.max(ogemv.rel_err(got, y_ref, den)) <= TOL, batch


SHAPES = [((64, 1024), 64, 0), ((130, 48), 16, 0), ((3, 64), 8, 0), ((200, 512), 128, 0), ((65, 96), 32, 0),
          ((1, 8), 8, 0), ((300, 2048), 64, 64), ((129, 1024), 64, 8), ((77, 512), 16, 32), ((19, 1024), 8, 1),
          ((256, 4096), 64, 0), ((100, 2048), 32, 0), ((40, 4096), 128, 0), ((50, 512), 16, 0)]


@pytest.mark.parametrize("shape,S,GR", SHAPES)
def test_decode_bit_exact(torch, shape, S, GR):
    print(f"fp16 decode {shape} S={S} GR={GR}", flush=True)
    w = random_fp16(shape, seed=shape[0] + S)
    blob = hl.encode(w, seg_len=S, grp_rows=GR, fp16=True)
    if w.size <= 1 << 16:
        assert bytes(blob) == codec.encode16(w, seg_len=S, grp_rows=GR or None)
    dt = hl.DeviceTensor(blob)
    assert dt.view.format == hl.HL_FORMAT_FP16
    assert np.array_equal(_decode(torch, dt), w)


@pytest.mark.parametrize("shape,S,GR", [s for s in SHAPES if (s[0][1] // s[1]) % 4 == 0 and s[2] in (0, 16)])
def test_gemv_vs_oracle(torch, shape, S, GR):
    print(f"fp16 gemv {shape} S={S}", flush=True)
    w = random_fp16(shape, seed=shape[0] * 3 + S)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=S, grp_rows=GR, fp16=True))
    assert dt.view.grp_rows == 16
    _check_gemv(torch, dt, w, (1, 3, 16), seed=S)


@pytest.mark.parametrize("batch", list(range(1, 17)))
def test_every_batch(torch, batch):
    print(f"fp16 gemv batch {batch}", flush=True)
    w = random_fp16((192, 4096), seed=batch)
    dt = hl.DeviceTensor(hl.encode(w, fp16=True))
    _check_gemv(torch, dt, w, (batch,), seed=5)


def test_no_workspace_and_split(torch):
    """Few rows: the blocks of a row block split the columns (workspace), or
    one block takes the whole row when no workspace is given."""
    print("fp16 split-k", flush=True)
    w = random_fp16((48, 8192), seed=3)
    dt = hl.DeviceTensor(hl.encode(w, fp16=True))
    x = random_x(4, 8192, seed=1, dtype="f16")
    y_ref, den = ogemv.gemv_rows(w, x, weights="fp16")
    for ws in (None, False):
        y = dt.gemv(_x(torch, x), workspace=ws).cpu().numpy()
        assert np.max(ogemv.rel_err(y, y_ref, den)) <= TOL
    # repeated calls leave the workspace ready
    y2 = dt.gemv(_x(torch, x)).cpu().numpy()
    assert np.max(ogemv.rel_err(y2, y_ref, den)) <= TOL


def _long_pairs(rows, cols, seed):
    """Exponent and low-mantissa codes long enough that code(ml) + code(e)
    often exceeds 13 bits."""
    rng = np.random.default_rng(seed)
    n = rows * cols
    e = np.minimum(rng.geometric(0.35, n), 30).astype(np.uint32)
    ml = np.minimum(rng.geometric(0.3, n) - 1, 31).astype(np.uint32)
    mh = rng.integers(0, 32, n).astype(np.uint32)
    return codec.join_fields16(rng.integers(0, 2, n), e, mh, ml).reshape(rows, cols)


def _window_overflow(rows, cols, seed):
    """Geometric fields (12-bit codes for the rarest values) and 24 planted
    pairs of adjacent weights, each weight holding the rarest value of all
    three fields: two such weights need more than the 62 new bits of a window."""
    rng = np.random.default_rng(seed)
    n = rows * cols
    e, mh, ml = (np.minimum(rng.geometric(0.5, n) - 1, 20).astype(np.uint32) for _ in range(3))
    idx = rng.choice(n // 2, 24, replace=False) * 2
    for f, top in ((e, 29), (mh, 31), (ml, 31)):
        f[idx], f[idx + 1] = top, top - 1
    return codec.join_fields16(rng.integers(0, 2, n), e, mh, ml).reshape(rows, cols)


@pytest.mark.parametrize("kind", ["all_patterns", "single_symbols", "long_pairs", "window_overflow"])
def test_code_shapes(torch, kind):
    print(f"fp16 codes {kind}", flush=True)
    if kind == "all_patterns":
        w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(64, 1024)
        w = np.random.default_rng(2).permutation(w.ravel()).reshape(64, 1024)
    elif kind == "single_symbols":
        rng = np.random.default_rng(1)
        w = (0x3C00 | (rng.integers(0, 32, (96, 1024)) << 5) | (rng.integers(0, 2, (96, 1024)) << 15))
        w = w.astype(np.uint16)                         # e = 15 and ml = 0 everywhere
    elif kind == "long_pairs":
        w = _long_pairs(96, 1024, seed=4)
    else:
        w = _window_overflow(96, 1024, seed=5)
    blob = hl.encode(w, fp16=True)
    h = codec.parse_header(bytes(blob))
    if kind == "single_symbols":
        assert h["cb16"][0][0] == 1 and h["cb16"][2][0] == 1
    if kind == "long_pairs":
        lens = [max(c[2]) for c in h["cb16"]]
        assert lens[0] + lens[2] > 13                   # e + ml: long codes together
    if kind == "window_overflow":
        _, e, mh, ml = codec.split_fields16(w)
        tot = sum(np.array(c[2])[f] for c, f in zip(h["cb16"], (e, mh, ml)))
        assert (tot.reshape(-1, 2).sum(axis=1) > 62).sum() == 24
    dt = hl.DeviceTensor(blob)
    assert np.array_equal(_decode(torch, dt), w)
    if kind == "all_patterns":
        return
    _check_gemv(torch, dt, w, (1, 16), seed=11)


def test_unsupported_requests(torch):
    w = random_fp16((64, 512), seed=1)
    dt = hl.DeviceTensor(hl.encode(w, fp16=True))
    for dtype in (torch.bfloat16, torch.float32):
        with pytest.raises(hl.HLError) as ei:
            dt.gemv(torch.zeros((1, 512), dtype=dtype, device="cuda"))
        assert ei.value.status == hl.HL_EUNSUPPORTED
    dt32 = hl.DeviceTensor(hl.encode(w, seg_len=64, grp_rows=32, fp16=True))
    with pytest.raises(hl.HLError) as ei:
        dt32.gemv(torch.zeros((1, 512), dtype=torch.float16, device="cuda"))
    assert ei.value.status == hl.HL_EUNSUPPORTED
    # a bf16 container with float16 activations
    from gen import random_bf16
    db = hl.DeviceTensor(hl.encode(random_bf16((64, 512), seed=1)))
    with pytest.raises(hl.HLError):
        db.gemv(torch.zeros((1, 512), dtype=torch.float16, device="cuda"))


@pytest.mark.parametrize("S,cols", [(64, 4096), (32, 2048)])
@pytest.mark.parametrize("kind", ["gaussian", "long_pairs", "window_overflow"])
def test_persistent_kernel(torch, S, cols, kind):
    """Matrices with two row blocks per CU and two groups per wave (8196
    rows: a ragged last row block) run the persistent kernel's float16 form: its
    product against a float64 product of the exact float16 values (every row)
    and the oracle (sampled rows) at batch 1, 5 and 16, and its decode form
    bit-exact. The planted window overflows take the bit-serial path inside
    the persistent loop."""
    rows = 8196
    print(f"fp16 persistent S={S} {rows}x{cols} {kind}", flush=True)
    if kind == "gaussian":
        w = random_fp16((rows, cols), seed=S + cols)
    elif kind == "long_pairs":
        w = _long_pairs(rows, cols, seed=S)
    else:
        w = _window_overflow(rows, cols, seed=S)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=S, fp16=True))
    assert dt.view.grp_rows == 16
    wf = w.view(np.float16).astype(np.float64)
    rng = np.random.default_rng(S)
    sample = sorted({0, 15, 16, rows - 5, rows - 4, rows - 1} | set(int(r) for r in rng.integers(0, rows, 10)))
    for batch in (1, 5, 16):
        x = random_x(batch, cols, seed=batch, dtype="f16")
        y = dt.gemv(_x(torch, x)).cpu().numpy().astype(np.float64)
        xf = x.astype(np.float64)
        err = np.abs(y - xf @ wf.T) / (np.abs(xf) @ np.abs(wf).T + 1e-30)
        assert err.max() <= TOL, (batch, float(err.max()))
        yo, do = ogemv.gemv_rows(w, x, rows=sample, weights="fp16")
        assert (np.abs(y[:, sample] - yo) / (do + 1e-30)).max() <= TOL
    assert np.array_equal(_decode(torch, dt), w)
