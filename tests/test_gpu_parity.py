"""GPU parity: the gfx950 decode and fused decode-GEMV against the oracle.

Decoded weights must equal the encoder's input bit for bit; the GEMV must meet
|y - y_ref| / (sum |w x| + 1e-30) <= 1e-3 per output against the oracle's
exactly rounded fp64 product. Every call goes through the C ABI.
"""
import numpy as np
import pytest

from gen import random_bf16, random_x
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


def _to_dev_x(torch, x):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(x).cuda()


def _decode(torch, dt):
    out = dt.decode()
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint16)


# (shape, segment length, group rows; 0 = the encoder's default)
SHAPES = [((64, 1024), 128, 0), ((130, 48), 16, 0), ((3, 64), 8, 0), ((200, 512), 512, 0), ((65, 96), 32, 0),
          ((1, 8), 8, 0), ((127, 136), 136, 0), ((300, 2048), 128, 0), ((64, 256), 256, 0),
          ((300, 2048), 64, 64), ((129, 1024), 64, 8), ((77, 512), 16, 32), ((19, 1024), 8, 1)]


@pytest.mark.parametrize("shape,S,GR", SHAPES)
def test_decode_bit_exact(torch, shape, S, GR):
    print(f"decode {shape} S={S} GR={GR}", flush=True)
    w = random_bf16(shape, seed=shape[0] * 7 + S)
    blob = hl.encode(w, seg_len=S, grp_rows=GR)
    if w.size <= 1 << 16:
        assert bytes(blob) == codec.encode(w, seg_len=S, grp_rows=GR or None)
    dt = hl.DeviceTensor(blob)
    assert np.array_equal(_decode(torch, dt), w)


@pytest.mark.parametrize("shape,S,GR", SHAPES)
@pytest.mark.parametrize("xdt", ["f32", "bf16"])
def test_gemv_vs_oracle(torch, shape, S, GR, xdt):
    print(f"gemv {shape} S={S} GR={GR} x={xdt}", flush=True)
    w = random_bf16(shape, seed=shape[0] * 5 + S)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=S, grp_rows=GR))
    for batch in (1, 3):
        x = random_x(batch, shape[1], seed=batch + S, dtype=xdt)
        y = dt.gemv(_to_dev_x(torch, x))
        torch.cuda.synchronize()
        y_ref, den = ogemv.gemv_rows(w, x)
        assert np.max(ogemv.rel_err(y.cpu().numpy(), y_ref, den)) <= TOL


@pytest.mark.parametrize("batch", list(range(1, 17)))
def test_gemv_every_batch(torch, batch):
    print(f"gemv batch {batch}", flush=True)
    w = random_bf16((192, 1024), seed=99)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=128))
    x = random_x(batch, 1024, seed=batch, dtype="bf16")
    y = dt.gemv(_to_dev_x(torch, x))
    torch.cuda.synchronize()
    y_ref, den = ogemv.gemv_rows(w, x)
    assert np.max(ogemv.rel_err(y.cpu().numpy(), y_ref, den)) <= TOL


def _geometric_matrix(rows, cols, seed, p=0.45):
    rng = np.random.default_rng(seed)
    n = rows * cols
    el = np.minimum(rng.geometric(p, n) - 1, 15)
    eh = rng.choice([3, 6, 7, 8], n, p=[0.02, 0.08, 0.8, 0.1])
    return codec.join_fields(rng.integers(0, 2, n), eh, el, rng.integers(0, 128, n)).reshape(rows, cols)


@pytest.mark.parametrize("lmax", [6, 12, 15])
def test_long_codes_take_the_slow_path(torch, lmax):
    """Code pairs longer than the 13-bit window (el codes up to 15 bits)."""
    print(f"long codes lmax={lmax}", flush=True)
    w = _geometric_matrix(96, 512, seed=lmax)
    # no joint limit of the pair: long pairs are the point here
    blob = hl.encode(w, seg_len=64, lmax=lmax, pair_max=0)
    assert bytes(blob) == codec.encode(w, seg_len=64, lmax=lmax, pair_max=0)
    h = codec.parse_header(bytes(blob))
    if lmax == 15:
        # el codes past the table window too (the bit-by-bit el decode)
        assert max(h["el_len"]) > 13 and max(h["el_len"]) + max(h["eh_len"]) > 13
    if lmax == 12:
        # pairs past the window whose el code fits in it (el from the table)
        assert max(h["el_len"]) <= 13 < max(h["el_len"]) + max(h["eh_len"])
    dt = hl.DeviceTensor(blob)
    assert np.array_equal(_decode(torch, dt), w)
    x = random_x(2, 512, seed=1, dtype="bf16")
    y = dt.gemv(_to_dev_x(torch, x))
    torch.cuda.synchronize()
    y_ref, den = ogemv.gemv_rows(w, x)
    assert np.max(ogemv.rel_err(y.cpu().numpy(), y_ref, den)) <= TOL


def test_single_symbol_fields(torch):
    print("single-symbol fields", flush=True)
    w = np.full((70, 64), 0x3F80, np.uint16)
    w[::3, ::5] = 0xBF80
    w = w | np.arange(64, dtype=np.uint16)[None, :] % 128
    dt = hl.DeviceTensor(hl.encode(w, seg_len=32))
    assert np.array_equal(_decode(torch, dt), w)
    x = random_x(1, 64, seed=2)
    y = dt.gemv(_to_dev_x(torch, x))
    torch.cuda.synchronize()
    y_ref, den = ogemv.gemv_rows(w, x)
    assert np.max(ogemv.rel_err(y.cpu().numpy(), y_ref, den)) <= TOL


def test_all_bf16_patterns_decode(torch):
    print("all patterns", flush=True)
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(128, 512)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=128))
    assert np.array_equal(_decode(torch, dt), w)


@pytest.mark.parametrize("xdt", ["f32", "bf16"])
def test_bf16_comparator(torch, xdt):
    print(f"bf16 comparator {xdt}", flush=True)
    w = random_bf16((257, 1024), seed=3)
    wd = torch.from_numpy(w.view(np.int16)).cuda()
    for batch in (1, 4, 16):
        x = random_x(batch, 1024, seed=batch, dtype=xdt)
        y = hl.gemv_bf16(wd, _to_dev_x(torch, x))
        torch.cuda.synchronize()
        y_ref, den = ogemv.gemv_rows(w, x)
        assert np.max(ogemv.rel_err(y.cpu().numpy(), y_ref, den)) <= TOL


def test_errors_are_reported(torch):
    w = random_bf16((64, 128), seed=1)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=128))
    x17 = torch.zeros((17, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        dt.gemv(x17)  # batch above 16: the binding refuses it, and so does the library
    import ctypes
    y = torch.empty((17, 64), dtype=torch.float32, device="cuda")
    assert hl.lib().hl_decode_gemv(ctypes.byref(dt.view), ctypes.c_void_p(x17.data_ptr()), hl.HL_BF16, 17,
                                   ctypes.c_void_p(y.data_ptr()), None, 0, None) == hl.HL_EINVAL
    with pytest.raises(ValueError):
        dt.gemv(torch.zeros((1, 64), dtype=torch.bfloat16, device="cuda"))


def test_misaligned_buffers_rejected(torch):
    # buffers the kernels access in 16-byte pieces must be 16-byte aligned:
    # a view 2 bytes into an allocation is refused on the host, nothing runs
    w = random_bf16((64, 256), seed=2)
    dt = hl.DeviceTensor(hl.encode(w))
    base = torch.zeros(64 * 256 + 8, dtype=torch.int16, device="cuda")
    with pytest.raises(hl.HLError):
        dt.decode(base[1:1 + 64 * 256].view(64, 256))
    xb = torch.zeros(256 + 8, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(hl.HLError):
        dt.gemv(xb[1:257].view(1, 256))
    # the aligned views of the same buffers work
    out = dt.decode(base[8:8 + 64 * 256].view(64, 256))
    assert np.array_equal(out.cpu().numpy().view(np.uint16), w)
    y = dt.gemv(xb[8:264].view(1, 256))
    torch.cuda.synchronize()
    assert np.all(y.cpu().numpy() == 0)


def test_device_copy(torch):
    # a device-to-device copy of a container and its table decodes and
    # multiplies exactly like the original, also after the original is gone
    print("device copy", flush=True)
    w = random_bf16((300, 2048), seed=21)
    dt = hl.DeviceTensor(hl.encode(w, seg_len=64))
    x = _to_dev_x(torch, random_x(3, 2048, seed=4, dtype="bf16"))
    y0 = dt.gemv(x).cpu().numpy()
    cp = dt.copy()
    assert cp.blob.data_ptr() != dt.blob.data_ptr() and cp.lut.data_ptr() != dt.lut.data_ptr()
    del dt
    torch.cuda.synchronize()
    assert np.array_equal(cp.gemv(x).cpu().numpy(), y0)
    assert np.array_equal(_decode(torch, cp), w)
