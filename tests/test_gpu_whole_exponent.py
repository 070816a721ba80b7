"""GPU parity of the whole-exponent format (one 256-symbol code per exponent
byte): the same decode and decode-GEMV kernels run on its decode table.

* decode equals the encoder's input bit for bit;
* decode-GEMV against the oracle's exactly rounded fp64 sums,
  |y - y_ref| <= 1e-3 * sum_k |w x|, for x in float32 and bf16, batch 1..16;
* the kernel variants all run: 16-row groups at S = 64 (matrix-core kernel,
  and the persistent one for a matrix of 4100 x 8192), 64- and 32-row groups,
  float32 activations (vector kernel);
* code shapes: one exponent value (no stream bits), 256 values with 8-bit
  codes (every bf16 pattern, so decode only), codes of exactly 13 bits (lmax 13 binding: four of them fill the
  decoder's 64-bit window but for 10 bits), log-uniform magnitudes.
"""
import numpy as np
import pytest

from gen import f32_to_bf16_bits, random_bf16, random_x
from oracle import codec, gemv as ogemv
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


def _to_dev_x(torch, x):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(x).cuda()


def _decode(torch, dt):
    out = dt.decode()
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint16)


def _check_gemv(torch, dt, w, batches, xdt, seed=0, rows=None):
    for batch in batches:
        x = random_x(batch, w.shape[1], seed=seed + batch, dtype=xdt)
        y = dt.gemv(_to_dev_x(torch, x))
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        y_ref, den = ogemv.gemv_rows(w, x, rows=rows)
        got = y if rows is None else y[:, rows]
        assert np.max(ogemv.rel_err(got, y_ref, den)) <= TOL, (batch, xdt)


def _log_uniform(shape, seed):
    rng = np.random.default_rng(seed)
    mag = np.exp2(rng.uniform(-60, 60, shape)).astype(np.float32)
    return f32_to_bf16_bits(mag * np.where(rng.random(shape) < 0.5, -1, 1).astype(np.float32))


SHAPES = [((64, 1024), 64, 0), ((130, 48), 16, 0), ((3, 64), 8, 0), ((200, 512), 512, 0), ((65, 96), 32, 0),
          ((1, 8), 8, 0), ((300, 2048), 64, 64), ((129, 1024), 64, 8), ((77, 512), 16, 32), ((19, 1024), 8, 1),
          ((256, 4096), 64, 0), ((100, 2048), 32, 0)]


@pytest.mark.parametrize("shape,S,GR", SHAPES)
def test_decode_and_gemv(torch, shape, S, GR):
    print(f"whole-exponent {shape} S={S} GR={GR}", flush=True)
    w = random_bf16(shape, seed=shape[0] * 3 + S)
    blob = hl.encode(w, seg_len=S, grp_rows=GR, whole_exponent=True)
    if w.size <= 1 << 16:
        assert bytes(blob) == codec.encode8(w, seg_len=S, grp_rows=GR or None)
    dt = hl.DeviceTensor(blob)
    assert dt.view.format == hl.HL_FORMAT_WHOLE_EXPONENT
    assert np.array_equal(_decode(torch, dt), w)
    _check_gemv(torch, dt, w, (1, 3), "bf16", seed=S)
    _check_gemv(torch, dt, w, (2,), "f32", seed=S)


@pytest.mark.parametrize("batch", [1, 4, 5, 8, 11, 16])
def test_every_kernel_batch(torch, batch):
    print(f"whole-exponent batch {batch}", flush=True)
    w = random_bf16((192, 4096), seed=batch)
    dt = hl.DeviceTensor(hl.encode(w, whole_exponent=True))
    _check_gemv(torch, dt, w, (batch,), "bf16", seed=7)


@pytest.mark.parametrize("kind", ["constant", "all_values", "lmax13", "log_uniform"])
def test_code_shapes(torch, kind):
    print(f"whole-exponent codes {kind}", flush=True)
    rows, cols, lmax = 96, 1024, 12
    if kind == "constant":
        rng = np.random.default_rng(1)
        w = (0x3F80 | rng.integers(0, 128, (rows, cols)) | (rng.integers(0, 2, (rows, cols)) << 15))
        w = w.astype(np.uint16)
    elif kind == "all_values":
        w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(64, 1024)
        w = np.random.default_rng(2).permutation(w.ravel()).reshape(64, 1024)
    elif kind == "lmax13":
        # counts 2, 2, 4, ..., 2^13 plus a uniform remainder: the unlimited code is
        # longer than 13 bits, the limited one has codes of exactly 13 bits
        rng = np.random.default_rng(3)
        e = [np.full(2, 60)] + [np.full(2 ** i, 60 + i) for i in range(1, 14)]
        e = np.concatenate(e + [rng.integers(120, 127, rows * cols - sum(map(len, e)))]).astype(np.uint32)
        e = rng.permutation(e)
        w = ((rng.integers(0, 2, e.size) << 15) | (e << 7) | rng.integers(0, 128, e.size)).astype(np.uint16)
        w = w.reshape(rows, cols)
        lmax = 13
    else:
        w = _log_uniform((rows, cols), seed=4)
    blob = hl.encode(w, lmax=lmax, whole_exponent=True)
    h = codec.parse_header(bytes(blob))
    if kind == "constant":
        assert h["nsym8"] == 1 and h["max_grp_units"] == 0
    if kind == "all_values":
        assert set(h["len8"]) == {8}
    if kind == "lmax13":
        assert max(h["len8"]) == 13
        assert max(codec.huffman_lengths(codec.histogram(codec.exponent_byte(w), 256))) > 13
    dt = hl.DeviceTensor(blob)
    assert np.array_equal(_decode(torch, dt), w)
    if kind == "all_values":
        return                  # holds infinities and NaNs: decode only
    _check_gemv(torch, dt, w, (1, 16), "bf16", seed=11)
    _check_gemv(torch, dt, w, (3,), "f32", seed=11)


@pytest.mark.parametrize("kind", ["gaussian", "log_uniform"])
def test_persistent_kernel(torch, kind):
    """4100 x 8192 at S = 64: at least one row block per CU, the persistent kernel."""
    rows, cols = 4100, 8192
    print(f"whole-exponent persistent {kind}", flush=True)
    w = random_bf16((rows, cols), seed=5) if kind == "gaussian" else _log_uniform((rows, cols), seed=5)
    dt = hl.DeviceTensor(hl.encode(w, whole_exponent=True))
    assert dt.view.grp_rows == 16 and dt.view.seg_len == 64
    assert np.array_equal(_decode(torch, dt), w)
    Wf = bf16_to_f64(w)
    for B in (1, 5, 16):
        xs = random_x(B, cols, seed=B, dtype="bf16")
        y = dt.gemv(_to_dev_x(torch, xs)).cpu().numpy().astype(np.float64)
        Xf = bf16_to_f64(xs)
        err = np.abs(y - Xf @ Wf.T) / (np.abs(Xf) @ np.abs(Wf).T + 1e-30)
        assert err.max() <= TOL, (B, float(err.max()))
        sample = [0, 15, 16, rows - 5, rows - 4, rows - 1, 1234]
        yo, do = ogemv.gemv_rows(w, xs, rows=sample)
        assert np.max(np.abs(y[:, sample] - yo) / (do + 1e-30)) <= TOL
    torch.cuda.synchronize()
