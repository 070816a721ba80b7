"""The persistent matrix-core decode-GEMV (chosen for 16-row groups at S = 32
or 64 when a matrix has at least one row block per CU and two groups per wave:
on a 256-CU MI355X, 4100 rows and 8192 (S = 64) or 4096 (S = 32) columns).

The rows leave a ragged last row block (4 rows). Three weight distributions
give short, typical and long codes, so that the kernel's instantiations for
different stream lengths all run:
* constant exponents (both fields single-symbol: no stream bits at all);
* N(0, 0.02) with outliers (the workloads' distribution);
* log-uniform magnitudes over 2^-60 .. 2^60 (long streams: about 7 code bits
  per weight, so two pairs often exceed a 14-bit window);
* a geometric low exponent nibble (codes up to the length limit: pairs past
  the 13-bit window);
* long moves: every pair fits the 13-bit window (no escapes), but every
  64th row holds pairs of 10 to 13 bits, so four pairs often move a lane's
  position past the four words it read and its second window is read from
  the column (the decode's rare wave-uniform branch);
* spread: the workloads' distribution with about one 64-column piece in 97
  log-uniform (long codes), so that some groups' segments span more than 255
  code bits and the shorter ones are padded to the group's base.
Each in the split format (code limit 12 and 15) and the whole-exponent
format. The full decode of each container (the same kernel storing the
weights) must be bit-exact. Outputs: every row against a float64 product of the exact bf16
values, and sampled rows against the oracle's exactly rounded sums, at batch
1, 5 and 16.
"""
import numpy as np
import pytest

from gen import f32_to_bf16_bits, random_bf16, random_x
from oracle import codec
from oracle import gemv as ogemv
from oracle.gemv import bf16_to_f64

hl = pytest.importorskip("paper_2502_00922_amd.hufflm")

pytestmark = pytest.mark.gpu
TOL = 1e-3


@pytest.fixture(scope="module")
def torch():
    t = pytest.importorskip("torch")
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _weights(kind, rows, cols, seed):
    rng = np.random.default_rng(seed)
    if kind == "constant_exponent":
        v = (1.0 + 0.96 * rng.random((rows, cols), dtype=np.float32)) * np.where(rng.random((rows, cols)) < 0.5, -1, 1)
        return f32_to_bf16_bits(v.astype(np.float32))
    if kind == "gaussian":
        return random_bf16((rows, cols), seed=seed)
    if kind == "geometric":
        # geometric low exponent nibble, a few high nibbles: codes up to the
        # length limit, pairs longer than the 13-bit window
        n = rows * cols
        el = np.minimum(rng.geometric(0.45, n) - 1, 15)
        eh = rng.choice([3, 6, 7, 8], n, p=[0.02, 0.08, 0.8, 0.1])
        bits = (rng.integers(0, 2, n) << 15) | (eh << 11) | (el << 7) | rng.integers(0, 128, n)
        return bits.astype(np.uint16).reshape(rows, cols)
    if kind == "long_moves":
        # eh uniform over 4..11 (3-bit codes); el geometric over 0..10 (codes
        # of 1..10 bits: the longest pair is exactly 13 bits), except in
        # every 64th row, where it is uniform over 7..10 (the longest codes)
        eh = rng.integers(4, 12, (rows, cols))
        el = np.minimum(rng.geometric(0.5, (rows, cols)) - 1, 10)
        el = np.where((np.arange(rows) % 64 == 0)[:, None], rng.integers(7, 11, (rows, cols)), el)
        bits = (rng.integers(0, 2, (rows, cols)) << 15) | (eh << 11) | (el << 7) | rng.integers(0, 128, (rows, cols))
        return bits.astype(np.uint16)
    mag = np.exp2(rng.uniform(-60, 60, (rows, cols))).astype(np.float32)
    wide = f32_to_bf16_bits(mag * np.where(rng.random((rows, cols)) < 0.5, -1, 1).astype(np.float32))
    if kind == "spread":
        piece = (np.arange(rows)[:, None] * 31 + np.arange(cols)[None, :] // 64) % 97 == 0
        return np.where(piece, wide, random_bf16((rows, cols), seed=seed))
    return wide


# container formats: (encoder keywords). The default split codes keep every
# weight's pair within 11 bits (at S = 64 the kernel's bounded-pair form:
# replicated 11-bit table, no escape or long-move branch); without the joint
# limit pairs reach 13 bits (long moves of the window) and with the longer
# limit el codes pass the 13-bit window (escape entries); whole exponents
# have codes of at most 13 bits (no escapes)
FORMATS = {"split": {}, "split_unbounded": {"pair_max": 0}, "split_lmax15": {"lmax": 15, "pair_max": 0},
           "whole": {"whole_exponent": True}}


@pytest.mark.parametrize("S,cols,fmt", [(64, 8192, "split"), (32, 4096, "split"), (64, 8192, "split_unbounded"),
                                        (64, 8192, "split_lmax15"), (64, 8192, "whole"), (32, 4096, "whole")])
@pytest.mark.parametrize("kind", ["constant_exponent", "gaussian", "log_uniform", "geometric", "long_moves", "spread"])
def test_persistent_kernel(torch, S, cols, fmt, kind):
    rows = 4100
    print(f"persistent S={S} {rows}x{cols} {fmt} {kind}", flush=True)
    W = _weights(kind, rows, cols, seed=S + cols)
    blob = hl.encode(W, seg_len=S, **FORMATS[fmt])
    if kind == "spread" and S == 64:
        # padded segments present: some stored length is 255 over its base
        h = codec.parse_header(bytes(blob))
        assert np.frombuffer(bytes(blob), np.uint8, h["n_seg"], h["off_seg_bits"]).max() == 255
    dt = hl.DeviceTensor(blob)
    assert dt.view.grp_rows == 16
    cb = dt.view.cb
    if kind == "long_moves" and fmt == "split_unbounded":
        # every pair fits the 13-bit window: long moves without escapes
        assert max(cb.eh.len) + max(cb.el.len) <= 13
    if fmt == "split":
        assert max(cb.eh.len) + max(cb.el.len) <= hl.PAIR_MAX
    Wf = bf16_to_f64(W)
    rng = np.random.default_rng(S)
    sample = sorted({0, 15, 16, rows - 5, rows - 4, rows - 1} | set(int(r) for r in rng.integers(0, rows, 10)))
    for B in (1, 5, 16):
        xs = random_x(B, cols, seed=B, dtype="bf16")
        x = torch.from_numpy(xs.view(np.int16)).cuda().view(torch.bfloat16)
        y = dt.gemv(x).cpu().numpy().astype(np.float64)
        Xf = bf16_to_f64(xs)
        ref = Xf @ Wf.T
        den = np.abs(Xf) @ np.abs(Wf).T
        err = np.abs(y - ref) / (den + 1e-30)
        assert err.max() <= TOL, (B, float(err.max()), int(np.argmax(err.max(0))))
        yo, do = ogemv.gemv_rows(W, xs, rows=sample)
        assert (np.abs(y[:, sample] - yo) / (do + 1e-30)).max() <= TOL
    # the full decode of the same container runs on the persistent kernel
    # too (its product replaced by stores): bit-exact
    assert np.array_equal(dt.decode().cpu().numpy().view(np.uint16), W)
    torch.cuda.synchronize()


def test_padded_segments_small(torch):
    """One 16 x 4 group whose segments span more than 255 code bits (the
    shorter ones padded to the group's base), on the non-persistent kernels:
    decode bit-exact, products against the oracle."""
    from test_oracle_pins import _spread_lengths_matrix
    W = _spread_lengths_matrix()
    dt = hl.DeviceTensor(hl.encode(W, seg_len=64, grp_rows=16))
    assert np.array_equal(dt.decode().cpu().numpy().view(np.uint16), W)
    for B in (1, 5):
        xs = random_x(B, W.shape[1], seed=B, dtype="bf16")
        x = torch.from_numpy(xs.view(np.int16)).cuda().view(torch.bfloat16)
        y = dt.gemv(x).cpu().numpy().astype(np.float64)
        yo, do = ogemv.gemv_rows(W, xs, rows=list(range(W.shape[0])))
        assert (np.abs(y - yo) / (do + 1e-30)).max() <= TOL
    torch.cuda.synchronize()
