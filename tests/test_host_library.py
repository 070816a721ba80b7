"""Host half of the library against the oracle (no GPU): codebooks, byte-identical
containers, validation of damaged containers, argument errors, and the C-ABI
exports declared in include/hufflm.h."""
import ctypes
import os
import re

import numpy as np
import pytest

from gen import random_bf16, random_fp16
from oracle import codec

hl = pytest.importorskip("paper_2502_00922_amd.hufflm")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    return hl.lib()


def test_exports_match_header(L):
    text = open(os.path.join(ROOT, "include", "hufflm.h")).read()
    names = set(re.findall(r"\b(hl_[a-z0-9_]+)\s*\(", text))
    assert names, "no declarations found"
    for n in sorted(names):
        assert hasattr(L, n), f"{n} declared in hufflm.h but not exported"
    assert set(hl.EXPORTS) == names


def test_binding_constants_match_header():
    # the binding allocates tables and checks batches with the header's sizes
    text = open(os.path.join(ROOT, "include", "hufflm.h")).read()
    defs = {k: int(v) for k, v in re.findall(r"#define (HL_[A-Z0-9_]+) (\d+)u?", text)}
    assert hl.LUT_BYTES == defs["HL_LUT_BYTES"]
    assert hl.MAX_BATCH == defs["HL_MAX_BATCH"]
    assert hl.HEADER_BYTES == defs["HL_HEADER_BYTES"]


def test_misaligned_pointers_rejected_before_device_work(L):
    # the alignment checks come before any device work, so fake device
    # addresses (never dereferenced) that are 2 bytes off a 16-byte boundary
    # give HL_EINVAL without a GPU
    import ctypes
    t = hl.TensorView()
    good, bad = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10002)
    assert L.hl_decode(ctypes.byref(t), bad, None) == hl.HL_EINVAL
    assert L.hl_decode_gemv(ctypes.byref(t), bad, hl.HL_BF16, 1, good, None, 0, None) == hl.HL_EINVAL
    assert L.hl_decode_gemv(ctypes.byref(t), good, hl.HL_BF16, 1, good, bad, 1 << 20, None) == hl.HL_EINVAL
    assert L.hl_decode_gemm(ctypes.byref(t), bad, hl.HL_BF16, 4, good, good, 1 << 20, None) == hl.HL_EINVAL
    assert L.hl_gemv_bf16(bad, 8, 8, good, hl.HL_BF16, 1, good, None) == hl.HL_EINVAL
    assert L.hl_gemv_bf16(good, 8, 8, good, hl.HL_BF16, 1, ctypes.c_void_p(0x10001), None) == hl.HL_EINVAL
    ts = (ctypes.POINTER(hl.TensorView) * 1)(ctypes.pointer(t))
    ys = (ctypes.c_void_p * 1)(0x10000)
    assert L.hl_decode_gemv_multi(ctypes.cast(ts, ctypes.c_void_p), 1, bad, hl.HL_BF16, 1,
                                  ctypes.cast(ys, ctypes.c_void_p), None, 0, None) == hl.HL_EINVAL
    assert L.hl_decode_gemv_noalloc(ctypes.byref(t), bad, hl.HL_BF16, 1, good, None) == hl.HL_EINVAL


def _codebook_lists(cb):
    return (cb.eh.nsym, cb.eh.single, list(cb.eh.len), cb.el.nsym, cb.el.single, list(cb.el.len))


@pytest.mark.parametrize("seed", range(6))
def test_codebook_equals_oracle(seed):
    rng = np.random.default_rng(seed)
    w = random_bf16((32, 256), seed, std=float(rng.choice([0.002, 0.02, 0.5])))
    cb = hl.build_codebook(w, lmax=12)
    ceh, cel = codec.build_codebooks(w, 12)
    assert _codebook_lists(cb) == (ceh.nsym, ceh.single, ceh.lengths, cel.nsym, cel.single, cel.lengths)


CASES = [
    ((64, 1024), 128, 12, 0), ((130, 48), 16, 12, 0), ((3, 64), 8, 12, 0), ((200, 512), 512, 12, 0),
    ((65, 96), 32, 12, 0), ((1, 8), 8, 12, 0), ((127, 136), 136, 12, 0), ((64, 1024), 256, 6, 0),
    ((130, 512), 64, 12, 64), ((130, 512), 64, 12, 8), ((37, 256), 32, 12, 32), ((21, 512), 8, 12, 1),
]


@pytest.mark.parametrize("shape,S,lmax,GR", CASES)
def test_byte_identical_to_oracle(shape, S, lmax, GR):
    w = random_bf16(shape, seed=sum(shape) + S)
    a = bytes(hl.encode(w, seg_len=S, lmax=lmax, grp_rows=GR))
    b = codec.encode(w, seg_len=S, lmax=lmax, grp_rows=GR or None)
    assert a == b
    assert hl.validate(a) == 0


def test_byte_identical_with_padded_segments():
    """A group whose segments' code bits span more than 255: the library pads
    the shorter segments to the group's base exactly as the oracle does."""
    from test_oracle_pins import _spread_lengths_matrix
    w = _spread_lengths_matrix()
    a = bytes(hl.encode(w, seg_len=64, grp_rows=16))
    assert a == codec.encode(w, seg_len=64, grp_rows=16)
    assert hl.validate(a) == 0
    h = codec.parse_header(a)
    assert max(a[h["off_seg_bits"]:h["off_seg_bits"] + 64]) == 255


def test_byte_identical_adversarial():
    rng = np.random.default_rng(9)
    # exponents drawn geometrically: el code would exceed lmax 8 -> package-merge
    el = np.minimum(rng.geometric(0.45, 128 * 64) - 1, 15)
    eh = rng.choice([3, 7, 8], 128 * 64, p=[0.01, 0.9, 0.09])
    w = codec.join_fields(rng.integers(0, 2, el.size), eh, el, rng.integers(0, 128, el.size)).reshape(128, 64)
    for lmax in (5, 8, 15):
        a = bytes(hl.encode(w, seg_len=32, lmax=lmax))
        assert a == codec.encode(w, seg_len=32, lmax=lmax)
    # every bf16 pattern once
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(128, 512)
    assert bytes(hl.encode(w, seg_len=64)) == codec.encode(w, seg_len=64)
    # one-symbol fields: empty streams
    w = np.full((70, 16), 0x3F80, np.uint16)
    w[5, 3] = 0xBF81
    assert bytes(hl.encode(w, seg_len=16)) == codec.encode(w, seg_len=16)


def test_thread_count_does_not_change_output():
    w = random_bf16((300, 256), seed=4)
    a = hl.encode(w, seg_len=64, nthreads=1)
    for t in (2, 3, 7, 16):
        assert np.array_equal(a, hl.encode(w, seg_len=64, nthreads=t))


def test_default_grp_rows():
    for cols, S in ((4096, 128), (11008, 344), (48, 16), (80, 8), (1024, 64)):
        assert hl.default_grp_rows(cols, S) == codec.default_grp_rows(cols, S)
    with pytest.raises(hl.HLError):
        hl.encode(random_bf16((4, 48), seed=1), seg_len=16, grp_rows=16)


def test_default_seg_len():
    # every projection width of the workloads: S = 64 with cols/S a multiple of 4
    assert [hl.default_seg_len(k) for k in (1024, 4096, 8192, 11008, 14336, 28672)] == [64] * 6
    assert hl.default_seg_len(24) == 24 and hl.default_seg_len(100) == 0 and hl.default_seg_len(8) == 8
    assert hl.default_seg_len(96) == 24            # 96/24 = 4
    assert hl.default_seg_len(48) == 48            # no quad split: nearest to 128
    assert hl.default_seg_len(1000) == 0 or 1000 % hl.default_seg_len(1000) == 0


def test_encode_errors():
    w = random_bf16((4, 100), seed=1)
    with pytest.raises(hl.HLError):
        hl.encode(w, seg_len=64)
    with pytest.raises(hl.HLError):
        hl.encode(random_bf16((4, 64), seed=1), seg_len=12)
    with pytest.raises(hl.HLError):
        hl.build_codebook(random_bf16((4, 64), seed=1), lmax=3)
    # a codebook that lacks a symbol present in the data
    w = random_bf16((8, 64), seed=2)
    other = hl.build_codebook(np.full((8, 64), 0x3F80, np.uint16))
    with pytest.raises(hl.HLError):
        hl.encode(w, seg_len=64, codebook=other)


def test_validate_rejects_damage():
    w = random_bf16((130, 256), seed=5)
    good = hl.encode(w, seg_len=64)
    assert hl.validate(good) == 0
    h = codec.parse_header(bytes(good))

    def damaged(offset, value, width=1):
        b = good.copy()
        b[offset:offset + width] = np.frombuffer(int(value).to_bytes(width, "little"), np.uint8)
        return b

    assert hl.validate(good[:-1]) == hl.HL_ECORRUPT                       # truncated
    assert hl.validate(damaged(0, 0x12345678, 4)) == hl.HL_ECORRUPT      # magic
    assert hl.validate(damaged(6, 3)) == hl.HL_ECORRUPT                  # lmax out of range
    assert hl.validate(damaged(24, 48, 4)) == hl.HL_ECORRUPT             # seg_len
    assert hl.validate(damaged(112 + 3, 1)) == hl.HL_ECORRUPT            # el lengths: Kraft != 1
    assert hl.validate(damaged(h["off_seg_bits"], 0xFFFF, 2)) == hl.HL_ECORRUPT   # seg_bits
    assert hl.validate(damaged(h["off_grp_off"] + 4, 0, 4)) == hl.HL_ECORRUPT     # grp_off
    assert hl.validate(damaged(88, h["max_grp_units"] + 1, 4)) == hl.HL_ECORRUPT


# ---------------------------------------------------------------- whole-exponent format
@pytest.mark.parametrize("seed", range(4))
def test_codebook8_equals_oracle(seed):
    rng = np.random.default_rng(seed)
    w = random_bf16((32, 256), seed, std=float(rng.choice([0.002, 0.02, 0.5])))
    for lmax in (8, 12, 13):
        cb = hl.build_codebook8(w, lmax=lmax)
        ref = codec.build_codebook8(w, lmax)
        assert (cb.nsym, cb.single, cb.lengths) == (ref.nsym, ref.single, ref.lengths)


CASES8 = [((64, 1024), 64, 12, 0), ((130, 48), 16, 12, 0), ((3, 64), 8, 8, 0), ((65, 96), 32, 13, 0),
          ((130, 512), 64, 12, 8), ((37, 256), 32, 10, 32), ((1, 8), 8, 12, 0), ((21, 512), 8, 12, 1)]


@pytest.mark.parametrize("shape,S,lmax,GR", CASES8)
def test_whole_exponent_byte_identical_to_oracle(shape, S, lmax, GR):
    w = random_bf16(shape, seed=sum(shape) + S + 1)
    a = bytes(hl.encode(w, seg_len=S, lmax=lmax, grp_rows=GR, whole_exponent=True))
    assert a == codec.encode8(w, seg_len=S, lmax=lmax, grp_rows=GR or None)
    assert hl.validate(a) == 0


def test_whole_exponent_adversarial():
    # every bf16 pattern once: all 256 exponent values, uniform -> 8-bit codes
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(128, 512)
    for lmax in (8, 13):
        assert bytes(hl.encode(w, seg_len=64, lmax=lmax, whole_exponent=True)) == codec.encode8(w, 64, lmax)
    # exponent counts 2, 2, 4, ..., 2^14: the unlimited code reaches 14 bits
    rng = np.random.default_rng(3)
    e = np.concatenate([np.full(2, 100)] + [np.full(2 ** i, 100 + i) for i in range(1, 15)]).astype(np.uint32)
    e = rng.permutation(e)
    w = ((rng.integers(0, 2, e.size) << 15) | (e << 7) | rng.integers(0, 128, e.size)).astype(np.uint16)
    w = w.reshape(128, 256)
    assert max(codec.huffman_lengths(codec.histogram(e, 256))) > 13
    for lmax in (8, 11, 13):
        a = bytes(hl.encode(w, seg_len=32, lmax=lmax, whole_exponent=True))
        assert a == codec.encode8(w, 32, lmax)
    # one exponent value: no stream bits
    w = np.full((70, 16), 0x3F80, np.uint16)
    w[5, 3] = 0xBF81
    a = bytes(hl.encode(w, seg_len=16, whole_exponent=True))
    assert a == codec.encode8(w, 16) and codec.parse_header(a)["max_grp_units"] == 0


def test_whole_exponent_threads_and_errors():
    w = random_bf16((300, 256), seed=6)
    a = hl.encode(w, seg_len=64, nthreads=1, whole_exponent=True)
    for t in (3, 16):
        assert np.array_equal(a, hl.encode(w, seg_len=64, nthreads=t, whole_exponent=True))
    for bad in (7, 14):
        with pytest.raises(hl.HLError):
            hl.build_codebook8(w, lmax=bad)
    other = hl.build_codebook8(np.full((8, 64), 0x3F80, np.uint16))
    with pytest.raises(hl.HLError):
        hl.encode(w, seg_len=64, codebook=other, whole_exponent=True)


def test_whole_exponent_validate_rejects_damage():
    w = random_bf16((130, 256), seed=7)
    good = hl.encode(w, seg_len=64, whole_exponent=True)
    assert hl.validate(good) == 0
    h = codec.parse_header(bytes(good))
    lens = h["len8"]
    s_long = max(range(256), key=lambda s: lens[s])

    def damaged(offset, value, width=1):
        b = good.copy()
        b[offset:offset + width] = np.frombuffer(int(value).to_bytes(width, "little"), np.uint8)
        return b

    assert hl.validate(good[:383]) == hl.HL_ECORRUPT                      # no room for the lengths
    assert hl.validate(damaged(7, 2)) == hl.HL_ECORRUPT                   # unknown format
    assert hl.validate(damaged(6, 14)) == hl.HL_ECORRUPT                  # lmax above the window
    assert hl.validate(damaged(6, 7)) == hl.HL_ECORRUPT                   # lmax below 8
    assert hl.validate(damaged(128 + s_long, lens[s_long] - 1)) == hl.HL_ECORRUPT   # Kraft > 1
    assert hl.validate(damaged(92, h["nsym8"] + 1, 2)) == hl.HL_ECORRUPT  # symbol count
    assert hl.validate(damaged(100, 1)) == hl.HL_ECORRUPT                 # reserved bytes
    assert hl.validate(damaged(48, 128, 8)) == hl.HL_ECORRUPT             # off_seg_bits of the split format
    assert hl.validate(damaged(h["off_seg_bits"], 0xFFFF, 2)) == hl.HL_ECORRUPT
    # a split-format header over the whole-exponent body
    assert hl.validate(damaged(7, 0)) == hl.HL_ECORRUPT


# ---------------------------------------------------------------- float16 format
def _cb16_lists(cb):
    return [(f.nsym, f.single, list(f.len)) for f in (cb.e, cb.mh, cb.ml)]


@pytest.mark.parametrize("seed", range(3))
def test_codebook16_equals_oracle(seed):
    w = random_fp16((32, 256), seed, std=[0.002, 0.02, 0.5][seed])
    for lmax in (5, 9, 12):
        cb = hl.build_codebook16(w, lmax=lmax)
        ref = codec.build_codebooks16(w, lmax)
        assert _cb16_lists(cb) == [(c.nsym, c.single, c.lengths if c.nsym > 1 else [0] * 32) for c in ref]


CASES16 = [((64, 1024), 64, 12, 0), ((130, 48), 16, 12, 0), ((3, 64), 8, 5, 0), ((65, 96), 32, 9, 0),
           ((130, 512), 64, 12, 8), ((37, 256), 32, 7, 32), ((1, 8), 8, 12, 0), ((21, 512), 8, 12, 1),
           ((200, 512), 512, 12, 0)]


@pytest.mark.parametrize("shape,S,lmax,GR", CASES16)
def test_fp16_byte_identical_to_oracle(shape, S, lmax, GR):
    w = random_fp16(shape, seed=sum(shape) + S + 2)
    a = bytes(hl.encode(w, seg_len=S, lmax=lmax, grp_rows=GR, fp16=True))
    assert a == codec.encode16(w, seg_len=S, lmax=lmax, grp_rows=GR or None)
    assert hl.validate(a) == 0


def test_fp16_adversarial_and_threads():
    # every float16 pattern once: all fields uniform over 32 symbols
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(128, 512)
    for lmax in (5, 12):
        assert bytes(hl.encode(w, seg_len=64, lmax=lmax, fp16=True)) == codec.encode16(w, 64, lmax)
    # geometric exponents with long codes cut by the limit; constant mantissa-low
    rng = np.random.default_rng(4)
    e = np.minimum(rng.geometric(0.4, 64 * 256), 30).astype(np.uint32)
    w = ((rng.integers(0, 2, e.size) << 15) | (e << 10) | (rng.integers(0, 32, e.size) << 5))
    w = w.astype(np.uint16).reshape(64, 256)
    for lmax in (5, 8, 12):
        assert bytes(hl.encode(w, seg_len=32, lmax=lmax, fp16=True)) == codec.encode16(w, 32, lmax)
    w = random_fp16((300, 256), seed=6)
    a = hl.encode(w, seg_len=64, nthreads=1, fp16=True)
    for t in (3, 16):
        assert np.array_equal(a, hl.encode(w, seg_len=64, nthreads=t, fp16=True))
    for bad in (4, 13):
        with pytest.raises(hl.HLError):
            hl.build_codebook16(w, lmax=bad)
    other = hl.build_codebook16(np.full((8, 64), 0x3C00, np.uint16))
    with pytest.raises(hl.HLError):
        hl.encode(w, seg_len=64, codebook=other, fp16=True)


def test_fp16_validate_rejects_damage():
    w = random_fp16((130, 256), seed=8)
    good = hl.encode(w, seg_len=64, fp16=True)
    assert hl.validate(good) == 0
    h = codec.parse_header(bytes(good))
    mh_lens = h["cb16"][1][2]
    s_long = max(range(32), key=lambda s: mh_lens[s])

    def damaged(offset, value, width=1):
        b = good.copy()
        b[offset:offset + width] = np.frombuffer(int(value).to_bytes(width, "little"), np.uint8)
        return b

    assert hl.validate(good[:-1]) == hl.HL_ECORRUPT                       # sign plane cut short
    assert hl.validate(good[:255]) == hl.HL_ECORRUPT
    assert hl.validate(damaged(7, 3)) == hl.HL_ECORRUPT                   # unknown format
    assert hl.validate(damaged(6, 13)) == hl.HL_ECORRUPT                  # lmax above 12
    assert hl.validate(damaged(6, 4)) == hl.HL_ECORRUPT                   # lmax below 5
    assert hl.validate(damaged(128 + 34 + 2 + s_long, mh_lens[s_long] - 1)) == hl.HL_ECORRUPT  # Kraft
    assert hl.validate(damaged(128 + 34, h["cb16"][1][0] + 1)) == hl.HL_ECORRUPT  # symbol count
    assert hl.validate(damaged(128 + 110, 1)) == hl.HL_ECORRUPT           # section padding
    assert hl.validate(damaged(93, 1)) == hl.HL_ECORRUPT                  # header bytes 92..127
    assert hl.validate(damaged(h["off_seg_bits"], 0xFFFF, 2)) == hl.HL_ECORRUPT
    assert hl.validate(damaged(7, 0)) == hl.HL_ECORRUPT                   # split header over the body


def test_view_rejects_misaligned_blob_and_table(L):
    # containers packed back to back may leave a blob 8 bytes off a 16-byte
    # boundary; the kernels copy blob and table in 16-byte pieces
    import ctypes
    w = random_bf16((16, 256), seed=3)
    blob = hl.encode(w, seg_len=64)
    t = hl.TensorView()
    good, bad = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x10008)
    assert L.hl_tensor_view(bad, blob.ctypes.data, blob.size, good, ctypes.byref(t)) == hl.HL_EINVAL
    assert L.hl_tensor_view(good, blob.ctypes.data, blob.size, bad, ctypes.byref(t)) == hl.HL_EINVAL
    assert L.hl_tensor_view(good, blob.ctypes.data, blob.size, good, ctypes.byref(t)) == hl.HL_OK


def _fake_tensor(rows, cols):
    # a view with shape only and a blob on the meta device: every check below
    # must raise before any library call could reach a kernel
    import torch
    dt = hl.DeviceTensor.__new__(hl.DeviceTensor)
    dt.view = hl.TensorView()
    dt.view.rows, dt.view.cols = rows, cols
    dt.blob = torch.empty(16, dtype=torch.uint8, device="meta")
    return dt


def test_binding_rejects_bad_buffers_before_launch():
    import torch
    dt = _fake_tensor(64, 128)
    x = torch.zeros((2, 128), dtype=torch.bfloat16)
    y = torch.zeros((2, 64), dtype=torch.float32)
    bad = [
        dict(x=torch.zeros((2, 127), dtype=torch.bfloat16)),             # wrong columns
        dict(x=torch.zeros((17, 128), dtype=torch.bfloat16)),            # batch above 16
        dict(x=torch.zeros((2, 128), dtype=torch.int32)),                # wrong dtype
        dict(x=torch.zeros((128, 2), dtype=torch.bfloat16).t()),         # not contiguous
        dict(y=torch.zeros((2, 63), dtype=torch.float32)),               # output too small
        dict(y=torch.zeros((2, 64), dtype=torch.float64)),               # output dtype
        dict(),                                                          # host tensors
    ]
    for kw in bad:
        args = dict(x=x, y=y)
        args.update(kw)
        with pytest.raises(ValueError):
            dt.gemv(args["x"], args["y"], workspace=False)
        with pytest.raises(ValueError):
            hl.gemv_multi([dt], args["x"], [args["y"]], workspace=False)
        with pytest.raises(ValueError):
            dt.gemv_noalloc(args["x"], args["y"])
    with pytest.raises(ValueError):
        dt.decode(out=torch.zeros((64, 127), dtype=torch.int16))
    with pytest.raises(ValueError):
        dt.decode(out=torch.zeros((64, 128), dtype=torch.float32))
    with pytest.raises(ValueError):
        dt.decode(out=torch.zeros((64, 128), dtype=torch.int16))  # host
    with pytest.raises(ValueError):
        dt.gemm(torch.zeros((5, 128), dtype=torch.float32))
    with pytest.raises(ValueError):
        dt.gemm(torch.zeros((5, 128), dtype=torch.bfloat16), torch.zeros((5, 10), dtype=torch.float32))
    w = torch.zeros((64, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        hl.gemv_bf16(w, torch.zeros((1, 100), dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        hl.gemv_bf16(w.float(), x)
    with pytest.raises(ValueError):
        hl.gemv_bf16(w, x, y)  # host tensors


@pytest.mark.parametrize("pair_max", [0, 7, 8, 9, 10, 11, 13, 30])
def test_pair_limited_codebook_equals_oracle(pair_max):
    # the joint limit of a weight's two codes binds on these weights (eh over
    # four values, el codes of up to 11 bits): codebooks and containers equal
    # the oracle's for limits from the smallest feasible one up
    from gen import workload_matrices, gen_matrix
    w = gen_matrix(workload_matrices(2)[0], rows=slice(0, 256))
    cb = hl.build_codebook(w, lmax=12, pair_max=pair_max)
    ceh, cel = codec.build_codebooks(w, 12, pair_max)
    assert _codebook_lists(cb) == (ceh.nsym, ceh.single, ceh.lengths, cel.nsym, cel.single, cel.lengths)
    if pair_max:
        assert max(cb.eh.len) + max(cb.el.len) <= pair_max
    assert bytes(hl.encode(w, pair_max=pair_max)) == codec.encode(w, seg_len=64, pair_max=pair_max)


def test_pair_limit_too_small_is_refused():
    from gen import workload_matrices, gen_matrix
    w = gen_matrix(workload_matrices(2)[0], rows=slice(0, 64))
    with pytest.raises(hl.HLError):
        hl.build_codebook(w, lmax=12, pair_max=3)
