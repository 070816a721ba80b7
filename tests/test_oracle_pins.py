"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks one oracle function against a closed form, a brute-force
search, a published worked example, a hand derivation or a library routine
computing the same definition another way.
"""
import collections
import itertools
import math
import os
import random
from fractions import Fraction

import numpy as np
import pytest

from gen import random_bf16, random_x, f32_to_bf16_bits
from oracle import codec, gemv

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- field split
def test_split_closed_form_all_patterns():
    """Eq. 1 (Sec. 2.1) with the bf16 bias B = 127: every finite normal pattern's
    value rebuilt from the split fields equals the float the bits denote."""
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    s, eh, el, m = codec.split_fields(w)
    assert (codec.join_fields(s, eh, el, m) == w).all()          # lossless concatenation
    e = (eh << 4) | el
    normal = (e > 0) & (e < 255)
    val = np.where(s == 1, -1.0, 1.0) * np.exp2(e.astype(np.float64) - 127) * (1 + m / 128.0)
    with np.errstate(invalid="ignore"):
        ref = (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.array_equal(val[normal], ref[normal])
    # subnormals / zero: exponent field 0, value 2^-126 * 0.M
    sub = e == 0
    val_sub = np.where(s == 1, -1.0, 1.0) * 2.0 ** -126 * (m / 128.0)
    assert np.array_equal(val_sub[sub], ref[sub])
    assert s.max() == 1 and eh.max() == 15 and el.max() == 15 and m.max() == 127


def test_raw_byte_layout():
    s, m = np.array([0, 1, 1]), np.array([5, 0, 127])
    assert codec.raw_byte(s, m).tolist() == [5, 128, 255]


# ---------------------------------------------------------------- histograms
def test_histogram_vs_counter():
    rng = np.random.default_rng(3)
    a = rng.integers(0, 16, 5000)
    h = codec.histogram(a)
    c = collections.Counter(a.tolist())
    assert h == [c.get(v, 0) for v in range(16)]
    assert sum(h) == a.size


# ---------------------------------------------------------------- Huffman
def _cost(f, l):
    return sum(a * b for a, b in zip(f, l))


def _brute_optimal_full(freqs, lmax=None):
    """Minimum cost over ALL length vectors (1..n-1 or 1..lmax) with Kraft <= 1."""
    idx = [i for i, f in enumerate(freqs) if f > 0]
    n = len(idx)
    top = n - 1 if lmax is None else min(lmax, n - 1 if n > 1 else 1)
    best = None
    for ls in itertools.product(range(1, max(top, 1) + 1), repeat=n):
        if sum(Fraction(1, 2 ** l) for l in ls) <= 1:
            c = sum(freqs[i] * l for i, l in zip(idx, ls))
            best = c if best is None else min(best, c)
    return best


def _brute_optimal_sorted(freqs, lmax=None):
    """Minimum cost over non-decreasing length multisets assigned to symbols in
    decreasing-frequency order (optimal for a fixed multiset by rearrangement)."""
    f = sorted((x for x in freqs if x > 0), reverse=True)
    n = len(f)
    top = n - 1 if lmax is None else lmax
    best = None
    for ls in itertools.combinations_with_replacement(range(1, top + 1), n):
        if sum(Fraction(1, 2 ** l) for l in ls) <= 1:
            c = sum(a * b for a, b in zip(f, ls))
            best = c if best is None else min(best, c)
    return best


@pytest.mark.parametrize("seed", range(40))
def test_huffman_optimal_bruteforce(seed):
    rnd = random.Random(seed)
    n = rnd.randint(2, 8)
    freqs = [0] * 16
    for s in rnd.sample(range(16), n):
        freqs[s] = rnd.choice([1, 1, 2, 3, 5, 8, 13, 100, rnd.randint(1, 1000)])
    l = codec.huffman_lengths(freqs)
    assert codec.kraft_sum(l) == 1
    assert all((l[i] > 0) == (freqs[i] > 0) for i in range(16))
    ref = _brute_optimal_full(freqs) if n <= 5 else _brute_optimal_sorted(freqs)
    assert _cost(freqs, l) == ref


def test_huffman_special_cases():
    # uniform over 2^k symbols -> all k
    for k in (1, 2, 3, 4):
        f = [7] * (2 ** k) + [0] * (16 - 2 ** k)
        assert codec.huffman_lengths(f)[: 2 ** k] == [k] * (2 ** k)
    # dyadic probabilities -> l = -log2 p and average length = entropy
    f = [8, 4, 2, 1, 1] + [0] * 11
    l = codec.huffman_lengths(f)
    assert l[:5] == [1, 2, 3, 4, 4]
    assert _cost(f, l) / sum(f) == codec.entropy_bits(f)
    # two symbols -> (1, 1); one symbol -> length 0 (no bits)
    assert codec.huffman_lengths([0, 5, 0, 9] + [0] * 12)[:4] == [0, 1, 0, 1]
    assert codec.huffman_lengths([0, 0, 42] + [0] * 13) == [0] * 16
    # frequencies 2^i -> lengths 1, 2, ..., n-1, n-1
    n = 10
    f = [2 ** i for i in range(n)] + [0] * (16 - n)
    l = codec.huffman_lengths(f)
    assert sorted(l[:n]) == sorted([n - 1] + list(range(1, n)))
    assert l[n - 1] == 1 and l[0] == n - 1 and l[1] == n - 1


@pytest.mark.parametrize("seed", range(25))
def test_average_length_shannon_bounds(seed):
    rng = np.random.default_rng(seed)
    f = (rng.pareto(1.0, 16) * 100).astype(int).tolist()
    f[seed % 16] += 1
    for lens in (codec.huffman_lengths(f),):
        if sum(1 for x in f if x) == 1:
            continue
        avg = _cost(f, lens) / sum(f)
        H = codec.entropy_bits(f)
        assert H - 1e-12 <= avg < H + 1


# ---------------------------------------------------------------- length limit
@pytest.mark.parametrize("seed", range(30))
def test_package_merge_optimal_bruteforce(seed):
    rnd = random.Random(100 + seed)
    n = rnd.randint(3, 8)
    L = rnd.choice([3, 4])
    if n > 2 ** L:
        n = 2 ** L
    freqs = [0] * 16
    for s in rnd.sample(range(16), n):
        freqs[s] = rnd.choice([1, 2, 4, 8, 16, 32, 64, 128, rnd.randint(1, 500)])
    l = codec.package_merge_lengths(freqs, L)
    assert max(l) <= L
    assert codec.kraft_sum(l) == 1
    ref = _brute_optimal_full(freqs, L) if n <= 5 else _brute_optimal_sorted(freqs, L)
    assert _cost(freqs, l) == ref


def test_package_merge_matches_huffman_cost_when_unconstrained():
    rnd = random.Random(7)
    for _ in range(30):
        f = [rnd.randint(0, 1000) for _ in range(16)]
        f[0] += 1
        f[1] += 1
        h = codec.huffman_lengths(f)
        pm = codec.package_merge_lengths(f, 15)
        assert _cost(f, pm) == _cost(f, h)
        lim = codec.limited_lengths(f, max(h))
        assert lim == h          # identity when the limit does not bind


def test_limit_binds_on_geometric_16():
    f = [2 ** i for i in range(16)]
    h = codec.huffman_lengths(f)
    assert max(h) == 15
    l = codec.limited_lengths(f, 12)
    assert max(l) == 12 and codec.kraft_sum(l) == 1
    assert _cost(f, l) >= _cost(f, h)


# ---------------------------------------------------------------- canonical codes
def _golden_rfc():
    rows = []
    with open(os.path.join(GOLDEN, "rfc1951_canonical.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                s, l, c = line.split()
                rows.append((int(s), int(l), c))
    return rows


def test_canonical_rfc1951_example():
    rows = _golden_rfc()
    lengths = [l for _, l, _ in rows]
    codes = codec.canonical_codes(lengths)
    for (s, l, c), code in zip(rows, codes):
        assert format(code, "0{}b".format(l)) == c


@pytest.mark.parametrize("seed", range(10))
def test_canonical_prefix_free_and_ordered(seed):
    rnd = random.Random(seed)
    f = [rnd.choice([0, rnd.randint(1, 10 ** rnd.randint(0, 5))]) for _ in range(16)]
    f[rnd.randrange(16)] += 1
    f[(seed + 3) % 16] += 2
    l = codec.limited_lengths(f, 12)
    c = codec.canonical_codes(l)
    words = [format(c[s], "0{}b".format(l[s])) for s in range(16) if l[s]]
    for a, b in itertools.permutations(words, 2):
        assert not b.startswith(a)
    for L in set(x for x in l if x):
        syms = [s for s in range(16) if l[s] == L]
        vals = [c[s] for s in syms]
        assert vals == list(range(vals[0], vals[0] + len(vals)))


# ---------------------------------------------------------------- container
def _golden_tiny():
    w, meta = [], {}
    with open(os.path.join(GOLDEN, "tiny_container.txt")) as fh:
        for line in fh:
            if not line.strip() or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "weight":
                w.append(tuple(int(p) for p in parts[1:]))
            else:
                meta[parts[0]] = parts[1:]
    return w, meta


def test_tiny_container_hand_derived():
    fields, meta = _golden_tiny()
    s, eh, el, m = (np.array(c) for c in zip(*fields))
    w = codec.join_fields(s, eh, el, m).reshape(1, 8)
    blob = codec.encode(w, seg_len=8)
    h = codec.parse_header(blob)
    # one segment in one group: its length is the group's base, its byte 0
    assert blob[h["off_seg_bits"]] == 0
    assert np.frombuffer(blob, np.uint32, 3, h["off_grp_off"]).tolist() == [0, int(meta["seg_bits"][0]), 1]
    stream = blob[h["off_stream"]:h["off_stream"] + 16]
    assert stream.hex() == "".join(meta["stream"])
    for key, field in (("eh_len", "eh_len"), ("el_len", "el_len")):
        want = {int(a): int(b) for a, b in (kv.split(":") for kv in meta[key])}
        got = {i: l for i, l in enumerate(h[field]) if l}
        assert got == want
    raw = np.frombuffer(blob, np.uint8, 8, h["off_raw"])
    assert raw.tolist() == ((s << 7) | m).tolist()
    assert (codec.decode(blob) == w).all()


def _cam_window_decode(bits, pos, fc, lmax):
    """Decoder of Sec. 3.2 written as a window match: take lmax bits from the
    start pointer and compare them against every codeword; advance by L."""
    if fc.nsym == 1:
        return fc.single, pos
    window = bits[pos:pos + lmax] + [0] * lmax
    for s in range(16):
        L = fc.lengths[s]
        if L and window[:L] == [int(b) for b in format(fc.codes[s], "0{}b".format(L))]:
            return s, pos + L
    raise AssertionError("no codeword matched")


@pytest.mark.parametrize("shape,S,GR", [((3, 64), 16, 64), ((70, 128), 128, 64), ((5, 96), 48, 32),
                                        ((130, 40), 8, 64), ((37, 256), 32, 16), ((20, 128), 16, 8)])
def test_roundtrip_and_window_match_decoder(shape, S, GR):
    w = random_bf16(shape, seed=S + GR)
    blob = codec.encode(w, seg_len=S, grp_rows=GR)
    assert (codec.decode(blob) == w).all()
    h = codec.parse_header(blob)
    assert h["grp_rows"] == GR
    ceh, cel = codec.header_codebooks(h)
    stored, grp = codec.segment_lengths(blob, h)
    _, eh, el, _ = codec.split_fields(w)
    # independent window-match decode of the first and the last group
    for g in (0, h["n_grp"] - 1):
        r0, G, c0, first, GC = codec.group_geometry(h["rows"], h["cols"], S, g, GR)
        bg = blob[h["off_stream"] + grp[g] * 16: h["off_stream"] + grp[g + 1] * 16]
        bits = np.unpackbits(np.frombuffer(bg, np.uint8), bitorder="little").tolist()
        pos = 0
        for mu in range(G * GC):
            r, c = r0 + mu % G, (c0 + mu // G) * S
            start = pos
            for t in range(S):
                b, pos = _cam_window_decode(bits, pos, cel, h["lmax"])
                a, pos = _cam_window_decode(bits, pos, ceh, h["lmax"])
                assert (a, b) == (eh[r, c + t], el[r, c + t])
            assert pos - start == stored[first + mu]   # no group here spans more than 255 bits
        assert (len(bits) - pos) < 128            # group padding below one 128-bit unit


def _spread_lengths_matrix():
    """16 x 256 bf16 (one 16 x 4 group at S = 64) whose segment (row 0,
    columns 0..63) holds rare exponents with long codes while every other
    weight is the common 1.0-like pattern: its segments' code bits span far
    more than 255 bits."""
    rng = np.random.default_rng(5)
    s = rng.integers(0, 2, (16, 256))
    m = rng.integers(0, 128, (16, 256))
    eh = np.full((16, 256), 7)
    el = np.full((16, 256), 15)
    el[:, ::2] = 14                                      # two common el values: 1-bit codes
    eh[0, :64] = rng.integers(0, 7, 64)                  # rare eh and el values in one segment
    el[0, :64] = rng.integers(0, 14, 64)
    return codec.join_fields(s, eh, el, m)


def test_segment_lengths_padded_to_the_group_base():
    """Stored segment lengths (the container's one-byte lengths): base = the
    least code-bit count of the group, or the greatest minus 255; shorter
    segments padded with zero bits to base. Checked against per-segment code
    bits computed from the code lengths alone, and by a window-match decode
    that steps over the padding."""
    w = _spread_lengths_matrix()
    blob = codec.encode(w, seg_len=64, grp_rows=16)
    h = codec.parse_header(blob)
    assert h["n_grp"] == 1
    ceh, cel = codec.header_codebooks(h)
    _, eh, el, _ = codec.split_fields(w)
    bits = np.array(ceh.lengths)[eh] + np.array(cel.lengths)[el]
    code = [int(bits[mu % 16, (mu // 16) * 64:(mu // 16 + 1) * 64].sum()) for mu in range(64)]
    assert max(code) - min(code) > 255
    base = max(code) - 255
    seg8 = np.frombuffer(blob, np.uint8, 64, h["off_seg_bits"])
    meta = np.frombuffer(blob, np.uint32, 3, h["off_grp_off"])
    assert meta[1] == base
    assert seg8.tolist() == [max(c, base) - base for c in code]
    assert seg8.max() == 255 and (seg8 == 0).sum() == sum(c <= base for c in code)
    stored, grp = codec.segment_lengths(blob, h)
    assert int(grp[1] - grp[0]) == (int(stored.sum()) + 127) // 128
    bg = blob[h["off_stream"]: h["off_stream"] + int(grp[1]) * 16]
    bits_l = np.unpackbits(np.frombuffer(bg, np.uint8), bitorder="little").tolist()
    pos = 0
    for mu in range(64):
        r, c = mu % 16, (mu // 16) * 64
        start = pos
        for t in range(64):
            b, pos = _cam_window_decode(bits_l, pos, cel, h["lmax"])
            a, pos = _cam_window_decode(bits_l, pos, ceh, h["lmax"])
            assert (a, b) == (eh[r, c + t], el[r, c + t])
        assert pos - start == code[mu]
        assert not any(bits_l[pos:start + int(stored[mu])])   # the padding is zero bits
        pos = start + int(stored[mu])
    assert (codec.decode(blob) == w).all()
    assert codec.container_size(w, 64, grp_rows=16)["total_bytes"] == len(blob)


@pytest.mark.parametrize("GR", [64, 32, 16, 8, 1])
def test_group_geometry_tiles_the_matrix(GR):
    rows, cols, S = 130, 512, 8
    seen = np.zeros((rows, cols), int)
    firsts = []
    for g in range(codec.layout(rows, cols, S, GR)["n_grp"]):
        r0, G, c0, first, GC = codec.group_geometry(rows, cols, S, g, GR)
        for mu in range(G * GC):
            r, c = r0 + mu % G, (c0 + mu // G) * S
            seen[r, c:c + S] += 1
        firsts.append((first, G * GC))
    assert (seen == 1).all()
    # group g's segments follow those of group g-1 with no gap
    for (f0, n0), (f1, _) in zip(firsts, firsts[1:]):
        assert f1 == f0 + n0


def test_default_group_rows():
    assert codec.default_grp_rows(4096, 128) == 16
    assert codec.default_grp_rows(11008, 344) == 16      # 32 segments per row
    assert codec.default_grp_rows(48, 16) == 64          # 3 segments per row
    assert codec.default_grp_rows(80, 8) == 32           # 10 segments per row
    with pytest.raises(ValueError):
        codec.encode(random_bf16((4, 48), seed=1), seg_len=16, grp_rows=16)


def test_size_accounting_and_ratio_identity():
    w = random_bf16((128, 512), seed=11)
    ceh, cel = codec.build_codebooks(w)
    blob = codec.encode(w, seg_len=128)
    h = codec.parse_header(blob)
    seg_bits, grp = codec.segment_lengths(blob, h)
    # per-field coded sizes add up to the stream (entropy-of-splits caption, Sec. 3.1)
    assert codec.payload_bits(w, ceh, cel) == seg_bits.sum() + 8 * w.size   # no padded segment here
    for g in range(h["n_grp"]):
        _, G, _, first, GC = codec.group_geometry(h["rows"], h["cols"], h["seg_len"], g, h["grp_rows"])
        bits = seg_bits[first: first + G * GC].sum()
        assert grp[g + 1] - grp[g] == (bits + 127) // 128
    # metadata: one byte per segment, two words per group and one more
    assert h["off_grp_off"] - h["off_seg_bits"] >= h["n_seg"]
    assert h["off_stream"] - h["off_grp_off"] >= 4 * (2 * h["n_grp"] + 1)
    assert h["total_bytes"] == len(blob) == h["off_raw"] + w.size
    ratio = 2 * w.size / len(blob)
    bits_per_param = 8 * len(blob) / w.size
    assert abs(bits_per_param - 16 / ratio) < 1e-12    # comp-ratio table caption identity


def test_single_symbol_fields_cost_no_bits():
    w = np.full((4, 64), 0x3F80, dtype=np.uint16)          # 1.0 everywhere
    w[0, 0] = 0xBF80                                        # -1.0: sign is raw
    blob = codec.encode(w, seg_len=32)
    h = codec.parse_header(blob)
    assert h["eh_nsym"] == 1 and h["el_nsym"] == 1
    assert h["max_grp_units"] == 0
    assert (codec.decode(blob) == w).all()


def test_all_patterns_roundtrip():
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(64, 1024)
    blob = codec.encode(w, seg_len=256, lmax=12)
    assert (codec.decode(blob) == w).all()


def test_lmax_binding_container_roundtrip():
    # skewed exponents so that the el code would exceed lmax without the limit
    rng = np.random.default_rng(5)
    el = np.minimum(rng.geometric(0.5, 4096) - 1, 15)
    eh = np.full(4096, 7)
    w = codec.join_fields(np.zeros(4096, int), eh, el, rng.integers(0, 128, 4096)).reshape(8, 512)
    f = codec.histogram(el)
    assert max(codec.huffman_lengths(f)) > 6
    blob = codec.encode(w, seg_len=64, lmax=6)
    h = codec.parse_header(blob)
    assert max(h["el_len"]) == 6
    assert (codec.decode(blob) == w).all()


@pytest.mark.parametrize("GR", [64, 16, 8])
def test_raw_plane_interleave_is_a_permutation(GR):
    for rows, cols, S in ((130, 64, 16), (64, 64, 8), (1, 96, 24), (200, 320, 40), (65, 256, 32)):
        if (cols // S) % (64 // GR):
            continue
        rr, cc = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
        p = codec.raw_pos(rr.ravel(), cc.ravel(), rows, cols, S, GR)
        assert np.array_equal(np.sort(p), np.arange(rows * cols))


def test_raw_plane_interleave_examples():
    # a full 64-row group (GR = 64): 8-byte runs of one row, rows interleaved
    p = codec.raw_pos(np.array([0, 0, 1, 0]), np.array([0, 7, 0, 8]), 64, 16, 16, 64)
    assert p.tolist() == [0, 7, 8, 512]
    # GR = 16: segment mu = j*16 + i; row 1 of the second segment is mu = 17
    p = codec.raw_pos(np.array([1, 0]), np.array([16, 8]), 16, 64, 16, 16)
    assert p.tolist() == [17 * 8, 64 * 8]


def test_encode_rejects_bad_shapes():
    w = random_bf16((4, 100), seed=1)
    with pytest.raises(ValueError):
        codec.encode(w, seg_len=64)        # 64 does not divide 100
    with pytest.raises(ValueError):
        codec.encode(w, seg_len=20)        # not a multiple of 8
    with pytest.raises(ValueError):
        codec.encode(random_bf16((4, 64), seed=1), seg_len=64, lmax=3)


# ---------------------------------------------------------------- fp64 GEMV
def test_gemv_exact_on_tiny_inputs():
    w = random_bf16((5, 24), seed=2)
    x = random_x(2, 24, seed=3)
    y, den = gemv.gemv_rows(w, x)
    W = gemv.bf16_to_f64(w)
    for b in range(2):
        for r in range(5):
            exact = sum(Fraction(float(W[r, k])) * Fraction(float(np.float32(x[b, k])))
                        for k in range(24))
            assert y[b, r] == float(exact)           # correctly rounded exact sum
            assert den[b, r] == float(sum(abs(Fraction(float(W[r, k])) *
                                              Fraction(float(np.float32(x[b, k])))) for k in range(24)))


def test_gemv_vs_numpy_float64():
    w = random_bf16((64, 1024), seed=4)
    xb = random_x(3, 1024, seed=5, dtype="bf16")
    y, den = gemv.gemv_rows(w, xb)
    ref = gemv.x_to_f64(xb) @ gemv.bf16_to_f64(w).T
    assert np.all(np.abs(y - ref) <= 1e-12 * den)


def test_bf16_conversion_matches_torch():
    import torch
    rng = np.random.default_rng(0)
    a = (rng.standard_normal(100000) * rng.choice([1e-3, 1, 1e3], 100000)).astype(np.float32)
    ours = f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(gemv.bf16_to_f64(ours),
                          torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).double().numpy())


@pytest.mark.parametrize("shape,S", [((130, 48), 16), ((64, 1024), 128), ((65, 96), 32), ((3, 64), 8),
                                     ((70, 512), 64)])
def test_container_size_matches_written_container(shape, S):
    w = random_bf16(shape, seed=shape[0])
    blob = codec.encode(w, seg_len=S)
    h = codec.parse_header(blob)
    cs = codec.container_size(w, S)
    assert cs["grp_rows"] == h["grp_rows"]
    assert cs["total_bytes"] == len(blob)
    assert cs["max_grp_units"] == h["max_grp_units"] and cs["off_raw"] == h["off_raw"]
    ceh, cel = codec.build_codebooks(w)
    assert cs["code_bits"] + 8 * w.size == codec.payload_bits(w, ceh, cel)


# ---- joint limit of a weight's two exponent codes (split format)

def _field_vectors(freqs, lmax):
    """Every complete prefix-code length vector of a field with lengths <= lmax
    (non-decreasing lengths given to symbols of non-increasing frequency:
    optimal for each multiset), as (cost, longest); a one-symbol field: (0, 0)."""
    f = sorted((x for x in freqs if x > 0), reverse=True)
    n = len(f)
    if n == 1:
        return [(0, 0)]
    out = []
    for ls in itertools.combinations_with_replacement(range(1, lmax + 1), n):
        if sum(Fraction(1, 2 ** l) for l in ls) == 1:
            out.append((sum(a * b for a, b in zip(f, ls)), max(ls)))
    return out


@pytest.mark.parametrize("seed", range(40))
def test_pair_limit_optimal_bruteforce(seed):
    # the cheapest pair of codes under both limits, by enumerating every pair
    # of complete length vectors (nothing of the oracle's rule is used)
    rnd = random.Random(500 + seed)
    feh, fel = [0] * 16, [0] * 16
    for s in rnd.sample(range(16), rnd.randint(1, 4)):
        feh[s] = rnd.choice([1, 3, 10, 1000, rnd.randint(1, 5000)])
    for s in rnd.sample(range(16), rnd.randint(2, 6)):
        fel[s] = rnd.choice([1, 2, 7, 60, 900, rnd.randint(1, 5000)])
    lmax = rnd.choice([4, 5, 6])
    J = rnd.randint(codec.min_limit(feh) + codec.min_limit(fel), 10)
    leh, lel = codec.pair_limited_lengths(feh, fel, lmax, J)
    assert max(leh) + max(lel) <= J and max(leh) <= lmax and max(lel) <= lmax
    for f, l in ((feh, leh), (fel, lel)):
        assert all((l[i] > 0) == (f[i] > 0) for i in range(16)) or sum(1 for x in f if x) == 1
        if sum(1 for x in f if x) > 1:
            assert codec.kraft_sum(l) == 1
    best = min(ca + cb for ca, ma in _field_vectors(feh, lmax) for cb, mb in _field_vectors(fel, lmax)
               if ma + mb <= J)
    assert _cost(feh, leh) + _cost(fel, lel) == best


def test_pair_limit_special_cases():
    rnd = random.Random(7)
    feh = [0] * 16
    feh[7], feh[6], feh[8] = 99000, 700, 300
    fel = [0] * 16
    for s in range(16):
        fel[s] = max(1, int(40000 * 0.5 ** abs(s - 9)))
    # no joint limit, or one that does not bind: the independent limited codes
    for J in (0, 30):
        assert codec.pair_limited_lengths(feh, fel, 12, J) == (codec.limited_lengths(feh, 12),
                                                                codec.limited_lengths(fel, 12))
    # a binding limit costs at least as much, never less, and meets the limit
    free = _cost(feh, codec.limited_lengths(feh, 12)) + _cost(fel, codec.limited_lengths(fel, 12))
    prev = free
    for J in range(20, 6, -1):
        leh, lel = codec.pair_limited_lengths(feh, fel, 12, J)
        c = _cost(feh, leh) + _cost(fel, lel)
        assert max(leh) + max(lel) <= J and c >= prev
        prev = c
    # one-symbol fields take no bits and leave the whole limit to the other
    one = [0] * 16
    one[5] = 10
    leh, lel = codec.pair_limited_lengths(one, fel, 12, 11)
    assert leh == [0] * 16 and lel == codec.limited_lengths(fel, 11)
    # a limit below what the alphabets need is refused
    with pytest.raises(ValueError):
        codec.pair_limited_lengths(feh, fel, 12, codec.min_limit(feh) + codec.min_limit(fel) - 1)
    del rnd
