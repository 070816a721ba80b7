"""Pins of the oracle's float16 {1,5,5,5} format (header flags 2), each
against a fact outside the oracle:

* the field split against numpy's float16 decoding of all 65,536 patterns
  (Eq. 1 of Sec. 2.1 with float16's 5-bit exponent, bias 15, 10-bit mantissa);
* a hand-derived 1x8 container (tests/golden/tiny_fp16.txt);
* an independent window-match decoder (three 5-bit decoders, Sec. 3.2) over
  written containers;
* the exact size from code lengths, and size additivity over the fields;
* the per-field entropies of float16 copies of bf16-trained weights against
  the paper's entropy-of-splits table (Sec. 3.1): the low mantissa field of
  such weights carries about 2 bits, because bf16 leaves its low three bits 0.
"""
import os

import numpy as np
import pytest

from gen import bf16_bits_to_f16_bits, workload_matrices, gen_matrix, random_fp16
from oracle import codec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_split16_matches_float16_decoding():
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    s, e, mh, ml = codec.split_fields16(w)
    m = (mh << 5) | ml
    finite = e < 31
    sign = np.where(s == 1, -1.0, 1.0)
    val = np.where(e == 0, sign * m.astype(np.float64) * 2.0 ** -24,
                   sign * (1.0 + m / 1024.0) * np.exp2(e.astype(np.float64) - 15))
    ref = w.view(np.float16).astype(np.float64)
    assert np.array_equal(val[finite], ref[finite])
    assert np.array_equal(codec.join_fields16(s, e, mh, ml), w)


def _golden():
    w, meta = [], {}
    with open(os.path.join(GOLDEN, "tiny_fp16.txt")) as fh:
        for line in fh:
            if not line.strip() or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "weight":
                w.append(tuple(int(p) for p in parts[1:]))
            else:
                meta[parts[0]] = parts[1:]
    return w, meta


def test_tiny_fp16_hand_derived():
    fields, meta = _golden()
    s, e, mh, ml = (np.array(c) for c in zip(*fields))
    w = codec.join_fields16(s, e, mh, ml).reshape(1, 8)
    blob = codec.encode16(w, seg_len=8)
    h = codec.parse_header(blob)
    assert h["flags"] == 2 and h["off_seg_bits"] == 256
    # one segment in one group: its length is the group's base, its byte 0
    assert blob[h["off_seg_bits"]] == 0
    assert np.frombuffer(blob, np.uint32, 3, h["off_grp_off"]).tolist()[:2] == [0, int(meta["seg_bits"][0])]
    assert blob[h["off_stream"]:h["off_stream"] + 16].hex() == "".join(meta["stream"])
    assert blob[h["off_raw"]:h["off_raw"] + 1].hex() == meta["signs"][0]
    assert len(blob) == h["off_raw"] + 1
    for (nsym, single, lens), key in zip(h["cb16"], ("e_len", "mh_len", "ml_len")):
        want = {int(a): int(b) for a, b in (kv.split(":") for kv in meta[key])}
        assert {i: l for i, l in enumerate(lens) if l} == want and nsym == len(want)
    assert (codec.decode(blob) == w).all()


def _window_decode(bits, pos, code, lmax):
    if code.nsym == 1:
        return code.single, pos
    window = bits[pos:pos + lmax] + [0] * lmax
    for v in range(32):
        L = code.lengths[v]
        if L and window[:L] == [int(b) for b in format(code.codes[v], "0{}b".format(L))]:
            return v, pos + L
    raise AssertionError("no codeword matched")


@pytest.mark.parametrize("shape,S,GR,lmax", [((37, 256), 32, 16, 12), ((5, 96), 48, 32, 6),
                                             ((70, 128), 128, 64, 12), ((20, 128), 16, 8, 9)])
def test_roundtrip_and_window_match_decoder(shape, S, GR, lmax):
    w = random_fp16(shape, seed=S + GR)
    blob = codec.encode16(w, seg_len=S, grp_rows=GR, lmax=lmax)
    assert (codec.decode(blob) == w).all()
    sz = codec.container_size16(w, S, lmax=lmax, grp_rows=GR)
    assert len(blob) == sz["total_bytes"]
    h = codec.parse_header(blob)
    ce, cmh, cml = codec.header_codebooks16(h)
    for c in (ce, cmh, cml):
        assert c.nsym == 1 or (max(c.lengths) <= lmax and codec.kraft_sum(c.lengths) == 1)
    seg_bits, grp = codec.segment_lengths(blob, h)
    signs = np.frombuffer(blob, np.uint8, w.size // 8, h["off_raw"])
    _, e, mh, ml = codec.split_fields16(w)
    for g in (0, h["n_grp"] - 1):
        r0, G, c0, first, GC = codec.group_geometry(h["rows"], h["cols"], S, g, GR)
        bg = blob[h["off_stream"] + grp[g] * 16: h["off_stream"] + grp[g + 1] * 16]
        bits = np.unpackbits(np.frombuffer(bg, np.uint8), bitorder="little").tolist()
        pos = 0
        for mu in range(G * GC):
            r, c = r0 + mu % G, (c0 + mu // G) * S
            start = pos
            for t in range(S):
                vl, pos = _window_decode(bits, pos, cml, lmax)
                ve, pos = _window_decode(bits, pos, ce, lmax)
                vh, pos = _window_decode(bits, pos, cmh, lmax)
                assert (ve, vh, vl) == (e[r, c + t], mh[r, c + t], ml[r, c + t])
                sb = (signs[(first + mu) * (S // 8) + t // 8] >> (t % 8)) & 1
                assert sb == w[r, c + t] >> 15
            assert pos - start == seg_bits[first + mu]   # no group here spans more than 255 bits
        assert len(bits) - pos < 128
    # size additivity: code bits = sum over fields of frequency x length
    tot = 0
    for c, f in ((ce, e), (cmh, mh), (cml, ml)):
        hist = codec.histogram(f, 32)
        tot += sum(a * (b if c.nsym > 1 else 0) for a, b in zip(hist, c.lengths))
    assert sz["code_bits"] == tot


def test_all_patterns_roundtrip():
    w = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(128, 512)
    blob = codec.encode16(w, 64)
    assert (codec.decode(blob) == w).all()
    assert all(nsym == 32 for nsym, _, _ in codec.parse_header(blob)["cb16"])


def test_entropies_against_the_split_table():
    """float16 copies of bf16-trained weights: per-field entropies near the
    paper's {1,5,5,5} row (1.00, 2.60, 4.97, 2.04 bits)."""
    w = bf16_bits_to_f16_bits(gen_matrix(workload_matrices(2)[0]))
    s, e, mh, ml = codec.split_fields16(w)
    H = [codec.entropy_bits(codec.histogram(f, n)) for f, n in ((s, 2), (e, 32), (mh, 32), (ml, 32))]
    for got, paper in zip(H, (1.00, 2.60, 4.97, 2.04)):
        assert abs(got - paper) < 0.1, (got, paper)
    # the structure behind the low-mantissa figure: normal float16 copies of
    # bf16 values keep the low three mantissa bits zero
    assert np.all((ml[e > 0] & 7) == 0)
    size = codec.container_size16(w[:512], 64)
    assert sum(H) - 0.05 < 8 * size["total_bytes"] / w[:512].size < sum(H) + 1.0


def test_rejects():
    w = random_fp16((4, 64), seed=1)
    for bad in (4, 13):
        with pytest.raises(ValueError):
            codec.encode16(w, 16, lmax=bad)


def test_gemv_fp16_weights_exact():
    """fp16 x fp16 products are exact in float64; the fsum is the exact sum
    rounded once: against exact rational arithmetic on a small case."""
    from fractions import Fraction
    from gen import random_x
    from oracle import gemv
    w = random_fp16((3, 64), seed=9)
    x = random_x(2, 64, seed=3, dtype="f16")
    y, den = gemv.gemv_rows(w, x, weights="fp16")
    W = w.view(np.float16)
    for b in range(2):
        for r in range(3):
            exact = sum(Fraction(float(W[r, k])) * Fraction(float(x[b, k])) for k in range(64))
            assert y[b, r] == float(exact)
    ref = x.astype(np.float64) @ W.astype(np.float64).T
    assert np.all(np.abs(y - ref) <= 1e-12 * den)
