"""Pins of the oracle's whole-exponent format (the 8 exponent bits as one
symbol of a 256-symbol per-matrix code, header flags 1), each against a fact
outside the oracle:

* a hand-derived 1x8 container (tests/golden/tiny_whole_exponent.txt);
* optimality of the length-limited code against an independent dynamic
  program over code trees built level by level (alphabets of up to 40
  symbols, limits that bind);
* Kraft sum exactly 1, the limit, and the Shannon bounds H <= average < H + 1
  when the limit does not bind;
* uniform alphabets of 2^k symbols (all lengths k), one symbol (no bits);
* an independent window-match decoder over the written container;
* the chain rule H(e) <= H(eh) + H(el): the whole-exponent code is never more
  than one bit per weight above the split code's entropy sum, and on the
  workloads' distribution it is shorter than the split code.
"""
import functools
import math
import os
import random

import numpy as np
import pytest

from gen import workload_matrices, gen_matrix, random_bf16
from oracle import codec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cost(f, l):
    return sum(a * b for a, b in zip(f, l))


def _dp_optimal(freqs, lmax):
    """Minimum of sum f*l over complete prefix codes with lengths <= lmax.

    Symbols sorted by decreasing frequency take non-decreasing lengths. The
    tree is built level by level: with i symbols placed and a open nodes at
    depth d, k of them become leaves and 2(a-k) nodes open at depth d+1. The
    cost counts, at each depth, the frequencies of all symbols not yet placed
    above it."""
    f = sorted((x for x in freqs if x > 0), reverse=True)
    n = len(f)
    suf = [0] * (n + 1)
    for i in range(n - 1, -1, -1):
        suf[i] = suf[i + 1] + f[i]

    @functools.lru_cache(maxsize=None)
    def best(d, i, a):
        if d > lmax:
            return math.inf
        here = suf[i]
        out = math.inf
        for k in range(0, min(a, n - i) + 1):
            rest, nodes = n - i - k, 2 * (a - k)
            if rest == 0 and nodes == 0:
                out = min(out, here)
            elif rest > 0 and 0 < nodes <= rest:
                out = min(out, here + best(d + 1, i + k, nodes))
        return out

    return best(1, 0, 2)


@pytest.mark.parametrize("seed", range(12))
def test_limited_code_optimal_vs_level_dp(seed):
    rnd = random.Random(500 + seed)
    n = rnd.randint(9, 40)
    freqs = [0] * 256
    for s in rnd.sample(range(256), n):
        freqs[s] = rnd.choice([1, 2, 3, 7, 50, 2 ** rnd.randint(0, 20), rnd.randint(1, 10 ** 6)])
    h = codec.huffman_lengths(freqs)
    L = rnd.randint(math.ceil(math.log2(n)), max(h) - 1)     # a limit that binds
    l = codec.limited_lengths(freqs, L)
    assert max(l) <= L and codec.kraft_sum(l) == 1
    assert all((l[s] > 0) == (freqs[s] > 0) for s in range(256))
    assert _cost(freqs, l) == _dp_optimal(freqs, L)
    assert _cost(freqs, h) == _dp_optimal(freqs, 64)         # unlimited Huffman is optimal too


def test_uniform_and_single_alphabets():
    for k in (1, 3, 8):
        f = [0] * 256
        for s in range(0, 256, 256 >> k):
            f[s] = 5
        l = codec.huffman_lengths(f)
        assert sorted(set(l) - {0}) == [k]
    w = np.full((4, 64), 0x3F80, np.uint16)                   # 1.0 everywhere
    c = codec.build_codebook8(w)
    assert c.nsym == 1 and c.single == 0x7F
    blob = codec.encode8(w, 16)
    h = codec.parse_header(blob)
    assert h["max_grp_units"] == 0 and (codec.decode(blob) == w).all()


@pytest.mark.parametrize("seed", range(8))
def test_kraft_limit_and_shannon_bounds_256(seed):
    rng = np.random.default_rng(seed)
    f = (rng.pareto(0.7, 256) * 50).astype(np.int64).tolist()
    f[seed] += 1
    f[200] += 1
    h = codec.huffman_lengths(f)
    H = codec.entropy_bits(f)
    assert codec.kraft_sum(h) == 1
    assert H - 1e-12 <= _cost(f, h) / sum(f) < H + 1
    for L in (8, 10, 12, 13):
        l = codec.limited_lengths(f, L)
        assert max(l) <= L and codec.kraft_sum(l) == 1
        assert _cost(f, l) >= _cost(f, h)
        if max(h) <= L:
            assert l == h


def _golden():
    w, meta = [], {}
    with open(os.path.join(GOLDEN, "tiny_whole_exponent.txt")) as fh:
        for line in fh:
            if not line.strip() or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "weight":
                w.append(tuple(int(p) for p in parts[1:]))
            else:
                meta[parts[0]] = parts[1:]
    return w, meta


def test_tiny_whole_exponent_hand_derived():
    fields, meta = _golden()
    s, e, m = (np.array(c, dtype=np.uint32) for c in zip(*fields))
    w = ((s << 15) | (e << 7) | m).astype(np.uint16).reshape(1, 8)
    blob = codec.encode8(w, seg_len=8)
    h = codec.parse_header(blob)
    assert h["flags"] == 1 and h["off_seg_bits"] == 384 and h["nsym8"] == 4
    # one segment in one group: its length is the group's base, its byte 0
    assert blob[h["off_seg_bits"]] == 0
    assert np.frombuffer(blob, np.uint32, 3, h["off_grp_off"]).tolist()[:2] == [0, int(meta["seg_bits"][0])]
    assert blob[h["off_stream"]:h["off_stream"] + 16].hex() == "".join(meta["stream"])
    want = {int(a): int(b) for a, b in (kv.split(":") for kv in meta["len"])}
    assert {i: l for i, l in enumerate(h["len8"]) if l} == want
    assert np.frombuffer(blob, np.uint8, 8, h["off_raw"]).tolist() == ((s << 7) | m).tolist()
    assert (codec.decode(blob) == w).all()


def _window_decode(bits, pos, lengths, codes, lmax):
    """Match the next lmax bits against every codeword (Sec. 3.2's window match)."""
    window = bits[pos:pos + lmax] + [0] * lmax
    for s in range(256):
        L = lengths[s]
        if L and window[:L] == [int(b) for b in format(codes[s], "0{}b".format(L))]:
            return s, pos + L
    raise AssertionError("no codeword matched")


@pytest.mark.parametrize("shape,S,GR,lmax", [((37, 256), 32, 16, 12), ((5, 96), 48, 32, 8),
                                             ((70, 128), 128, 64, 13), ((20, 128), 16, 8, 10)])
def test_roundtrip_and_window_match_decoder(shape, S, GR, lmax):
    rng = np.random.default_rng(S)
    w = random_bf16(shape, seed=S + GR)
    w[rng.random(shape) < 0.05] ^= np.uint16(0x2000)          # widen the exponent alphabet
    blob = codec.encode8(w, seg_len=S, grp_rows=GR, lmax=lmax)
    assert (codec.decode(blob) == w).all()
    assert len(blob) == codec.container_size8(w, S, lmax=lmax, grp_rows=GR)["total_bytes"]
    h = codec.parse_header(blob)
    lengths = h["len8"]
    assert max(lengths) <= lmax and codec.kraft_sum(lengths) == 1
    codes = codec.canonical_codes(lengths)
    seg_bits, grp = codec.segment_lengths(blob, h)
    e = codec.exponent_byte(w)
    for g in (0, h["n_grp"] - 1):
        r0, G, c0, first, GC = codec.group_geometry(h["rows"], h["cols"], S, g, GR)
        bg = blob[h["off_stream"] + grp[g] * 16: h["off_stream"] + grp[g + 1] * 16]
        bits = np.unpackbits(np.frombuffer(bg, np.uint8), bitorder="little").tolist()
        pos = 0
        for mu in range(G * GC):
            r, c = r0 + mu % G, (c0 + mu // G) * S
            start = pos
            for t in range(S):
                v, pos = _window_decode(bits, pos, lengths, codes, lmax)
                assert v == e[r, c + t]
            assert pos - start == seg_bits[first + mu]   # no group here spans more than 255 bits
        assert len(bits) - pos < 128


def test_chain_rule_and_workload_ratio():
    spec = workload_matrices(1)[0]
    w = gen_matrix(spec)
    _, eh, el, _ = codec.split_fields(w)
    e = codec.exponent_byte(w)
    He = codec.entropy_bits(codec.histogram(e, 256))
    Hs = codec.entropy_bits(codec.histogram(eh)) + codec.entropy_bits(codec.histogram(el))
    assert He <= Hs + 1e-12
    whole = codec.container_size8(w, 64)
    split = codec.container_size(w, 64)
    n = w.size
    assert He <= whole["code_bits"] / n < He + 1
    assert whole["code_bits"] < split["code_bits"]
    h = codec.huffman_lengths(codec.histogram(e, 256))
    assert max(h) > 12                                         # the limit binds on this distribution
    assert max(codec.build_codebook8(w).lengths) == 12


def test_rejects():
    w = random_bf16((4, 64), seed=1)
    for bad in (7, 14):
        with pytest.raises(ValueError):
            codec.encode8(w, 16, lmax=bad)
    c = codec.build_codebook8(w[:1])
    if any(c.lengths[v] == 0 for v in np.unique(codec.exponent_byte(w)).tolist()):
        with pytest.raises(ValueError):
            codec.encode8(w, 16, codebook=c)
