"""Plain CPU oracle of the Huff-LLM bf16 weight codec (HLF1 container).

TEST INFRASTRUCTURE ONLY: this module exists to check the product path. Only
the tests, the smoke entry point and the benchmark's CPU-baseline leg may
import it; the library never does, and it shares no code with the library.

What it computes, following the paper (Huff-LLM, arXiv 2502.00922):

* Sec. 2.1, Eq. 1: a float is sign, biased exponent and mantissa fields.
* Sec. 5.1 (compression experiments): bf16 weights are split 1-4-4-7: the
  sign and the 7 mantissa bits stay raw, the 8 exponent bits become two 4-bit
  groups, each Huffman coded. Codebooks are per weight matrix.
* Sec. 3.1: the split fields are Huffman coded once, offline, on a CPU.
* Sec. 3.2: the decoder matches a window of L_max bits against the codebook,
  emits the symbol and advances its start pointer by the code length; the
  sign is passed through and the fields are concatenated back to 16 bits.

Readings where the paper is silent (each is written down in the design notes):
code-length limit L_max = 12 by default (Sec. 3.2 / 5.2 report 12 as the
empirical maximum); textbook heap Huffman with ties broken leaf-before-node,
leaves by symbol, nodes by creation order; package-merge when the Huffman code
is longer than L_max; canonical code values in the RFC 1951 Sec. 3.2.2 order;
each weight's pair stored as code(el) then code(eh); codes emitted
most-significant bit first into a stream packed least-significant bit first;
a one-symbol field gets code length 0; segments of S weights along a
row are the unit of independent decoding.

Tiling: segment (r, cs) holds W[r, cs*S : cs*S+S] (L = cols/S segments per
row). A group is GR rows x GC consecutive column segments (GR*GC = 64): row
block rb holds rows GR*rb .. GR*rb+G-1 (G = GR except maybe in the last
block), column block cb holds segments cb*GC .. cb*GC+GC-1, and group
g = rb*(L/GC) + cb. Its G*GC segments are numbered mu = j*G + i for row
offset i < G and segment offset j < GC.

Container layout (little-endian; sections start at 64-byte boundaries):
  header (128 B), seg_len u8[n_seg] in group order, grp_meta u32[2*n_grp + 1],
  stream (one 16-byte aligned bit stream per group, its segments concatenated
  in mu order), raw u8[n] (sign<<7 | mantissa; group g's bytes start at S
  times the number of segments before it; weight t of segment mu at
  ((t // 8) * N + mu) * 8 + t % 8, N = G*GC).
Segment lengths (ours: the paper's decoder reads its stream serially, Sec.
3.2, and needs none; segments here decode in parallel from their own starts): a
segment occupies base + seg_len[k] bits of its group's stream, its codes
first, then zero bits; grp_meta[2g] is group g's stream start in 16-byte
units, grp_meta[2g + 1] its base, grp_meta[2*n_grp] the end of the last
stream. base is the group's shortest code-bit count, or its longest minus 255
when the counts span more than 255 (the shorter segments are then padded to
base), so that every length fits one byte (stored_lengths).

Whole-exponent variant (header flags = 1): the 8 exponent bits of a weight
are one symbol of a single per-matrix 256-symbol Huffman code (the {1,8,7}
split; Sec. 3.1 weighs the size of the symbol alphabet against the cost of a
single-cycle CAM match, which a table lookup in local memory does not pay).
Code lengths are limited to lmax in [8, 13]; the 256 lengths are stored in a
256-byte section right after the header. Tiling, stream order (one code per
weight, MSB-first, packed LSB-first), group padding and the raw plane are
those of the split format.

FP16 format (header flags = 2), the paper's own {1,5,5,5} split (Sec. 3.1,
entropy-of-splits table and Huffman-flow figure; Sec. 3.2 decoder with three
5-bit Huffman decoders): a float16 weight is sign (bit 15, kept raw), exponent
e (bits 14..10), mantissa-high mh (bits 9..5) and mantissa-low ml (bits 4..0);
e, mh and ml each get a per-matrix 32-symbol code, lmax in [5, 12]. Each
weight's codes go into the stream as code(ml), code(e), code(mh). The three
code-length tables (each: symbol count, single symbol, 32 lengths) follow the
header in a 128-byte section. The raw plane holds the sign bits only: byte
(segment number) * S/8 + t/8, bit t % 8, for weight t of a segment, segments
numbered in group order.
"""
from __future__ import annotations

import heapq
import math
import struct
from fractions import Fraction
from typing import Dict, List, Sequence, Tuple

import numpy as np

MAGIC = 0x31464C48          # 'HLF1'
VERSION = 2                 # one-byte segment lengths over a per-group base
HEADER_BYTES = 128
GROUP_SEGS = 64             # segments per group (one per lane of a 64-wide wavefront)
RAW_UNIT = 8                # bytes of one segment's raw plane stored contiguously
UNIT_BYTES = 16             # group streams are padded to 128 bits
SECTION_ALIGN = 64
NSYM = 16                   # both exponent groups are 4-bit symbols
NSYM8 = 256                 # the whole exponent as one symbol
FLAG_SPLIT = 0              # header flags: two 4-bit exponent codes
FLAG_WHOLE_EXPONENT = 1     # header flags: one 8-bit exponent code
LEN8_BYTES = 256            # whole-exponent code lengths, after the header
LMAX8_MIN, LMAX8_MAX = 8, 13
FLAG_FP16 = 2               # header flags: float16 {1,5,5,5}
NSYM5 = 32                  # 5-bit fields of the float16 split
CB16_BYTES = 128            # float16 code tables, after the header
LMAX16_MIN, LMAX16_MAX = 5, 12


# --------------------------------------------------------------------------
# Field split (Sec. 2.1 Eq. 1; bf16 1-4-4-7 split of Sec. 5.1)
# --------------------------------------------------------------------------

def split_fields(w: np.ndarray):
    """bf16 bit patterns -> (sign, exponent-high nibble, exponent-low nibble, mantissa).

    bf16 = sign (bit 15) | exponent (bits 14..7) | mantissa (bits 6..0); the
    1-4-4-7 split reads the fields most-significant first."""
    w = np.asarray(w, dtype=np.uint16).astype(np.uint32)
    s = (w >> 15) & 0x1
    eh = (w >> 11) & 0xF
    el = (w >> 7) & 0xF
    m = w & 0x7F
    return s, eh, el, m


def join_fields(s, eh, el, m) -> np.ndarray:
    """Concatenate the fields back into the 16-bit weight (Sec. 3.2)."""
    s, eh, el, m = (np.asarray(a, dtype=np.uint32) for a in (s, eh, el, m))
    return ((s << 15) | (eh << 11) | (el << 7) | m).astype(np.uint16)


def raw_byte(s, m) -> np.ndarray:
    """The raw (uncompressed) part of a weight: sign above the 7 mantissa bits."""
    return ((np.asarray(s, np.uint32) << 7) | np.asarray(m, np.uint32)).astype(np.uint8)


# --------------------------------------------------------------------------
# Histograms and entropy (Sec. 3.1, entropy-of-splits table)
# --------------------------------------------------------------------------

def histogram(sym: np.ndarray, nsym: int = NSYM) -> List[int]:
    sym = np.asarray(sym).ravel()
    return [int(np.count_nonzero(sym == v)) for v in range(nsym)]


def entropy_bits(freqs: Sequence[int]) -> float:
    """Empirical entropy in bits per symbol."""
    n = sum(freqs)
    h = 0.0
    for f in freqs:
        if f:
            p = f / n
            h -= p * math.log2(p)
    return h


def kraft_sum(lengths: Sequence[int]) -> Fraction:
    return sum((Fraction(1, 2 ** l) for l in lengths if l > 0), Fraction(0))


# --------------------------------------------------------------------------
# Huffman code lengths, length limit, canonical codes
# --------------------------------------------------------------------------

def huffman_lengths(freqs: Sequence[int]) -> List[int]:
    """Textbook Huffman: repeatedly merge the two lightest nodes.

    Heap key (weight, kind, id): leaves (kind 0, id = symbol) pop before
    internal nodes (kind 1, id = creation order) of equal weight. A code
    length is the depth of the symbol's leaf. Absent symbols get length 0;
    a field with a single present symbol gets length 0 (no bits)."""
    present = [s for s, f in enumerate(freqs) if f > 0]
    if not present:
        raise ValueError("empty alphabet")
    lengths = [0] * len(freqs)
    if len(present) == 1:
        return lengths
    heap = [(freqs[s], 0, s) for s in present]
    heapq.heapify(heap)
    children: Dict[Tuple[int, int], Tuple[Tuple[int, int], Tuple[int, int]]] = {}
    next_id = 0
    while len(heap) > 1:
        a = heapq.heappop(heap)
        b = heapq.heappop(heap)
        node = (a[0] + b[0], 1, next_id)
        children[(1, next_id)] = ((a[1], a[2]), (b[1], b[2]))
        next_id += 1
        heapq.heappush(heap, node)
    root = (heap[0][1], heap[0][2])
    stack = [(root, 0)]
    while stack:
        (kind, ident), depth = stack.pop()
        if kind == 0:
            lengths[ident] = depth
        else:
            left, right = children[(kind, ident)]
            stack.append((left, depth + 1))
            stack.append((right, depth + 1))
    return lengths


def package_merge_lengths(freqs: Sequence[int], lmax: int) -> List[int]:
    """Optimal prefix-code lengths with every length <= lmax (package-merge).

    Items are the present symbols sorted by (weight, symbol). Starting from
    that list, lmax - 1 times: pair consecutive items into packages (an odd
    last item is dropped) and merge them with the leaves by weight, a leaf
    before a package on equal weight. The first 2(n-1) items of the final list
    are selected; a symbol's length is the number of selected items holding it."""
    present = sorted((f, s) for s, f in enumerate(freqs) if f > 0)
    n = len(present)
    lengths = [0] * len(freqs)
    if n == 0:
        raise ValueError("empty alphabet")
    if n == 1:
        return lengths
    if n > 2 ** lmax:
        raise ValueError("alphabet too large for lmax")
    leaves = [(f, 0, (s,)) for f, s in present]
    cur = list(leaves)
    for _ in range(lmax - 1):
        packages = [(cur[2 * i][0] + cur[2 * i + 1][0], 1, cur[2 * i][2] + cur[2 * i + 1][2])
                    for i in range(len(cur) // 2)]
        cur = sorted(leaves + packages, key=lambda it: (it[0], it[1]))   # stable
    for item in cur[: 2 * (n - 1)]:
        for s in item[2]:
            lengths[s] += 1
    return lengths


def limited_lengths(freqs: Sequence[int], lmax: int) -> List[int]:
    """Huffman lengths, replaced by package-merge lengths if any exceeds lmax."""
    h = huffman_lengths(freqs)
    if max(h) <= lmax:
        return h
    return package_merge_lengths(freqs, lmax)


def min_limit(freqs: Sequence[int]) -> int:
    """Smallest length limit a prefix code of the present symbols can meet:
    0 for one symbol (no bits), else ceil(log2(count))."""
    n = sum(1 for f in freqs if f > 0)
    return 0 if n <= 1 else (n - 1).bit_length()


def code_cost(freqs: Sequence[int], lengths: Sequence[int]) -> int:
    """Total code bits: sum of frequency times length."""
    return sum(f * l for f, l in zip(freqs, lengths))


def pair_limited_lengths(feh: Sequence[int], fel: Sequence[int], lmax: int,
                         pair_max: int) -> Tuple[List[int], List[int]]:
    """Lengths of the two exponent codes of the split format: each code at
    most lmax bits long and, with pair_max > 0, the longest eh code plus the
    longest el code at most pair_max bits, so that every weight's two codes
    fit one decoder window of pair_max bits (the window match of Sec. 3.2,
    applied to the pair that one table lookup decodes).

    Any pair of codes meeting the joint limit has some longest eh code a, so
    its cost is at least that of the optimal codes limited to a and to
    pair_max - a (each length-limited optimum by the rule of limited_lengths).
    The result is therefore the cheapest of those splits, a = 0 .. lmax; on
    equal cost the smallest a. pair_max = 0: each code limited to lmax only."""
    if not pair_max:
        return limited_lengths(feh, lmax), limited_lengths(fel, lmax)
    best = None
    for a in range(0, lmax + 1):
        b = min(lmax, pair_max - a)
        if b < min_limit(fel):
            break
        if a < min_limit(feh):
            continue
        le = limited_lengths(feh, a) if a else [0] * len(feh)
        ll = limited_lengths(fel, b) if b else [0] * len(fel)
        cost = code_cost(feh, le) + code_cost(fel, ll)
        if best is None or cost < best[0]:
            best = (cost, le, ll)
    if best is None:
        raise ValueError("pair limit too small for the alphabets")
    return best[1], best[2]


def canonical_codes(lengths: Sequence[int]) -> List[int]:
    """Canonical code values (RFC 1951 Sec. 3.2.2): shorter codes first, equal
    lengths in increasing symbol order. Entries with length 0 get code 0."""
    maxl = max(lengths) if lengths else 0
    bl_count = [0] * (maxl + 1)
    for l in lengths:
        if l:
            bl_count[l] += 1
    next_code = [0] * (maxl + 2)
    code = 0
    for bits in range(1, maxl + 1):
        code = (code + bl_count[bits - 1]) << 1
        next_code[bits] = code
    codes = [0] * len(lengths)
    for s, l in enumerate(lengths):
        if l:
            codes[s] = next_code[l]
            next_code[l] += 1
    return codes


class FieldCode:
    """One field's codebook: lengths, canonical codes and a bit-serial decoder."""

    def __init__(self, lengths: Sequence[int], nsym_present: int, single: int):
        self.lengths = list(lengths)
        self.nsym = nsym_present
        self.single = single
        self.codes = canonical_codes(self.lengths)
        # Decoder tables: for each length, the first code value and its symbols.
        maxl = max(self.lengths) if any(self.lengths) else 0
        self.by_len: Dict[int, Tuple[int, List[int]]] = {}
        for l in range(1, maxl + 1):
            syms = [s for s in range(len(self.lengths)) if self.lengths[s] == l]
            if syms:
                self.by_len[l] = (self.codes[syms[0]], syms)
        self.maxl = maxl

    @classmethod
    def from_freqs(cls, freqs: Sequence[int], lmax: int) -> "FieldCode":
        return cls.from_lengths(limited_lengths(freqs, lmax), freqs)

    @classmethod
    def from_lengths(cls, lengths: Sequence[int], freqs: Sequence[int]) -> "FieldCode":
        present = [s for s, f in enumerate(freqs) if f > 0]
        return cls(lengths, len(present), present[0] if len(present) == 1 else 0)

    def decode_one(self, bits: List[int], pos: int) -> Tuple[int, int]:
        """Read one code MSB-first starting at bit ``pos``; returns (symbol, new pos)."""
        if self.nsym == 1:
            return self.single, pos
        code = 0
        for l in range(1, self.maxl + 1):
            code = (code << 1) | bits[pos]
            pos += 1
            if l in self.by_len:
                first, syms = self.by_len[l]
                if 0 <= code - first < len(syms):
                    return syms[code - first], pos
        raise ValueError("invalid code in stream")


def bit_reverse(value: int, nbits: int) -> int:
    r = 0
    for i in range(nbits):
        r = (r << 1) | ((value >> i) & 1)
    return r


# --------------------------------------------------------------------------
# Container (HLF1)
# --------------------------------------------------------------------------

def _align(x: int, a: int = SECTION_ALIGN) -> int:
    return (x + a - 1) // a * a


def default_grp_rows(cols: int, seg_len: int) -> int:
    """16 rows x 4 segments when the segments per row allow it, else 32 x 2, else 64 x 1."""
    L = cols // seg_len
    for gc in (4, 2, 1):
        if L % gc == 0:
            return GROUP_SEGS // gc
    return GROUP_SEGS


def layout(rows: int, cols: int, seg_len: int, grp_rows: int = GROUP_SEGS,
           flags: int = FLAG_SPLIT) -> Dict[str, int]:
    n = rows * cols
    n_seg = n // seg_len
    L = cols // seg_len
    GC = GROUP_SEGS // grp_rows
    n_grp = (rows + grp_rows - 1) // grp_rows * (L // GC)
    extra = {FLAG_SPLIT: 0, FLAG_WHOLE_EXPONENT: LEN8_BYTES, FLAG_FP16: CB16_BYTES}[flags]
    off_seg_bits = _align(HEADER_BYTES + extra)      # seg_len u8[n_seg]
    off_grp_off = _align(off_seg_bits + n_seg)        # grp_meta u32[2*n_grp + 1]
    off_stream = _align(off_grp_off + 4 * (2 * n_grp + 1))
    return dict(n=n, n_seg=n_seg, n_grp=n_grp, L=L, GC=GC, off_seg_bits=off_seg_bits,
                off_grp_off=off_grp_off, off_stream=off_stream)


def group_geometry(rows: int, cols: int, seg_len: int, g: int,
                   grp_rows: int = GROUP_SEGS) -> Tuple[int, int, int, int, int]:
    """(first row r0, rows G, first column segment, first segment number, GC) of group g.

    Segment mu of the group is (r0 + mu % G, first column segment + mu // G)."""
    L = cols // seg_len
    GC = GROUP_SEGS // grp_rows
    rb, cb = divmod(g, L // GC)
    r0 = rb * grp_rows
    G = min(grp_rows, rows - r0)
    return r0, G, cb * GC, r0 * L + cb * GC * G, GC


def check_shape(rows: int, cols: int, seg_len: int, lmax: int, grp_rows: int = GROUP_SEGS,
                flags: int = FLAG_SPLIT) -> None:
    if rows < 1 or cols < 1:
        raise ValueError("empty matrix")
    if flags == FLAG_WHOLE_EXPONENT:
        if not (LMAX8_MIN <= lmax <= LMAX8_MAX):
            raise ValueError("lmax must be in [8, 13] for the whole-exponent code")
    elif flags == FLAG_FP16:
        if not (LMAX16_MIN <= lmax <= LMAX16_MAX):
            raise ValueError("lmax must be in [5, 12] for the float16 codes")
    elif not (4 <= lmax <= 15):
        raise ValueError("lmax must be in [4, 15]")
    if seg_len < 8 or seg_len > 512 or seg_len % 8 or cols % seg_len:
        raise ValueError("segment length must be a multiple of 8 in [8, 512] dividing cols")
    if grp_rows not in (1, 2, 4, 8, 16, 32, 64) or (cols // seg_len) % (GROUP_SEGS // grp_rows):
        raise ValueError("group rows must be a power of two whose 64/GR divides the segments per row")


def raw_pos(r: np.ndarray, c: np.ndarray, rows: int, cols: int, seg_len: int,
            grp_rows: int = GROUP_SEGS) -> np.ndarray:
    """Byte offset in the raw plane of weight (r, c)."""
    r = np.asarray(r, dtype=np.int64)
    c = np.asarray(c, dtype=np.int64)
    L = cols // seg_len
    GC = GROUP_SEGS // grp_rows
    rb, i = r // grp_rows, r % grp_rows
    cs, t = c // seg_len, c % seg_len
    cb, j = cs // GC, cs % GC
    G = np.minimum(grp_rows, rows - rb * grp_rows)
    mu = j * G + i
    first_seg = rb * grp_rows * L + cb * GC * G
    return first_seg * seg_len + ((t // RAW_UNIT) * (G * GC) + mu) * RAW_UNIT + (t % RAW_UNIT)


def raw_plane(w: np.ndarray, seg_len: int, grp_rows: int) -> np.ndarray:
    """Raw plane of the bf16 formats: (sign<<7 | mantissa) of every weight at raw_pos."""
    rows, cols = w.shape
    s, _, _, m = split_fields(w)
    rr, cc = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    raw = np.zeros(rows * cols, dtype=np.uint8)
    raw[raw_pos(rr.ravel(), cc.ravel(), rows, cols, seg_len, grp_rows)] = raw_byte(s, m).ravel()
    return raw


def segment_number(r, c, rows: int, cols: int, seg_len: int, grp_rows: int) -> np.ndarray:
    """Group-order number of the segment holding weight (r, c)."""
    r = np.asarray(r, dtype=np.int64)
    c = np.asarray(c, dtype=np.int64)
    L = cols // seg_len
    GC = GROUP_SEGS // grp_rows
    rb, i = r // grp_rows, r % grp_rows
    cb, j = (c // seg_len) // GC, (c // seg_len) % GC
    G = np.minimum(grp_rows, rows - rb * grp_rows)
    return rb * grp_rows * L + cb * GC * G + j * G + i


def sign_plane(w: np.ndarray, seg_len: int, grp_rows: int) -> np.ndarray:
    """Raw plane of the float16 format: one sign bit per weight, S/8 bytes per
    segment in group order; bit t % 8 of byte t // 8 is weight t's sign."""
    rows, cols = w.shape
    sgn = (np.asarray(w, np.uint16) >> 15).astype(np.uint8)
    rr, cc = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    seg = segment_number(rr, cc, rows, cols, seg_len, grp_rows)
    t = cc % seg_len
    byte = (seg * (seg_len // 8) + t // 8).ravel()
    plane = np.zeros(rows * cols // 8, dtype=np.uint8)
    np.bitwise_or.at(plane, byte, (sgn.ravel() << (t.ravel() % 8)).astype(np.uint8))
    return plane


PAIR_MAX = 11              # default joint limit of a weight's two exponent codes


def build_codebooks(w: np.ndarray, lmax: int = 12, pair_max: int = PAIR_MAX) -> Tuple[FieldCode, FieldCode]:
    """Per-matrix codebooks for the two exponent nibbles (Sec. 5.1), each
    code limited to lmax bits and the pair to pair_max (pair_limited_lengths)."""
    _, eh, el, _ = split_fields(w)
    feh, fel = histogram(eh), histogram(el)
    leh, lel = pair_limited_lengths(feh, fel, lmax, pair_max)
    return FieldCode.from_lengths(leh, feh), FieldCode.from_lengths(lel, fel)


def segment_stream(eh_seg, el_seg, ceh: FieldCode, cel: FieldCode) -> Tuple[int, int]:
    """Bit stream of one segment as (integer, bit count).

    For each weight in order: code(el) then code(eh), each emitted MSB-first;
    stream bit k is bit k of the integer (least-significant first)."""
    rev_eh = [bit_reverse(ceh.codes[v], ceh.lengths[v]) for v in range(NSYM)]
    rev_el = [bit_reverse(cel.codes[v], cel.lengths[v]) for v in range(NSYM)]
    acc = 0
    pos = 0
    for a, b in zip(eh_seg, el_seg):
        la = ceh.lengths[a] if ceh.nsym > 1 else 0
        lb = cel.lengths[b] if cel.nsym > 1 else 0
        acc |= (rev_el[b] | (rev_eh[a] << lb)) << pos
        pos += la + lb
    return acc, pos


def encode(w: np.ndarray, seg_len: int, lmax: int = 12,
           codebooks: Tuple[FieldCode, FieldCode] = None, grp_rows: int = None,
           pair_max: int = PAIR_MAX) -> bytes:
    """Compress a bf16 matrix [rows, cols] (uint16 bit patterns) into HLF1 bytes."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    rows, cols = w.shape
    GR = default_grp_rows(cols, seg_len) if grp_rows is None else grp_rows
    check_shape(rows, cols, seg_len, lmax, GR)
    ceh, cel = codebooks if codebooks is not None else build_codebooks(w, lmax, pair_max)
    _, eh, el, _ = split_fields(w)

    def seg_stream(r, a, S):
        return segment_stream(eh[r, a:a + S].tolist(), el[r, a:a + S].tolist(), ceh, cel)

    def header(*geo):
        return pack_header(rows, cols, seg_len, lmax, GR, *geo, ceh, cel)

    return _assemble(w, seg_len, GR, FLAG_SPLIT, seg_stream, header, b"")


SEG_LEN_SPAN = 255          # one-byte segment lengths over the group's base


def stored_lengths(code_bits: Sequence[int]) -> Tuple[int, List[int]]:
    """(base, stored bit counts) of one group's segments from their code-bit
    counts: base is the least count, or the greatest minus 255 when the counts
    span more than that; a segment shorter than base is padded to it."""
    base = max(min(code_bits), max(code_bits) - SEG_LEN_SPAN)
    return base, [max(c, base) for c in code_bits]


def _assemble(w, seg_len, GR, flags, seg_stream, header, codebook_section) -> bytes:
    """Container bytes from a per-segment stream function (all formats)."""
    rows, cols = w.shape
    lay = layout(rows, cols, seg_len, GR, flags)
    n, n_seg, n_grp = lay["n"], lay["n_seg"], lay["n_grp"]
    S = seg_len

    seg_len8 = np.zeros(n_seg, dtype=np.uint8)
    grp_meta = np.zeros(2 * n_grp + 1, dtype=np.uint32)
    chunks: List[bytes] = []
    units_total = 0
    max_units = 0
    for g in range(n_grp):
        r0, G, c0, first, GC = group_geometry(rows, cols, S, g, GR)
        segs = [seg_stream(r0 + mu % G, (c0 + mu // G) * S, S) for mu in range(G * GC)]
        base, stored = stored_lengths([nb for _, nb in segs])
        gacc, gpos = 0, 0
        for mu, (acc, nb) in enumerate(segs):
            seg_len8[first + mu] = stored[mu] - base
            gacc |= acc << gpos            # codes, then zero bits up to the stored length
            gpos += stored[mu]
        units = (gpos + 127) // 128
        chunks.append(gacc.to_bytes(units * UNIT_BYTES, "little"))
        grp_meta[2 * g] = units_total
        grp_meta[2 * g + 1] = base
        units_total += units
        max_units = max(max_units, units)
    grp_meta[2 * n_grp] = units_total
    stream = b"".join(chunks)

    off_raw = _align(lay["off_stream"] + len(stream))
    raw = sign_plane(w, S, GR) if flags == FLAG_FP16 else raw_plane(w, S, GR)
    total = off_raw + raw.size

    out = bytearray(total)
    out[0:HEADER_BYTES] = header(n_seg, n_grp, lay["off_seg_bits"], lay["off_grp_off"],
                                 lay["off_stream"], off_raw, total, max_units)
    out[HEADER_BYTES:HEADER_BYTES + len(codebook_section)] = codebook_section
    out[lay["off_seg_bits"]:lay["off_seg_bits"] + n_seg] = seg_len8.tobytes()
    out[lay["off_grp_off"]:lay["off_grp_off"] + 4 * (2 * n_grp + 1)] = grp_meta.tobytes()
    out[lay["off_stream"]:lay["off_stream"] + len(stream)] = stream
    out[off_raw:off_raw + n] = raw.tobytes()
    return bytes(out)


# --------------------------------------------------------------------------
# Whole-exponent variant (flags = 1)
# --------------------------------------------------------------------------

def exponent_byte(w: np.ndarray) -> np.ndarray:
    """The 8-bit biased exponent of bf16 bit patterns (Sec. 2.1, Eq. 1)."""
    return (np.asarray(w, dtype=np.uint16).astype(np.uint32) >> 7) & 0xFF


def build_codebook8(w: np.ndarray, lmax: int = 12) -> FieldCode:
    """Per-matrix 256-symbol code of the whole exponent, lengths <= lmax."""
    if not (LMAX8_MIN <= lmax <= LMAX8_MAX):
        raise ValueError("lmax must be in [8, 13] for the whole-exponent code")
    return FieldCode.from_freqs(histogram(exponent_byte(w), NSYM8), lmax)


def segment_stream8(e_seg, code: FieldCode) -> Tuple[int, int]:
    """Bit stream of one segment, one code per weight, each MSB-first; stream
    bit k is bit k of the integer."""
    acc = 0
    pos = 0
    for e in e_seg:
        l = code.lengths[e] if code.nsym > 1 else 0
        acc |= bit_reverse(code.codes[e], l) << pos
        pos += l
    return acc, pos


def encode8(w: np.ndarray, seg_len: int, lmax: int = 12, codebook: FieldCode = None,
            grp_rows: int = None) -> bytes:
    """Compress a bf16 matrix into an HLF1 container of the whole-exponent format."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    rows, cols = w.shape
    GR = default_grp_rows(cols, seg_len) if grp_rows is None else grp_rows
    check_shape(rows, cols, seg_len, lmax, GR, FLAG_WHOLE_EXPONENT)
    code = codebook if codebook is not None else build_codebook8(w, lmax)
    if code.nsym > 1 and (max(code.lengths) > lmax or len(code.lengths) != NSYM8):
        raise ValueError("codebook does not fit lmax")
    e = exponent_byte(w)
    for v in np.unique(e).tolist():
        if (code.lengths[v] == 0) if code.nsym > 1 else (v != code.single):
            raise ValueError("exponent without a code")

    def seg_stream(r, a, S):
        return segment_stream8(e[r, a:a + S].tolist(), code)

    def header(n_seg, n_grp, off_sb, off_go, off_st, off_raw, total, max_units):
        return struct.pack(HEADER_FMT, MAGIC, VERSION, lmax, FLAG_WHOLE_EXPONENT, rows, cols, seg_len, GR,
                           n_seg, n_grp, off_sb, off_go, off_st, off_raw, total, max_units,
                           code.nsym & 0xFF, code.nsym >> 8, code.single, 0, bytes(16), bytes(16))

    lens = bytes(code.lengths) if code.nsym > 1 else bytes(NSYM8)
    return _assemble(w, seg_len, GR, FLAG_WHOLE_EXPONENT, seg_stream, header, lens)


def header_codebook8(h) -> FieldCode:
    return FieldCode(h["len8"], h["nsym8"], h["single8"])


def container_size8(w: np.ndarray, seg_len: int, lmax: int = 12, codebook: FieldCode = None,
                    grp_rows: int = None) -> Dict[str, int]:
    """Exact size of ``encode8(w, ...)`` from the code lengths alone."""
    w = np.asarray(w, dtype=np.uint16)
    code = codebook if codebook is not None else build_codebook8(w, lmax)
    le = np.array(code.lengths if code.nsym > 1 else [0] * NSYM8, dtype=np.int64)
    return _size_from_bits(le[exponent_byte(w)], w.shape, seg_len, lmax, grp_rows, FLAG_WHOLE_EXPONENT)


# --------------------------------------------------------------------------
# FP16 {1,5,5,5} format (flags = 2)
# --------------------------------------------------------------------------

def split_fields16(w: np.ndarray):
    """float16 bit patterns -> (sign, exponent, mantissa-high, mantissa-low):
    float16 = sign (bit 15) | exponent (bits 14..10) | mantissa (bits 9..0),
    the mantissa halved into its high and low 5 bits (the {1,5,5,5} split)."""
    w = np.asarray(w, dtype=np.uint16).astype(np.uint32)
    return (w >> 15) & 1, (w >> 10) & 0x1F, (w >> 5) & 0x1F, w & 0x1F


def join_fields16(s, e, mh, ml) -> np.ndarray:
    s, e, mh, ml = (np.asarray(a, dtype=np.uint32) for a in (s, e, mh, ml))
    return ((s << 15) | (e << 10) | (mh << 5) | ml).astype(np.uint16)


def build_codebooks16(w: np.ndarray, lmax: int = 12) -> Tuple[FieldCode, FieldCode, FieldCode]:
    """Per-matrix codes of the three 5-bit fields (exponent, mantissa-high, mantissa-low)."""
    if not (LMAX16_MIN <= lmax <= LMAX16_MAX):
        raise ValueError("lmax must be in [5, 12] for the float16 codes")
    _, e, mh, ml = split_fields16(w)
    return tuple(FieldCode.from_freqs(histogram(f, NSYM5), lmax) for f in (e, mh, ml))


def segment_stream16(e_seg, mh_seg, ml_seg, ce: FieldCode, cmh: FieldCode, cml: FieldCode) -> Tuple[int, int]:
    """Bit stream of one segment: per weight code(ml), code(e), code(mh), each
    MSB-first; stream bit k is bit k of the integer."""
    acc, pos = 0, 0
    for e, mh, ml in zip(e_seg, mh_seg, ml_seg):
        for code, v in ((cml, ml), (ce, e), (cmh, mh)):
            l = code.lengths[v] if code.nsym > 1 else 0
            acc |= bit_reverse(code.codes[v], l) << pos
            pos += l
    return acc, pos


def _codebook16_section(codes) -> bytes:
    out = bytearray(CB16_BYTES)
    for f, c in enumerate(codes):
        rec = bytes([c.nsym, c.single]) + (bytes(c.lengths) if c.nsym > 1 else bytes(NSYM5))
        out[f * 34:(f + 1) * 34] = rec
    return bytes(out)


def encode16(w: np.ndarray, seg_len: int, lmax: int = 12, codebooks=None, grp_rows: int = None) -> bytes:
    """Compress a float16 matrix [rows, cols] (uint16 bit patterns) into an HLF1
    container of the float16 format."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    rows, cols = w.shape
    GR = default_grp_rows(cols, seg_len) if grp_rows is None else grp_rows
    check_shape(rows, cols, seg_len, lmax, GR, FLAG_FP16)
    codes = codebooks if codebooks is not None else build_codebooks16(w, lmax)
    ce, cmh, cml = codes
    _, e, mh, ml = split_fields16(w)
    for c, f in ((ce, e), (cmh, mh), (cml, ml)):
        if c.nsym > 1 and max(c.lengths) > lmax:
            raise ValueError("codebook does not fit lmax")
        for v in np.unique(f).tolist():
            if (c.lengths[v] == 0) if c.nsym > 1 else (v != c.single):
                raise ValueError("field value without a code")

    def seg_stream(r, a, S):
        return segment_stream16(e[r, a:a + S].tolist(), mh[r, a:a + S].tolist(), ml[r, a:a + S].tolist(),
                                ce, cmh, cml)

    def header(n_seg, n_grp, off_sb, off_go, off_st, off_raw, total, max_units):
        return struct.pack(HEADER_FMT, MAGIC, VERSION, lmax, FLAG_FP16, rows, cols, seg_len, GR,
                           n_seg, n_grp, off_sb, off_go, off_st, off_raw, total, max_units,
                           0, 0, 0, 0, bytes(16), bytes(16))

    return _assemble(w, seg_len, GR, FLAG_FP16, seg_stream, header, _codebook16_section(codes))


def header_codebooks16(h) -> Tuple[FieldCode, FieldCode, FieldCode]:
    return tuple(FieldCode(lens, nsym, single) for nsym, single, lens in h["cb16"])


def container_size16(w: np.ndarray, seg_len: int, lmax: int = 12, codebooks=None,
                     grp_rows: int = None) -> Dict[str, int]:
    """Exact size of ``encode16(w, ...)`` from the code lengths alone."""
    w = np.asarray(w, dtype=np.uint16)
    codes = codebooks if codebooks is not None else build_codebooks16(w, lmax)
    _, e, mh, ml = split_fields16(w)
    bits = 0
    for c, f in zip(codes, (e, mh, ml)):
        bits = bits + np.array(c.lengths if c.nsym > 1 else [0] * NSYM5, dtype=np.int64)[f]
    return _size_from_bits(bits, w.shape, seg_len, lmax, grp_rows, FLAG_FP16)


HEADER_FMT = "<IHBBQQIIQQQQQQQIBBBB16s16s"


def pack_header(rows, cols, seg_len, lmax, grp_rows, n_seg, n_grp, off_sb, off_go, off_st, off_raw, total,
                max_units, ceh: FieldCode, cel: FieldCode) -> bytes:
    h = struct.pack(HEADER_FMT, MAGIC, VERSION, lmax, FLAG_SPLIT, rows, cols, seg_len, grp_rows,
                    n_seg, n_grp, off_sb, off_go, off_st, off_raw, total, max_units,
                    ceh.nsym, cel.nsym, ceh.single, cel.single,
                    bytes(ceh.lengths), bytes(cel.lengths))
    assert len(h) == HEADER_BYTES
    return h


def parse_header(blob: bytes) -> Dict[str, object]:
    f = struct.unpack(HEADER_FMT, blob[:HEADER_BYTES])
    keys = ["magic", "version", "lmax", "flags", "rows", "cols", "seg_len", "grp_rows", "n_seg",
            "n_grp", "off_seg_bits", "off_grp_off", "off_stream", "off_raw", "total_bytes",
            "max_grp_units", "eh_nsym", "el_nsym", "eh_single", "el_single", "eh_len", "el_len"]
    h = dict(zip(keys, f))
    h["eh_len"] = list(h["eh_len"])
    h["el_len"] = list(h["el_len"])
    if h["magic"] != MAGIC or h["version"] != VERSION:
        raise ValueError("not an HLF1 container")
    if h["flags"] == FLAG_WHOLE_EXPONENT:
        # bytes 92..93: u16 symbol count; byte 94: the symbol when it is the only one
        h["nsym8"] = h["eh_nsym"] | (h["el_nsym"] << 8)
        h["single8"] = h["eh_single"]
        h["len8"] = list(blob[HEADER_BYTES:HEADER_BYTES + LEN8_BYTES])
    elif h["flags"] == FLAG_FP16:
        # three records (exponent, mantissa-high, mantissa-low): nsym, single, 32 lengths
        sec = blob[HEADER_BYTES:HEADER_BYTES + CB16_BYTES]
        h["cb16"] = [(sec[f * 34], sec[f * 34 + 1], list(sec[f * 34 + 2:f * 34 + 34])) for f in range(3)]
    elif h["flags"] != FLAG_SPLIT:
        raise ValueError("unknown format flags")
    return h


def header_codebooks(h) -> Tuple[FieldCode, FieldCode]:
    return (FieldCode(h["eh_len"], h["eh_nsym"], h["eh_single"]),
            FieldCode(h["el_len"], h["el_nsym"], h["el_single"]))


def segment_lengths(blob: bytes, h=None) -> Tuple[np.ndarray, np.ndarray]:
    """(stored bit count of every segment in group order, group stream starts
    in 16-byte units with the end of the last appended) from the container's
    one-byte lengths and per-group bases."""
    h = parse_header(blob) if h is None else h
    n_seg, n_grp = h["n_seg"], h["n_grp"]
    rows, cols, S, GR = h["rows"], h["cols"], h["seg_len"], h["grp_rows"]
    seg8 = np.frombuffer(blob, np.uint8, n_seg, h["off_seg_bits"]).astype(np.int64)
    meta = np.frombuffer(blob, np.uint32, 2 * n_grp + 1, h["off_grp_off"]).astype(np.int64)
    stored = np.zeros(n_seg, dtype=np.int64)
    for g in range(n_grp):
        _, G, _, first, GC = group_geometry(rows, cols, S, g, GR)
        stored[first:first + G * GC] = seg8[first:first + G * GC] + meta[2 * g + 1]
    return stored, meta[0::2]


def _segment_end(bits: List[int], start: int, pos: int, stored: int) -> int:
    """The next segment's start: a segment's codes take at most its stored
    length (less only where it was padded to its group's base), and any
    padding is zero bits."""
    if pos - start > stored or any(bits[pos:start + stored]):
        raise ValueError("segment length mismatch")
    return start + stored


def decode_group(blob: bytes, g: int) -> Tuple[int, int, int, int, np.ndarray]:
    """Bit-serial decode of one group.

    Returns (first row r0, rows G, first column segment, GC, uint16[G, GC*S])."""
    h = parse_header(blob)
    if h["flags"] == FLAG_FP16:
        return _decode_group16(blob, h, g)
    whole = h["flags"] == FLAG_WHOLE_EXPONENT
    if whole:
        code8 = header_codebook8(h)
    else:
        ceh, cel = header_codebooks(h)
    rows, cols, S, GR = h["rows"], h["cols"], h["seg_len"], h["grp_rows"]
    stored, grp_off = segment_lengths(blob, h)
    raw_plane = np.frombuffer(blob, np.uint8, rows * cols, h["off_raw"])
    r0, G, c0, first, GC = group_geometry(rows, cols, S, g, GR)
    a = h["off_stream"] + int(grp_off[g]) * UNIT_BYTES
    b = h["off_stream"] + int(grp_off[g + 1]) * UNIT_BYTES
    bits = np.unpackbits(np.frombuffer(blob[a:b], np.uint8), bitorder="little").tolist()
    out = np.zeros((G, GC * S), dtype=np.uint16)
    pos = 0
    for mu in range(G * GC):
        i, j = mu % G, mu // G
        start = pos
        eh = np.zeros(S, np.uint32)
        el = np.zeros(S, np.uint32)
        for t in range(S):
            if whole:                       # one 8-bit symbol: eh, el are its nibbles
                e, pos = code8.decode_one(bits, pos)
                eh[t], el[t] = e >> 4, e & 15
            else:
                el[t], pos = cel.decode_one(bits, pos)
                eh[t], pos = ceh.decode_one(bits, pos)
        pos = _segment_end(bits, start, pos, int(stored[first + mu]))
        cols_of = (c0 + j) * S + np.arange(S)
        rp = raw_pos(np.full(S, r0 + i), cols_of, rows, cols, S, GR)
        r = raw_plane[rp].astype(np.uint32)
        out[i, j * S:(j + 1) * S] = join_fields(r >> 7, eh, el, r & 0x7F)
    return r0, G, c0, GC, out


def _decode_group16(blob: bytes, h, g: int):
    """decode_group for the float16 format."""
    ce, cmh, cml = header_codebooks16(h)
    rows, cols, S, GR = h["rows"], h["cols"], h["seg_len"], h["grp_rows"]
    stored, grp_off = segment_lengths(blob, h)
    signs = np.frombuffer(blob, np.uint8, rows * cols // 8, h["off_raw"])
    r0, G, c0, first, GC = group_geometry(rows, cols, S, g, GR)
    a = h["off_stream"] + int(grp_off[g]) * UNIT_BYTES
    b = h["off_stream"] + int(grp_off[g + 1]) * UNIT_BYTES
    bits = np.unpackbits(np.frombuffer(blob[a:b], np.uint8), bitorder="little").tolist()
    out = np.zeros((G, GC * S), dtype=np.uint16)
    pos = 0
    for mu in range(G * GC):
        i, j = mu % G, mu // G
        start = pos
        f = np.zeros((3, S), np.uint32)
        for t in range(S):
            f[2, t], pos = cml.decode_one(bits, pos)
            f[0, t], pos = ce.decode_one(bits, pos)
            f[1, t], pos = cmh.decode_one(bits, pos)
        pos = _segment_end(bits, start, pos, int(stored[first + mu]))
        t = np.arange(S)
        sb = signs[(first + mu) * (S // 8) + t // 8]
        out[i, j * S:(j + 1) * S] = join_fields16((sb >> (t % 8)) & 1, f[0], f[1], f[2])
    return r0, G, c0, GC, out


def decode(blob: bytes) -> np.ndarray:
    """Decompress a whole HLF1 container back to the bf16 matrix (uint16)."""
    h = parse_header(blob)
    w = np.zeros((h["rows"], h["cols"]), dtype=np.uint16)
    S = h["seg_len"]
    for g in range(h["n_grp"]):
        r0, G, c0, GC, part = decode_group(blob, g)
        w[r0:r0 + G, c0 * S:(c0 + GC) * S] = part
    return w


def payload_bits(w: np.ndarray, ceh: FieldCode, cel: FieldCode) -> int:
    """Sum of code lengths plus 8 raw bits per weight (size without metadata)."""
    _, eh, el, _ = split_fields(w)
    he, hl = histogram(eh), histogram(el)
    le = ceh.lengths if ceh.nsym > 1 else [0] * NSYM
    ll = cel.lengths if cel.nsym > 1 else [0] * NSYM
    return sum(f * l for f, l in zip(he, le)) + sum(f * l for f, l in zip(hl, ll)) + 8 * int(np.size(w))


def container_size(w: np.ndarray, seg_len: int, lmax: int = 12,
                   codebooks: Tuple[FieldCode, FieldCode] = None, grp_rows: int = None,
                   pair_max: int = PAIR_MAX) -> Dict[str, int]:
    """Exact container size of ``encode(w, seg_len, lmax, grp_rows=...)`` from the
    code lengths alone (sum of code lengths per segment, 128-bit padding per
    group, section alignment), without building the stream."""
    w = np.asarray(w, dtype=np.uint16)
    ceh, cel = codebooks if codebooks is not None else build_codebooks(w, lmax, pair_max)
    _, eh, el, _ = split_fields(w)
    le = np.array(ceh.lengths if ceh.nsym > 1 else [0] * NSYM, dtype=np.int64)
    ll = np.array(cel.lengths if cel.nsym > 1 else [0] * NSYM, dtype=np.int64)
    return _size_from_bits(le[eh] + ll[el], w.shape, seg_len, lmax, grp_rows, FLAG_SPLIT)


def _size_from_bits(bits, shape, seg_len, lmax, grp_rows, flags) -> Dict[str, int]:
    """Container size from the code bits of every weight ([rows, cols])."""
    rows, cols = shape
    GR = default_grp_rows(cols, seg_len) if grp_rows is None else grp_rows
    check_shape(rows, cols, seg_len, lmax, GR, flags)
    L = cols // seg_len
    GC = GROUP_SEGS // GR
    seg = bits.reshape(rows, L, seg_len).sum(axis=2)                      # [rows, L]
    units = 0
    max_units = 0
    for rb in range(0, rows, GR):
        blk = seg[rb:rb + GR].reshape(-1, L // GC, GC).transpose(1, 0, 2).reshape(L // GC, -1)  # [CB, G*GC]
        base = np.maximum(blk.min(axis=1), blk.max(axis=1) - SEG_LEN_SPAN)  # stored_lengths, per group
        per_grp = np.maximum(blk, base[:, None]).sum(axis=1)
        u = (per_grp + 127) // 128
        units += int(u.sum())
        max_units = max(max_units, int(u.max()))
    lay = layout(rows, cols, seg_len, GR, flags)
    off_raw = _align(lay["off_stream"] + units * UNIT_BYTES)
    raw_bytes = rows * cols // 8 if flags == FLAG_FP16 else rows * cols
    return dict(total_bytes=off_raw + raw_bytes, stream_units=units, max_grp_units=max_units,
                code_bits=int(seg.sum()), off_raw=off_raw, grp_rows=GR)
