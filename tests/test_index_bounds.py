"""Host model of the fused kernels' address arithmetic (CPU).

The kernels take no bounds checks per access; they keep every read inside the
container by clamping. This model restates, in plain Python, the index
arithmetic of the persistent decode-GEMV for one group (the metadata loads,
the clamps of the group's stream start and length, each lane's first stream
word from the prefix sum of the segment lengths, the words it loads, the raw
bytes, the four column rows of every 8-weight step and the table index), and
checks every address against the container and the LDS regions while the
inputs are damaged at random: segment length bytes, group starts and bases
replaced by arbitrary values, and every table entry's length field arbitrary (stream bits
that decode to anything). Geometry comes from real containers."""
import numpy as np
import pytest

from gen import random_bf16
from oracle import codec

hl = pytest.importorskip("paper_2502_00922_amd.hufflm")

KCOL = 64          # column row stride (words)
POS_MASK = 0x7FFFFF


def _model_group(h, seg8, grp_meta, g, JT, rng, bounded):
    """Byte ranges the group's wave reads from the container, and the LDS
    column rows it touches; the position entries are arbitrary."""
    S, GR, rows, cols = h["seg_len"], h["grp_rows"], h["rows"], h["cols"]
    L = cols // S
    GC = 64 // GR
    CB = L // GC
    rb, cb = divmod(g, CB)
    r0, c0 = rb * GR, cb * GC
    G = min(GR, rows - r0)
    N = G * GC
    first = r0 * L + c0 * G
    stream_units = (h["off_raw"] - h["off_stream"]) // 16
    max_units = h["max_grp_units"]
    reads = []
    # metadata: the dword of each lane's one-byte length; the group's start,
    # base and end (lanes 0, 2, 1; the other lanes reload the start)
    for lane in range(64):
        reads.append((h["off_seg_bits"] + ((first + min(lane, N - 1)) >> 2) * 4, 4))
        reads.append((h["off_grp_off"] + (2 * g + {1: 2, 2: 1}.get(lane, 0)) * 4, 4))
    v0 = min(int(grp_meta[2 * g]), stream_units)
    v1 = min(max(int(grp_meta[2 * g + 2]), v0), stream_units)
    base = int(grp_meta[2 * g + 1])
    units = min(v1 - v0, max_units)
    # 32-bit lane arithmetic, as in the kernel (a damaged base wraps)
    nb = [(base + int(seg8[first + min(l, N - 1)])) & 0xFFFFFFFF if l < N else 0 for l in range(64)]
    incl = np.cumsum(np.array(nb, dtype=np.uint64)) & 0xFFFFFFFF
    rows_used = []
    for lane in range(64):
        start = min((int(incl[lane]) - nb[lane]) & 0xFFFFFFFF, units * 128)
        ws, bit0 = start >> 5, start & 31
        if units:
            base = h["off_stream"] + (v0 * 4 + ws) * 4
        else:
            base = h["off_raw"] + first * S
        reads.append((base, JT * 4))
        # raw bytes of each step: 8 per lane per step
        for k in range(S // 8):
            reads.append((h["off_raw"] + first * S + (k * N + min(lane, N - 1)) * 8, 8))
        # the decode: positions advance by arbitrary entry lengths (bits 0..4)
        p = (27 if bounded else 30) + bit0
        kRows = JT + 1
        jmax = kRows - 3
        for _ in range(S // 8):
            j = min((p & POS_MASK) >> 5, jmax - 1)
            rows_used.extend([j, j + 3])
            for _ in range(8):
                p += int(rng.integers(0, 32))
            p &= 0xFFFFFFFF
    return reads, rows_used, JT + 1


@pytest.mark.parametrize("seed", range(6))
def test_persistent_kernel_reads_stay_in_bounds(seed):
    rng = np.random.default_rng(seed)
    w = random_bf16((48, 1024), seed=seed)
    blob = bytes(codec.encode(w, seg_len=64))
    h = codec.parse_header(blob)
    n_seg, n_grp = h["n_seg"], h["n_grp"]
    off_sb, off_go = h["off_seg_bits"], h["off_grp_off"]
    seg8 = np.frombuffer(blob, np.uint8, n_seg, off_sb).copy()
    grp_meta = np.frombuffer(blob, np.uint32, 2 * n_grp + 1, off_go).copy()
    max_seg = int(codec.segment_lengths(blob, h)[0].max())
    col_rows = 1 + ((31 + max_seg + 31) >> 5) + 3
    JT = next(j for j in (12, 16, 20) if j >= col_rows - 1)
    for trial in range(40):
        sb, go = seg8.copy(), grp_meta.copy()
        if trial % 2:
            sb = rng.integers(0, 1 << 8, n_seg).astype(np.uint8)
            go = rng.integers(0, 1 << 32, 2 * n_grp + 1, dtype=np.uint64).astype(np.uint32)
        for g in range(n_grp):
            reads, rows_used, krows = _model_group(h, sb, go, g, JT, rng, bounded=bool(trial % 4 < 2))
            for off, size in reads:
                assert 0 <= off and off + size <= len(blob), (trial, g, off, size, len(blob))
            assert min(rows_used) >= 0 and max(rows_used) < krows
