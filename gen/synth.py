"""Seeded synthetic LLM-shaped bf16 weights and decode-step activations.

Recipe (every draw is float32 from numpy's PCG64 ``default_rng``):

* weights ~ N(0, std) with std = 0.02 unless a workload says otherwise;
* an independent Bernoulli(0.001) outlier mask multiplies the selected
  weights by 20 (before rounding);
* optional per-row scale exp(0.3 * z_r), z_r ~ N(0, 1)  (LogNormal(0, 0.3));
* optional per-matrix layer scale u ~ U[1, 4] giving std = 0.02 / sqrt(u);
* float32 -> bfloat16 by round-to-nearest-even on the bit pattern;
* activations x ~ N(0, 1), as float32 or rounded to bfloat16.

Seeds: the 1024x1024 single-matrix workload uses ``default_rng(0)`` and draws
W, then the mask, then x, in that order. Every other matrix draws its values
and its outlier mask per block of 256 rows, from the independent streams
``default_rng([0, cfg, layer, matrix, k, block])`` with k = 0 for the values
and 2 for the mask, and its x and scales from ``default_rng([0, cfg, layer,
matrix, k])`` with k = 1 for x and 3 for the scales. A matrix or any row range
of it can thus be regenerated alone, and the row blocks in parallel.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

OUTLIER_P = 0.001
OUTLIER_MUL = 20.0
BASE_STD = 0.02


@dataclass(frozen=True)
class MatrixSpec:
    cfg: int
    layer: int
    index: int
    name: str
    rows: int
    cols: int
    row_scale: bool = False      # LogNormal(0, 0.3) per-row scale
    layer_scale: bool = False    # std = 0.02 / sqrt(U[1, 4]) per matrix


def _llama7b_mlp():
    return [("gate", 11008, 4096), ("up", 11008, 4096), ("down", 4096, 11008)]


def _llama8b_layer():
    return [("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096),
            ("o", 4096, 4096), ("gate", 14336, 4096), ("up", 14336, 4096),
            ("down", 4096, 14336)]


def _llama70b_layer():
    return [("q", 8192, 8192), ("k", 1024, 8192), ("v", 1024, 8192),
            ("o", 8192, 8192), ("gate", 28672, 8192), ("up", 28672, 8192),
            ("down", 8192, 28672)]


# Workloads: 1 = one 1024x1024 matrix, 2 = one 4096x4096 projection with
# per-row scales, 3 = a 7B-shaped MLP triple, 4 = one 8B-shaped decoder layer
# with per-matrix scale, 5 = an 80-layer 70B-shaped stack.
WORKLOADS = {
    1: dict(batches=(1,), x_dtype="f32", layers=1),
    2: dict(batches=(1, 4), x_dtype="bf16", layers=1),
    3: dict(batches=(1, 4, 16), x_dtype="bf16", layers=1),
    4: dict(batches=tuple(range(1, 17)), x_dtype="bf16", layers=1),
    5: dict(batches=(1,), x_dtype="bf16", layers=80),
}


def workload_matrices(cfg: int, layer: int = 0) -> List[MatrixSpec]:
    if cfg == 1:
        return [MatrixSpec(1, 0, 0, "w", 1024, 1024)]
    if cfg == 2:
        return [MatrixSpec(2, 0, 0, "q", 4096, 4096, row_scale=True)]
    if cfg == 3:
        return [MatrixSpec(3, 0, i, n, r, c) for i, (n, r, c) in enumerate(_llama7b_mlp())]
    if cfg == 4:
        return [MatrixSpec(4, 0, i, n, r, c, layer_scale=True)
                for i, (n, r, c) in enumerate(_llama8b_layer())]
    if cfg == 5:
        return [MatrixSpec(5, layer, i, n, r, c) for i, (n, r, c) in enumerate(_llama70b_layer())]
    raise ValueError(f"unknown workload {cfg}")


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits.

    Finite inputs only (the generator never produces Inf/NaN)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f16_bits(b: np.ndarray) -> np.ndarray:
    """The float16 copy of bf16 weights (float16 rounding, nearest-even): the
    FP16 release of a model trained in bf16. Returns uint16 bits."""
    return bf16_bits_to_f32(b).astype(np.float16).view(np.uint16)


ROW_BLOCK = 256


def _stream(spec: MatrixSpec, k: int, block: Optional[int] = None) -> np.random.Generator:
    key = [0, spec.cfg, spec.layer, spec.index, k]
    return np.random.default_rng(key if block is None else key + [block])


def _row_block(spec: MatrixSpec, b: int, std: np.float32, scale: Optional[np.ndarray]) -> np.ndarray:
    """Rows [b*ROW_BLOCK, min(rows, (b+1)*ROW_BLOCK)) as float32."""
    R, K = spec.rows, spec.cols
    n = min(R, (b + 1) * ROW_BLOCK) - b * ROW_BLOCK
    w = _stream(spec, 0, b).standard_normal(n * K, dtype=np.float32) * std
    mask = _stream(spec, 2, b).random(n * K, dtype=np.float32) < OUTLIER_P
    w[mask] *= np.float32(OUTLIER_MUL)
    w = w.reshape(n, K)
    if scale is not None:
        w *= scale[b * ROW_BLOCK:b * ROW_BLOCK + n, None]
    return w


def gen_matrix(spec: MatrixSpec, rows: Optional[slice] = None, threads: int = 0) -> np.ndarray:
    """bf16 bit patterns (uint16, shape [rows, cols]) of one matrix.

    ``rows`` selects a contiguous row range; the values equal the same rows of
    the full matrix (workload 1 is always drawn whole). Row blocks are drawn on
    ``threads`` threads (0: all cores); the result does not depend on it."""
    R, K = spec.rows, spec.cols
    if spec.cfg == 1:
        rng = np.random.default_rng(0)
        w = rng.standard_normal((R, K), dtype=np.float32) * np.float32(BASE_STD)
        mask = rng.random((R, K), dtype=np.float32) < OUTLIER_P
        w[mask] *= np.float32(OUTLIER_MUL)
        out = f32_to_bf16_bits(w)
        return out if rows is None else out[rows]
    r0, r1 = (0, R) if rows is None else (rows.start or 0, rows.stop if rows.stop is not None else R)
    std = np.float32(BASE_STD)
    if spec.layer_scale:
        u = _stream(spec, 3).uniform(1.0, 4.0)
        std = np.float32(BASE_STD / np.sqrt(u))
    scale = None
    if spec.row_scale:
        z = _stream(spec, 3).standard_normal(R, dtype=np.float32)
        scale = np.exp(np.float32(0.3) * z).astype(np.float32)
    out = np.empty((r1 - r0, K), dtype=np.uint16)
    b0, b1 = r0 // ROW_BLOCK, (r1 + ROW_BLOCK - 1) // ROW_BLOCK

    def one(b):
        lo = b * ROW_BLOCK
        w = _row_block(spec, b, std, scale)
        a, e = max(r0, lo), min(r1, lo + w.shape[0])
        out[a - r0:e - r0] = f32_to_bf16_bits(w[a - lo:e - lo])

    nt = threads or min(32, os.cpu_count() or 1)
    if nt <= 1 or b1 - b0 <= 1:
        for b in range(b0, b1):
            one(b)
    else:
        with ThreadPoolExecutor(nt) as ex:
            list(ex.map(one, range(b0, b1)))
    return out


def device_seed(spec: MatrixSpec) -> int:
    """63-bit seed of a matrix for gen_matrix_device, from (0, cfg, layer, matrix)."""
    key = np.random.SeedSequence([0, spec.cfg, spec.layer, spec.index, 9]).generate_state(2, np.uint32)
    return int(key[0]) | (int(key[1] & np.uint32(0x7FFFFFFF)) << 32)


def gen_matrix_device(spec: MatrixSpec, torch, device="cuda"):
    """The same distribution as gen_matrix, drawn on the GPU (torch's seeded
    Philox generator) for stacks too large to draw on the host in reasonable
    time: values N(0, std) (std as in gen_matrix), then an independent
    Bernoulli(0.001) mask from the same generator multiplying by 20, the
    per-row or per-matrix scales of gen_matrix (drawn on the host from the
    same streams), float32 -> bfloat16 round-to-nearest-even (torch's cast).
    Returns a bfloat16 tensor [rows, cols] on `device`. The values are
    deterministic for a given seed, torch version and device model; they
    differ from gen_matrix's (another generator)."""
    R, K = spec.rows, spec.cols
    g = torch.Generator(device=device)
    g.manual_seed(device_seed(spec))
    std = np.float32(BASE_STD)
    if spec.layer_scale:
        std = np.float32(BASE_STD / np.sqrt(_stream(spec, 3).uniform(1.0, 4.0)))
    w = torch.randn((R, K), generator=g, device=device, dtype=torch.float32)
    w.mul_(float(std))
    mask = torch.rand((R, K), generator=g, device=device, dtype=torch.float32) < OUTLIER_P
    w = torch.where(mask, w * np.float32(OUTLIER_MUL), w)
    del mask
    if spec.row_scale:
        z = _stream(spec, 3).standard_normal(R, dtype=np.float32)
        w.mul_(torch.from_numpy(np.exp(np.float32(0.3) * z).astype(np.float32)).to(device)[:, None])
    return w.to(torch.bfloat16)


def gen_x(spec: MatrixSpec, batch: int, dtype: str) -> np.ndarray:
    """Activation rows x[batch][cols]: float32, bf16 bits (uint16) if dtype ==
    'bf16', or float16 values if dtype == 'f16'."""
    if spec.cfg == 1:
        rng = np.random.default_rng(0)
        rng.standard_normal((spec.rows, spec.cols), dtype=np.float32)
        rng.random((spec.rows, spec.cols), dtype=np.float32)
        x = rng.standard_normal((batch, spec.cols), dtype=np.float32)
    else:
        x = _stream(spec, 1).standard_normal((batch, spec.cols), dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return x.astype(np.float16)
    raise ValueError(dtype)


def random_bf16(shape, seed: int, std: float = BASE_STD, outliers: bool = True) -> np.ndarray:
    """Small seeded bf16 matrix of the same distribution, for tests of any shape."""
    rng = np.random.default_rng([7, seed])
    w = rng.standard_normal(shape, dtype=np.float32) * np.float32(std)
    if outliers:
        mask = rng.random(shape, dtype=np.float32) < OUTLIER_P
        w[mask] *= np.float32(OUTLIER_MUL)
    return f32_to_bf16_bits(w)


def random_fp16(shape, seed: int, std: float = BASE_STD, outliers: bool = True) -> np.ndarray:
    """FP16 bits of random_bf16's matrix (see bf16_bits_to_f16_bits)."""
    return bf16_bits_to_f16_bits(random_bf16(shape, seed, std, outliers))


def random_x(batch: int, cols: int, seed: int, dtype: str = "f32") -> np.ndarray:
    """float32, bf16 bits (uint16) or float16 values."""
    rng = np.random.default_rng([8, seed])
    x = rng.standard_normal((batch, cols), dtype=np.float32)
    if dtype == "f16":
        return x.astype(np.float16)
    return x if dtype == "f32" else f32_to_bf16_bits(x)
