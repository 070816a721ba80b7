"""MI355X-native Huff-LLM: lossless bf16 weight compression with decoding
fused into the decode-step GEMV on gfx950."""
from .hufflm import (HLError, Codebook, DeviceTensor, build_codebook, default_grp_rows, default_seg_len, encode,
                     gemv_bf16, gemv_multi, lib, status_str, validate)

__all__ = ["HLError", "Codebook", "DeviceTensor", "build_codebook", "default_grp_rows", "default_seg_len", "encode",
           "gemv_bf16", "gemv_multi", "lib", "status_str", "validate"]
