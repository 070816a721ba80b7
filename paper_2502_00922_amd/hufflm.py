"""ctypes binding of libhufflm.so (argument marshalling only).

Every step of the codec runs in the library: the host encoder in C++, decoding
and the fused decode-GEMV in gfx950 kernels. PyTorch only provides device
memory and the current HIP stream. There is no fallback: if the library is
missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhufflm.so")

HL_OK, HL_EINVAL, HL_ENOMEM, HL_ECORRUPT, HL_EUNSUPPORTED, HL_EHIP = range(6)
HL_F32, HL_BF16, HL_F16 = 0, 1, 2
HL_FORMAT_SPLIT, HL_FORMAT_WHOLE_EXPONENT, HL_FORMAT_FP16 = 0, 1, 2
HEADER_BYTES = 128
LUT_BYTES = 49440
MAX_BATCH = 16


class HLError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} ({status})")


class FieldCode(ctypes.Structure):
    _fields_ = [("nsym", ctypes.c_uint8), ("single", ctypes.c_uint8), ("len", ctypes.c_uint8 * 16)]

    @property
    def lengths(self):
        return list(self.len)


class Codebook(ctypes.Structure):
    _fields_ = [("lmax", ctypes.c_uint32), ("eh", FieldCode), ("el", FieldCode)]


class Codebook8(ctypes.Structure):
    _fields_ = [("lmax", ctypes.c_uint32), ("nsym", ctypes.c_uint16), ("single", ctypes.c_uint8),
                ("reserved", ctypes.c_uint8), ("len", ctypes.c_uint8 * 256)]

    @property
    def lengths(self):
        return list(self.len)


class FieldCode5(ctypes.Structure):
    _fields_ = [("nsym", ctypes.c_uint8), ("single", ctypes.c_uint8), ("len", ctypes.c_uint8 * 32)]

    @property
    def lengths(self):
        return list(self.len)


class Codebook16(ctypes.Structure):
    _fields_ = [("lmax", ctypes.c_uint32), ("e", FieldCode5), ("mh", FieldCode5), ("ml", FieldCode5)]


class TensorView(ctypes.Structure):
    _fields_ = [("blob_dev", ctypes.c_void_p), ("lut_dev", ctypes.c_void_p),
                ("rows", ctypes.c_uint64), ("cols", ctypes.c_uint64), ("n_seg", ctypes.c_uint64),
                ("n_grp", ctypes.c_uint64), ("total_bytes", ctypes.c_uint64),
                ("off_seg_bits", ctypes.c_uint64), ("off_grp_off", ctypes.c_uint64),
                ("off_stream", ctypes.c_uint64), ("off_raw", ctypes.c_uint64),
                ("seg_len", ctypes.c_uint32), ("grp_rows", ctypes.c_uint32), ("lmax", ctypes.c_uint32),
                ("max_grp_units", ctypes.c_uint32), ("max_seg_bits", ctypes.c_uint32),
                ("format", ctypes.c_uint32),
                ("cb", Codebook), ("cb8", Codebook8), ("cb16", Codebook16)]


_lib = None

EXPORTS = ["hl_status_str", "hl_default_seg_len", "hl_default_grp_rows", "hl_build_codebook", "hl_encode",
           "hl_build_codebook8", "hl_encode8", "hl_build_codebook16", "hl_encode16", "hl_validate",
           "hl_tensor_view", "hl_tensor_prepare", "hl_decode", "hl_gemv_workspace_bytes",
           "hl_decode_gemv", "hl_decode_gemv_noalloc", "hl_decode_gemv_multi", "hl_gemm_workspace_bytes",
           "hl_decode_gemm",
           "hl_gemv_bf16"]


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2502_00922_amd/build.py")
    L = ctypes.CDLL(LIB_PATH)
    c = ctypes
    L.hl_status_str.restype = c.c_char_p
    L.hl_status_str.argtypes = [c.c_int]
    L.hl_default_seg_len.restype = c.c_uint32
    L.hl_default_seg_len.argtypes = [c.c_uint64]
    L.hl_default_grp_rows.restype = c.c_uint32
    L.hl_default_grp_rows.argtypes = [c.c_uint64, c.c_uint32]
    L.hl_build_codebook.restype = c.c_int
    L.hl_build_codebook.argtypes = [c.c_void_p, c.c_size_t, c.c_uint32, c.c_uint32, c.POINTER(Codebook)]
    L.hl_encode.restype = c.c_int
    L.hl_encode.argtypes = [c.c_void_p, c.c_uint64, c.c_uint64, c.POINTER(Codebook), c.c_uint32,
                            c.c_uint32, c.c_uint32, c.c_void_p, c.POINTER(c.c_size_t)]
    L.hl_build_codebook8.restype = c.c_int
    L.hl_build_codebook8.argtypes = [c.c_void_p, c.c_size_t, c.c_uint32, c.POINTER(Codebook8)]
    L.hl_encode8.restype = c.c_int
    L.hl_encode8.argtypes = [c.c_void_p, c.c_uint64, c.c_uint64, c.POINTER(Codebook8), c.c_uint32,
                             c.c_uint32, c.c_uint32, c.c_void_p, c.POINTER(c.c_size_t)]
    L.hl_build_codebook16.restype = c.c_int
    L.hl_build_codebook16.argtypes = [c.c_void_p, c.c_size_t, c.c_uint32, c.POINTER(Codebook16)]
    L.hl_encode16.restype = c.c_int
    L.hl_encode16.argtypes = [c.c_void_p, c.c_uint64, c.c_uint64, c.POINTER(Codebook16), c.c_uint32,
                              c.c_uint32, c.c_uint32, c.c_void_p, c.POINTER(c.c_size_t)]
    L.hl_validate.restype = c.c_int
    L.hl_validate.argtypes = [c.c_void_p, c.c_size_t]
    L.hl_tensor_view.restype = c.c_int
    L.hl_tensor_view.argtypes = [c.c_void_p, c.c_void_p, c.c_size_t, c.c_void_p, c.POINTER(TensorView)]
    L.hl_tensor_prepare.restype = c.c_int
    L.hl_tensor_prepare.argtypes = [c.POINTER(TensorView), c.c_void_p]
    L.hl_decode.restype = c.c_int
    L.hl_decode.argtypes = [c.POINTER(TensorView), c.c_void_p, c.c_void_p]
    L.hl_gemv_workspace_bytes.restype = c.c_size_t
    L.hl_gemv_workspace_bytes.argtypes = [c.POINTER(TensorView), c.c_uint32]
    L.hl_decode_gemv.restype = c.c_int
    L.hl_decode_gemv.argtypes = [c.POINTER(TensorView), c.c_void_p, c.c_int, c.c_uint32, c.c_void_p,
                                 c.c_void_p, c.c_size_t, c.c_void_p]
    L.hl_decode_gemv_noalloc.restype = c.c_int
    L.hl_decode_gemv_noalloc.argtypes = [c.POINTER(TensorView), c.c_void_p, c.c_int, c.c_uint32, c.c_void_p,
                                         c.c_void_p]
    L.hl_decode_gemv_multi.restype = c.c_int
    L.hl_decode_gemv_multi.argtypes = [c.c_void_p, c.c_uint32, c.c_void_p, c.c_int, c.c_uint32, c.c_void_p,
                                       c.c_void_p, c.c_size_t, c.c_void_p]
    L.hl_gemm_workspace_bytes.restype = c.c_size_t
    L.hl_gemm_workspace_bytes.argtypes = [c.POINTER(TensorView), c.c_uint32]
    L.hl_decode_gemm.restype = c.c_int
    L.hl_decode_gemm.argtypes = [c.POINTER(TensorView), c.c_void_p, c.c_int, c.c_uint32, c.c_void_p,
                                 c.c_void_p, c.c_size_t, c.c_void_p]
    L.hl_gemv_bf16.restype = c.c_int
    L.hl_gemv_bf16.argtypes = [c.c_void_p, c.c_uint64, c.c_uint64, c.c_void_p, c.c_int, c.c_uint32,
                               c.c_void_p, c.c_void_p]
    _lib = L
    return L


def status_str(s: int) -> str:
    return lib().hl_status_str(s).decode()


def _check(s: int, where: str) -> None:
    if s != HL_OK:
        raise HLError(s, where)


def default_seg_len(cols: int) -> int:
    return int(lib().hl_default_seg_len(cols))


PAIR_MAX = 11  # default joint limit of a weight's two exponent codes (the fused kernel's table window)


def build_codebook(w: np.ndarray, lmax: int = 12, pair_max: int = PAIR_MAX) -> Codebook:
    """Codes of the two exponent fields: each at most lmax bits, the pair at
    most pair_max bits (0: no joint limit)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    cb = Codebook()
    _check(lib().hl_build_codebook(w.ctypes.data, w.size, lmax, pair_max, ctypes.byref(cb)), "hl_build_codebook")
    return cb


def build_codebook8(w: np.ndarray, lmax: int = 12) -> Codebook8:
    """Whole-exponent code: one 256-symbol code over the exponent bytes."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    cb = Codebook8()
    _check(lib().hl_build_codebook8(w.ctypes.data, w.size, lmax, ctypes.byref(cb)), "hl_build_codebook8")
    return cb


def build_codebook16(w: np.ndarray, lmax: int = 12) -> Codebook16:
    """Float16 codes: one 32-symbol code per 5-bit field (exponent, mantissa halves)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    cb = Codebook16()
    _check(lib().hl_build_codebook16(w.ctypes.data, w.size, lmax, ctypes.byref(cb)), "hl_build_codebook16")
    return cb


def default_grp_rows(cols: int, seg_len: int = 0) -> int:
    return int(lib().hl_default_grp_rows(cols, seg_len))


def encode(w: np.ndarray, seg_len: int = 0, lmax: int = 12, codebook=None,
           nthreads: int = 0, grp_rows: int = 0, whole_exponent: bool = False, fp16: bool = False,
           pair_max: int = PAIR_MAX) -> np.ndarray:
    """HLF1 container (uint8 array) of a bf16 matrix given as uint16 bits [rows, cols].

    whole_exponent selects the format with one 256-symbol exponent code
    (``codebook`` then is a Codebook8); fp16 takes float16 bits and selects the
    {1,5,5,5} format (``codebook``: a Codebook16). pair_max (split format):
    joint limit of a weight's two exponent codes, 0 for none."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    if w.ndim != 2:
        raise ValueError("expected a 2-D matrix")
    L = lib()
    if fp16:
        cb = codebook if codebook is not None else build_codebook16(w, lmax)
        fn, name = L.hl_encode16, "hl_encode16"
    elif whole_exponent:
        cb = codebook if codebook is not None else build_codebook8(w, lmax)
        fn, name = L.hl_encode8, "hl_encode8"
    else:
        cb = codebook if codebook is not None else build_codebook(w, lmax, pair_max)
        fn, name = L.hl_encode, "hl_encode"
    n = ctypes.c_size_t(0)
    _check(fn(w.ctypes.data, w.shape[0], w.shape[1], ctypes.byref(cb), seg_len, grp_rows, nthreads,
              None, ctypes.byref(n)), name + "(size)")
    out = np.empty(n.value, dtype=np.uint8)
    _check(fn(w.ctypes.data, w.shape[0], w.shape[1], ctypes.byref(cb), seg_len, grp_rows, nthreads,
              out.ctypes.data, ctypes.byref(n)), name)
    return out


def validate(blob) -> int:
    b = np.frombuffer(blob, dtype=np.uint8) if not isinstance(blob, np.ndarray) else blob
    b = np.ascontiguousarray(b)
    return int(lib().hl_validate(b.ctypes.data, b.size))


def _stream_ptr(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev_arg(t, name: str, dtypes=None, shape=None, numel: int = 0):
    """Checks a device buffer's dtype, shape (or at least `numel` elements)
    and contiguity before it reaches a kernel. The C ABI takes no sizes for
    these buffers, so a wrong one would be read or written out of bounds on
    the device; raises ValueError instead."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype} not in {tuple(dtypes)}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {numel} needed")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _on_device(device, **bufs):
    """Every given buffer lives on `device`, a GPU (else ValueError): a host
    pointer would reach the kernel as a device address."""
    for name, t in bufs.items():
        if t is None or t is False:
            continue
        if not t.is_cuda or (device is not None and t.device != device):
            raise ValueError(f"{name} must be on {device if device is not None else 'the GPU'}, not {t.device}")


def _x_dtype(x):
    import torch
    dt = {torch.float32: HL_F32, torch.bfloat16: HL_BF16, torch.float16: HL_F16}.get(x.dtype)
    if dt is None:
        raise ValueError("x must be float32, bfloat16 or float16")
    return dt


def _check_x(x, K: int):
    """x as a [batch, K] tensor of a supported dtype, batch in 1..16."""
    import torch
    if x.dim() == 1:
        x = x.unsqueeze(0)
    if x.dim() != 2 or x.shape[1] != K or not 1 <= x.shape[0] <= MAX_BATCH:
        raise ValueError(f"x must be [batch <= {MAX_BATCH}, {K}], got {tuple(x.shape)}")
    _dev_arg(x, "x", (torch.float32, torch.bfloat16, torch.float16))
    return x


def _check_ws(ws):
    if ws is False or ws is None:
        return ws
    return _dev_arg(ws, "workspace")


class DeviceTensor:
    """A container resident in device memory plus its decode table."""

    def __init__(self, blob: np.ndarray, device="cuda", stream=None):
        import torch
        blob = np.ascontiguousarray(blob, dtype=np.uint8)
        self.blob = torch.from_numpy(blob).to(device)
        self.lut = torch.empty(LUT_BYTES // 4, dtype=torch.int32, device=device)
        self.view = TensorView()
        _check(lib().hl_tensor_view(ctypes.c_void_p(self.blob.data_ptr()), blob.ctypes.data, blob.size,
                                    ctypes.c_void_p(self.lut.data_ptr()), ctypes.byref(self.view)),
               "hl_tensor_view")
        _check(lib().hl_tensor_prepare(ctypes.byref(self.view), _stream_ptr(stream)), "hl_tensor_prepare")

    def copy(self):
        """Another resident copy of the same container and table (device to
        device; the host-side validation of the container is not repeated)."""
        t = DeviceTensor.__new__(DeviceTensor)
        t.blob = self.blob.clone()
        t.lut = self.lut.clone()
        t.view = TensorView.from_buffer_copy(self.view)
        t.view.blob_dev = t.blob.data_ptr()
        t.view.lut_dev = t.lut.data_ptr()
        return t

    @property
    def shape(self):
        return int(self.view.rows), int(self.view.cols)

    @property
    def nbytes(self) -> int:
        return int(self.view.total_bytes)

    def decode(self, out=None, stream=None):
        """Weight bit patterns (bf16, or float16 for the float16 format) as a torch.int16 tensor [rows, cols] on the device."""
        import torch
        R, K = self.shape
        if out is None:
            out = torch.empty((R, K), dtype=torch.int16, device=self.blob.device)
        _dev_arg(out, "out", (torch.int16, torch.bfloat16, torch.float16), numel=R * K)
        _on_device(self.blob.device, out=out)
        _check(lib().hl_decode(ctypes.byref(self.view), ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)),
               "hl_decode")
        return out

    def workspace(self, batch: int = MAX_BATCH):
        """Zeroed device workspace for gemv at up to ``batch`` rows (cached)."""
        import torch
        need = int(lib().hl_gemv_workspace_bytes(ctypes.byref(self.view), batch))
        ws = getattr(self, "_ws", None)
        if ws is None or ws.numel() < need:
            ws = torch.zeros(max(need, 4), dtype=torch.uint8, device=self.blob.device)
            self._ws = ws
        return ws

    def gemv(self, x, y=None, stream=None, workspace=None):
        """y[b, r] = sum_k W[r, k] x[b, k]; x: [batch, cols] float32 or bfloat16 (device).

        ``workspace`` defaults to a cached zeroed buffer owned by this tensor;
        pass False to run without one."""
        import torch
        R, K = self.shape
        dev = self.blob.device
        x = _check_x(x, K)
        dt = _x_dtype(x)
        if y is None:
            y = torch.empty((x.shape[0], R), dtype=torch.float32, device=x.device)
        _dev_arg(y, "y", (torch.float32,), numel=x.shape[0] * R)
        _check_ws(workspace)
        _on_device(dev, x=x, y=y, workspace=workspace)
        if workspace is None:
            workspace = self.workspace()
        ws_ptr, ws_n = (None, 0) if workspace is False else (ctypes.c_void_p(workspace.data_ptr()),
                                                              workspace.numel() * workspace.element_size())
        _check(lib().hl_decode_gemv(ctypes.byref(self.view), ctypes.c_void_p(x.data_ptr()), dt, x.shape[0],
                                    ctypes.c_void_p(y.data_ptr()), ws_ptr, ws_n, _stream_ptr(stream)),
               "hl_decode_gemv")
        return y

    def gemv_noalloc(self, x, y, stream=None):
        """The product of gemv without a workspace (hl_decode_gemv_noalloc):
        the library's per-GPU scratch holds the partial sums. y must be given."""
        import torch
        R, K = self.shape
        x = _check_x(x, K)
        _dev_arg(y, "y", (torch.float32,), numel=x.shape[0] * R)
        _on_device(self.blob.device, x=x, y=y)
        _check(lib().hl_decode_gemv_noalloc(ctypes.byref(self.view), ctypes.c_void_p(x.data_ptr()), _x_dtype(x),
                                            x.shape[0], ctypes.c_void_p(y.data_ptr()), _stream_ptr(stream)),
               "hl_decode_gemv_noalloc")
        return y

    def gemm(self, x, y=None, stream=None):
        """Y[n, r] = sum_k W[r, k] X[n, k]; X: [tokens, cols] bfloat16 (device).
        Uses a cached zeroed workspace owned by the tensor, grown as needed."""
        import torch
        R, K = self.shape
        dev = self.blob.device
        if x.dim() != 2 or x.shape[1] != K or x.shape[0] < 1:
            raise ValueError(f"x must be [tokens, {K}], got {tuple(x.shape)}")
        _dev_arg(x, "x", (torch.bfloat16,))
        T = x.shape[0]
        if y is None:
            y = torch.empty((T, R), dtype=torch.float32, device=x.device)
        _dev_arg(y, "y", (torch.float32,), numel=T * R)
        _on_device(dev, x=x, y=y)
        need = int(lib().hl_gemm_workspace_bytes(ctypes.byref(self.view), T))
        ws = getattr(self, "_gemm_ws", None)
        if ws is None or ws.numel() < need:
            ws = torch.zeros(max(need, 4), dtype=torch.uint8, device=self.blob.device)
            self._gemm_ws = ws
        _check(lib().hl_decode_gemm(ctypes.byref(self.view), ctypes.c_void_p(x.data_ptr()), HL_BF16, T,
                                    ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                                    _stream_ptr(stream)), "hl_decode_gemm")
        return y


def gemv_multi(tensors, x, ys=None, stream=None, workspace=None):
    """ys[m][b, r] = sum_k W_m[r, k] x[b, k] for up to 4 DeviceTensors with the
    same columns that share x (one grouped launch where the library can).

    ``workspace`` defaults to the largest of the tensors' cached workspaces;
    pass False to run without one."""
    import torch
    if not 1 <= len(tensors) <= 4:
        raise ValueError("one to four tensors")
    K = tensors[0].shape[1]
    dev = tensors[0].blob.device
    if any(t.shape[1] != K or t.blob.device != dev for t in tensors):
        raise ValueError("the tensors must have the same columns and device")
    x = _check_x(x, K)
    dt = _x_dtype(x)
    if ys is None:
        ys = [torch.empty((x.shape[0], t.shape[0]), dtype=torch.float32, device=x.device) for t in tensors]
    if len(ys) != len(tensors):
        raise ValueError("one output per tensor")
    for m, (t, y) in enumerate(zip(tensors, ys)):
        _dev_arg(y, f"ys[{m}]", (torch.float32,), numel=x.shape[0] * t.shape[0])
    _check_ws(workspace)
    _on_device(dev, x=x, workspace=workspace, **{f"ys[{m}]": y for m, y in enumerate(ys)})
    if workspace is None:
        workspace = max((t.workspace() for t in tensors), key=lambda w: w.numel())
    ws_ptr, ws_n = (None, 0) if workspace is False else (ctypes.c_void_p(workspace.data_ptr()),
                                                          workspace.numel() * workspace.element_size())
    views = (ctypes.POINTER(TensorView) * len(tensors))(*[ctypes.pointer(t.view) for t in tensors])
    outs = (ctypes.c_void_p * len(tensors))(*[y.data_ptr() for y in ys])
    _check(lib().hl_decode_gemv_multi(ctypes.cast(views, ctypes.c_void_p), len(tensors),
                                      ctypes.c_void_p(x.data_ptr()), dt, x.shape[0],
                                      ctypes.cast(outs, ctypes.c_void_p), ws_ptr, ws_n, _stream_ptr(stream)),
           "hl_decode_gemv_multi")
    return ys


def gemv_bf16(w, x, y=None, stream=None):
    """Uncompressed comparator: w [rows, cols] bf16 (or int16 bits) on the device."""
    import torch
    if w.dim() != 2:
        raise ValueError("w must be [rows, cols]")
    R, K = w.shape
    _dev_arg(w, "w", (torch.bfloat16, torch.int16))
    x = _check_x(x, K)
    if x.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("x must be float32 or bfloat16")
    dt = _x_dtype(x)
    if y is None:
        y = torch.empty((x.shape[0], R), dtype=torch.float32, device=x.device)
    _dev_arg(y, "y", (torch.float32,), numel=x.shape[0] * R)
    _on_device(w.device if w.is_cuda else None, w=w, x=x, y=y)
    _check(lib().hl_gemv_bf16(ctypes.c_void_p(w.data_ptr()), R, K, ctypes.c_void_p(x.data_ptr()), dt,
                              x.shape[0], ctypes.c_void_p(y.data_ptr()), _stream_ptr(stream)), "hl_gemv_bf16")
    return y
