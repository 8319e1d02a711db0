"""Python binding of ``liblutgemm.so`` (LUT-based mixed-precision GEMM for gfx950).

Argument marshalling only: every step of the computation runs in the HIP kernels
behind the C ABI declared in ``include/lutgemm.h``.  PyTorch is used for device
memory and streams.  If the shared library has not been built, importing this
package raises ``ImportError`` -- there is no CPU fallback.

Low-level functions mirror the C entry points (``validate``, ``packed_weight_size``,
``table_size``, ``table_offsets``, ``workspace_size``, ``pack_weights``,
``precompute``, ``mpgemm``, ``fused_workspace_size``, ``mpgemm_fused``, ``dequant_workspace_size``, ``mpgemm_dequant``); ``LutGemm`` is a small holder that
allocates the packed weights, tables and workspace with torch and calls them.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

# Load PyTorch's HIP runtime before the library: liblutgemm.so needs
# libamdhip64.so.7, and the dynamic loader then binds it to the runtime already
# in the process, so torch's streams and allocations are valid in our calls.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblutgemm.so")

# enums of include/lutgemm.h
SUCCESS, ERROR_INVALID_VALUE, ERROR_NOT_SUPPORTED, ERROR_INSUFFICIENT_SIZE, ERROR_HIP = 0, 1, 2, 3, 4
WFMT_UINT, WFMT_BINARY, WFMT_TERNARY, WFMT_TERNARY_3IN5 = 0, 1, 2, 3
ACT_FP16, ACT_INT8, ACT_FP16_LUT8 = 0, 1, 2
OUT_FP16, OUT_FP32, OUT_INT32 = 0, 1, 2
WORKSPACE_ZERO_BYTES = 1 << 20  # LUTGEMM_WORKSPACE_ZERO_BYTES

EXPORTS = [
    "lutgemm_status_string", "lutgemm_version", "lutgemm_last_error", "lutgemm_validate", "lutgemm_packed_weight_size",
    "lutgemm_table_size", "lutgemm_table_offsets", "lutgemm_workspace_size", "lutgemm_pack_weights",
    "lutgemm_precompute", "lutgemm_mpgemm", "lutgemm_mpgemm_dequant", "lutgemm_dequant_workspace_size", "lutgemm_dequant_plan",
    "lutgemm_calibrate_stream_read",
    "lutgemm_fused_workspace_size", "lutgemm_mpgemm_fused", "lutgemm_calibrate_stream_read_ex",
    "lutgemm_set_tuning", "lutgemm_get_tuning", "lutgemm_mpgemm_noalloc",
]

# planner overrides (LUTGEMM_TUNE_*), for tests and experiments
TUNE = {"TARGET_BLOCKS": 0, "WHOLEK_MAX_KB": 1, "GEMV_KIND": 2, "GEMV_CFG": 3, "SPLITS": 4, "KBS": 5,
        "MT16": 6, "MT_TARGET": 7, "MT_SPLITS": 8, "MT_ORDER": 9, "DEQUANT_KIND": 10, "LOG": 11,
        "SPLIT_PRE": 12, "DEQUANT_SPLITS": 13, "MT_FUSED": 14, "MT4": 15, "SPLIT_EXACT": 16}


class Problem(ctypes.Structure):
    """``lutgemm_problem_t``."""
    _fields_ = [("K", ctypes.c_int64), ("N", ctypes.c_int64), ("w_bits", ctypes.c_int32),
                ("wfmt", ctypes.c_int32), ("group_size", ctypes.c_int32), ("scale_fp32", ctypes.c_int32),
                ("act", ctypes.c_int32), ("reserved", ctypes.c_int32)]

    def __repr__(self):
        return (f"Problem(K={self.K}, N={self.N}, w_bits={self.w_bits}, wfmt={self.wfmt}, "
                f"group_size={self.group_size}, scale_fp32={self.scale_fp32}, act={self.act})")


class LutGemmError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = f"{where}: {status_string(status)}"
        if status == ERROR_HIP:
            msg += f" [{lib.lutgemm_last_error().decode()}]"
        super().__init__(msg)
        self.status = status


def _load(path: str = LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() "
                          "(or python paper_2408_06003_amd/build.py) first")
    L = ctypes.CDLL(path)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    PP = ctypes.POINTER(Problem)
    L.lutgemm_status_string.restype = ctypes.c_char_p
    L.lutgemm_status_string.argtypes = [ctypes.c_int]
    L.lutgemm_version.restype = ctypes.c_char_p
    L.lutgemm_version.argtypes = []
    L.lutgemm_last_error.restype = ctypes.c_char_p
    L.lutgemm_last_error.argtypes = []
    L.lutgemm_validate.restype = ctypes.c_int
    L.lutgemm_validate.argtypes = [PP, I64]
    L.lutgemm_packed_weight_size.restype = SZ
    L.lutgemm_packed_weight_size.argtypes = [PP]
    L.lutgemm_table_size.restype = SZ
    L.lutgemm_table_size.argtypes = [PP, I64]
    L.lutgemm_table_offsets.restype = ctypes.c_int
    L.lutgemm_table_offsets.argtypes = [PP, I64, ctypes.POINTER(SZ), ctypes.POINTER(SZ)]
    L.lutgemm_workspace_size.restype = SZ
    L.lutgemm_workspace_size.argtypes = [PP, I64]
    L.lutgemm_pack_weights.restype = ctypes.c_int
    L.lutgemm_pack_weights.argtypes = [PP, P, P, P, P, SZ, P]
    L.lutgemm_precompute.restype = ctypes.c_int
    L.lutgemm_precompute.argtypes = [PP, I64, P, P, SZ, P]
    L.lutgemm_mpgemm.restype = ctypes.c_int
    L.lutgemm_mpgemm.argtypes = [PP, I64, P, P, P, I32, I32, P, SZ, P]
    L.lutgemm_mpgemm_dequant.restype = ctypes.c_int
    L.lutgemm_mpgemm_dequant.argtypes = [PP, I64, P, P, P, I32, I32, P, SZ, P]
    L.lutgemm_dequant_workspace_size.restype = ctypes.c_size_t
    L.lutgemm_dequant_workspace_size.argtypes = [PP, I64]
    L.lutgemm_dequant_plan.restype = ctypes.c_int
    L.lutgemm_dequant_plan.argtypes = [PP, I64, ctypes.POINTER(I32), ctypes.POINTER(I32)]
    L.lutgemm_fused_workspace_size.restype = SZ
    L.lutgemm_fused_workspace_size.argtypes = [PP, I64]
    L.lutgemm_mpgemm_fused.restype = ctypes.c_int
    L.lutgemm_mpgemm_fused.argtypes = [PP, I64, P, P, P, I32, I32, P, SZ, P]
    L.lutgemm_calibrate_stream_read.restype = ctypes.c_int
    L.lutgemm_calibrate_stream_read.argtypes = [P, SZ, P, I32, P]
    L.lutgemm_mpgemm_noalloc.restype = ctypes.c_int
    L.lutgemm_mpgemm_noalloc.argtypes = [PP, I64, P, P, P, I32, I32, P]
    L.lutgemm_set_tuning.restype = ctypes.c_int
    L.lutgemm_set_tuning.argtypes = [I32, I32]
    L.lutgemm_get_tuning.restype = ctypes.c_int32
    L.lutgemm_get_tuning.argtypes = [I32]
    L.lutgemm_calibrate_stream_read_ex.restype = ctypes.c_int
    L.lutgemm_calibrate_stream_read_ex.argtypes = [P, SZ, P, I32, I32, I32, P]
    return L


lib = _load()


def status_string(status: int) -> str:
    return lib.lutgemm_status_string(int(status)).decode()


def version() -> str:
    return lib.lutgemm_version().decode()


def problem(K: int, N: int, w_bits: int, wfmt: int, group_size: int, act: int = ACT_FP16,
            scale_fp32: bool = False) -> Problem:
    return Problem(K, N, w_bits, wfmt, group_size, 1 if scale_fp32 else 0, act, 0)


def _ptr(x) -> Optional[int]:
    """Device (or host) address of a torch tensor, an int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != SUCCESS:
        raise LutGemmError(status, where)


def validate(p: Problem, M: int = 1) -> int:
    return lib.lutgemm_validate(ctypes.byref(p), M)


def packed_weight_size(p: Problem) -> int:
    return lib.lutgemm_packed_weight_size(ctypes.byref(p))


def table_size(p: Problem, M: int) -> int:
    return lib.lutgemm_table_size(ctypes.byref(p), M)


def table_offsets(p: Problem, M: int):
    s, t = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib.lutgemm_table_offsets(ctypes.byref(p), M, ctypes.byref(s), ctypes.byref(t)), "table_offsets")
    return s.value, t.value


def workspace_size(p: Problem, M: int) -> int:
    return lib.lutgemm_workspace_size(ctypes.byref(p), M)


def pack_weights(p: Problem, codes, scales, zeros, packed, stream=None, packed_bytes=None):
    nbytes = packed_bytes if packed_bytes is not None else packed.numel() * packed.element_size()
    _check(lib.lutgemm_pack_weights(ctypes.byref(p), _ptr(codes), _ptr(scales), _ptr(zeros), _ptr(packed),
                                    nbytes, _stream(stream)), "lutgemm_pack_weights")


def precompute(p: Problem, M: int, act, tables, stream=None, table_bytes=None):
    nbytes = table_bytes if table_bytes is not None else tables.numel() * tables.element_size()
    _check(lib.lutgemm_precompute(ctypes.byref(p), M, _ptr(act), _ptr(tables), nbytes, _stream(stream)),
           "lutgemm_precompute")


def mpgemm(p: Problem, M: int, tables, packed, out, out_dtype: int, accumulate: bool = False,
           workspace=None, stream=None, workspace_bytes=None):
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.lutgemm_mpgemm(ctypes.byref(p), M, _ptr(tables), _ptr(packed), _ptr(out), out_dtype,
                              1 if accumulate else 0, _ptr(workspace), workspace_bytes, _stream(stream)),
           "lutgemm_mpgemm")


def mpgemm_noalloc(p: Problem, M: int, tables, packed, out, out_dtype: int, accumulate: bool = False,
                   stream=None):
    """lutgemm_mpgemm with the library's static scratch array instead of a workspace."""
    _check(lib.lutgemm_mpgemm_noalloc(ctypes.byref(p), M, _ptr(tables), _ptr(packed), _ptr(out), out_dtype,
                                      1 if accumulate else 0, _stream(stream)), "lutgemm_mpgemm_noalloc")


def fused_workspace_size(p: Problem, M: int) -> int:
    return lib.lutgemm_fused_workspace_size(ctypes.byref(p), M)


def mpgemm_fused(p: Problem, M: int, act, packed, out, out_dtype: int, accumulate: bool = False,
                 workspace=None, stream=None, workspace_bytes=None):
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.lutgemm_mpgemm_fused(ctypes.byref(p), M, _ptr(act), _ptr(packed), _ptr(out), out_dtype,
                                    1 if accumulate else 0, _ptr(workspace), workspace_bytes, _stream(stream)),
           "lutgemm_mpgemm_fused")


def dequant_workspace_size(p: Problem, M: int) -> int:
    return lib.lutgemm_dequant_workspace_size(ctypes.byref(p), M)


def dequant_plan(p: Problem, M: int):
    """(kernel, splits) of the comparison path for M tokens: kernel 0 = 128x128 tiles,
    1 = pipelined 256x256 tiles, 2 = 16-token slabs."""
    k, s = ctypes.c_int32(), ctypes.c_int32()
    _check(lib.lutgemm_dequant_plan(ctypes.byref(p), M, ctypes.byref(k), ctypes.byref(s)), "lutgemm_dequant_plan")
    return k.value, s.value


def mpgemm_dequant(p: Problem, M: int, act, packed, out, out_dtype: int, accumulate: bool = False,
                   workspace=None, stream=None, workspace_bytes=None):
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.lutgemm_mpgemm_dequant(ctypes.byref(p), M, _ptr(act), _ptr(packed), _ptr(out), out_dtype,
                                      1 if accumulate else 0, _ptr(workspace), workspace_bytes,
                                      _stream(stream)), "lutgemm_mpgemm_dequant")


def calibrate_stream_read(src, nbytes: int, sink, blocks: int, stream=None):
    """Launch the streaming-read calibration kernel over ``nbytes`` of ``src``."""
    _check(lib.lutgemm_calibrate_stream_read(_ptr(src), nbytes, _ptr(sink), blocks, _stream(stream)),
           "lutgemm_calibrate_stream_read")


def set_tuning(name: str, value: int):
    """Planner override ``name`` (a key of ``TUNE``) to ``value`` (-1 restores its default)."""
    _check(lib.lutgemm_set_tuning(TUNE[name], int(value)), "lutgemm_set_tuning")


def get_tuning(name: str) -> int:
    return int(lib.lutgemm_get_tuning(TUNE[name]))


def calibrate_stream_read_ex(src, nbytes: int, sink, blocks: int, unroll: int = 4, flags: int = 0,
                             stream=None):
    """Streaming-read calibration with a chosen read pattern (unroll, nontemporal / contiguous flags)."""
    _check(lib.lutgemm_calibrate_stream_read_ex(_ptr(src), nbytes, _ptr(sink), blocks, unroll, flags,
                                                _stream(stream)), "lutgemm_calibrate_stream_read_ex")


class LutGemm:
    """Packed low-bit weights plus the buffers one mpGEMM call needs (torch allocations).

    ``codes``, ``scales``, ``zeros`` are device tensors in the layout of
    ``lutgemm_pack_weights``; packing is enqueued on the current stream.
    """

    def __init__(self, p: Problem, codes, scales, zeros=None, device="cuda"):
        import torch
        st = validate(p, 1)
        _check(st, "lutgemm_validate")
        self.p = p
        self.device = torch.device(device)
        self.packed = torch.empty(packed_weight_size(p), dtype=torch.uint8, device=self.device)
        pack_weights(p, codes, scales, zeros, self.packed)
        self._tables = {}
        self._ws = {}

    def tables(self, M: int):
        import torch
        if M not in self._tables:
            self._tables[M] = torch.empty(table_size(self.p, M), dtype=torch.uint8, device=self.device)
        return self._tables[M]

    def workspace(self, M: int):
        import torch
        n = workspace_size(self.p, M)
        if n == 0:
            return None
        if M not in self._ws or self._ws[M].numel() < n:  # (the size follows the tuning keys)
            self._ws[M] = torch.zeros(n, dtype=torch.uint8, device=self.device)
        return self._ws[M]

    def out_dtype_code(self, dtype) -> int:
        import torch
        return {torch.float16: OUT_FP16, torch.float32: OUT_FP32, torch.int32: OUT_INT32}[dtype]

    def __call__(self, act, out=None, out_dtype=None, accumulate=False, stream=None):
        """out[M, N] (=|+=) act[M, K] x W^T through precompute + LUT mpGEMM."""
        import torch
        M = act.shape[0]
        if out is None:
            out = torch.empty((M, self.p.N), dtype=out_dtype or torch.float16, device=self.device)
        t = self.tables(M)
        precompute(self.p, M, act, t, stream=stream)
        mpgemm(self.p, M, t, self.packed, out, self.out_dtype_code(out.dtype), accumulate,
               workspace=self.workspace(M), stream=stream)
        return out

    def fused_workspace(self, M: int):
        import torch
        n = fused_workspace_size(self.p, M)
        if n == 0:
            return None
        key = ("fused", M)
        if key not in self._ws or self._ws[key].numel() < n:
            self._ws[key] = torch.zeros(n, dtype=torch.uint8, device=self.device)
        return self._ws[key]

    def fused(self, act, out=None, out_dtype=None, accumulate=False, stream=None):
        """Same product through lutgemm_mpgemm_fused (tables built inside the LUT kernel)."""
        import torch
        M = act.shape[0]
        if out is None:
            out = torch.empty((M, self.p.N), dtype=out_dtype or torch.float16, device=self.device)
        mpgemm_fused(self.p, M, act, self.packed, out, self.out_dtype_code(out.dtype), accumulate,
                     workspace=self.fused_workspace(M), stream=stream)
        return out

    def dequant(self, act, out=None, out_dtype=None, accumulate=False, stream=None):
        """Comparison path: dequantize to FP16 + matrix cores."""
        import torch
        M = act.shape[0]
        if out is None:
            out = torch.empty((M, self.p.N), dtype=out_dtype or torch.float16, device=self.device)
        mpgemm_dequant(self.p, M, act, self.packed, out, self.out_dtype_code(out.dtype), accumulate,
                       workspace=self.dequant_workspace(M), stream=stream)
        return out

    def dequant_workspace(self, M: int):
        import torch
        n = dequant_workspace_size(self.p, M)
        if n == 0:
            return None
        key = ("dequant", M)
        if key not in self._ws or self._ws[key].numel() < n:
            self._ws[key] = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self._ws[key]
