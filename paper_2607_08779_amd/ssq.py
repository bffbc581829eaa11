"""Thin Python binding of libssq's C ABI (argument marshalling only).

Every step of the quantize / matmul path runs in the HIP kernels behind
``libssq.so``; this module only checks tensor dtypes and shapes, allocates
output tensors with torch and passes device pointers and the current stream.
It fails loudly if the library has not been built: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

SIGNED_SYM, UNSIGNED_SYM, ASYM = 0, 1, 2
ASYM_MIN = 3    # min-max grid in the fp16-minimum layout (the ssq_*_min entry points)
MODES = {"signed_sym": SIGNED_SYM, "unsigned_sym": UNSIGNED_SYM, "asym": ASYM, "asym_min": ASYM_MIN}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libssq.so")

_EXPORTS = {
    "ssq_quantize": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p]),
    "ssq_quantize_f32": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p]),
    "ssq_matmul": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                  ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
    "ssq_matmul_f32": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                      ctypes.c_void_p]),
    "ssq_matmul_workspace_size": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                                     ctypes.c_int, ctypes.c_int]),
    "ssq_matmul_ws": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_size_t, ctypes.c_void_p]),
    "ssq_strerror": (ctypes.c_char_p, [ctypes.c_int]),
}
_EXPORTS["ssq_matmul_noalloc"] = _EXPORTS["ssq_matmul"]
_Q_MIN = (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p])
_EXPORTS["ssq_quantize_min"] = _Q_MIN
_EXPORTS["ssq_quantize_min_f32"] = _Q_MIN
for _name in ("ssq_matmul_min", "ssq_matmul_min_f32", "ssq_matmul_min_ws"):
    _EXPORTS[_name] = (ctypes.c_int, list(_EXPORTS[_name.replace("_min", "")][1]))
_EXPORTS["ssq_sign_diagnostics"] = _Q_MIN
_EXPORTS["ssq_sign_diagnostics_f32"] = _Q_MIN
_EXPORTS["ssq_quantize_diag"] = (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                                ctypes.c_int] + [ctypes.c_void_p] * 4)
_EXPORTS["ssq_quantize_diag_f32"] = _EXPORTS["ssq_quantize_diag"]
_EXPORTS["ssq_quantize_act_q8"] = (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p])
_EXPORTS["ssq_matmul_q8"] = (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p] + _EXPORTS["ssq_matmul"][1][1:])
_EXPORTS["ssq_matmul_q8_min"] = _EXPORTS["ssq_matmul_q8"]
_EXPORTS["ssq_export_gguf"] = (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                              ctypes.c_void_p])
_EXPORTS["ssq_gguf_block_bytes"] = (ctypes.c_int64, [ctypes.c_int, ctypes.c_int])

_lib: Optional[ctypes.CDLL] = None


class SSQError(RuntimeError):
    """A libssq call returned a non-zero ssq_status."""

    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {ssq_strerror(status)} (status {status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libssq.so (once) and declare its signatures; raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_08779_amd.build` (no fallback exists)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _EXPORTS.items():
            fn = getattr(handle, name)
            fn.restype, fn.argtypes = res, args
        _lib = handle
    return _lib


def ssq_strerror(status: int) -> str:
    return lib().ssq_strerror(int(status)).decode()


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    """Device address of a GPU tensor; a host tensor would hand a kernel a host pointer."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("ssq kernels take GPU tensors only (got a tensor on %s)" % t.device)
    return t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise SSQError(fn, status)


class _OnNullStream:
    """Orders a null-stream entry point (ssq_quantize*, the diagnostics) with the caller's
    current torch stream: the null stream waits for the work already queued on the
    current stream, and the current stream waits for the launch.  PyTorch's side streams
    are non-blocking, so without this a call inside ``torch.cuda.stream(s)`` could read
    W before s has written it, and s could read the outputs before they are written."""

    def __init__(self, device: torch.device):
        self.other = False
        if device.type == "cuda":        # a host tensor is refused by _ptr inside the block
            self.cur = torch.cuda.current_stream(device)
            self.null = torch.cuda.default_stream(device)
            self.other = self.cur.cuda_stream != self.null.cuda_stream

    def __enter__(self):
        if self.other:
            self.null.wait_stream(self.cur)
        return self

    def __exit__(self, *exc):
        if self.other:
            self.cur.wait_stream(self.null)
        return False


def ssq_quantize(W: torch.Tensor, group: int, q: int, mode: int,
                 out: Optional[Tuple[torch.Tensor, torch.Tensor, Optional[torch.Tensor]]] = None):
    """Quantize W [rows, cols] (bf16 or fp32, on the GPU) group-wise.

    Returns (codes u8 [rows, cols*q/8], scales int16 [rows, cols/group] holding
    binary16 bit patterns, zp u8 [rows, cols/group] for ASYM, the binary16 minimums
    as int16 [rows, cols/group] for ASYM_MIN, else None).
    Runs on the null stream, like the C entry point, ordered after the work queued on
    the current stream and before the work queued on it afterwards.
    """
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D tensor")
    if W.dtype == torch.bfloat16:
        fn = "ssq_quantize"
    elif W.dtype == torch.float32:
        fn = "ssq_quantize_f32"
    else:
        raise TypeError("W must be bfloat16 or float32")
    rows, cols = W.shape
    if out is None:
        codes = torch.empty((rows, cols * q // 8), dtype=torch.uint8, device=W.device)
        scales = torch.empty((rows, cols // group if group else 0), dtype=torch.int16, device=W.device)
        meta_dtype = {ASYM: torch.uint8, ASYM_MIN: torch.int16}.get(mode)
        zp = (torch.empty((rows, cols // group if group else 0), dtype=meta_dtype, device=W.device)
              if meta_dtype is not None else None)
    else:
        codes, scales, zp = out
    with _OnNullStream(W.device):
        if mode == ASYM_MIN:
            fn = fn.replace("ssq_quantize", "ssq_quantize_min")
            st = getattr(lib(), fn)(_ptr(W), rows, cols, group, q, _ptr(codes), _ptr(scales), _ptr(zp))
        else:
            st = getattr(lib(), fn)(_ptr(W), rows, cols, group, q, mode, _ptr(codes), _ptr(scales), _ptr(zp))
    _check(fn, st)
    return codes, scales, zp


def ssq_matmul_workspace_size(M: int, N: int, K: int, group: int, q: int) -> int:
    """Bytes of workspace that let ssq_matmul_ws split the reduction (0: no benefit)."""
    return int(lib().ssq_matmul_workspace_size(M, N, K, group, q))


def ssq_matmul_workspace(M: int, N: int, K: int, group: int, q: int,
                         device=None) -> Optional[torch.Tensor]:
    """A zero-filled workspace tensor for ssq_matmul(..., workspace=...), or None."""
    n = ssq_matmul_workspace_size(M, N, K, group, q)
    return torch.zeros(n, dtype=torch.uint8, device=device or "cuda") if n else None


def ssq_matmul(x: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor,
               zp: Optional[torch.Tensor], N: int, K: int, group: int, q: int,
               out: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y [M, N] = x [M, K] @ dequant(codes, scales, zp)^T on the current stream.

    x bf16 gives y bf16 (``ssq_matmul``, or ``ssq_matmul_ws`` when a workspace is
    given); x fp32 gives y fp32 (``ssq_matmul_f32``).  A ``zp`` of dtype int16
    holds binary16 minimums (the ASYM_MIN layout) and selects the ``*_min`` entry
    points; uint8 is the integer zero point; None the symmetric formats.
    """
    if x.dim() != 2 or not x.is_contiguous() or x.shape[1] != K:
        raise ValueError("x must be a contiguous [M, K] tensor")
    if x.dtype == torch.bfloat16:
        fn = "ssq_matmul"
    elif x.dtype == torch.float32:
        fn = "ssq_matmul_f32"
    else:
        raise TypeError("x must be bfloat16 or float32")
    if zp is not None and zp.dtype not in (torch.uint8, torch.int16):
        raise TypeError("zp must be uint8 zero points or int16 binary16 minimums")
    suffix = "_min" if zp is not None and zp.dtype == torch.int16 else ""
    M = x.shape[0]
    y = torch.empty((M, N), dtype=x.dtype, device=x.device) if out is None else out
    if workspace is not None and fn == "ssq_matmul":
        fn = "ssq_matmul" + suffix + "_ws"
        st = getattr(lib(), fn)(_ptr(x), M, _ptr(codes), _ptr(scales), _ptr(zp), N, K, group, q,
                                _ptr(y), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                _stream(x.device))
    else:
        fn = fn.replace("ssq_matmul", "ssq_matmul" + suffix)
        st = getattr(lib(), fn)(_ptr(x), M, _ptr(codes), _ptr(scales), _ptr(zp), N, K, group, q,
                                _ptr(y), _stream(x.device))
    _check(fn, st)
    return y


def ssq_matmul_noalloc(x: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor,
                       zp: Optional[torch.Tensor], N: int, K: int, group: int, q: int,
                       out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """ssq_matmul for bf16 x whose split reduction uses the library's static scratch
    (``ssq_matmul_noalloc``) instead of a workspace; symmetric or u8 zero-point weights.
    With ``out`` given, the call allocates nothing."""
    if x.dim() != 2 or not x.is_contiguous() or x.shape[1] != K or x.dtype != torch.bfloat16:
        raise ValueError("x must be a contiguous bfloat16 [M, K] tensor")
    if zp is not None and zp.dtype != torch.uint8:
        raise TypeError("zp must be uint8 zero points or None")
    M = x.shape[0]
    y = torch.empty((M, N), dtype=x.dtype, device=x.device) if out is None else out
    st = lib().ssq_matmul_noalloc(_ptr(x), M, _ptr(codes), _ptr(scales), _ptr(zp), N, K, group, q,
                                  _ptr(y), _stream(x.device))
    _check("ssq_matmul_noalloc", st)
    return y


def ssq_sign_diagnostics(W: torch.Tensor, group: int, q: int, tally: bool = True, out=None):
    """Sec. 4 Remark 1 statistics of the signed absmax grid for every group of W.

    Returns (margin int16 [rows, cols/group] = |C_{-g*}| - |C_{g*}|, gain float32
    [rows, cols/group] = realised l2 gain of gamma* over -gamma*, tally int64 [3, 3]
    of groups by (sign margin, sign gain) or None).  `out` = (margin, gain, tally[9] or
    None) reuses buffers.  Runs on the null stream.
    """
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D tensor")
    if W.dtype == torch.bfloat16:
        fn = "ssq_sign_diagnostics"
    elif W.dtype == torch.float32:
        fn = "ssq_sign_diagnostics_f32"
    else:
        raise TypeError("W must be bfloat16 or float32")
    rows, cols = W.shape
    shape = (rows, cols // group if group else 0)
    if out is not None:
        margin, gain, t = out
        if (margin.dtype != torch.int16 or gain.dtype != torch.float32 or tuple(margin.shape) != shape
                or tuple(gain.shape) != shape or not (margin.is_contiguous() and gain.is_contiguous())
                or (t is not None and (t.dtype != torch.int64 or t.numel() != 9))):
            raise ValueError("out must be (int16 margin, float32 gain) of shape rows x cols/group "
                             "and an int64 tally of 9 elements or None")
    else:
        margin = torch.empty(shape, dtype=torch.int16, device=W.device)
        gain = torch.empty(shape, dtype=torch.float32, device=W.device)
        t = torch.empty(9, dtype=torch.int64, device=W.device) if tally else None
    with _OnNullStream(W.device):
        st = getattr(lib(), fn)(_ptr(W), rows, cols, group, q, _ptr(margin), _ptr(gain), _ptr(t))
    _check(fn, st)
    return margin, gain, (t.view(3, 3) if t is not None else None)


def ssq_quantize_act_q8(x: torch.Tensor, out=None):
    """Dynamic Q8_0 quantization of bf16 activations x [M, K] (App. C) on the current
    stream: returns (codes int8 [M, K], scales int16 [M, K/32] holding binary16 bits).
    ``out`` = (codes, scales) reuses buffers."""
    if x.dim() != 2 or not x.is_contiguous() or x.dtype != torch.bfloat16:
        raise ValueError("x must be a contiguous bfloat16 [M, K] tensor")
    M, K = x.shape
    if out is None:
        qx = torch.empty((M, K), dtype=torch.int8, device=x.device)
        dx = torch.empty((M, K // 32), dtype=torch.int16, device=x.device)
    else:
        qx, dx = out
    _check("ssq_quantize_act_q8", lib().ssq_quantize_act_q8(_ptr(x), M, K, _ptr(qx), _ptr(dx), _stream(x.device)))
    return qx, dx


def ssq_matmul_q8(qx: torch.Tensor, dx: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor,
                  zp: Optional[torch.Tensor], N: int, K: int, group: int, q: int,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y [M, N] bf16 from Q8_0 activations (``ssq_quantize_act_q8``) and packed weights
    by integer dot products (App. B.3), on the current stream.  ``zp``: None
    (symmetric), uint8 zero points, or int16 binary16 minimums (``ssq_matmul_q8_min``)."""
    if qx.dim() != 2 or not qx.is_contiguous() or qx.dtype != torch.int8 or qx.shape[1] != K:
        raise ValueError("qx must be a contiguous int8 [M, K] tensor")
    if zp is not None and zp.dtype not in (torch.uint8, torch.int16):
        raise TypeError("zp must be uint8 zero points or int16 binary16 minimums")
    fn = "ssq_matmul_q8_min" if zp is not None and zp.dtype == torch.int16 else "ssq_matmul_q8"
    M = qx.shape[0]
    y = torch.empty((M, N), dtype=torch.bfloat16, device=qx.device) if out is None else out
    st = getattr(lib(), fn)(_ptr(qx), _ptr(dx), M, _ptr(codes), _ptr(scales), _ptr(zp), N, K, group, q,
                            _ptr(y), _stream(qx.device))
    _check(fn, st)
    return y


def ssq_export_gguf(codes: torch.Tensor, scales: torch.Tensor, mins: Optional[torch.Tensor], rows: int,
                    cols: int, group: int, q: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The packed weights as GGUF blocks (uint8 [rows, cols/32, block bytes]: Q4_0/Q4_0s,
    Q4_1, Q2_0/Q2_0s or Q2_1 by q and whether ``mins`` is given), on the current stream."""
    if mins is not None and mins.dtype != torch.int16:
        raise TypeError("mins must be int16 binary16 minimums (ssq_quantize_min)")
    nbytes = int(lib().ssq_gguf_block_bytes(q, int(mins is not None)))
    if out is None:
        out = torch.empty((rows, cols // 32, max(nbytes, 1)), dtype=torch.uint8, device=codes.device)
    _check("ssq_export_gguf", lib().ssq_export_gguf(_ptr(codes), _ptr(scales), _ptr(mins), rows, cols, group, q,
                                                    _ptr(out), _stream(codes.device)))
    return out


def ssq_quantize_diag(W: torch.Tensor, group: int, q: int):
    """Signed-symmetric quantization fused with the sign-rule statistics (Sec. 4
    Remark 1): returns (codes, scales, margin int16, gain float32) in one pass over W,
    on the null stream."""
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D tensor")
    if W.dtype == torch.bfloat16:
        fn = "ssq_quantize_diag"
    elif W.dtype == torch.float32:
        fn = "ssq_quantize_diag_f32"
    else:
        raise TypeError("W must be bfloat16 or float32")
    rows, cols = W.shape
    groups = cols // group if group else 0
    codes = torch.empty((rows, cols * q // 8), dtype=torch.uint8, device=W.device)
    scales = torch.empty((rows, groups), dtype=torch.int16, device=W.device)
    margin = torch.empty((rows, groups), dtype=torch.int16, device=W.device)
    gain = torch.empty((rows, groups), dtype=torch.float32, device=W.device)
    with _OnNullStream(W.device):
        st = getattr(lib(), fn)(_ptr(W), rows, cols, group, q, _ptr(codes), _ptr(scales), _ptr(margin), _ptr(gain))
    _check(fn, st)
    return codes, scales, margin, gain
