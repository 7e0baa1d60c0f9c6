"""ctypes binding of libfqvit (include/fqvit.h).

Argument marshalling only: each function checks dtypes, devices, shapes and
contiguity of torch tensors, passes their device pointers and the current HIP
stream to the C ABI entry point of the same name, and raises ``FqError`` on a
non-zero status.  Every step of the computation runs in the HIP kernels; there
is no fallback.  If libfqvit.so is not built the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfqvit.so")

(FQ_OK, FQ_ERR_NULL, FQ_ERR_SHAPE, FQ_ERR_PARAM, FQ_ERR_HEADROOM, FQ_ERR_HIP,
 FQ_ERR_SCRATCH) = range(7)
# Bytes of the library's fixed device scratch (FQ_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 8 << 20

# Entry points declared in include/fqvit.h and their C argument types.
_P = ctypes.c_void_p
_I32, _I64, _F32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
SIGNATURES = {
    "ptf_layernorm_int8": [_P, _I64, _I32, _I32, _P, _I32, _P, _P, _F32, _I32, _I32, _P, _P],
    "lis_softmax_log4": [_P, _I64, _I32, _I32, _P, _I32, _F32, _I32, _I32, _P, _I32, _P],
    "lis_attn_v_shift": [_P, _I32, _P, _I32, _I64, _I32, _I32, _I32, _I32, _P, _P],
    "lis_attn_v_shift_wide": [_P, _I32, _P, _I32, _I64, _I32, _I32, _I32, _I32, _P, _P],
    "lis_attention_head": [_P, _P, _I32, _I64, _I32, _I32, _F32, _I32, _I32, _P, _I32, _I32, _P,
                           _P, _I32, _P],
    "lis_attention_qk": [_P, _P, _I32, _I32, _I32, _P, _I32, _I64, _I32, _I32, _F32, _I32, _I32,
                         _P, _I32, _I32, _P, _P],
    "ptf_calibrate": [_P, _I64, _I32, _I32, _I32, _P, _P, _P, _P, ctypes.c_size_t, _P],
    "ptf_calibrate_noalloc": [_P, _I64, _I32, _I32, _I32, _P, _P, _P, _P],
    "ptf_quantize_int8": [_P, _I64, _I32, _P, _P, _P, _I32, _P, _P],
    "requant_dyadic_int8": [_P, _I64, _F32, _F32, _I32, _I32, _P, _P],
}


class FqError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {status_str(status)}")


_lib: Optional[ctypes.CDLL] = None


def load(path: str) -> ctypes.CDLL:
    """Open a build of libfqvit at `path` and declare its entry points' C types."""
    L = ctypes.CDLL(path)
    for name, args in SIGNATURES.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int32
    L.fq_status_str.argtypes = [ctypes.c_int]
    L.fq_status_str.restype = ctypes.c_char_p
    L.fq_version.argtypes = []
    L.fq_version.restype = ctypes.c_int32
    L.fq_time_next_call.argtypes = [_P, _P]
    L.fq_time_next_call.restype = ctypes.c_int32
    L.fq_ptf_calibrate_workspace_bytes.argtypes = [_I64, _I32, _I32]
    L.fq_ptf_calibrate_workspace_bytes.restype = ctypes.c_size_t
    return L


def lib() -> ctypes.CDLL:
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c "
                               f"'import __graft_entry__ as g; g.build()'` (no fallback exists)")
        _lib = load(LIB_PATH)
    return _lib


def status_str(status: int) -> str:
    return lib().fq_status_str(int(status)).decode()


def version() -> int:
    return lib().fq_version()


def time_next_call(start_event: int, stop_event: int) -> None:
    """Attach two hipEvent_t handles (ints) to the kernel of the next call on
    this thread: they record that kernel's own start and end."""
    lib().fq_time_next_call(start_event or None, stop_event or None)


def _stream(stream, like) -> int:
    """Raw hipStream_t: the given torch stream, else torch's current stream on
    the device of tensor `like` (read without creating a Stream object)."""
    if stream is not None:
        return stream.cuda_stream
    import torch
    return torch._C._cuda_getCurrentRawStream(like.device.index)


def _dev_ptr(t, dtype, name: str, ndim: Optional[int] = None):
    if t is None:
        return None
    try:
        ok = (t.dtype is dtype and t.is_cuda and (ndim is None or t.dim() == ndim)
              and t.is_contiguous())
    except AttributeError:
        raise TypeError(f"{name} must be a torch.Tensor") from None
    if not ok:
        if t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")
    return t.data_ptr()


def _check(fn: str, status: int) -> None:
    if status != FQ_OK:
        raise FqError(fn, status)


class Prepared:
    """A validated call with its arguments already converted to C types:
    calling it only enters the library (for launch loops where Python
    marshalling would otherwise dominate).  The stream is the one current when
    the call was prepared; the tensors are kept alive by the object."""

    __slots__ = ("_name", "_fn", "_args", "_keep")

    def __init__(self, name: str, args, keep):
        self._name = name
        self._fn = getattr(lib(), name)
        self._args = tuple(t(a) if a is not None else None
                           for t, a in zip(SIGNATURES[name], args))
        self._keep = keep

    def __call__(self) -> None:
        st = self._fn(*self._args)
        if st != FQ_OK:
            raise FqError(self._name, st)


def _invoke(name: str, args, keep, prepare: bool, result):
    """Run the entry point now, or return it prepared for repeated calls."""
    if prepare:
        return Prepared(name, args, keep)
    _check(name, getattr(lib(), name)(*args))
    return result


def ptf_layernorm_int8(x_q, zp_in: int, alpha, K: int, gamma, beta, s_out: float, zp_out: int,
                       bits: int = 8, y_q=None, stream=None, prepare: bool = False):
    """PTF LayerNorm of an int8 [T, C] tensor; returns (or fills) int8 [T, C].
    With prepare=True returns a Prepared call instead of running it."""
    import torch
    T, C = x_q.shape
    if y_q is None:
        y_q = torch.empty_like(x_q)
    if alpha.shape != (C,) or gamma.shape != (C,) or beta.shape != (C,) or y_q.shape != (T, C):
        raise ValueError("alpha, gamma, beta must be [C] and y_q [T, C]")
    args = (_dev_ptr(x_q, torch.int8, "x_q", 2), T, C, zp_in,
            _dev_ptr(alpha, torch.uint8, "alpha", 1), K,
            _dev_ptr(gamma, torch.float32, "gamma", 1),
            _dev_ptr(beta, torch.float32, "beta", 1), s_out, zp_out, bits,
            _dev_ptr(y_q, torch.int8, "y_q", 2), _stream(stream, x_q))
    return _invoke("ptf_layernorm_int8", args, (x_q, alpha, gamma, beta, y_q), prepare, y_q)


def codes_ld(Lk: int, bits: int = 4) -> int:
    """Bytes per row of stored codes: two per byte up to 4 bits, else one."""
    return (Lk + 1) // 2 if bits <= 4 else Lk


def lis_softmax_log4(logits, s_logit: float, bits: int = 4, exp_n: int = 20, bias=None,
                     codes=None, stream=None, prepare: bool = False):
    """Log-Int-Softmax codes [G, Lq, ld] of int32 logits [G, Lq, Lk]: packed two
    per byte for bits <= 4, one per byte for bits in [5, 8]."""
    import torch
    G, Lq, Lk = logits.shape
    if codes is None:
        codes = torch.zeros((G, Lq, codes_ld(Lk, bits)), dtype=torch.uint8, device=logits.device)
    if codes.dim() != 3 or codes.shape[:2] != (G, Lq):
        raise ValueError("codes must be [G, Lq, ld_codes]")
    Hb = 0
    if bias is not None:
        if bias.dim() != 3 or bias.shape[1:] != (Lq, Lk):
            raise ValueError("bias must be [Hb, Lq, Lk]")
        Hb = bias.shape[0]
    args = (_dev_ptr(logits, torch.int32, "logits", 3), G, Lq, Lk,
            _dev_ptr(bias, torch.int32, "bias", 3), Hb, s_logit, bits, exp_n,
            _dev_ptr(codes, torch.uint8, "codes", 3), codes.shape[2], _stream(stream, logits))
    return _invoke("lis_softmax_log4", args, (logits, bias, codes), prepare, codes)


def lis_attn_v_shift(codes, v, Lk: int, zp_v: int = 0, bits: int = 4, out=None, stream=None,
                     prepare: bool = False):
    """BitShift Attn x V: int32 [G, Lq, d] from packed codes [G, Lq, ld] and int8 V [G, Lk, d]."""
    import torch
    G, Lq, ld = codes.shape
    d = v.shape[2]
    if v.dim() != 3 or v.shape[:2] != (G, Lk):
        raise ValueError("v must be [G, Lk, d]")
    if out is None:
        out = torch.empty((G, Lq, d), dtype=torch.int32, device=v.device)
    if out.shape != (G, Lq, d):
        raise ValueError("out must be [G, Lq, d]")
    args = (_dev_ptr(codes, torch.uint8, "codes", 3), ld, _dev_ptr(v, torch.int8, "v", 3), zp_v,
            G, Lq, Lk, d, bits, _dev_ptr(out, torch.int32, "out", 3), _stream(stream, v))
    return _invoke("lis_attn_v_shift", args, (codes, v, out), prepare, out)


def lis_attn_v_shift_wide(codes, v, Lk: int, zp_v: int = 0, bits: int = 8, out=None, stream=None,
                          prepare: bool = False):
    """BitShift Attn x V for codes of any width b in [1, 8] (nibbles for b <= 4,
    bytes above): int64 [G, Lq, d] at scale s_V / 2^min(2^b - 1, 44)."""
    import torch
    G, Lq, ld = codes.shape
    d = v.shape[2]
    if v.dim() != 3 or v.shape[:2] != (G, Lk):
        raise ValueError("v must be [G, Lk, d]")
    if out is None:
        out = torch.empty((G, Lq, d), dtype=torch.int64, device=v.device)
    if out.shape != (G, Lq, d):
        raise ValueError("out must be [G, Lq, d]")
    args = (_dev_ptr(codes, torch.uint8, "codes", 3), ld, _dev_ptr(v, torch.int8, "v", 3), zp_v,
            G, Lq, Lk, d, bits, _dev_ptr(out, torch.int64, "out", 3), _stream(stream, v))
    return _invoke("lis_attn_v_shift_wide", args, (codes, v, out), prepare, out)


def lis_attention_head(logits, v, s_logit: float, bits: int = 4, exp_n: int = 20, zp_v: int = 0,
                       bias=None, out=None, codes_out=None, stream=None, prepare: bool = False):
    """Fused Log-Int-Softmax + BitShift Attn x V; returns int32 [G, Lq, d]."""
    import torch
    G, Lq, Lk = logits.shape
    d = v.shape[2]
    if v.dim() != 3 or v.shape[:2] != (G, Lk):
        raise ValueError("v must be [G, Lk, d]")
    if out is None:
        out = torch.empty((G, Lq, d), dtype=torch.int32, device=logits.device)
    if out.shape != (G, Lq, d):
        raise ValueError("out must be [G, Lq, d]")
    Hb = 0
    if bias is not None:
        if bias.dim() != 3 or bias.shape[1:] != (Lq, Lk):
            raise ValueError("bias must be [Hb, Lq, Lk]")
        Hb = bias.shape[0]
    ld = 0
    if codes_out is not None:
        if codes_out.dim() != 3 or codes_out.shape[:2] != (G, Lq):
            raise ValueError("codes_out must be [G, Lq, ld_codes]")
        ld = codes_out.shape[2]
    args = (_dev_ptr(logits, torch.int32, "logits", 3), _dev_ptr(bias, torch.int32, "bias", 3), Hb,
            G, Lq, Lk, s_logit, bits, exp_n, _dev_ptr(v, torch.int8, "v", 3), zp_v, d,
            _dev_ptr(out, torch.int32, "out", 3),
            _dev_ptr(codes_out, torch.uint8, "codes_out", 3), ld, _stream(stream, logits))
    return _invoke("lis_attention_head", args, (logits, bias, v, out, codes_out), prepare, out)


def ptf_calibrate_workspace_bytes(T: int, C: int, K: int = 3) -> int:
    """Bytes of device scratch that ptf_calibrate needs (0 for invalid sizes)."""
    return int(lib().fq_ptf_calibrate_workspace_bytes(T, C, K))


def ptf_calibrate(x, bits: int = 8, K: int = 3, s=None, zp=None, alpha=None, workspace=None,
                  stream=None, prepare: bool = False):
    """PTF calibration of a float [T, C] tensor: returns (s, zp, alpha) as device
    tensors (float64 [1], int32 [1] in container form, uint8 [C]).  The
    workspace is allocated here with torch when not given."""
    import torch
    T, C = x.shape
    dev = x.device
    s = torch.empty(1, dtype=torch.float64, device=dev) if s is None else s
    zp = torch.empty(1, dtype=torch.int32, device=dev) if zp is None else zp
    alpha = torch.empty(C, dtype=torch.uint8, device=dev) if alpha is None else alpha
    need = ptf_calibrate_workspace_bytes(T, C, K) if T > 0 else 0
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    args = (_dev_ptr(x, torch.float32, "x", 2), T, C, bits, K,
            _dev_ptr(s, torch.float64, "s", 1), _dev_ptr(zp, torch.int32, "zp", 1),
            _dev_ptr(alpha, torch.uint8, "alpha", 1), _dev_ptr(workspace, torch.uint8, "workspace", 1),
            workspace.numel(), _stream(stream, x))
    return _invoke("ptf_calibrate", args, (x, s, zp, alpha, workspace), prepare, (s, zp, alpha))


def ptf_calibrate_noalloc(x, bits: int = 8, K: int = 3, s=None, zp=None, alpha=None,
                          stream=None, prepare: bool = False):
    """ptf_calibrate with the workspace in the library's fixed device scratch:
    the entry point allocates nothing (outputs not given are allocated here,
    by torch, before the call)."""
    import torch
    T, C = x.shape
    dev = x.device
    s = torch.empty(1, dtype=torch.float64, device=dev) if s is None else s
    zp = torch.empty(1, dtype=torch.int32, device=dev) if zp is None else zp
    alpha = torch.empty(C, dtype=torch.uint8, device=dev) if alpha is None else alpha
    args = (_dev_ptr(x, torch.float32, "x", 2), T, C, bits, K,
            _dev_ptr(s, torch.float64, "s", 1), _dev_ptr(zp, torch.int32, "zp", 1),
            _dev_ptr(alpha, torch.uint8, "alpha", 1), _stream(stream, x))
    return _invoke("ptf_calibrate_noalloc", args, (x, s, zp, alpha), prepare, (s, zp, alpha))


def ptf_quantize_int8(x, s, zp, alpha, bits: int = 8, x_q=None, stream=None,
                      prepare: bool = False):
    """PTF quantization of a float [T, C] tensor with device scalars s, zp (as
    returned by ptf_calibrate) and alpha [C]; returns (or fills) int8 [T, C]."""
    import torch
    T, C = x.shape
    if x_q is None:
        x_q = torch.empty((T, C), dtype=torch.int8, device=x.device)
    if alpha.shape != (C,) or x_q.shape != (T, C):
        raise ValueError("alpha must be [C] and x_q [T, C]")
    args = (_dev_ptr(x, torch.float32, "x", 2), T, C, _dev_ptr(s, torch.float64, "s", 1),
            _dev_ptr(zp, torch.int32, "zp", 1), _dev_ptr(alpha, torch.uint8, "alpha", 1), bits,
            _dev_ptr(x_q, torch.int8, "x_q", 2), _stream(stream, x))
    return _invoke("ptf_quantize_int8", args, (x, s, zp, alpha, x_q), prepare, x_q)


def requant_dyadic_int8(q, s_in: float, s_out: float, zp_out: int, bits: int = 8, y=None,
                        stream=None, prepare: bool = False):
    """Dyadic requantization of an int32 tensor (any shape, contiguous) to the
    int8 container; returns (or fills) int8 of the same shape."""
    import torch
    if y is None:
        y = torch.empty(q.shape, dtype=torch.int8, device=q.device)
    if y.shape != q.shape:
        raise ValueError("y must have the shape of q")
    args = (_dev_ptr(q, torch.int32, "q"), q.numel(), s_in, s_out, zp_out, bits,
            _dev_ptr(y, torch.int8, "y"), _stream(stream, q))
    return _invoke("requant_dyadic_int8", args, (q, y), prepare, y)


def lis_attention_qk(q, k, v, s_logit: float, zp_q: int = 0, zp_k: int = 0, bits: int = 4,
                     exp_n: int = 20, zp_v: int = 0, bias=None, out=None, stream=None,
                     prepare: bool = False):
    """Integer-only attention from int8 q [G, Lq, dk], k [G, Lk, dk] and
    v [G, Lk, d]; returns (or fills) int32 [G, Lq, d]."""
    import torch
    G, Lq, dk = q.shape
    Lk = k.shape[1]
    d = v.shape[2]
    if k.shape != (G, Lk, dk) or v.shape[:2] != (G, Lk):
        raise ValueError("k must be [G, Lk, dk] and v [G, Lk, d]")
    if out is None:
        out = torch.empty((G, Lq, d), dtype=torch.int32, device=q.device)
    Hb = bias.shape[0] if bias is not None else 0
    args = (_dev_ptr(q, torch.int8, "q", 3), _dev_ptr(k, torch.int8, "k", 3), zp_q, zp_k, dk,
            _dev_ptr(bias, torch.int32, "bias", 3), Hb, G, Lq, Lk, s_logit, bits, exp_n,
            _dev_ptr(v, torch.int8, "v", 3), zp_v, d, _dev_ptr(out, torch.int32, "out", 3),
            _stream(stream, q))
    return _invoke("lis_attention_qk", args, (q, k, v, bias, out), prepare, out)
