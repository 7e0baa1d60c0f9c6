"""CPU oracle for FQ-ViT's integer hot path (PTF LayerNorm, Log-Int-Softmax,
BitShift Attn x V).

TEST INFRASTRUCTURE ONLY.  The plain scalar C implementation in
``fqvit_oracle.c`` follows the paper step by step; this module compiles it with
gcc and calls it through ctypes on numpy arrays.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package.  The HIP library never calls into it and shares no code with it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fqvit_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test may point the loader at another build of the same source (for example
# a copy with a planted mistake) through this variable.
_LIB_OVERRIDE = os.environ.get("FQVIT_ORACLE_LIB")

CFLAGS = ["-std=gnu11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra"]

OK, ERR_ARG, ERR_RANGE = 0, 1, 2


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile liboracle.so next to its source with gcc."""
    if src != _SRC or out != _LIB:
        subprocess.run(["gcc", *CFLAGS, "-I", _HERE, src, "-o", out, "-lm"], check=True)
        return out
    if _LIB_OVERRIDE:
        return _LIB_OVERRIDE
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class IExpConsts(ctypes.Structure):
    _fields_ = [("q_ln2", ctypes.c_int64), ("q_b", ctypes.c_int64), ("q_c", ctypes.c_int64),
                ("s_L", ctypes.c_double), ("n", ctypes.c_int32)]


_lib: Optional[ctypes.CDLL] = None

_P = ctypes.c_void_p
_I32, _I64, _F32, _F64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double

_SIGS = {
    "oracle_minmax_params": [_P, _I64, _I32, _P, _P],
    "oracle_minmax_quantize": [_P, _I64, _F64, _I32, _I32, _P],
    "oracle_ptf_params": [_P, _I64, _I32, _I32, _I32, _P, _P],
    "oracle_ptf_alpha": [_P, _I64, _I32, _F64, _I32, _I32, _I32, _P],
    "oracle_ptf_alpha_errors": [_P, _I64, _I32, _F64, _I32, _I32, _I32, _P, _P],
    "oracle_ptf_quantize": [_P, _I64, _I32, _F64, _I32, _P, _I32, _P],
    "oracle_ptf_layernorm_int8": [_P, _I64, _I32, _I32, _P, _I32, _P, _P, _F32, _I32, _I32, _P],
    "oracle_iexp_constants": [_F64, _I32, _P],
    "oracle_ilog2": [ctypes.c_uint64],
    "oracle_lis_softmax_log4": [_P, _I64, _I32, _I32, _P, _I32, _F32, _I32, _I32, _P, _I32],
    "oracle_lis_row_exp": [_P, _P, _I32, _F32, _I32, _P, _P],
    "oracle_lis_attn_v_shift": [_P, _I32, _P, _I32, _I64, _I32, _I32, _I32, _I32, _P],
    "oracle_lis_attn_v_shift_wide": [_P, _I32, _P, _I32, _I64, _I32, _I32, _I32, _I32, _P],
    "oracle_lis_attention_head": [_P, _P, _I32, _I64, _I32, _I32, _F32, _I32, _I32, _P, _I32,
                                  _I32, _P, _P, _I32],
    "oracle_requant_dyadic_int8": [_P, _I64, _F32, _F32, _I32, _I32, _P],
    "oracle_qk_logits": [_P, _P, _I32, _I32, _I64, _I32, _I32, _I32, _P],
    "oracle_lis_attention_qk": [_P, _P, _I32, _I32, _I32, _P, _I32, _I64, _I32, _I32, _F32, _I32,
                                _I32, _P, _I32, _I32, _P],
}


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        path = _LIB_OVERRIDE or _LIB
        if not _LIB_OVERRIDE and (not os.path.exists(_LIB)
                                  or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build(force=True)
        L = ctypes.CDLL(path)
        for name, args in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int32
        L.oracle_iexp.argtypes = [_I64, _P, _P, _P]
        L.oracle_iexp.restype = _I64
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise ValueError(f"{what}: oracle returned {rc}")


# ---- Sec. 3.1: MinMax ------------------------------------------------------

def minmax_params(x: np.ndarray, b: int = 8):
    x = np.ascontiguousarray(x, dtype=np.float64)
    s, zp = ctypes.c_double(), ctypes.c_int32()
    _check(lib().oracle_minmax_params(_ptr(x), x.size, b, ctypes.byref(s), ctypes.byref(zp)),
           "minmax_params")
    return s.value, zp.value


def minmax_quantize(x: np.ndarray, s: float, zp: int, b: int = 8) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    q = np.empty(x.shape, dtype=np.int32)
    _check(lib().oracle_minmax_quantize(_ptr(x), x.size, s, zp, b, _ptr(q)), "minmax_quantize")
    return q


# ---- Sec. 3.2: PTF quantizer ----------------------------------------------

def ptf_params(x: np.ndarray, b: int = 8, K: int = 3):
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, C = x.shape
    s, zp = ctypes.c_double(), ctypes.c_int32()
    _check(lib().oracle_ptf_params(_ptr(x), T, C, b, K, ctypes.byref(s), ctypes.byref(zp)),
           "ptf_params")
    return s.value, zp.value


def ptf_alpha(x: np.ndarray, s: float, zp: int, b: int = 8, K: int = 3) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, C = x.shape
    alpha = np.empty(C, dtype=np.uint8)
    _check(lib().oracle_ptf_alpha(_ptr(x), T, C, s, zp, b, K, _ptr(alpha)), "ptf_alpha")
    return alpha


def ptf_alpha_errors(x: np.ndarray, s: float, zp: int, b: int = 8, K: int = 3,
                     with_lo: bool = False):
    """[C, K + 1] exact errors of eq. (11), rounded to binary64; with_lo: also
    the [C, K + 1] remainders (hi + lo is the exact value to about 106 bits)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, C = x.shape
    err = np.empty((C, K + 1), dtype=np.float64)
    lo = np.empty((C, K + 1), dtype=np.float64) if with_lo else None
    _check(lib().oracle_ptf_alpha_errors(_ptr(x), T, C, s, zp, b, K, _ptr(err), _ptr(lo)),
           "ptf_alpha_errors")
    return (err, lo) if with_lo else err


def ptf_quantize(x: np.ndarray, s: float, zp: int, alpha: np.ndarray, b: int = 8) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    alpha = np.ascontiguousarray(alpha, dtype=np.uint8)
    T, C = x.shape
    q = np.empty((T, C), dtype=np.int32)
    _check(lib().oracle_ptf_quantize(_ptr(x), T, C, s, zp, _ptr(alpha), b, _ptr(q)),
           "ptf_quantize")
    return q


# ---- Dyadic requantization ----------------------------------------------------

def requant_dyadic_int8(q: np.ndarray, s_in: float, s_out: float, zp_out: int,
                        bits: int = 8) -> np.ndarray:
    """int32 accumulator of scale s_in -> b-bit activation of scale s_out in the
    int8 container (value - 2^(b-1)), through the 31-bit dyadic form of s_in/s_out."""
    q = np.ascontiguousarray(q, dtype=np.int32)
    y = np.empty(q.shape, dtype=np.int8)
    _check(lib().oracle_requant_dyadic_int8(_ptr(q), q.size, s_in, s_out, zp_out, bits, _ptr(y)),
           "requant_dyadic_int8")
    return y


# ---- Supplement A.1: integer LayerNorm --------------------------------------

def ptf_layernorm_int8(x_q, zp_in, alpha, K, gamma, beta, s_out, zp_out, bits=8) -> np.ndarray:
    x_q = np.ascontiguousarray(x_q, dtype=np.int8)
    T, C = x_q.shape
    alpha = np.ascontiguousarray(alpha, dtype=np.uint8)
    gamma = np.ascontiguousarray(gamma, dtype=np.float32)
    beta = np.ascontiguousarray(beta, dtype=np.float32)
    y = np.empty((T, C), dtype=np.int8)
    _check(lib().oracle_ptf_layernorm_int8(_ptr(x_q), T, C, zp_in, _ptr(alpha), K, _ptr(gamma),
                                           _ptr(beta), s_out, zp_out, bits, _ptr(y)),
           "ptf_layernorm_int8")
    return y


# ---- Supplement A.2: I-Exp, I-Log2, LIS -------------------------------------

def iexp_constants(s: float, n: int = 20) -> IExpConsts:
    k = IExpConsts()
    _check(lib().oracle_iexp_constants(float(s), n, ctypes.byref(k)), "iexp_constants")
    return k


def iexp(q: int, k: IExpConsts):
    """Return (q_out, z, q_p) for one non-positive input."""
    z, qp = ctypes.c_int64(), ctypes.c_int64()
    out = lib().oracle_iexp(int(q), ctypes.byref(k), ctypes.byref(z), ctypes.byref(qp))
    return out, z.value, qp.value


def ilog2(q: int) -> int:
    return lib().oracle_ilog2(int(q))


def codes_ld(Lk: int, bits: int = 4) -> int:
    return (Lk + 1) // 2 if bits <= 4 else Lk


def unpack_codes(packed: np.ndarray, Lk: int, bits: int = 4) -> np.ndarray:
    """[..., ld] stored codes -> [..., Lk] codes: nibbles (even key in the low
    nibble) for bits <= 4, one byte per code above."""
    if bits > 4:
        return packed[..., :Lk]
    lo = packed & 15
    hi = packed >> 4
    out = np.stack([lo, hi], axis=-1).reshape(*packed.shape[:-1], packed.shape[-1] * 2)
    return out[..., :Lk]


def lis_softmax_log4(logits, s_logit, bits=4, exp_n=20, bias=None, ld_codes=None) -> np.ndarray:
    logits = np.ascontiguousarray(logits, dtype=np.int32)
    G, Lq, Lk = logits.shape
    ld = codes_ld(Lk, bits) if ld_codes is None else ld_codes
    Hb = 0
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.int32)
        Hb = bias.shape[0]
    codes = np.zeros((G, Lq, ld), dtype=np.uint8)
    _check(lib().oracle_lis_softmax_log4(_ptr(logits), G, Lq, Lk, _ptr(bias), Hb, s_logit, bits,
                                         exp_n, _ptr(codes), ld), "lis_softmax_log4")
    return codes


def lis_row_exp(row, s_logit, exp_n=20, bias_row=None):
    row = np.ascontiguousarray(row, dtype=np.int32)
    if bias_row is not None:
        bias_row = np.ascontiguousarray(bias_row, dtype=np.int32)
    e = np.empty(row.shape[0], dtype=np.int64)
    ssum = ctypes.c_double()
    _check(lib().oracle_lis_row_exp(_ptr(row), _ptr(bias_row), row.shape[0], s_logit, exp_n,
                                    _ptr(e), ctypes.byref(ssum)), "lis_row_exp")
    return e, ssum.value


def lis_attn_v_shift(codes, v, zp_v=0, bits=4, Lk=None) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    v = np.ascontiguousarray(v, dtype=np.int8)
    G, Lk_v, d = v.shape
    Lk = Lk_v if Lk is None else Lk
    Gc, Lq, ld = codes.shape
    assert Gc == G
    out = np.empty((G, Lq, d), dtype=np.int32)
    _check(lib().oracle_lis_attn_v_shift(_ptr(codes), ld, _ptr(v), zp_v, G, Lq, Lk, d, bits,
                                         _ptr(out)), "lis_attn_v_shift")
    return out


def lis_attn_v_shift_wide(codes, v, zp_v=0, bits=8, Lk=None) -> np.ndarray:
    """int64 [G, Lq, d] product at scale s_V / 2^min(2^bits - 1, 44)."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    v = np.ascontiguousarray(v, dtype=np.int8)
    G, Lk_v, d = v.shape
    Lk = Lk_v if Lk is None else Lk
    Gc, Lq, ld = codes.shape
    assert Gc == G
    out = np.empty((G, Lq, d), dtype=np.int64)
    _check(lib().oracle_lis_attn_v_shift_wide(_ptr(codes), ld, _ptr(v), zp_v, G, Lq, Lk, d, bits,
                                              _ptr(out)), "lis_attn_v_shift_wide")
    return out


def lis_attention_head(logits, v, s_logit, bits=4, exp_n=20, zp_v=0, bias=None,
                       want_codes=False):
    logits = np.ascontiguousarray(logits, dtype=np.int32)
    v = np.ascontiguousarray(v, dtype=np.int8)
    G, Lq, Lk = logits.shape
    d = v.shape[2]
    Hb = 0
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.int32)
        Hb = bias.shape[0]
    out = np.empty((G, Lq, d), dtype=np.int32)
    ld = codes_ld(Lk)
    codes = np.zeros((G, Lq, ld), dtype=np.uint8) if want_codes else None
    _check(lib().oracle_lis_attention_head(_ptr(logits), _ptr(bias), Hb, G, Lq, Lk, s_logit, bits,
                                           exp_n, _ptr(v), zp_v, d, _ptr(out), _ptr(codes), ld),
           "lis_attention_head")
    return (out, codes) if want_codes else out


# ---- Sec. 3.3, Fig. 4: integer-only MSA from int8 Q and K --------------------

def qk_logits(q, k, zp_q=0, zp_k=0) -> np.ndarray:
    """int32 logits [G, Lq, Lk] = (q - zp_q)(k - zp_k)^T per unit, exact."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    k = np.ascontiguousarray(k, dtype=np.int8)
    G, Lq, dk = q.shape
    Lk = k.shape[1]
    out = np.empty((G, Lq, Lk), dtype=np.int32)
    _check(lib().oracle_qk_logits(_ptr(q), _ptr(k), zp_q, zp_k, G, Lq, Lk, dk, _ptr(out)),
           "qk_logits")
    return out


def lis_attention_qk(q, k, v, s_logit, zp_q=0, zp_k=0, bits=4, exp_n=20, zp_v=0, bias=None):
    """int8 Q K^T, Log-Int-Softmax and BitShift Attn x V; returns int32 [G, Lq, d]."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    k = np.ascontiguousarray(k, dtype=np.int8)
    v = np.ascontiguousarray(v, dtype=np.int8)
    G, Lq, dk = q.shape
    Lk = k.shape[1]
    d = v.shape[2]
    Hb = 0
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.int32)
        Hb = bias.shape[0]
    out = np.empty((G, Lq, d), dtype=np.int32)
    _check(lib().oracle_lis_attention_qk(_ptr(q), _ptr(k), zp_q, zp_k, dk, _ptr(bias), Hb, G, Lq,
                                         Lk, s_logit, bits, exp_n, _ptr(v), zp_v, d, _ptr(out)),
           "lis_attention_qk")
    return out
