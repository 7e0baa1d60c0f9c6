"""The C ABI library loads, exports every entry point its header declares, and
rejects invalid arguments on the host before anything is enqueued.  No test
here launches a kernel or needs a GPU: every call below fails validation (or
is empty) before the first HIP runtime call."""
import ctypes
import os
import re

import pytest

from paper_2111_13824_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fqvit.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\**\s+\**([a-z_][a-z0-9_]*)\s*\(",
                      text, flags=re.M)


# A test build of the C ABI's host code (tests/test_sanitizers.py: built with
# AddressSanitizer and UndefinedBehaviorSanitizer and linked against counting
# stand-ins for the kernel launchers) can be named here instead of libfqvit.
STUB_LIB = os.environ.get("FQVIT_ABI_TEST_LIB")


@pytest.fixture(scope="module")
def lib():
    if STUB_LIB:
        saved = B._lib
        B._lib = B.load(STUB_LIB)
        B._lib.fq_test_launch_count.restype = ctypes.c_int
        yield B._lib
        B._lib = saved
        return
    if not os.path.exists(B.LIB_PATH):
        from paper_2111_13824_amd import build
        build.build()
    yield B.lib()


def test_header_symbols_exported(lib):
    names = _declared_functions()
    assert set(names) >= {"ptf_layernorm_int8", "lis_softmax_log4", "lis_attn_v_shift",
                          "lis_attention_head", "fq_status_str", "fq_version",
                          "fq_time_next_call", "ptf_calibrate", "fq_ptf_calibrate_workspace_bytes",
                          "ptf_quantize_int8", "requant_dyadic_int8", "lis_attention_qk",
                          "lis_attn_v_shift_wide", "ptf_calibrate_noalloc"}
    for n in names:
        assert hasattr(lib, n), f"{n} declared in fqvit.h but not exported"
    # the binding exposes the compute entry points under the same names
    for n in B.SIGNATURES:
        assert n in names


def test_time_next_call_is_host_only(lib):
    # setting and clearing the events touches no HIP state; a call that fails
    # validation consumes them without enqueueing anything
    assert lib.fq_time_next_call(None, None) == 0
    assert lib.fq_time_next_call(ctypes.c_void_p(16), ctypes.c_void_p(32)) == 0
    assert lib.ptf_layernorm_int8(None, 4, 0, 0, None, 3, None, None, ctypes.c_float(1.0), 0, 8,
                                  None, None) == 2
    assert lib.fq_time_next_call(None, None) == 0


def test_prepared_call_reports_status(lib):
    # a prepared call that fails host validation raises like a direct call
    call = B.Prepared("ptf_layernorm_int8",
                      (None, 4, 0, 0, None, 3, None, None, 1.0, 0, 8, None, None), ())
    with pytest.raises(B.FqError) as ei:
        call()
    assert ei.value.status == B.FQ_ERR_SHAPE


def test_status_strings(lib):
    for s in range(7):
        assert B.status_str(s).startswith("FQ_")
    assert "unknown" in B.status_str(99)
    assert B.version() == 100


NULL = None


def test_layernorm_validation(lib):
    f = lib.ptf_layernorm_int8
    args = dict(x=1, T=4, C=8, zp=0, alpha=1, K=3, g=1, b=1, s=0.1, zpo=0, bits=8, y=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["x"], a["T"], a["C"], a["zp"], a["alpha"], a["K"], a["g"], a["b"], a["s"],
                 a["zpo"], a["bits"], a["y"], NULL)

    assert call(C=0) == B.FQ_ERR_SHAPE
    assert call(C=8193) == B.FQ_ERR_SHAPE
    assert call(T=-1) == B.FQ_ERR_SHAPE
    assert call(bits=9) == B.FQ_ERR_PARAM
    assert call(bits=1) == B.FQ_ERR_PARAM
    assert call(K=8) == B.FQ_ERR_PARAM
    assert call(K=-1) == B.FQ_ERR_PARAM
    assert call(s=0.0) == B.FQ_ERR_PARAM
    assert call(s=float("inf")) == B.FQ_ERR_PARAM
    assert call(s=float("nan")) == B.FQ_ERR_PARAM
    assert call(zp=128) == B.FQ_ERR_PARAM
    assert call(zpo=-129) == B.FQ_ERR_PARAM
    assert call(bits=4, zp=8) == B.FQ_ERR_PARAM
    assert call(x=NULL) == B.FQ_ERR_NULL
    assert call(y=NULL) == B.FQ_ERR_NULL
    assert call(alpha=NULL) == B.FQ_ERR_NULL
    assert call(T=0, x=NULL, y=NULL) == B.FQ_OK     # empty: nothing enqueued


def test_lis_validation(lib):
    f = lib.lis_softmax_log4
    args = dict(lg=1, G=2, Lq=3, Lk=5, bias=NULL, Hb=0, s=2.0 ** -10, bits=4, n=20, codes=1, ld=3)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["lg"], a["G"], a["Lq"], a["Lk"], a["bias"], a["Hb"], a["s"], a["bits"], a["n"],
                 a["codes"], a["ld"], NULL)

    assert call(Lk=0) == B.FQ_ERR_SHAPE
    assert call(Lk=4097, ld=2049) == B.FQ_ERR_SHAPE
    assert call(ld=2) == B.FQ_ERR_SHAPE
    assert call(G=-1) == B.FQ_ERR_SHAPE
    assert call(bias=1, Hb=0) == B.FQ_ERR_SHAPE
    assert call(bits=0) == B.FQ_ERR_PARAM
    assert call(bits=9) == B.FQ_ERR_PARAM
    assert call(bits=5, ld=4) == B.FQ_ERR_SHAPE      # one byte per code above 4 bits
    assert call(n=0) == B.FQ_ERR_PARAM
    assert call(n=31) == B.FQ_ERR_PARAM
    assert call(s=0.6) == B.FQ_ERR_PARAM
    assert call(s=5e-5) == B.FQ_ERR_PARAM
    assert call(s=1e-4, n=30, Lk=4096, ld=2048) == B.FQ_ERR_HEADROOM
    assert call(lg=NULL) == B.FQ_ERR_NULL
    assert call(codes=NULL) == B.FQ_ERR_NULL
    assert call(G=0, lg=NULL, codes=NULL) == B.FQ_OK
    assert call(Lq=0, lg=NULL, codes=NULL) == B.FQ_OK


def test_attn_v_validation(lib):
    f = lib.lis_attn_v_shift
    args = dict(codes=1, ld=3, v=1, zp=0, G=2, Lq=3, Lk=5, d=64, bits=4, out=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["codes"], a["ld"], a["v"], a["zp"], a["G"], a["Lq"], a["Lk"], a["d"], a["bits"],
                 a["out"], NULL)

    assert call(d=0) == B.FQ_ERR_SHAPE
    assert call(d=257) == B.FQ_ERR_SHAPE
    assert call(ld=2) == B.FQ_ERR_SHAPE
    assert call(bits=5) == B.FQ_ERR_PARAM
    assert call(zp=128) == B.FQ_ERR_PARAM
    assert call(out=NULL) == B.FQ_ERR_NULL
    assert call(v=NULL) == B.FQ_ERR_NULL
    assert call(G=0, codes=NULL, v=NULL, out=NULL) == B.FQ_OK


def test_attn_v_wide_validation(lib):
    f = lib.lis_attn_v_shift_wide
    args = dict(c=1, ld=7, v=1, zp=0, G=2, Lq=5, Lk=7, d=64, bits=8, out=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["c"], a["ld"], a["v"], a["zp"], a["G"], a["Lq"], a["Lk"], a["d"], a["bits"],
                 a["out"], NULL)

    assert call(G=-1) == B.FQ_ERR_SHAPE
    assert call(Lk=0) == B.FQ_ERR_SHAPE
    assert call(Lk=4097, ld=4097) == B.FQ_ERR_SHAPE
    assert call(d=0) == B.FQ_ERR_SHAPE
    assert call(d=257) == B.FQ_ERR_SHAPE
    assert call(ld=6) == B.FQ_ERR_SHAPE              # one byte per code at 8 bits
    assert call(bits=4, ld=3) == B.FQ_ERR_SHAPE      # nibbles: ceil(7 / 2) = 4 bytes
    assert call(bits=0) == B.FQ_ERR_PARAM
    assert call(bits=9) == B.FQ_ERR_PARAM
    assert call(zp=128) == B.FQ_ERR_PARAM
    for k in ("c", "v", "out"):
        assert call(**{k: None}) == B.FQ_ERR_NULL
    assert call(G=0, c=None, v=None, out=None) == B.FQ_OK


def test_head_validation(lib):
    f = lib.lis_attention_head
    args = dict(lg=1, bias=NULL, Hb=0, G=2, Lq=3, Lk=5, s=2.0 ** -10, bits=4, n=20, v=1, zp=0,
                d=64, out=1, codes=NULL, ld=0)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["lg"], a["bias"], a["Hb"], a["G"], a["Lq"], a["Lk"], a["s"], a["bits"], a["n"],
                 a["v"], a["zp"], a["d"], a["out"], a["codes"], a["ld"], NULL)

    assert call(d=300) == B.FQ_ERR_SHAPE
    assert call(codes=1, ld=2) == B.FQ_ERR_SHAPE
    assert call(bias=1, Hb=0) == B.FQ_ERR_SHAPE
    assert call(zp=-200) == B.FQ_ERR_PARAM
    assert call(s=0.0) == B.FQ_ERR_PARAM
    assert call(bits=0) == B.FQ_ERR_PARAM
    assert call(v=NULL) == B.FQ_ERR_NULL
    assert call(out=NULL) == B.FQ_ERR_NULL
    assert call(Lq=0, lg=NULL, v=NULL, out=NULL) == B.FQ_OK


@pytest.mark.skipif(bool(STUB_LIB), reason="tests the binding's own loader")
def test_binding_requires_library(monkeypatch):
    """The binding refuses to run without the HIP library instead of falling back."""
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", "/nonexistent/libfqvit.so")
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()


def test_calibrate_workspace_size(lib):
    f = B.ptf_calibrate_workspace_bytes
    assert f(0, 768, 3) == 0 and f(10, 0, 3) == 0 and f(10, 768, 8) == 0
    # min/max partials, per-block error sums, per-channel error totals
    assert f(12608, 768, 3) == 1024 * 8 + 4 * 197 * 768 * 8 + 4 * 768 * 8
    assert f(64, 5, 0) == 1024 * 8 + 1 * 1 * 5 * 8 + 1 * 5 * 8
    assert f(65, 5, 7) == 1024 * 8 + 8 * 2 * 5 * 8 + 8 * 5 * 8


def test_calibrate_validation(lib):
    f = lib.ptf_calibrate
    need = B.ptf_calibrate_workspace_bytes(100, 16, 3)
    args = dict(x=1, T=100, C=16, bits=8, K=3, s=1, zp=1, alpha=1, ws=1, wsb=need)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["x"], a["T"], a["C"], a["bits"], a["K"], a["s"], a["zp"], a["alpha"], a["ws"],
                 a["wsb"], NULL)

    assert call(T=-1) == B.FQ_ERR_SHAPE
    assert call(T=65535 * 64 + 1) == B.FQ_ERR_SHAPE
    assert call(C=0) == B.FQ_ERR_SHAPE
    assert call(C=8193) == B.FQ_ERR_SHAPE
    assert call(bits=1) == B.FQ_ERR_PARAM
    assert call(bits=9) == B.FQ_ERR_PARAM
    assert call(K=8) == B.FQ_ERR_PARAM
    assert call(wsb=need - 1) == B.FQ_ERR_PARAM
    for k in ("x", "s", "zp", "alpha", "ws"):
        assert call(**{k: None}) == B.FQ_ERR_NULL
    assert call(T=0, x=None, s=None) == B.FQ_OK      # empty: nothing enqueued


def test_calibrate_noalloc_validation(lib):
    """Host-side checks of the entry point that allocates nothing: the same
    argument checks as ptf_calibrate, and sizes whose workspace exceeds the
    fixed device scratch rejected with FQ_ERR_SCRATCH before any HIP call."""
    f = lib.ptf_calibrate_noalloc
    args = dict(x=1, T=100, C=16, bits=8, K=3, s=1, zp=1, alpha=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["x"], a["T"], a["C"], a["bits"], a["K"], a["s"], a["zp"], a["alpha"], NULL)

    assert call(T=-1) == B.FQ_ERR_SHAPE
    assert call(C=8193) == B.FQ_ERR_SHAPE
    assert call(bits=9) == B.FQ_ERR_PARAM
    assert call(K=8) == B.FQ_ERR_PARAM
    for k in ("x", "s", "zp", "alpha"):
        assert call(**{k: None}) == B.FQ_ERR_NULL
    assert call(T=0, x=None) == B.FQ_OK
    # the largest workloads' calibrations fit; a larger one does not
    for T, C in ((12608, 768), (9232, 1024), (100352, 96)):
        assert B.ptf_calibrate_workspace_bytes(T, C, 3) <= B.NOALLOC_SCRATCH_BYTES
    assert B.ptf_calibrate_workspace_bytes(200000, 768, 3) > B.NOALLOC_SCRATCH_BYTES
    assert call(T=200000, C=768) == B.FQ_ERR_SCRATCH
    assert "scratch" in B.status_str(B.FQ_ERR_SCRATCH)


def test_quantize_validation(lib):
    f = lib.ptf_quantize_int8
    args = dict(x=1, T=10, C=16, s=1, zp=1, alpha=1, bits=8, y=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["x"], a["T"], a["C"], a["s"], a["zp"], a["alpha"], a["bits"], a["y"], NULL)

    assert call(T=-1) == B.FQ_ERR_SHAPE
    assert call(C=0) == B.FQ_ERR_SHAPE
    assert call(bits=1) == B.FQ_ERR_PARAM
    assert call(bits=9) == B.FQ_ERR_PARAM
    for k in ("x", "s", "zp", "alpha", "y"):
        assert call(**{k: None}) == B.FQ_ERR_NULL
    assert call(T=0, x=None) == B.FQ_OK


def test_requant_validation(lib):
    f = lib.requant_dyadic_int8
    args = dict(q=1, n=10, si=0.5, so=0.25, zp=0, bits=8, y=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["q"], a["n"], a["si"], a["so"], a["zp"], a["bits"], a["y"], NULL)

    assert call(n=-1) == B.FQ_ERR_SHAPE
    assert call(bits=1) == B.FQ_ERR_PARAM
    assert call(bits=9) == B.FQ_ERR_PARAM
    for k, v in (("si", 0.0), ("si", float("nan")), ("so", -1.0), ("so", float("inf"))):
        assert call(**{k: v}) == B.FQ_ERR_PARAM
    assert call(zp=128) == B.FQ_ERR_PARAM
    assert call(bits=4, zp=8) == B.FQ_ERR_PARAM
    assert call(bits=4, zp=-9) == B.FQ_ERR_PARAM
    assert call(q=None) == B.FQ_ERR_NULL
    assert call(y=None) == B.FQ_ERR_NULL
    assert call(n=0, q=None, y=None) == B.FQ_OK


def test_qk_validation(lib):
    f = lib.lis_attention_qk
    args = dict(q=16, k=16, zq=0, zk=0, dk=64, bias=None, Hb=0, G=2, Lq=5, Lk=7, s=0.001, bits=4,
                n=20, v=1, zv=0, d=64, out=1)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["q"], a["k"], a["zq"], a["zk"], a["dk"], a["bias"], a["Hb"], a["G"], a["Lq"],
                 a["Lk"], a["s"], a["bits"], a["n"], a["v"], a["zv"], a["d"], a["out"], NULL)

    assert call(G=-1) == B.FQ_ERR_SHAPE
    assert call(Lk=0) == B.FQ_ERR_SHAPE
    assert call(Lk=641) == B.FQ_ERR_SHAPE
    assert call(d=65) == B.FQ_ERR_SHAPE
    assert call(d=0) == B.FQ_ERR_SHAPE
    assert call(dk=48) == B.FQ_ERR_SHAPE
    assert call(dk=128) == B.FQ_ERR_SHAPE
    assert call(bias=16, Hb=0) == B.FQ_ERR_SHAPE
    assert call(zq=128) == B.FQ_ERR_PARAM
    assert call(zk=-129) == B.FQ_ERR_PARAM
    assert call(zv=200) == B.FQ_ERR_PARAM
    assert call(bits=5) == B.FQ_ERR_PARAM
    assert call(s=1.0) == B.FQ_ERR_PARAM
    assert call(n=0) == B.FQ_ERR_PARAM
    assert call(q=8) == B.FQ_ERR_PARAM           # q not 16-byte aligned
    assert call(k=24) == B.FQ_ERR_PARAM
    for key in ("q", "k", "v", "out"):
        assert call(**{key: None}) == B.FQ_ERR_NULL
    assert call(G=0, q=None) == B.FQ_OK
    assert call(Lq=0, out=None) == B.FQ_OK


@pytest.mark.skipif(not STUB_LIB, reason="needs the host-only test build (counting launchers)")
def test_valid_calls_reach_exactly_one_launch(lib):
    """With the launchers replaced by counters: every valid call reaches its
    launcher once and returns FQ_OK; a rejected or empty call reaches none."""
    count = lib.fq_test_launch_count

    def launches(fn, *args):
        n0 = count()
        rc = fn(*args)
        return rc, count() - n0

    f32 = ctypes.c_float
    assert launches(lib.ptf_layernorm_int8, 1, 4, 8, 0, 1, 3, 1, 1, f32(0.1), 0, 8, 1, None) == (0, 1)
    assert launches(lib.ptf_layernorm_int8, 1, 4, 8, 0, 1, 3, 1, 1, f32(0.0), 0, 8, 1, None)[1] == 0
    assert launches(lib.ptf_layernorm_int8, 1, 0, 8, 0, 1, 3, 1, 1, f32(0.1), 0, 8, 1, None) == (0, 0)
    assert launches(lib.lis_softmax_log4, 1, 2, 5, 7, None, 0, f32(0.001), 4, 20, 1, 4, None) == (0, 1)
    assert launches(lib.lis_softmax_log4, 1, 2, 5, 7, None, 0, f32(0.001), 4, 20, 1, 3, None)[1] == 0
    assert launches(lib.lis_attn_v_shift, 1, 4, 1, 0, 2, 5, 7, 64, 4, 1, None) == (0, 1)
    assert launches(lib.lis_attn_v_shift_wide, 1, 7, 1, 0, 2, 5, 7, 64, 8, 1, None) == (0, 1)
    assert launches(lib.lis_attn_v_shift_wide, 1, 4, 1, 0, 2, 5, 7, 64, 4, 1, None) == (0, 1)
    assert launches(lib.lis_attention_head, 1, None, 0, 2, 5, 7, f32(0.001), 4, 20, 1, 0, 64, 1,
                    None, 0, None) == (0, 1)
    assert launches(lib.lis_attention_qk, 16, 16, 0, 0, 64, None, 0, 2, 5, 7, f32(0.001), 4, 20,
                    1, 0, 64, 1, None) == (0, 1)
    need = lib.fq_ptf_calibrate_workspace_bytes(100, 16, 3)
    assert launches(lib.ptf_calibrate, 1, 100, 16, 8, 3, 1, 1, 1, 1, need, None) == (0, 1)
    assert launches(lib.ptf_calibrate, 1, 100, 16, 8, 3, 1, 1, 1, 1, need - 1, None)[1] == 0
    assert launches(lib.ptf_calibrate_noalloc, 1, 100, 16, 8, 3, 1, 1, 1, None) == (0, 1)
    assert launches(lib.ptf_calibrate_noalloc, 1, 200000, 768, 8, 3, 1, 1, 1, None) == (6, 0)
    assert launches(lib.ptf_quantize_int8, 1, 10, 16, 1, 1, 1, 8, 1, None) == (0, 1)
    assert launches(lib.requant_dyadic_int8, 1, 10, f32(0.5), f32(0.25), 0, 8, 1, None) == (0, 1)
