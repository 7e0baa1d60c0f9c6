"""The float-path form of I-Exp and of the LIS code, as the fused kernels
evaluate it (24-bit integer I-Exp steps ending in a binary32 value, the code
from binary64 bit patterns and a binary32 comparison), against the oracle's
integer definitions.

The GPU parity tests compare the kernels with the oracle on sampled inputs;
these tests establish, on the CPU, that the formulation itself equals the
definition on every input the I-Exp can see and at the exact code
thresholds."""
import numpy as np
import pytest


def _float_consts(k):
    d = -k.q_ln2
    pre = 0
    while (d << pre) <= 256:
        pre += 1
    dp = d << pre
    return dict(d=d, qb=int(k.q_b), qc=int(k.q_c), n=k.n, umax=np.uint64(k.n * d), pre=pre,
                magic=(1 << 32) // dp + 1, ok=k.n * dp * dp < 2 ** 32 and k.n * dp < 2 ** 24)


def _iexp_float(u_raw, f):
    """e = qL 2^(n - z) from u = -q by the kernel's steps: z by the 24-bit
    multiply-high with the magic constant, q_p + q_b and qL by 24-bit
    multiply-adds, then a binary32 conversion and ldexp."""
    u = np.minimum(u_raw.astype(np.uint64), f["umax"])
    z = (((u << np.uint64(f["pre"])) & np.uint64(0xFFFFFF)) * np.uint64(f["magic"])) >> np.uint64(32)
    w = (z * np.uint64(f["d"]) + np.uint64(f["qb"]) - u) & np.uint64(0xFFFFFFFF)
    qL = (w * w + np.uint64(f["qc"])) & np.uint64(0xFFFFFFFF)
    assert np.all(qL < 2 ** 24)
    shift = np.int64(f["n"]) - z.astype(np.int64)
    return np.ldexp(qL.astype(np.float32).astype(np.float64), shift)


@pytest.mark.parametrize("s", [0.5, 0.05, 2.0 ** -10, 0.0005])
@pytest.mark.parametrize("n", [1, 8, 20, 30])
def test_iexp_float_form_exhaustive(orc, s, n):
    k = orc.iexp_constants(s, n)
    d = -k.q_ln2
    if k.q_b ** 2 + k.q_c >= 2 ** 24:
        pytest.skip("outside the float path's bound")
    f = _float_consts(k)
    if not f["ok"]:
        pytest.skip("outside the magic division's bound")
    u = np.arange(n * d + 4, dtype=np.int64)          # every clamped input, plus beyond the clamp
    got = _iexp_float(u, f)
    ref = np.array([orc.iexp(-int(x), k)[0] for x in u], dtype=np.float64)
    assert np.array_equal(got, ref)


SCALE = 2.0 ** -1000


def _shr27(v):
    """floor(bits(v) / 2^27) mod 2^32 (the funnel shift of the two words)."""
    return (v.view(np.uint64) >> np.uint64(27)) & np.uint64(0xFFFFFFFF)


def _third_floor_f32(S2):
    """Largest binary32 value <= floor(S2 / 3), as the kernel forms it:
    q0 = floor(S2 RN(1/3)), plus one when the exact remainder S2 - 3 q0 is 3
    or more; then converted to nearest and stepped down when above."""
    q0 = np.floor(S2 * (1.0 / 3.0))
    r = np.array([int(a) - 3 * int(b) for a, b in zip(S2, q0)], dtype=object)
    q = np.where(r >= 3, q0 + 1.0, q0)
    exact = np.array([int(a) // 3 for a in S2], dtype=object)
    assert np.all(np.array([int(v) for v in q], dtype=object) == exact)
    f = q.astype(np.float32)
    down = (f.astype(np.float64) > q)
    f = np.where(down, (f.view(np.int32) - 1).view(np.float32), f)
    return f.astype(np.float32)


def _code_parts(S2, e):
    """(m, t) as the kernel computes them: m from the funnel-shifted patterns
    of (2S + e) 2^-1000 and 1.5 e 2^-1000, t = [e > tau]."""
    X = (S2 * SCALE) + e * SCALE          # one rounding of an exact value
    Y = e * (1.5 * SCALE)
    ax, ay = _shr27(X), _shr27(Y)
    m = (((ax - ay) & np.uint64(0xFFFFFFFF)) >> np.uint64(25)).astype(np.int64)
    t = (e.astype(np.float32) > _third_floor_f32(S2)).astype(np.int64)
    return ax, ay, m, t


def _code_float(S2, e, top):
    _, _, m, t = _code_parts(S2, e)
    return np.minimum(m, top) - t


def _code_rev_float(S2, e, top):
    """top - code as the fused kernel forms it: the saturated difference
    (top + 1) 2^25 - 1 + ay - ax, shifted right by 25, plus t."""
    ax, ay, _, t = _code_parts(S2, e)
    kr = np.uint64(((top + 1) << 25) - 1)
    a = (ay + kr).astype(np.int64)
    assert np.all(a < 2 ** 32)
    s = np.maximum(a - ax.astype(np.int64), 0)
    return (s >> 25) + t


def test_code_float_form_at_thresholds(orc):
    """2S = c_k e + delta for every threshold c_k and small delta, i.e. exactly
    where round(S / e) crosses an I-Log2 step."""
    rng = np.random.default_rng(7)
    cases = []
    for _ in range(4000):
        qL = int(rng.integers(1, 2 ** 24))
        sh = int(rng.integers(0, 31))
        e = qL << sh
        k = int(rng.integers(1, 16))
        ck = 3 if k == 1 else 3 * 2 ** (k - 1) - 1
        for delta in (-2, -1, 0, 1, 2):
            S2 = ck * e + delta
            S2 += S2 & 1                                  # 2S is even
            if S2 < 2 * e or S2 + e + 1 >= 2 ** 52:
                continue
            cases.append((S2, e))
    S2 = np.array([c[0] for c in cases], dtype=np.float64)
    e = np.array([c[1] for c in cases], dtype=np.float64)
    for top in (1, 3, 7, 15, 31, 255):
        got = _code_float(S2, e, top)
        ref = np.array([min(orc.ilog2((a + b) // (2 * b)), top) for a, b in cases])
        assert np.array_equal(got, ref)
        if top <= 15:
            assert np.array_equal(_code_rev_float(S2, e, top), top - ref)


def test_code_float_form_on_rows(orc):
    """Whole rows through the oracle's I-Exp: codes from the float form equal
    the oracle's codes."""
    rng = np.random.default_rng(3)
    for sigma, Lk in [(1.0, 197), (3.0, 197), (6.0, 577), (0.2, 49)]:
        row = np.rint(rng.standard_normal(Lk) * sigma / 2.0 ** -10).astype(np.int32)
        e, ssum = orc.lis_row_exp(row, 2.0 ** -10, 20)
        S2 = 2.0 * float(np.sum(e))
        codes = orc.unpack_codes(orc.lis_softmax_log4(row[None, None, :], 2.0 ** -10), Lk)[0, 0]
        got = _code_float(np.full(Lk, S2), e.astype(np.float64), 15)
        assert np.array_equal(got, codes.astype(np.int64))
        got = _code_rev_float(np.full(Lk, S2), e.astype(np.float64), 15)
        assert np.array_equal(got, 15 - codes.astype(np.int64))
