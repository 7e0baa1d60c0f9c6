"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test ties an oracle function to something other than itself: a value the
paper prints, a closed form, an invariant, a special case that reduces to a
textbook routine or a library primitive, or the paper's error bound.  None of
these tests touches the GPU.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
S = 2.0 ** -10


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def ilog2_closed_form(r: int) -> int:
    """M + chi with chi the bit below the leading one is the integer k with
    3 * 2^k <= 4 r < 3 * 2^(k+1), i.e. floor(log2(4 r / 3)): rounding log2 at
    1.5 * 2^M.  Written with exact integers."""
    k = 0
    while 3 * 2 ** (k + 1) <= 4 * r:
        k += 1
    return k


# ---------------------------------------------------------------------------
# I-Log2 (Algorithm 2)
# ---------------------------------------------------------------------------

def test_ilog2_worked_example(orc):
    (binary, M, chi, result), = _golden("ilog2_worked_example.txt")
    q = int(binary, 2)
    assert q == 3500
    assert orc.ilog2(q) == int(result) == int(M) + int(chi)


def test_ilog2_closed_form_exhaustive(orc):
    # every r < 2^16 exhaustively, then a strided sweep to 2^20 and powers of two
    rs = list(range(1, 1 << 16)) + list(range(1 << 16, 1 << 20, 97))
    rs += [1 << k for k in range(0, 62)] + [(1 << k) - 1 for k in range(2, 62)]
    rs += [3 << k for k in range(0, 60)] + [(3 << k) - 1 for k in range(1, 60)]
    bad = [r for r in rs if orc.ilog2(r) != ilog2_closed_form(r)]
    assert not bad, bad[:10]


# ---------------------------------------------------------------------------
# I-Exp (Algorithm 1)
# ---------------------------------------------------------------------------

def test_iexp_constants_golden(orc):
    g = {k: int(v) for k, v in _golden("iexp_constants_s2m10.txt")}
    k = orc.iexp_constants(S, 20)
    assert (k.q_ln2, k.q_b, k.q_c) == (g["q_ln2"], g["q_b"], g["q_c"])
    assert orc.iexp(0, k)[0] == g["iexp0_n20"]
    poly = {k_: float(v) for k_, v in _golden("iexp_polynomial.txt")}
    assert math.isclose(k.s_L, poly["a"] * S * S, rel_tol=1e-15)


def _iexp_table(orc, s, n):
    k = orc.iexp_constants(s, n)
    ts = np.arange(n * k.q_ln2 - 3 * abs(k.q_ln2), 1)
    e = np.array([orc.iexp(int(t), k)[0] for t in ts], dtype=np.float64)
    return k, ts, e


@pytest.mark.parametrize("s", [2.0 ** -10, 1e-3, 2.0 ** -12, 1.2e-4])
def test_iexp_error_bound(orc, s):
    """|s_L e / 2^n - exp(s t)| stays within the polynomial's gap.  The paper
    states 1.9e-3; its own polynomial peaks at 2.13e-3 near p = -0.138, so the
    bound tested is 2.2e-3 (the floors of q_b, q_c add < 1e-4 at these scales)."""
    n = 20
    k, ts, e = _iexp_table(orc, s, n)
    approx = k.s_L * e / 2.0 ** n
    err = np.abs(approx - np.exp(s * ts))
    assert err.max() <= 2.2e-3
    # the continuous polynomial itself: its max gap on (-ln2, 0] is above the stated value
    p = np.linspace(-math.log(2), 0, 200001)
    gap = np.abs(0.3585 * (p + 1.353) ** 2 + 0.344 - np.exp(p)).max()
    assert 1.9e-3 < gap < 2.2e-3


def test_iexp_halves_per_ln2_step(orc):
    """i-exp = L(p) >> z: moving the input down by |q_ln2| keeps p and adds one to
    z, so the output halves exactly (until the clamp at n q_ln2)."""
    n = 20
    k = orc.iexp_constants(S, n)
    for t in range(-5 * abs(k.q_ln2), 1, 7):
        t2 = t + k.q_ln2
        if t2 < n * k.q_ln2:
            continue
        e1, z1, p1 = orc.iexp(t, k)
        e2, z2, p2 = orc.iexp(t2, k)
        assert (z2, p2) == (z1 + 1, p1)
        assert e1 == 2 * e2


def test_iexp_decomposition_and_monotone(orc):
    """t = z q_ln2 + q_p with z >= 0 and q_p in (q_ln2, 0]; outputs are
    non-decreasing in t; below n q_ln2 the input is clamped."""
    n = 20
    k, ts, e = _iexp_table(orc, S, n)
    for t in ts[:: 13]:
        out, z, qp = orc.iexp(int(t), k)
        tc = max(int(t), n * k.q_ln2)
        assert z >= 0 and k.q_ln2 < qp <= 0
        assert tc == z * k.q_ln2 + qp
        assert out == ((qp + k.q_b) ** 2 + k.q_c) * 2 ** (n - z)
    assert np.all(np.diff(e) >= 0)
    assert orc.iexp(n * k.q_ln2 - 12345, k)[0] == orc.iexp(n * k.q_ln2, k)[0]


# ---------------------------------------------------------------------------
# Log-Int-Softmax (Algorithm 2 + the clip of the LIS equation)
# ---------------------------------------------------------------------------

def test_lis_flat_rows_golden(orc):
    for Lk, code in _golden("lis_flat_rows.txt"):
        Lk, code = int(Lk), int(code)
        for val in (0, 12345, -777777):
            row = np.full((1, 3, Lk), val, dtype=np.int32)
            c = orc.unpack_codes(orc.lis_softmax_log4(row, S), Lk)
            assert np.all(c == code), (Lk, val)


def test_lis_dominant_max(orc):
    """A max far above the rest: the max gets Attn_Q = 0, every clamped entry 15."""
    rng = np.random.default_rng(5)
    for Lk in (2, 9, 49, 197, 577):
        row = rng.integers(-100000, -50000, size=(1, 4, Lk)).astype(np.int32)
        j = rng.integers(0, Lk, size=4)
        row[0, np.arange(4), j] = 10 ** 6
        c = orc.unpack_codes(orc.lis_softmax_log4(row, S), Lk)[0]
        assert np.all(c[np.arange(4), j] == 0)
        mask = np.ones_like(c, dtype=bool)
        mask[np.arange(4), j] = False
        assert np.all(c[mask] == 15)


def _codes_and_e(orc, logits, s=S, n=20, bias=None):
    G, Lq, Lk = logits.shape
    codes = orc.unpack_codes(orc.lis_softmax_log4(logits, s, exp_n=n, bias=bias), Lk)
    return codes


def test_lis_reciprocal_and_log2_steps_exact(orc):
    """From the oracle's i-exp values, recompute q_rev = round(sum/e) (ties up)
    as an exact Fraction and Attn_Q with the closed form of I-Log2."""
    a = W.attn_inputs(3, 16, 37, 8, seed=11, heads=3, sigma=(1.0, 3.0, 6.0))
    codes = _codes_and_e(orc, a["logits"])
    for g in range(3):
        for i in range(16):
            e, _ = orc.lis_row_exp(a["logits"][g, i], S)
            tot = int(e.astype(object).sum())
            for j in range(37):
                frac = Fraction(tot, int(e[j]))
                q_rev = math.floor(frac + Fraction(1, 2))
                assert codes[g, i, j] == min(ilog2_closed_form(q_rev), 15)


def test_lis_range_monotone_argmax(orc):
    """Codes lie in [0, 15], never increase with the logit, and the row maximum
    gets the row's smallest code."""
    for cfg in W.CONFIGS:
        a = W.attn_inputs(4, min(cfg.Lq, 64), cfg.Lk, 8, seed=cfg.seed, heads=cfg.heads,
                          sigma=cfg.sigma, bias=cfg.bias)
        lg = a["logits"].astype(np.int64)
        if a["bias"] is not None:
            lg = lg + a["bias"][np.arange(4) % a["Hb"]][:, : lg.shape[1]]
            a["bias"] = np.ascontiguousarray(a["bias"][:, : lg.shape[1]])
        c = _codes_and_e(orc, a["logits"], bias=a["bias"])
        assert c.min() >= 0 and c.max() <= 15
        order = np.argsort(lg, axis=-1, kind="stable")
        cs = np.take_along_axis(c, order, axis=-1)
        assert np.all(np.diff(cs.astype(np.int64), axis=-1) <= 0)
        am = lg.argmax(-1)
        assert np.all(np.take_along_axis(c, am[..., None], -1)[..., 0] == c.min(-1))


def test_lis_shift_and_bias_invariance(orc):
    """Subtracting the row max makes LIS invariant to a per-row constant, and the
    bias is part of the logit (adding it in the input is the same)."""
    a = W.attn_inputs(6, 20, 49, 8, seed=3, heads=3, bias=True)
    base = _codes_and_e(orc, a["logits"], bias=a["bias"])
    shifted = (a["logits"].astype(np.int64) + np.arange(20)[None, :, None] * 12345 - 4242)
    c2 = _codes_and_e(orc, shifted.astype(np.int32), bias=a["bias"])
    assert np.array_equal(base, c2)
    folded = a["logits"] + a["bias"][np.arange(6) % 3]
    c3 = _codes_and_e(orc, folded.astype(np.int32))
    assert np.array_equal(base, c3)


def test_lis_row_sum_bound(orc):
    """0.625 (1 - (Lk-1)/49151.5) <= sum_j 2^-Attn_Q < 1.5 + (Lk-1)/32768: each
    unclipped entry lies within [0.625, 1.5) of its i-exp probability and each
    clipped entry is 2^-15."""
    for cfg in W.CONFIGS:
        a = W.attn_inputs(4, min(cfg.Lq, 96), cfg.Lk, 8, seed=cfg.seed, heads=cfg.heads,
                          sigma=cfg.sigma)
        c = _codes_and_e(orc, a["logits"])
        rs = (2.0 ** -c.astype(np.float64)).sum(-1)
        Lk = cfg.Lk
        assert rs.min() >= 0.625 * (1 - (Lk - 1) / 49151.5)
        assert rs.max() < 1.5 + (Lk - 1) / 32768


def test_lis_against_float_softmax(orc):
    """Secondary checks: the i-exp probabilities e/sum are within L1 0.05 of the
    float softmax per row, and Attn_Q is within 1 of the float log2 quantizer
    clip(round(-log2 softmax), 0, 15) of Sec. 3.3."""
    worst_l1, worst_code = 0.0, 0
    for cfg in W.CONFIGS:
        a = W.attn_inputs(2, min(cfg.Lq, 48), cfg.Lk, 8, seed=cfg.seed, heads=cfg.heads,
                          sigma=cfg.sigma)
        c = _codes_and_e(orc, a["logits"])
        for g in range(2):
            for i in range(a["logits"].shape[1]):
                row = a["logits"][g, i].astype(np.float64) * S
                sm = np.exp(row - row.max())
                sm /= sm.sum()
                e, tot = orc.lis_row_exp(a["logits"][g, i], S)
                l1 = np.abs(e / e.sum() - sm).sum()
                worst_l1 = max(worst_l1, l1)
                fq = np.clip(np.rint(-np.log2(np.maximum(sm, 1e-300))), 0, 15)
                worst_code = max(worst_code, int(np.abs(fq - c[g, i]).max()))
    assert worst_l1 <= 0.05
    assert worst_code <= 1


def test_lis_lower_bits_clip(orc):
    """With b-bit codes the clip is at 2^b - 1 and agrees with the 4-bit codes below it."""
    a = W.attn_inputs(2, 10, 49, 8, seed=9)
    c4 = _codes_and_e(orc, a["logits"])
    for bits in (1, 2, 3):
        cb = orc.unpack_codes(orc.lis_softmax_log4(a["logits"], S, bits=bits), 49)
        assert np.array_equal(cb, np.minimum(c4, 2 ** bits - 1))


def test_lis_wide_codes_exact(orc):
    """Codes of 5 to 8 bits (one per byte): exact rational q_rev = round(sum/e)
    (ties up) through the closed form of I-Log2, clipped at 2^b - 1; below 15
    they agree with the 4-bit codes, and rows wide enough in spread reach codes
    above 15.  Bytes past Lk in a wider row stride are left alone."""
    a = W.attn_inputs(2, 12, 41, 8, seed=13, heads=2, sigma=(6.0, 9.0))
    c4 = _codes_and_e(orc, a["logits"])
    seen_wide = False
    for bits in (5, 6, 8):
        stored = orc.lis_softmax_log4(a["logits"], S, bits=bits, ld_codes=44)
        assert np.all(stored[..., 41:] == 0)
        cb = orc.unpack_codes(stored, 41, bits)
        assert np.array_equal(np.minimum(cb, 15), c4)
        for g in range(2):
            for i in range(12):
                e, _ = orc.lis_row_exp(a["logits"][g, i], S)
                tot = int(e.astype(object).sum())
                for j in range(41):
                    q_rev = math.floor(Fraction(tot, int(e[j])) + Fraction(1, 2))
                    assert cb[g, i, j] == min(ilog2_closed_form(q_rev), 2 ** bits - 1)
        seen_wide |= bool((cb > 15).any())
    assert seen_wide


def test_lis_packing_layout(orc):
    """Two codes per byte, even key in the low nibble; bytes past ceil(Lk/2) in a
    wider row stride are left alone; an odd tail's high nibble is zero."""
    a = W.attn_inputs(2, 5, 9, 8, seed=1)
    dense = orc.lis_softmax_log4(a["logits"], S)
    wide = orc.lis_softmax_log4(a["logits"], S, ld_codes=8)
    assert np.array_equal(wide[..., :5], dense)
    assert np.all(wide[..., 5:] == 0)
    assert np.all((dense[..., -1] >> 4) == 0)
    c = orc.unpack_codes(dense, 9)
    assert np.array_equal(dense[..., 0], c[..., 0] | (c[..., 1] << 4))


# ---------------------------------------------------------------------------
# BitShift Attn x V (Sec. 3.3, Supplement A.2)
# ---------------------------------------------------------------------------

def test_attn_v_equals_power_of_two_matmul(orc):
    """Shift-accumulate equals the integer matrix product P (V - zp_V) with
    P_ij = 2^(N - Attn_Q_ij), computed by numpy's int64 matmul."""
    rng = np.random.default_rng(4)
    for (G, Lq, Lk, d, bits, zp) in [(3, 7, 9, 5, 4, 0), (2, 17, 33, 16, 4, -3),
                                     (1, 5, 1, 3, 4, 7), (2, 6, 11, 4, 2, 1)]:
        v = rng.integers(-128, 128, size=(G, Lk, d)).astype(np.int8)
        codes = rng.integers(0, 2 ** bits, size=(G, Lq, Lk))
        # keep the sums inside int32
        codes[:, :, :] = np.maximum(codes, 0)
        ld = (Lk + 1) // 2
        packed = np.zeros((G, Lq, ld), dtype=np.uint8)
        for j in range(Lk):
            packed[..., j // 2] |= (codes[..., j] << (4 * (j % 2))).astype(np.uint8)
        out = orc.lis_attn_v_shift(packed, v, zp_v=zp, bits=bits, Lk=Lk)
        N = 2 ** bits - 1
        P = (2 ** (N - codes)).astype(np.int64)
        ref = np.matmul(P, v.astype(np.int64) - zp)
        assert np.array_equal(out.astype(np.int64), ref)


def test_attn_v_single_element_exhaustive(orc):
    """Every (code, V, zp_V) for one key: out = (V - zp_V) * 2^(15 - code)."""
    vals = np.arange(-128, 128, dtype=np.int64)
    for zp in (-128, -1, 0, 5, 127):
        for code in range(16):
            v = vals.astype(np.int8).reshape(1, 1, 256)
            packed = np.full((1, 1, 1), code, dtype=np.uint8)
            out = orc.lis_attn_v_shift(packed, v, zp_v=zp, bits=4, Lk=1)
            assert np.array_equal(out[0, 0].astype(np.int64), (vals - zp) << (15 - code))


def test_head_is_lis_then_attn_v(orc):
    a = W.attn_inputs(5, 13, 49, 32, seed=7, heads=3, bias=True)
    out, codes = orc.lis_attention_head(a["logits"], a["v"], S, bias=a["bias"], want_codes=True)
    c2 = orc.lis_softmax_log4(a["logits"], S, bias=a["bias"])
    assert np.array_equal(codes, c2)
    assert np.array_equal(out, orc.lis_attn_v_shift(c2, a["v"], Lk=49))


# ---------------------------------------------------------------------------
# BitShift Attn x V for wide codes (b in [5, 8])
# ---------------------------------------------------------------------------

def _pack(codes, bits):
    """[..., Lk] codes -> stored form: nibbles (even key low) for bits <= 4, bytes above."""
    if bits > 4:
        return np.ascontiguousarray(codes.astype(np.uint8))
    Lk = codes.shape[-1]
    ld = (Lk + 1) // 2
    packed = np.zeros(codes.shape[:-1] + (ld,), dtype=np.uint8)
    for j in range(Lk):
        packed[..., j // 2] |= (codes[..., j] << (4 * (j % 2))).astype(np.uint8)
    return packed


def _wide_w(bits):
    return min(2 ** bits - 1, 44)


def test_attn_v_wide_equals_narrow_for_4_bits_or_less(orc):
    rng = np.random.default_rng(61)
    for bits in (1, 2, 3, 4):
        codes = rng.integers(0, 2 ** bits, size=(3, 7, 33))
        v = rng.integers(-128, 128, size=(3, 33, 20)).astype(np.int8)
        pk = _pack(codes, bits)
        narrow = orc.lis_attn_v_shift(pk, v, zp_v=5, bits=bits, Lk=33).astype(np.int64)
        assert np.array_equal(orc.lis_attn_v_shift_wide(pk, v, zp_v=5, bits=bits, Lk=33), narrow)


@pytest.mark.parametrize("bits", [5, 6, 8])
def test_attn_v_wide_single_element_exhaustive(orc, bits):
    """One key, one column: every code the storage holds (0 .. 2^b - 1) times
    every byte value and three zero points, against the floor of the exact
    product (v - zp) 2^(W - code) in Python integers (>> floors)."""
    W = _wide_w(bits)
    codes = np.arange(2 ** bits)
    vals = np.arange(-128, 128)
    for zp in (0, -7, 127):
        cc = np.repeat(codes, vals.size).reshape(1, -1, 1)          # rows = (code, v) pairs
        vv = np.tile(vals, codes.size)
        # unit g = pair: 1 query row, 1 key, 1 column
        G = cc.shape[1]
        got = orc.lis_attn_v_shift_wide(_pack(cc.reshape(G, 1, 1), bits),
                                        vv.astype(np.int8).reshape(G, 1, 1), zp_v=zp, bits=bits, Lk=1)
        want = [((int(v) - zp) << (W - int(c))) if c <= W else ((int(v) - zp) >> (int(c) - W))
                for c, v in zip(cc.ravel(), vv)]
        assert np.array_equal(got.ravel(), np.array(want, dtype=np.int64)), (bits, zp)


def test_attn_v_wide_on_lis_codes_is_exact(orc):
    """8-bit Log-Int-Softmax codes of spread rows never exceed W = 44, and the
    product is then the integer matrix product P (V - zp) with
    P = 2^(44 - code) (numpy int64, a textbook routine); the row sums of
    2^-code stay below 1.5 (no clip acts at 8 bits)."""
    for s, n, sigma in ((2.0 ** -10, 20, 9.0), (2e-4, 30, 9.0), (0.05, 30, 60.0)):
        a = W.attn_inputs(3, 20, 577, 48, seed=17, sigma=(sigma,), s_logit=s, v_lo=-128, v_hi=127)
        pk = orc.lis_softmax_log4(a["logits"], s, bits=8, exp_n=n)
        codes = pk[..., :577].astype(np.int64)
        assert codes.max() <= 44 and codes.max() > 15
        assert np.sum(np.ldexp(1.0, -codes), axis=-1).max() < 1.5
        got = orc.lis_attn_v_shift_wide(pk, a["v"], zp_v=-3, bits=8, Lk=577)
        P = np.left_shift(np.int64(1), 44 - codes)
        ref = np.matmul(P, a["v"].astype(np.int64) + 3)
        assert np.array_equal(got, ref), (s, n)


def test_lis_code_bound_44_at_extreme_parameters(orc):
    """The largest codes Log-Int-Softmax produces within the accepted
    parameters: Lk = 4096 keys, all at the maximum but one far below it.  That
    key is clamped (z = n, p = 0), so its I-Exp value equals q_b^2 + q_c while
    every other key has (q_b^2 + q_c) 2^n: round(S / e) = 4095 2^n exactly,
    whose leading one is bit n + 11 with the bit below it set, so its code is
    n + 12 (42 at n = 30, the deepest clamp, with s = 0.5, the coarsest scale;
    32 at n = 20).  Both stay within the wide product's exponent W = 44."""
    for s, n in ((0.5, 30), (2.0 ** -10, 20), (1e-3, 25)):
        lg = np.zeros((1, 1, 4096), dtype=np.int32)
        lg[0, 0, 0] = -(2 ** 29)
        pk = orc.lis_softmax_log4(lg, s, bits=8, exp_n=n)
        assert int(pk[0, 0, 0]) == n + 12 <= 44, (s, n, int(pk[0, 0, 0]))


# ---------------------------------------------------------------------------
# PTF quantizer (Sec. 3.2)
# ---------------------------------------------------------------------------

def test_ptf_K0_is_minmax(orc):
    """K = 0 makes eq. (9)-(10) the MinMax parameters of eq. (5), and eq. (8) with
    alpha = 0 the uniform quantizer of eq. (3), bit for bit."""
    X = W.ln_inputs(64, 48, seed=0)["x_float"]
    s_p, zp_p = orc.ptf_params(X, b=8, K=0)
    s_m, zp_m = orc.minmax_params(X, b=8)
    assert (s_p, zp_p) == (s_m, zp_m)
    q_p = orc.ptf_quantize(X, s_p, zp_p, np.zeros(48, np.uint8))
    q_m = orc.minmax_quantize(X, s_m, zp_m)
    assert np.array_equal(q_p, q_m)


def test_ptf_alpha_K_is_minmax(orc):
    """alpha = K on every channel puts every channel on the MinMax grid 2^K s."""
    X = W.ln_inputs(64, 48, seed=1)["x_float"]
    s_p, zp_p = orc.ptf_params(X, b=8, K=3)
    s_m, zp_m = orc.minmax_params(X, b=8)
    assert zp_p == zp_m and s_p * 8 == s_m
    q_p = orc.ptf_quantize(X, s_p, zp_p, np.full(48, 3, np.uint8))
    assert np.array_equal(q_p, orc.minmax_quantize(X, s_m, zp_m))


def test_ptf_alpha_search_outliers(orc):
    """The argmin of eq. (11) gives the widest channels the largest factor and
    narrow channels the finest grid; a narrower grid never loses on a channel
    that it holds without clipping."""
    ln = W.ln_inputs(197, 96, seed=2, outliers=4)
    X = ln["x_float"]
    s, zp = orc.ptf_params(X, b=8, K=3)
    alpha = orc.ptf_alpha(X, s, zp, b=8, K=3)
    rng_c = X.max(0) - X.min(0)
    widest = np.argsort(rng_c)[-4:]
    assert np.all(alpha[widest] == 3)
    narrow = rng_c < 0.5 * np.median(rng_c)
    assert np.all(alpha[narrow] == 0)
    assert np.all(np.diff(alpha[np.argsort(rng_c)].astype(int)) >= -1)


def _exact_ptf_errors(x, s, zp, K, b=8):
    """Exact rational errors of eq. (11) per channel and alpha, [C][K+1]: the
    quantized value of eq. (8) from the binary64 quotient x / (2^alpha s)
    rounded half to even (Python's float division and round() are both
    IEEE), then the exact squared residual, summed exactly."""
    from fractions import Fraction as F
    levels = 2 ** b - 1
    T, C = x.shape
    err = [[F(0)] * (K + 1) for _ in range(C)]
    for c in range(C):
        for a in range(K + 1):
            step = F(s) * 2 ** a
            step_d = s * 2.0 ** a
            tot = F(0)
            for t in range(T):
                xd = float(x[t, c])
                q = min(max(round(xd / step_d) + zp, 0), levels)
                tot += (F(xd) - (q - zp) * step) ** 2
            err[c][a] = tot
    return err


def _exact_argmin(errs):
    """argmin with ties to the smallest index."""
    best = 0
    for a in range(1, len(errs)):
        if errs[a] < errs[best]:
            best = a
    return best


def test_ptf_alpha_matches_exact_argmin(orc):
    """The alpha search against exact rational arithmetic on every channel:
    the oracle's argmin is the exact argmin (ties to the smallest alpha) and
    its reported errors are the exact ones rounded to binary64 (one unit in
    the last place).  Channel 0 holds all its information in its last rows,
    channel 1 is all zeros (every alpha exact: the tie goes to alpha = 0),
    channel 4 is an outlier channel."""
    rng = np.random.default_rng(41)
    T, C, K = 150, 12, 3
    x = (rng.standard_normal((T, C)) * np.exp(rng.uniform(np.log(0.05), np.log(2.5), C))).astype(np.float32)
    x[:, 4] *= 40.0
    x[:128, 0] = 0.0
    x[128:, 0] = rng.uniform(-30, 30, T - 128).astype(np.float32)
    x[:, 1] = 0.0
    xd = x.astype(np.float64)
    s, zp = orc.ptf_params(xd, b=8, K=K)
    alpha = orc.ptf_alpha(xd, s, zp, b=8, K=K)
    got_err, got_lo = orc.ptf_alpha_errors(xd, s, zp, b=8, K=K, with_lo=True)
    err = _exact_ptf_errors(xd, s, zp, K)
    from fractions import Fraction as F
    for c in range(C):
        assert alpha[c] == _exact_argmin(err[c]), (c, [float(e) for e in err[c]])
        for a in range(K + 1):
            want = float(err[c][a])
            assert abs(got_err[c, a] - want) <= np.spacing(want), (c, a, got_err[c, a], want)
            # hi + lo carries the exact value to about 106 bits
            assert abs(F(got_err[c, a]) + F(got_lo[c, a]) - err[c][a]) <= err[c][a] * F(1, 2 ** 100)
    assert alpha[1] == 0 and alpha[4] >= 2
    assert alpha[0] != 0          # decided by the last rows alone


def _near_tie_channel(rng, eps_units, s, n_common=600):
    """One channel (values in units of s, all exact binary64 with s a power of
    two) on which alpha = 0 and alpha = 1 of eq. (11) (b = 8, zp = 250, so the
    grid of alpha = 0 ends at 5 s) have errors that differ by exactly
    2 eps_units s^2:
      * common rows (2m + f) s, |f| < 1/2: the same nearest point on both
        grids, the same residual;
      * two rows (2m + 1.25) s: residual 0.25 s on the grid s, 0.75 s on 2 s;
      * one row (6 + eps_units) s above the grid of alpha = 0: clipped to 5 s
        there (residual (1 + eps) s), residual eps s on the grid 2 s.
    The two rows cost alpha = 1 exactly s^2 more, the last row costs alpha = 0
    (1 + eps)^2 s^2 - eps^2 s^2 = (1 + 2 eps) s^2 more: the errors tie for
    eps = 0 and differ by 2 eps s^2 otherwise."""
    m = rng.integers(-100, 3, size=n_common)
    f = rng.choice([-0.375, -0.25, -0.125, 0.125, 0.25, 0.375], size=n_common)
    vals = list((2 * m + f) * s)
    vals += [(2 * -7 + 1.25) * s, (2 * 1 + 1.25) * s]
    vals.append((6.0 + eps_units) * s)
    return np.array(vals, dtype=np.float64)


def test_ptf_alpha_exact_ties_and_near_ties(orc):
    """eq. (11) evaluated exactly: an exact tie between alpha = 0 and alpha = 1
    (both errors non-zero) goes to alpha = 0, and errors that differ by a
    less than one unit in the last place of their binary64 value (a plain
    binary64 sum of the terms, in row order, reversed or in 64-row blocks,
    orders them wrongly or ties them) are ordered by their exact values.  The expected alphas come
    from the construction and are re-derived in Fractions."""
    s, zp, K = 2.0 ** -7, 250, 1
    rng = np.random.default_rng(7)
    # 6 + eps is exact in binary64 for these eps (its unit in the last place is 2^-50)
    eps = [0.0, 2.0 ** -50, -2.0 ** -50, 2.0 ** -49, -2.0 ** -48]
    cols = [_near_tie_channel(rng, e, s) for e in eps]
    x = np.stack(cols, axis=1)
    alpha = orc.ptf_alpha(x, s, zp, b=8, K=K)
    want = [0, 1, 0, 1, 0]
    err = _exact_ptf_errors(x, s, zp, K)
    for c, e in enumerate(eps):
        gap = err[c][0] - err[c][1]
        from fractions import Fraction as F
        assert gap == 2 * F(e) * F(s) ** 2, (c, gap)
        assert err[c][0] > 0 and err[c][1] > 0
        assert _exact_argmin(err[c]) == want[c]
        if e != 0.0:
            # below one unit in the last place of the binary64 total: any
            # rounded sum of the squared residuals sees a tie or the wrong order
            assert abs(gap) <= np.spacing(float(err[c][0]))
    assert list(alpha) == want


# ---------------------------------------------------------------------------
# Integer Q K^T (Sec. 3.1 int MatMul feeding Sec. 3.3)
# ---------------------------------------------------------------------------

def test_qk_logits_is_integer_matmul(orc):
    """A textbook special case: the logits are the batched int64 matrix product
    of the zero-point-centred operands (numpy), for every zero point pair."""
    rng = np.random.default_rng(51)
    q = rng.integers(-128, 128, size=(3, 17, 64)).astype(np.int8)
    k = rng.integers(-128, 128, size=(3, 29, 64)).astype(np.int8)
    for zq, zk in ((0, 0), (5, -7), (-128, 127)):
        ref = np.matmul(q.astype(np.int64) - zq, np.swapaxes(k.astype(np.int64) - zk, 1, 2))
        assert np.array_equal(orc.qk_logits(q, k, zq, zk).astype(np.int64), ref)


def test_qk_logits_zero_point_shift_invariance(orc):
    """Moving the container grid (values and zero point by the same amount)
    leaves the logits unchanged; q = zp_q gives zero logits."""
    rng = np.random.default_rng(52)
    q = rng.integers(-100, 100, size=(2, 9, 32)).astype(np.int8)
    k = rng.integers(-100, 100, size=(2, 11, 32)).astype(np.int8)
    base = orc.qk_logits(q, k, 3, -4)
    assert np.array_equal(orc.qk_logits((q + 20).astype(np.int8), k, 23, -4), base)
    assert np.array_equal(orc.qk_logits(q, (k - 20).astype(np.int8), 3, -24), base)
    assert not orc.qk_logits(np.full_like(q, 7), k, 7, -4).any()


def test_qk_head_is_logits_then_head(orc):
    """The integer-only MSA from Q, K equals the logits followed by the fused
    Log-Int-Softmax / BitShift head."""
    rng = np.random.default_rng(53)
    q = rng.integers(-128, 128, size=(2, 13, 64)).astype(np.int8)
    k = rng.integers(-128, 128, size=(2, 21, 64)).astype(np.int8)
    v = rng.integers(-127, 128, size=(2, 21, 16)).astype(np.int8)
    s = 1.0 / 1800.0
    out = orc.lis_attention_qk(q, k, v, s, zp_q=2, zp_k=-3)
    assert np.array_equal(out, orc.lis_attention_head(orc.qk_logits(q, k, 2, -3), v, s))


# ---------------------------------------------------------------------------
# Dyadic requantization
# ---------------------------------------------------------------------------

def _round_half_up(fr):
    return (fr + Fraction(1, 2)).numerator // (fr + Fraction(1, 2)).denominator


def test_requant_power_of_two_is_exact(orc):
    """A power-of-two multiplier has an exact dyadic form: the output is the
    exact q 2^k rounded half up, plus zp, clipped to the b-bit grid."""
    q = np.arange(-70000, 70000, 7, dtype=np.int32)
    for k in (-12, -5, -1, 0, 1, 3):
        for bits, zp in ((8, 0), (8, -100), (8, 127), (4, -3), (2, 1)):
            y = orc.requant_dyadic_int8(q, float(2.0 ** k), 1.0, zp, bits)
            half, levels = 2 ** (bits - 1), 2 ** bits - 1
            ref = [min(max(_round_half_up(Fraction(int(v)) * Fraction(2) ** k) + zp + half, 0), levels) - half
                   for v in q]
            assert np.array_equal(y.astype(np.int64), np.array(ref)), (k, bits, zp)


def test_requant_matches_exact_product_within_31_bits(orc):
    """For any multiplier M = s_in / s_out, the output equals round-half-up of
    the exact q M wherever q M + 1/2 is farther than |q| M 2^-30 (the bound of
    a 31-bit truncation of M) from an integer, and is never more than one
    step from it.  q is drawn so that q M covers the output range."""
    rng = np.random.default_rng(43)
    for s_in, s_out in ((0.02 / 32768, 0.013), (3.0e-7, 0.5), (1.0, 3.0), (7.0, 0.001)):
        s_in32, s_out32 = np.float32(s_in), np.float32(s_out)
        M = Fraction(float(s_in32)) / Fraction(float(s_out32))
        span = rng.uniform(-300.0, 300.0, size=3000) / float(M)
        q = np.clip(np.rint(span), -(2 ** 31), 2 ** 31 - 1).astype(np.int64).astype(np.int32)
        q[:4] = [0, 1, -1, 2 ** 31 - 1]
        for zp in (0, -17):
            y = orc.requant_dyadic_int8(q, float(s_in32), float(s_out32), zp).astype(np.int64)
            n_exact = 0
            for v, got in zip(q, y):
                exact = Fraction(int(v)) * M
                r = _round_half_up(exact)
                ref = min(max(r + zp + 128, 0), 255) - 128
                assert abs(got - ref) <= 1
                f = exact + Fraction(1, 2) - r          # in [0, 1)
                if min(f, 1 - f) > abs(int(v)) * M * Fraction(1, 2 ** 30):
                    assert got == ref, (s_in, s_out, int(v))
                    n_exact += 1
            assert n_exact > 0.99 * len(q)


# ---------------------------------------------------------------------------
# Integer LayerNorm with PTF (Supplement A.1)
# ---------------------------------------------------------------------------

def float_ln_requant(x_q, zp_in, alpha, s_in, gamma, beta, s_out, zp_out, bits=8, eps=1e-6):
    """fp64 LayerNorm (Sec. 3.2, eq. 7) of the dequantized PTF input, quantized
    with (s_out, zp_out) onto the int8 container."""
    half = 2 ** (bits - 1)
    X = (x_q.astype(np.float64) - zp_in) * (2.0 ** alpha.astype(np.float64)) * s_in
    mu = X.mean(-1, keepdims=True)
    var = X.var(-1, keepdims=True)
    Y = (X - mu) / np.sqrt(var + eps) * gamma.astype(np.float64) + beta.astype(np.float64)
    return np.clip(np.rint(Y / float(np.float32(s_out))) + zp_out + half, 0, 2 ** bits - 1) - half


def _ln(orc, d, x_q=None, alpha=None, gamma=None, beta=None, zp_in=None):
    return orc.ptf_layernorm_int8(d["x_q"] if x_q is None else x_q,
                                  d["zp_in"] if zp_in is None else zp_in,
                                  d["alpha"] if alpha is None else alpha, d["K"],
                                  d["gamma"] if gamma is None else gamma,
                                  d["beta"] if beta is None else beta,
                                  d["s_out"], d["zp_out"], d["bits"])


@pytest.mark.parametrize("cfg", W.CONFIGS, ids=lambda c: c.name)
def test_ln_within_2lsb_of_float(orc, cfg):
    d = W.ln_inputs(min(cfg.T, 1024), cfg.channels, cfg.seed, outliers=cfg.outliers,
                    alpha_uniform=cfg.alpha_uniform)
    y = _ln(orc, d)
    ref = float_ln_requant(d["x_q"], d["zp_in"], d["alpha"], d["s_in"], d["gamma"],
                           d["beta"], d["s_out"], d["zp_out"])
    diff = np.abs(y.astype(np.int64) - ref)
    assert diff.max() <= 2
    assert diff.mean() < 0.05


def test_ln_constant_row_and_zero_gamma(orc):
    """A row whose shifted values X^_Q are all equal has zero variance: its output
    is round(beta/s_out) + zp_out.  A channel with gamma = 0 gives the same value
    on every row."""
    d = W.ln_inputs(16, 64, seed=3)
    x = d["x_q"].copy()
    x[3, :] = (d["zp_in"] + (8 >> np.minimum(d["alpha"], 3))).astype(np.int8)
    x[9, :] = d["zp_in"]
    gamma = d["gamma"].copy()
    gamma[[0, 5, 63]] = 0.0
    y = _ln(orc, d, x_q=x, gamma=gamma)
    expect = np.clip(np.rint(d["beta"].astype(np.float64) / np.float64(np.float32(d["s_out"])))
                     + d["zp_out"], -128, 127)
    assert np.array_equal(y[3], expect.astype(np.int8))
    assert np.array_equal(y[9], expect.astype(np.int8))
    for c in (0, 5, 63):
        assert np.all(y[:, c] == expect[c])


def test_ln_uniform_alpha_is_scale_free(orc):
    """The same alpha = k on every channel scales X^_Q, sqrt(C M2 - M1^2) and hence
    A by exact powers of two: N2 and A X^_Q are unchanged and N1 grows by k.  Only
    round(B 2^N1) moves to a 2^k finer grid, so the output stays within 1 LSB of
    the alpha = 0 output and is almost always identical."""
    d = W.ln_inputs(256, 96, seed=4)
    y0 = _ln(orc, d, alpha=np.zeros(96, np.uint8)).astype(np.int64)
    for k in (1, 2, 3):
        yk = _ln(orc, d, alpha=np.full(96, k, np.uint8)).astype(np.int64)
        assert np.abs(yk - y0).max() <= 1
        assert np.mean(yk != y0) < 0.01


def test_ln_zero_point_shift(orc):
    """Only X_Q - zp enters: shifting the input and its zero point together changes nothing."""
    d = W.ln_inputs(32, 64, seed=5)
    x = d["x_q"].astype(np.int64)
    x = np.clip(x, -100, 100)
    y0 = _ln(orc, d, x_q=x.astype(np.int8))
    y1 = _ln(orc, d, x_q=(x + 20).astype(np.int8), zp_in=d["zp_in"] + 20)
    assert np.array_equal(y0, y1)


def test_ln_alpha_clamped_to_K(orc):
    d = W.ln_inputs(16, 32, seed=6)
    a = d["alpha"].copy()
    a[::3] = 7
    a2 = np.minimum(a, d["K"])
    assert np.array_equal(_ln(orc, d, alpha=a), _ln(orc, d, alpha=a2))


def test_ln_exhaustive_alpha_4x8(orc):
    """All 4^8 alpha vectors on 4 tokens x 8 channels: within 2 LSB of the float
    LayerNorm of the dequantized input."""
    rng = np.random.default_rng(8)
    x_q = rng.integers(-128, 128, size=(4, 8)).astype(np.int8)
    gamma = (1 + 0.5 * rng.standard_normal(8)).astype(np.float32)
    beta = (0.5 * rng.standard_normal(8)).astype(np.float32)
    s_out, zp_out, zp_in = 0.03, -3, 2
    alphas = np.array(np.meshgrid(*[np.arange(4)] * 8, indexing="ij")).reshape(8, -1).T
    worst = 0
    for a in alphas.astype(np.uint8):
        y = orc.ptf_layernorm_int8(x_q, zp_in, a, 3, gamma, beta, s_out, zp_out, 8)
        ref = float_ln_requant(x_q, zp_in, a, 1.0, gamma, beta, s_out, zp_out, eps=0.0)
        worst = max(worst, int(np.abs(y.astype(np.int64) - ref).max()))
    assert worst <= 2


def test_ln_worked_examples_golden(orc):
    """Two one-row examples worked by hand from the Supplement A.1 formulas: the
    b-bit dyadic form of A (N1, N2), round(B 2^N1) and the half-up outer rounding."""
    x_q = np.array([[-126, 126]], dtype=np.int8)
    alpha = np.array([3, 3], dtype=np.uint8)
    gamma = np.array([1.57421875, 1.57421875], dtype=np.float32)
    for beta, y0, y1 in _golden("ln_worked_examples.txt"):
        b = np.array([float(beta)] * 2, dtype=np.float32)
        y = orc.ptf_layernorm_int8(x_q, 0, alpha, 3, gamma, b, 0.015625, 0, 8)
        assert y.tolist() == [[int(y0), int(y1)]]
