"""Parity of the HIP library with the CPU oracle, element by element.

Every integer output must be bit-exact.  Small cases span several tiles and
ragged tails; the full-size configs run the exact launch the benchmark times
and compare every LayerNorm row and every attention unit.  Each case prints
its name before its GPU step."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

S = 2.0 ** -10


@pytest.fixture(scope="module")
def fq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2111_13824_amd as fq
    return fq


def dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def say(*a):
    print("CASE", *a, flush=True)


# ---------------------------------------------------------------------------
# PTF LayerNorm
# ---------------------------------------------------------------------------

def _ln_gpu(fq, d, **over):
    p = dict(d, **over)
    return host(fq.ptf_layernorm_int8(dev(p["x_q"]), p["zp_in"], dev(p["alpha"]), p["K"],
                                      dev(p["gamma"]), dev(p["beta"]), p["s_out"], p["zp_out"],
                                      p["bits"]))


def _ln_ref(orc, d, **over):
    p = dict(d, **over)
    return orc.ptf_layernorm_int8(p["x_q"], p["zp_in"], p["alpha"], p["K"], p["gamma"], p["beta"],
                                  p["s_out"], p["zp_out"], p["bits"])


LN_SHAPES = [(1, 192), (7, 96), (197, 192), (333, 384), (64, 768), (100, 1024), (37, 100),
             (9, 13), (5, 2048), (3, 4096), (2, 8192), (65, 4), (3, 1), (70, 2000),
             # row-batch kernel (256 <= C <= 1024): one row, partial batches,
             # several batches per wavefront, idle lanes in the last dword
             (1, 768), (5, 256), (4099, 260), (20000, 256), (9001, 1020), (16400, 512),
             # rows of < 64 dwords: 8, 16 or 32 lanes per row, four passes per
             # batch, partial batches and idle lanes
             (1001, 96), (50, 128), (3000, 64), (77, 32), (4099, 192), (130, 112)]


@pytest.mark.parametrize("T,C", LN_SHAPES)
def test_ln_shapes(fq, orc, T, C):
    say("ln", T, C)
    d = W.ln_inputs(T, C, seed=T * 31 + C)
    assert np.array_equal(_ln_gpu(fq, d), _ln_ref(orc, d))


# (7001, 512) and (13001, 256) take the row-batch kernel's workgroups of one
# per CU, with two-row and four-row batches
@pytest.mark.parametrize("T,C", [(100, 1024), (7, 768), (13, 256), (101, 512), (4099, 768), (37, 96),
                                 (7001, 512), (13001, 256), (1001, 96), (333, 192), (130, 112)])
def test_ln_writes_only_its_rows(fq, orc, T, C):
    """Every row count, including a last batch of fewer rows than the one
    before it: the output matches and the bytes after it (a guard region in
    the same allocation) are untouched."""
    import torch
    say("ln guard", T, C)
    d = W.ln_inputs(T, C, seed=T + 3 * C)
    buf = torch.full(((T + 16) * C,), 0x5A, dtype=torch.int8, device="cuda:0")
    y = buf[:T * C].view(T, C)
    fq.ptf_layernorm_int8(dev(d["x_q"]), d["zp_in"], dev(d["alpha"]), d["K"], dev(d["gamma"]),
                          dev(d["beta"]), d["s_out"], d["zp_out"], d["bits"], y_q=y)
    out = host(buf)
    assert np.array_equal(out[:T * C].reshape(T, C), _ln_ref(orc, d))
    assert np.all(out[T * C:] == 0x5A)


@pytest.mark.parametrize("K,bits", [(0, 8), (3, 8), (7, 8), (5, 8), (3, 4), (2, 2), (6, 6)])
def test_ln_params(fq, orc, K, bits):
    say("ln params", K, bits)
    rng = np.random.default_rng(K * 10 + bits)
    d = W.ln_inputs(150, 768, seed=5)
    half = 2 ** (bits - 1)
    x = rng.integers(-half, half, size=(150, 768)).astype(np.int8)
    alpha = rng.integers(0, 8, size=768).astype(np.uint8)
    zp = int(rng.integers(-half, half))
    zpo = int(rng.integers(-half, half))
    over = dict(x_q=x, alpha=alpha, K=K, bits=bits, zp_in=zp, zp_out=zpo)
    assert np.array_equal(_ln_gpu(fq, d, **over), _ln_ref(orc, d, **over))


@pytest.mark.parametrize("C", [96, 192, 128])
@pytest.mark.parametrize("K,bits", [(0, 8), (3, 4), (5, 8), (6, 8), (7, 6), (2, 2)])
def test_ln_params_small_rows(fq, orc, C, K, bits):
    """Rows of fewer than 256 channels: the batched-factor kernel while the
    per-lane sums of squares fit 32 bits (K <= 5 at C = 96), the per-lane
    factor kernel beyond."""
    say("ln params small rows", C, K, bits)
    rng = np.random.default_rng(K * 100 + bits * 10 + C)
    T = 777
    d = W.ln_inputs(T, C, seed=C + K)
    half = 2 ** (bits - 1)
    x = rng.integers(-half, half, size=(T, C)).astype(np.int8)
    alpha = rng.integers(0, 8, size=C).astype(np.uint8)
    zp = int(rng.integers(-half, half))
    zpo = int(rng.integers(-half, half))
    over = dict(x_q=x, alpha=alpha, K=K, bits=bits, zp_in=zp, zp_out=zpo)
    assert np.array_equal(_ln_gpu(fq, d, **over), _ln_ref(orc, d, **over))


@pytest.mark.parametrize("C", [384, 96, 768, 1024])
def test_ln_edge_rows(fq, orc, C):
    """Constant rows (zero variance), rows at the zero point, gamma = 0, extreme
    affine values, tiny and huge s_out."""
    say("ln edges", C)
    d = W.ln_inputs(64, C, seed=9)
    x = d["x_q"].copy()
    x[0] = d["zp_in"]
    x[1] = (d["zp_in"] + (8 >> np.minimum(d["alpha"].astype(np.int32), 3))).astype(np.int8)
    x[2] = 127
    x[3] = -128
    gamma = d["gamma"].copy()
    beta = d["beta"].copy()
    gamma[:5] = 0.0
    gamma[5] = -gamma[5]
    gamma[6] = 1e-30
    gamma[7] = 3e4
    beta[8] = 1e6
    beta[9] = -1e6
    for s_out in (d["s_out"], 1e-6, 1e3, 0.5):
        over = dict(x_q=x, gamma=gamma, beta=beta, s_out=s_out)
        assert np.array_equal(_ln_gpu(fq, d, **over), _ln_ref(orc, d, **over)), s_out


@pytest.mark.parametrize("T,C", [(4099, 768), (7001, 768), (13001, 768), (5003, 96), (2001, 192)])
def test_ln_mixed_fast_and_general_rows(fq, orc, T, C):
    """Rows whose factors leave the fast range (near-constant rows: tiny
    variance, huge 1/sigma) between ordinary rows, so that batches of rows
    mix both output paths (T and C pick the kernel, its batch size and its
    workgroup shape)."""
    say("ln mixed rows", T, C)
    d = W.ln_inputs(T, C, seed=12)
    x = d["x_q"].copy()
    rng = np.random.default_rng(12)
    unshifted = np.flatnonzero(np.minimum(d["alpha"], d["K"]) == 0)
    assert unshifted.size > 0
    for i in rng.choice(T, size=300, replace=False):
        x[i] = d["zp_in"]
        x[i, int(rng.choice(unshifted))] += 1 if d["zp_in"] < 127 else -1
    over = dict(x_q=x)
    assert np.array_equal(_ln_gpu(fq, d, **over), _ln_ref(orc, d, **over))


@pytest.mark.parametrize("cfg", W.CONFIGS, ids=lambda c: c.name)
def test_ln_full_config(fq, orc, cfg):
    say("ln full", cfg.name)
    d = W.config_inputs(cfg, "ln")["ln"]
    assert np.array_equal(_ln_gpu(fq, d), _ln_ref(orc, d))


def test_ln_unaligned_pointers(fq, orc):
    """A row-major view starting one byte into an allocation takes the general path."""
    import torch
    say("ln unaligned")
    d = W.ln_inputs(40, 192, seed=2)
    xb = torch.zeros(40 * 192 + 1, dtype=torch.int8, device="cuda:0")
    xb[1:] = dev(d["x_q"]).reshape(-1)
    yb = torch.zeros(40 * 192 + 1, dtype=torch.int8, device="cuda:0")
    x = xb[1:].view(40, 192)
    y = yb[1:].view(40, 192)
    fq.ptf_layernorm_int8(x, d["zp_in"], dev(d["alpha"]), d["K"], dev(d["gamma"]),
                          dev(d["beta"]), d["s_out"], d["zp_out"], d["bits"], y_q=y)
    assert np.array_equal(host(y), _ln_ref(orc, d))


# ---------------------------------------------------------------------------
# Log-Int-Softmax codes
# ---------------------------------------------------------------------------

LIS_SHAPES = [(3, 5, 1), (2, 17, 2), (2, 17, 33), (3, 64, 197), (2, 70, 197), (1, 65, 577),
              (4, 49, 49), (2, 3, 640), (1, 3, 700), (1, 2, 4096), (5, 1, 31), (2, 130, 96)]


@pytest.mark.parametrize("G,Lq,Lk", LIS_SHAPES)
def test_lis_codes_shapes(fq, orc, G, Lq, Lk):
    say("lis", G, Lq, Lk)
    a = W.attn_inputs(G, Lq, Lk, 8, seed=G + Lq + Lk, heads=G, sigma=(1.0, 3.0, 6.0))
    got = host(fq.lis_softmax_log4(dev(a["logits"]), S))
    assert np.array_equal(got, orc.lis_softmax_log4(a["logits"], S))


@pytest.mark.parametrize("s", [0.5, 1e-2, 1e-3, 2.0 ** -10, 2.0 ** -12, 1.2e-4, 1e-4])
@pytest.mark.parametrize("n", [1, 20, 30])
def test_lis_codes_scales(fq, orc, s, n):
    say("lis scale", s, n)
    a = W.attn_inputs(2, 40, 197, 8, seed=3, sigma=(3.0,), s_logit=s)
    try:
        got = host(fq.lis_softmax_log4(dev(a["logits"]), s, exp_n=n))
    except fq.FqError as e:
        assert e.status == 4 and n == 30  # headroom rejection at the deepest clamp
        return
    assert np.array_equal(got, orc.lis_softmax_log4(a["logits"], s, exp_n=n))


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6, 7, 8])
def test_lis_codes_bits(fq, orc, bits):
    say("lis bits", bits)
    a = W.attn_inputs(3, 33, 77, 8, seed=bits)
    got = host(fq.lis_softmax_log4(dev(a["logits"]), S, bits=bits))
    assert np.array_equal(got, orc.lis_softmax_log4(a["logits"], S, bits=bits))


@pytest.mark.parametrize("G,Lq,Lk,bits,sigma", [
    (1024, 17, 197, 8, 9.0),     # unit kernel (enough units for it)
    (6, 40, 300, 6, 6.0),        # tile kernel
    (2, 9, 900, 5, 9.0),         # stream kernel (long rows)
    (1024, 16, 49, 8, 9.0),
])
def test_lis_wide_codes_each_kernel(fq, orc, G, Lq, Lk, bits, sigma):
    """Codes of 5 to 8 bits, one per byte, from every kernel that writes codes,
    on rows spread enough for codes above 15, in a wider row stride whose extra
    bytes stay untouched; integer and float paths."""
    import torch
    say("lis wide codes", G, Lq, Lk, bits)
    a = W.attn_inputs(G, Lq, Lk, 8, seed=G + Lk, sigma=(sigma,))
    for s in (S, 2e-4):
        codes = torch.full((G, Lq, Lk + 3), 0xAB, dtype=torch.uint8, device="cuda:0")
        fq.lis_softmax_log4(dev(a["logits"]), s, bits=bits, codes=codes)
        got = host(codes)
        ref = orc.lis_softmax_log4(a["logits"], s, bits=bits)
        assert np.array_equal(got[..., :Lk], ref), s
        assert np.all(got[..., Lk:] == 0xAB)
        assert got[..., :Lk].max() > 15


def test_lis_codes_bias_and_stride(fq, orc):
    """Swin relative-position bias (head g % Hb) and a wider code row stride whose
    extra bytes must stay untouched."""
    import torch
    say("lis bias stride")
    a = W.attn_inputs(12, 49, 49, 8, seed=4, heads=3, bias=True)
    codes = torch.full((12, 49, 32), 0xAB, dtype=torch.uint8, device="cuda:0")
    fq.lis_softmax_log4(dev(a["logits"]), S, bias=dev(a["bias"]), codes=codes)
    got = host(codes)
    ref = orc.lis_softmax_log4(a["logits"], S, bias=a["bias"])
    assert np.array_equal(got[..., :25], ref)
    assert np.all(got[..., 25:] == 0xAB)


def test_lis_extreme_logits(fq, orc):
    """Logits near +-2^30, flat rows, one-hot rows, rows mixing both ends."""
    say("lis extreme")
    rng = np.random.default_rng(1)
    lg = rng.integers(-(2 ** 30) + 1, 2 ** 30, size=(4, 20, 197)).astype(np.int32)
    lg[0, :5] = 12345
    lg[1, :, :] = -(2 ** 30) + 1
    lg[1, np.arange(20), np.arange(20)] = 2 ** 30 - 1
    lg[2, :, ::2] = 0
    got = host(fq.lis_softmax_log4(dev(lg), S))
    assert np.array_equal(got, orc.lis_softmax_log4(lg, S))


# ---------------------------------------------------------------------------
# BitShift Attn x V and the fused head
# ---------------------------------------------------------------------------

def _random_codes(rng, G, Lq, Lk, bits=4):
    codes = rng.integers(0, 2 ** bits, size=(G, Lq, Lk))
    ld = (Lk + 1) // 2
    packed = np.zeros((G, Lq, ld), dtype=np.uint8)
    for j in range(Lk):
        packed[..., j // 2] |= (codes[..., j] << (4 * (j % 2))).astype(np.uint8)
    return packed


@pytest.mark.parametrize("G,Lq,Lk,d,zp", [(2, 5, 1, 64, 0), (3, 17, 33, 16, 3), (2, 64, 197, 64, 0),
                                          (2, 70, 197, 17, -7), (1, 9, 577, 64, 0),
                                          (4, 49, 49, 32, 0), (1, 3, 700, 256, 1), (2, 20, 96, 100, 0)])
def test_attn_v_shift(fq, orc, G, Lq, Lk, d, zp):
    say("av", G, Lq, Lk, d, zp)
    rng = np.random.default_rng(G * Lk + d)
    a = W.attn_inputs(G, Lq, Lk, d, seed=7, v_lo=-128, v_hi=127)
    codes = orc.lis_softmax_log4(a["logits"], S) if Lk > 1 else _random_codes(rng, G, Lq, Lk)
    got = host(fq.lis_attn_v_shift(dev(codes), dev(a["v"]), Lk, zp_v=zp))
    assert np.array_equal(got, orc.lis_attn_v_shift(codes, a["v"], zp_v=zp, Lk=Lk))


def test_attn_v_shift_any_codes(fq, orc):
    """Arbitrary codes (not from LIS), including small-bit widths."""
    say("av any codes")
    rng = np.random.default_rng(3)
    for bits in (1, 2, 3, 4):
        codes = _random_codes(rng, 2, 33, 65, bits)
        v = rng.integers(-128, 128, size=(2, 65, 48)).astype(np.int8)
        got = host(fq.lis_attn_v_shift(dev(codes), dev(v), 65, zp_v=-3, bits=bits))
        assert np.array_equal(got, orc.lis_attn_v_shift(codes, v, zp_v=-3, bits=bits, Lk=65))


# The product on the int8 matrix cores (rows of up to 1024 keys, d <= 64):
# code rows that start at every byte alignment and with padded strides, key
# counts on and around the 64-key steps, one- to four-range splits of P
# (bits 1..4), row counts that leave ragged tiles, every zero point sign;
# rows of more than 1024 keys or d > 64 take the vector-ALU kernel.
AV_MFMA = [(3, 33, 64, 64, 4, 0, 5), (2, 17, 65, 48, 4, 1, -128), (2, 40, 127, 20, 3, 2, 127),
           (5, 16, 128, 64, 2, 3, 0), (2, 9, 1024, 32, 4, 5, -1), (3, 20, 300, 64, 1, 0, 9),
           (2, 50, 197, 33, 4, 7, -4), (2, 3, 1025, 64, 4, 0, 2), (2, 10, 200, 80, 4, 1, 3)]


@pytest.mark.parametrize("G,Lq,Lk,d,bits,shift,zp", AV_MFMA)
def test_attn_v_shift_layouts(fq, orc, G, Lq, Lk, d, bits, shift, zp):
    """Arbitrary codes of b bits in a buffer whose rows start `shift` bytes
    into an allocation and are `shift` bytes longer than ceil(Lk/2) (the
    bytes between rows and the unused high nibble of an odd row hold
    garbage)."""
    import torch
    say("av layouts", G, Lq, Lk, d, bits, shift, zp)
    rng = np.random.default_rng(Lk * 7 + d + bits)
    nb = (Lk + 1) // 2
    ld = nb + shift
    codes = rng.integers(0, 2 ** bits, size=(G, Lq, Lk))
    packed = rng.integers(0, 256, size=(G, Lq, ld)).astype(np.uint8)
    packed[..., :nb] = 0
    for j in range(Lk):
        packed[..., j // 2] |= (codes[..., j] << (4 * (j % 2))).astype(np.uint8)
    if Lk % 2:
        packed[..., nb - 1] |= (rng.integers(0, 16, size=(G, Lq)) << 4).astype(np.uint8)
    v = rng.integers(-128, 128, size=(G, Lk, d)).astype(np.int8)
    buf = torch.zeros(G * Lq * ld + shift + 64, dtype=torch.uint8, device="cuda")
    buf[shift:shift + G * Lq * ld] = dev(packed.reshape(-1))
    view = buf[shift:shift + G * Lq * ld].view(G, Lq, ld)
    got = host(fq.lis_attn_v_shift(view, dev(v), Lk, zp_v=zp, bits=bits))
    assert np.array_equal(got, orc.lis_attn_v_shift(packed, v, zp_v=zp, bits=bits, Lk=Lk))


def test_attn_v_shift_full_vit_base(fq, orc):
    """The unfused head of the ViT-B/16 batch-64 workload: GPU codes, then the
    standalone product, against the oracle on every unit (threads)."""
    import concurrent.futures as cf
    import os
    say("av full vit_b")
    cfg = W.BY_NAME["vit_base16_224_b64"]
    a = W.config_inputs(cfg, "attn")["attn"]
    codes = fq.lis_softmax_log4(dev(a["logits"]), a["s_logit"])
    got = host(fq.lis_attn_v_shift(codes, dev(a["v"]), cfg.Lk, zp_v=a["zp_v"]))
    ch = host(codes)
    parts = np.array_split(np.arange(cfg.G), min(16, os.cpu_count() or 1))
    def one(ix):
        return orc.lis_attn_v_shift(np.ascontiguousarray(ch[ix]), np.ascontiguousarray(a["v"][ix]),
                                    zp_v=a["zp_v"], Lk=cfg.Lk)
    with cf.ThreadPoolExecutor(len(parts)) as ex:
        ref = np.concatenate(list(ex.map(one, parts)))
    assert np.array_equal(got, ref)


def _stored_codes(codes, bits):
    """[..., Lk] codes -> stored form (nibbles for bits <= 4, bytes above)."""
    if bits > 4:
        return np.ascontiguousarray(codes.astype(np.uint8))
    Lk = codes.shape[-1]
    packed = np.zeros(codes.shape[:-1] + ((Lk + 1) // 2,), dtype=np.uint8)
    for j in range(Lk):
        packed[..., j // 2] |= (codes[..., j] << (4 * (j % 2))).astype(np.uint8)
    return packed


@pytest.mark.parametrize("G,Lq,Lk,d,bits", [(2, 5, 1, 64, 8), (3, 17, 33, 16, 8), (2, 64, 197, 64, 8),
                                            (2, 70, 197, 17, 6), (1, 9, 577, 64, 8), (4, 49, 49, 32, 5),
                                            (1, 3, 700, 256, 8), (2, 20, 96, 100, 7),
                                            (2, 33, 65, 48, 4), (2, 30, 40, 8, 2)])
def test_attn_v_shift_wide(fq, orc, G, Lq, Lk, d, bits):
    """The wide BitShift product on Log-Int-Softmax codes of b bits (spread rows,
    so that 8-bit codes pass 15) and on arbitrary codes of every stored value,
    above the output exponent W = min(2^b - 1, 44) too (the floor path)."""
    say("av wide", G, Lq, Lk, d, bits)
    rng = np.random.default_rng(G * Lk + d + bits)
    a = W.attn_inputs(G, Lq, Lk, d, seed=13, sigma=(9.0,), s_logit=2e-4, v_lo=-128, v_hi=127)
    lis = orc.lis_softmax_log4(a["logits"], 2e-4, bits=bits, exp_n=30) if Lk > 1 else None
    anyc = _stored_codes(rng.integers(0, 2 ** bits, size=(G, Lq, Lk)), bits)
    for codes in ([lis] if lis is not None else []) + [anyc]:
        got = host(fq.lis_attn_v_shift_wide(dev(codes), dev(a["v"]), Lk, zp_v=-5, bits=bits))
        assert got.dtype == np.int64
        assert np.array_equal(got, orc.lis_attn_v_shift_wide(codes, a["v"], zp_v=-5, bits=bits, Lk=Lk))


@pytest.mark.parametrize("bits,d", [(1, 1), (2, 4), (3, 40)])
def test_attn_v_wide_nibbles_above_N(fq, orc, bits, d):
    """Nibble codes of b <= 3 bits with stored values above N = 2^b - 1 (never
    written by Log-Int-Softmax): the units holding one are computed again
    term by term (the floor of the shifted value), beside units without."""
    say("av wide nibbles above N", bits, d)
    rng = np.random.default_rng(90 + bits)
    G, Lq, Lk = 6, 21, 130
    codes = rng.integers(0, 2 ** bits, size=(G, Lq, Lk))
    codes[1, 3, 7] = 15
    codes[4, :, 100:] = rng.integers(0, 16, size=(Lq, Lk - 100))
    pk = _stored_codes(codes, 4)
    v = rng.integers(-128, 128, size=(G, Lk, d)).astype(np.int8)
    got = host(fq.lis_attn_v_shift_wide(dev(pk), dev(v), Lk, zp_v=6, bits=bits))
    assert np.array_equal(got, orc.lis_attn_v_shift_wide(pk, v, zp_v=6, bits=bits, Lk=Lk))


@pytest.mark.parametrize("d,zp", [(1, 0), (4, -3), (8, 7)])
def test_attn_v_shift_small_head_dims(fq, orc, d, zp):
    """Head dimensions that take the byte-wise V^T staging and the scalar
    output stores of the matrix-core product."""
    say("av small d", d, zp)
    rng = np.random.default_rng(d + 40)
    a = W.attn_inputs(3, 37, 150, d, seed=d, v_lo=-128, v_hi=127)
    codes = orc.lis_softmax_log4(a["logits"], S)
    got = host(fq.lis_attn_v_shift(dev(codes), dev(a["v"]), 150, zp_v=zp))
    assert np.array_equal(got, orc.lis_attn_v_shift(codes, a["v"], zp_v=zp, Lk=150))
    anyc = _random_codes(rng, 3, 37, 150)
    got = host(fq.lis_attn_v_shift(dev(anyc), dev(a["v"]), 150, zp_v=zp))
    assert np.array_equal(got, orc.lis_attn_v_shift(anyc, a["v"], zp_v=zp, Lk=150))


def test_attention_888_full_vit_base(fq, orc):
    """The 8/8/8 attention of the ViT-B/16 batch-64 workload: 8-bit
    Log-Int-Softmax codes on the GPU, then the wide BitShift product, against
    the same chain in the oracle (every unit; oracle split over host threads)."""
    import concurrent.futures as cf
    import os
    say("attention 8/8/8 full vit_b")
    cfg = W.BY_NAME["vit_base16_224_b64"]
    a = W.config_inputs(cfg, "attn")["attn"]
    codes = fq.lis_softmax_log4(dev(a["logits"]), a["s_logit"], bits=8, exp_n=a["exp_n"])
    out = host(fq.lis_attn_v_shift_wide(codes, dev(a["v"]), cfg.Lk, zp_v=a["zp_v"], bits=8))
    got_codes = host(codes)
    G = cfg.G
    bounds = np.linspace(0, G, 65).astype(int)

    def run(k):
        g0, g1 = bounds[k], bounds[k + 1]
        c = orc.lis_softmax_log4(a["logits"][g0:g1], a["s_logit"], bits=8, exp_n=a["exp_n"])
        return c, orc.lis_attn_v_shift_wide(c, a["v"][g0:g1], zp_v=a["zp_v"], bits=8)

    with cf.ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        parts = list(ex.map(run, range(64)))
    assert np.array_equal(got_codes, np.concatenate([p[0] for p in parts]))
    assert got_codes.max() > 15
    assert np.array_equal(out, np.concatenate([p[1] for p in parts]))


# (2, 40, 288, 64) and (2, 33, 270, 32): the longest rows of the fused tile
# kernels (9 chunks of 32 keys); (2, 40, 290, 64): the shortest that takes the
# stream kernel, with (2, 40, 350, 64), (2, 33, 384, 32) and (2, 40, 400, 64)
HEAD_SHAPES = [(3, 5, 1, 64), (2, 17, 33, 16), (3, 64, 197, 64), (2, 70, 197, 64), (1, 65, 577, 64),
               (12, 49, 49, 32), (2, 3, 640, 64), (1, 3, 700, 64), (1, 2, 4096, 32), (2, 20, 96, 100),
               (2, 33, 65, 256), (2, 19, 129, 1), (2, 40, 288, 64), (2, 33, 270, 32),
               (2, 40, 290, 64), (2, 40, 350, 64), (2, 33, 384, 32), (2, 40, 400, 64)]


@pytest.mark.parametrize("G,Lq,Lk,d", HEAD_SHAPES)
def test_head_shapes(fq, orc, G, Lq, Lk, d):
    say("head", G, Lq, Lk, d)
    a = W.attn_inputs(G, Lq, Lk, d, seed=G * 7 + Lk, heads=G, sigma=(1.0, 3.0, 6.0), v_lo=-128,
                      v_hi=127)
    got = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, zp_v=-2))
    ref = orc.lis_attention_head(a["logits"], a["v"], S, zp_v=-2)
    assert np.array_equal(got, ref)


# Long rows (10 to 20 chunks of 32 keys) take the long-row kernel: logits read
# once, I-Exp from an LDS table.
LONG_SHAPES = [(3, 70, 577, 64, 0), (2, 33, 289, 32, 0), (2, 17, 640, 64, 2), (3, 50, 400, 17, 3),
               (2, 40, 313, 48, 2), (4, 16, 336, 64, 0), (2, 1, 600, 8, 0)]


@pytest.mark.parametrize("G,Lq,Lk,d,Hb", LONG_SHAPES)
def test_head_long_rows(fq, orc, G, Lq, Lk, d, Hb):
    say("head long", G, Lq, Lk, d, Hb)
    a = W.attn_inputs(G, Lq, Lk, d, seed=G + Lq + Lk, heads=max(Hb, 1), sigma=(1.0, 3.0, 6.0),
                      v_lo=-128, v_hi=127, bias=Hb > 0)
    bias = dev(a["bias"]) if Hb else None
    got = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, zp_v=-4, bias=bias))
    assert np.array_equal(got, orc.lis_attention_head(a["logits"], a["v"], S, zp_v=-4, bias=a["bias"]))


def test_head_long_rows_wide_span(fq, orc):
    """Rows whose logits span more than 2^15 units (a tile holding one of them
    is computed from the logits again), beside ordinary tiles, in units whose
    first chunk does not hold the row maximum."""
    say("head long wide span")
    a = W.attn_inputs(3, 100, 577, 64, seed=31, sigma=(3.0,), v_lo=-128, v_hi=127)
    lg = a["logits"].copy()
    lg[0, 5, 500] = 2 ** 24                  # tile 0 of unit 0
    lg[1, 40, 300] = lg[1, 40].max() + 40000  # tile 2 of unit 1
    lg[2, :, 400:] += 20000                  # every row: maximum far from the first chunk
    lg[2, 99, 0] = -(2 ** 29)
    got = host(fq.lis_attention_head(dev(lg), dev(a["v"]), S))
    assert np.array_equal(got, orc.lis_attention_head(lg, a["v"], S))


@pytest.mark.parametrize("n", [23, 25])
def test_head_long_rows_clamp_depth(fq, orc, n):
    """n = 23: an I-Exp table of 16331 entries (65 KB of LDS beside V^T); n = 25:
    beyond the table's 16-bit offsets, the stream kernel."""
    say("head long depth", n)
    a = W.attn_inputs(2, 40, 577, 64, seed=n, sigma=(6.0,))
    got = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, exp_n=n))
    assert np.array_equal(got, orc.lis_attention_head(a["logits"], a["v"], S, exp_n=n))


# Shapes with enough units that the launch takes the one-workgroup-per-unit
# kernel (G * min(4, ceil(Lq / 16)) >= 2048): half and full last chunks, waves
# with several 16-row tiles, head dimensions that take the byte-wise V loads
# (d % 16 != 0) and the scalar output stores (d % 4 != 0).
UNIT_SHAPES = [(1024, 17, 16, 64), (1024, 17, 17, 64), (1024, 20, 100, 64), (512, 70, 197, 64),
               (600, 49, 49, 32), (512, 65, 224, 64), (700, 33, 120, 48), (700, 33, 120, 20),
               (2048, 2, 40, 17), (2048, 1, 5, 64),
               # rows of five to seven chunks, whose fused kernels mask the last
               # chunk at its use and prefetch two chunks ahead
               (512, 50, 150, 32), (512, 64, 170, 64), (520, 49, 180, 20), (512, 70, 200, 16)]


@pytest.mark.parametrize("G,Lq,Lk,d", UNIT_SHAPES)
def test_head_unit_kernel(fq, orc, G, Lq, Lk, d):
    say("head unit", G, Lq, Lk, d)
    a = W.attn_inputs(G, Lq, Lk, d, seed=G + Lk + d, heads=G, sigma=(1.0, 3.0, 6.0), v_lo=-128,
                      v_hi=127)
    got = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, zp_v=3))
    ref = orc.lis_attention_head(a["logits"], a["v"], S, zp_v=3)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("G,Lq,Lk,bits,shift", [(512, 70, 197, 4, 1), (1024, 20, 100, 8, 3),
                                                 (600, 33, 197, 8, 2), (2048, 1, 33, 5, 1),
                                                 (512, 17, 63, 4, 0)])
def test_codes_unit_kernel_dense_rows(fq, orc, G, Lq, Lk, bits, shift):
    """Dense code rows (ld_codes = row bytes) are gathered per 16-row tile in
    LDS and written as one span: a codes tensor starting 0..3 bytes past a
    dword boundary, guard bytes before and after it left untouched."""
    import torch
    say("codes unit dense", G, Lq, Lk, bits, shift)
    a = W.attn_inputs(G, Lq, Lk, 1, seed=5 * G + Lk + bits, heads=G, sigma=(1.0, 3.0, 6.0))
    nb = Lk if bits > 4 else (Lk + 1) // 2
    n = G * Lq * nb
    buf = torch.full((n + shift + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    codes = buf[shift:shift + n].view(G, Lq, nb)
    fq.lis_softmax_log4(dev(a["logits"]), S, bits=bits, codes=codes)
    got = host(buf)
    assert np.all(got[:shift] == 0xA5) and np.all(got[shift + n:] == 0xA5)
    ref = orc.lis_softmax_log4(a["logits"], S, bits=bits)
    assert np.array_equal(got[shift:shift + n].reshape(G, Lq, nb), ref[..., :nb])


@pytest.mark.parametrize("G,Lq,Lk", [(1024, 17, 16), (1024, 20, 100), (512, 70, 197),
                                     (2048, 1, 33)])
def test_codes_unit_kernel(fq, orc, G, Lq, Lk):
    say("codes unit", G, Lq, Lk)
    a = W.attn_inputs(G, Lq, Lk, 1, seed=3 * G + Lk, heads=G, sigma=(1.0, 3.0, 6.0))
    got = host(fq.lis_softmax_log4(dev(a["logits"]), S))
    assert np.array_equal(got, orc.lis_softmax_log4(a["logits"], S))


@pytest.mark.parametrize("s", [1e-4, 0.5, 0.0009765625])
def test_head_integer_and_float_paths(fq, orc, s):
    """s = 1e-4 exceeds the float path's 2^24 bound on q_b^2 + q_c and runs the
    integer path; the others run the float path, on both kernels."""
    for G, Lq, Lk, d in [(3, 40, 197, 64), (1024, 17, 100, 64)]:
        say("head path", s, G, Lq, Lk, d)
        a = W.attn_inputs(G, Lq, Lk, d, seed=5 + G, heads=G, s_logit=s, sigma=(0.5, 2.0, 8.0))
        got = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), s))
        assert np.array_equal(got, orc.lis_attention_head(a["logits"], a["v"], s))


def test_prepared_calls_match_direct(fq, orc):
    import torch
    say("prepared")
    a = W.attn_inputs(1024, 17, 100, 64, seed=9, heads=4)
    lg, v = dev(a["logits"]), dev(a["v"])
    out = torch.empty((1024, 17, 64), dtype=torch.int32, device="cuda:0")
    call = fq.lis_attention_head(lg, v, S, out=out, prepare=True)
    call()
    assert np.array_equal(host(out), host(fq.lis_attention_head(lg, v, S)))
    d = W.ln_inputs(100, 768, seed=4)
    y = torch.empty((100, 768), dtype=torch.int8, device="cuda:0")
    fq.ptf_layernorm_int8(dev(d["x_q"]), d["zp_in"], dev(d["alpha"]), d["K"], dev(d["gamma"]),
                          dev(d["beta"]), d["s_out"], d["zp_out"], d["bits"], y_q=y, prepare=True)()
    assert np.array_equal(host(y), _ln_ref(orc, d))


def test_swin_shifted_window_mask_in_bias(fq, orc):
    """A shifted-window mask folds into the bias planes: with units ordered
    (image, window, head), the bias is mask[window] + relative-position
    bias[head], passed as [windows x heads, Lq, Lk]."""
    say("swin shifted-window mask as bias")
    H, nW, B = 3, 4, 2
    a = W.attn_inputs(B * nW * H, 49, 49, 32, seed=21, heads=H, bias=True)
    mask = W.shifted_window_mask(14, 7, 3, -int(100 / S))
    comb = (mask[:, None, :, :] + a["bias"][None, :, :, :]).reshape(nW * H, 49, 49)
    comb = np.ascontiguousarray(comb.astype(np.int32))
    out = fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, bias=dev(comb))
    assert np.array_equal(host(out), orc.lis_attention_head(a["logits"], a["v"], S, bias=comb))
    codes = fq.lis_softmax_log4(dev(a["logits"]), S, bias=dev(comb))
    assert np.array_equal(host(codes), orc.lis_softmax_log4(a["logits"], S, bias=comb))


def test_head_codes_out_and_unfused_equal(fq, orc):
    """The fused head writes the same codes as lis_softmax_log4, and its output
    equals lis_attn_v_shift of those codes (MFMA product vs VALU shifts)."""
    import torch
    say("head vs unfused")
    a = W.attn_inputs(12, 49, 49, 32, seed=11, heads=3, bias=True)
    codes = torch.zeros((12, 49, 25), dtype=torch.uint8, device="cuda:0")
    out = fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), S, bias=dev(a["bias"]),
                                codes_out=codes)
    c2 = fq.lis_softmax_log4(dev(a["logits"]), S, bias=dev(a["bias"]))
    out2 = fq.lis_attn_v_shift(c2, dev(a["v"]), 49)
    assert np.array_equal(host(codes), host(c2))
    assert np.array_equal(host(out), host(out2))
    assert np.array_equal(host(out), orc.lis_attention_head(a["logits"], a["v"], S, bias=a["bias"]))


def test_head_dominant_rows_saturate_exactly(fq, orc):
    """Rows whose codes are all 0 but one produce the largest sums the LIS bound
    allows; the MFMA accumulation must stay exact there."""
    say("head dominant")
    lg = np.full((2, 64, 197), -(2 ** 29), dtype=np.int32)
    lg[:, np.arange(64), np.arange(64)] = 2 ** 29
    v = np.full((2, 197, 64), 127, dtype=np.int8)
    v[1] = -128
    got = host(fq.lis_attention_head(dev(lg), dev(v), S, zp_v=127))
    assert np.array_equal(got, orc.lis_attention_head(lg, v, S, zp_v=127))


def test_empty_calls_are_noops(fq):
    import torch
    say("empty")
    z = torch.zeros((0, 5, 7), dtype=torch.int32, device="cuda:0")
    v = torch.zeros((0, 7, 8), dtype=torch.int8, device="cuda:0")
    assert fq.lis_attention_head(z, v, S).shape == (0, 5, 8)
    x = torch.zeros((0, 16), dtype=torch.int8, device="cuda:0")
    al = torch.zeros(16, dtype=torch.uint8, device="cuda:0")
    gm = torch.ones(16, dtype=torch.float32, device="cuda:0")
    assert fq.ptf_layernorm_int8(x, 0, al, 3, gm, gm, 0.1, 0).shape == (0, 16)


# ---------------------------------------------------------------------------
# Full-size configs (the benchmark's launch), every unit
# ---------------------------------------------------------------------------

def oracle_head_threads(orc, a, workers=None):
    """The oracle's fused head over all units, split into contiguous unit
    ranges run on host threads (ctypes releases the GIL during each call).
    A range starting at unit g0 gets the bias planes (g0 .. g1 - 1) % Hb, so
    each unit keeps its own head's plane."""
    import concurrent.futures as cf
    import os
    G = a["logits"].shape[0]
    workers = workers or max(1, min(16, os.cpu_count() or 1))
    bounds = np.linspace(0, G, min(G, 4 * workers) + 1).astype(int)

    def run(k):
        g0, g1 = bounds[k], bounds[k + 1]
        b = None
        if a["bias"] is not None:
            b = np.ascontiguousarray(a["bias"][np.arange(g0, g1) % a["bias"].shape[0]])
        return orc.lis_attention_head(a["logits"][g0:g1], a["v"][g0:g1], a["s_logit"], a["bits"],
                                      a["exp_n"], a["zp_v"], bias=b)

    with cf.ThreadPoolExecutor(workers) as ex:
        parts = list(ex.map(run, range(len(bounds) - 1)))
    return np.concatenate(parts, axis=0)


@pytest.mark.parametrize("cfg", W.CONFIGS, ids=lambda c: c.name)
def test_head_full_config(fq, orc, cfg):
    say("head full", cfg.name)
    a = W.config_inputs(cfg, "attn")["attn"]
    bias = dev(a["bias"]) if a["bias"] is not None else None
    out = host(fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), a["s_logit"], a["bits"],
                                     a["exp_n"], a["zp_v"], bias=bias))
    ref = oracle_head_threads(orc, a)
    assert out.shape == ref.shape
    bad = np.argwhere(np.any(out != ref, axis=(1, 2))).ravel()
    assert bad.size == 0, f"{bad.size} of {cfg.G} units differ, first {bad[:8]}"
