"""Parity of the GPU PTF calibration, PTF quantizer and dyadic requantization
with the CPU oracle: the scale and the zero point bit for bit, every channel's
alpha under the stated tie rule (check_alpha), every quantized and
requantized element.  Inputs are the generator's
float activations (log-uniform channel scales, optional outlier channels)
rounded to binary32; the oracle sees the same values in binary64."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


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


def acts(T, C, seed, outliers=0):
    return W.ln_inputs(T, C, seed=seed, outliers=outliers)["x_float"].astype(np.float32)


U = 2.0 ** -53


def alpha_error_bounds(x64, s, zp, bits, K):
    """[C, K + 1] bound on how far the GPU's value of each candidate's error
    (every term rounded in binary64: the dequantized value, the residual and
    its square, then a sum of T terms in any order) can be from the exact one:
    (T + 8) u sum_t (|x| + 2 |deq|)^2, u = 2^-53.  Per term the three
    roundings move the square by at most 3.1 u (|x - deq| + |deq|)^2 and the
    sum adds at most (T - 1) u times the sum of the terms; |x - deq| + |deq|
    <= |x| + 2 |deq|.  The margin of 1.01 covers numpy's own rounding here."""
    T = x64.shape[0]
    levels = 2 ** bits - 1
    bound = np.empty((x64.shape[1], K + 1))
    for a in range(K + 1):
        step = s * 2.0 ** a
        q = np.clip(np.rint(x64 / step) + zp, 0, levels)
        deq = (q - zp) * step
        bound[:, a] = (T + 8) * U * np.sum((np.abs(x64) + 2 * np.abs(deq)) ** 2, axis=0) * 1.01
    return bound


def check_alpha(got, x64, s, zp, bits, K, orc):
    """The tie rule of the GPU's alpha: it must be the oracle's (the exact
    argmin of eq. 11, ties to the smallest alpha) unless the exact errors of
    the two candidates are within the sum of their bounds, where either is
    accepted.  Returns the number of channels decided inside that band."""
    ref = orc.ptf_alpha(x64, s, zp, b=bits, K=K)
    err = orc.ptf_alpha_errors(x64, s, zp, b=bits, K=K)
    bound = alpha_error_bounds(x64, s, zp, bits, K)
    in_band = 0
    for c in range(got.size):
        g, r = int(got[c]), int(ref[c])
        near = [a for a in range(K + 1)
                if a != r and err[c, a] - err[c, r] <= bound[c, a] + bound[c, r]]
        in_band += bool(near)
        if g != r:
            assert g in near, (c, g, r, err[c], bound[c])
    return ref, in_band


def _calib_check(fq, orc, x, bits, K):
    s, zp, alpha = fq.ptf_calibrate(dev(x), bits=bits, K=K)
    x64 = x.astype(np.float64)
    s_ref, zp_ref = orc.ptf_params(x64, b=bits, K=K)
    assert host(s)[0] == s_ref                      # binary64, bit for bit
    assert host(zp)[0] == zp_ref - 2 ** (bits - 1)  # container form
    alpha_ref, in_band = check_alpha(host(alpha), x64, s_ref, zp_ref, bits, K, orc)
    print(f"alpha: {x.shape[1]} channels, {in_band} with a candidate inside the rounding band",
          flush=True)
    return s, zp, alpha, s_ref, zp_ref, alpha_ref


# (20000, 40): 313 row blocks, more than one LDS pass of the per-channel sums
CAL_SHAPES = [(1, 5, 0), (65, 13, 0), (197, 192, 0), (150, 96, 4), (1576, 384, 0),
              (4099, 768, 8), (130, 1000, 2), (20000, 40, 1)]


@pytest.mark.parametrize("T,C,outliers", CAL_SHAPES)
def test_calibrate_shapes(fq, orc, T, C, outliers):
    say("calibrate", T, C, outliers)
    _calib_check(fq, orc, acts(T, C, seed=T + C, outliers=outliers), 8, 3)


@pytest.mark.parametrize("bits,K", [(8, 0), (8, 7), (4, 3), (2, 1), (6, 5)])
def test_calibrate_params(fq, orc, bits, K):
    say("calibrate params", bits, K)
    _calib_check(fq, orc, acts(300, 160, seed=bits * 10 + K, outliers=3), bits, K)


def test_calibrate_full_vit_base(fq, orc):
    """The ViT-B/16 batch-64 LayerNorm input: 12608 x 768 with 8 outlier channels."""
    say("calibrate full vit_b")
    cfg = W.BY_NAME["vit_base16_224_b64"]
    x = acts(cfg.T, cfg.channels, seed=2, outliers=cfg.outliers)
    _, _, alpha, _, _, _ = _calib_check(fq, orc, x, 8, 3)
    assert host(alpha).max() == 3


def test_calibrate_degenerate_and_ties(fq, orc):
    """A constant tensor gets s = 0, zp = 0 on the paper's grid and alpha = 0;
    an all-zero channel ties every alpha (0 wins); a channel whose only data
    sits in the partial last 64-row block is decided by that block."""
    say("calibrate degenerate")
    x = np.full((70, 9), 1.25, dtype=np.float32)
    s, zp, alpha = fq.ptf_calibrate(dev(x), bits=8, K=3)
    assert host(s)[0] == 0.0 and host(zp)[0] == -128 and not host(alpha).any()
    x = acts(150, 12, seed=41)
    x[:, 1] = 0.0
    x[:128, 0] = 0.0
    x[128:, 0] = np.linspace(-30, 30, 22, dtype=np.float32)
    _calib_check(fq, orc, x, 8, 3)


def test_calibrate_reused_workspace(fq, orc):
    """The workspace's contents on entry do not matter: two different tensors
    through one workspace, the second smaller."""
    import torch
    say("calibrate workspace reuse")
    ws = torch.full((fq.ptf_calibrate_workspace_bytes(900, 200, 3),), 0x7F, dtype=torch.uint8,
                    device="cuda:0")
    for T, C, seed in ((900, 200, 1), (333, 150, 2)):
        x = acts(T, C, seed=seed, outliers=2)
        s, zp, alpha = fq.ptf_calibrate(dev(x), bits=8, K=3, workspace=ws)
        s_ref, zp_ref = orc.ptf_params(x.astype(np.float64))
        assert host(s)[0] == s_ref and host(zp)[0] == zp_ref - 128
        check_alpha(host(alpha), x.astype(np.float64), s_ref, zp_ref, 8, 3, orc)


@pytest.mark.parametrize("T,C", [(1, 4), (7, 13), (197, 192), (1000, 768), (33, 1001)])
def test_quantize(fq, orc, T, C):
    say("quantize", T, C)
    x = acts(T, C, seed=C, outliers=min(4, C // 8))
    s, zp, alpha, s_ref, zp_ref, alpha_ref = _calib_check(fq, orc, x, 8, 3)
    got = host(fq.ptf_quantize_int8(dev(x), s, zp, alpha))
    # the quantizer given the alphas the GPU chose (equal to the oracle's
    # outside the tie band checked above)
    ref = orc.ptf_quantize(x.astype(np.float64), s_ref, zp_ref, host(alpha)) - 128
    assert np.array_equal(got.astype(np.int64), ref)


def test_quantize_any_alpha_and_bits(fq, orc):
    """alpha as given (also above K), b = 4, and a view that starts 4 bytes into
    its allocation (scalar path)."""
    import torch
    say("quantize alpha bits")
    T, C = 64, 100
    x = acts(T, C, seed=5)
    rng = np.random.default_rng(5)
    alpha = rng.integers(0, 10, size=C).astype(np.uint8)
    s_ref, zp_ref = orc.ptf_params(x.astype(np.float64), b=4, K=3)
    s = torch.tensor([s_ref], dtype=torch.float64, device="cuda:0")
    zp = torch.tensor([zp_ref - 8], dtype=torch.int32, device="cuda:0")
    xb = torch.zeros(T * C + 1, dtype=torch.float32, device="cuda:0")
    xb[1:] = dev(x).reshape(-1)
    got = host(fq.ptf_quantize_int8(xb[1:].view(T, C), s, zp, dev(alpha), bits=4))
    ref = orc.ptf_quantize(x.astype(np.float64), s_ref, zp_ref, alpha, b=4) - 8
    assert np.array_equal(got.astype(np.int64), ref)


def test_calibrate_quantize_layernorm_chain(fq, orc):
    """Float activations -> calibration -> PTF quantization -> PTF LayerNorm,
    all on the GPU, against the same chain in the oracle."""
    say("calibrate-quantize-ln chain")
    d = W.ln_inputs(2000, 768, seed=9, outliers=8)
    x = d["x_float"].astype(np.float32)
    s, zp, alpha, s_ref, zp_ref, alpha_ref = _calib_check(fq, orc, x, 8, 3)
    xq = fq.ptf_quantize_int8(dev(x), s, zp, alpha)
    zp_c = int(host(zp)[0])
    y = host(fq.ptf_layernorm_int8(xq, zp_c, alpha, 3, dev(d["gamma"]), dev(d["beta"]),
                                   d["s_out"], d["zp_out"]))
    a_gpu = host(alpha)      # the oracle's outside the tie band (checked above)
    xq_ref = (orc.ptf_quantize(x.astype(np.float64), s_ref, zp_ref, a_gpu) - 128).astype(np.int8)
    y_ref = orc.ptf_layernorm_int8(xq_ref, zp_ref - 128, a_gpu, 3, d["gamma"], d["beta"],
                                   d["s_out"], d["zp_out"])
    assert np.array_equal(y, y_ref)


@pytest.mark.parametrize("cfg", [c for c in W.CONFIGS if not c.alpha_uniform], ids=lambda c: c.name)
def test_calibrated_chain_full_config(fq, orc, cfg):
    """The full LayerNorm input of each workload whose alphas come from eq. (11)
    (all but ViT-L, whose recipe draws them uniformly), as float activations:
    GPU calibration -> PTF quantization -> PTF LayerNorm against the oracle's
    chain, every element."""
    say("calibrated chain full", cfg.name)
    d = W.config_inputs(cfg, "ln")["ln"]
    x = d["x_float"].astype(np.float32)
    s, zp, alpha, s_ref, zp_ref, _ = _calib_check(fq, orc, x, 8, 3)
    xq = fq.ptf_quantize_int8(dev(x), s, zp, alpha)
    y = host(fq.ptf_layernorm_int8(xq, int(host(zp)[0]), alpha, 3, dev(d["gamma"]),
                                   dev(d["beta"]), d["s_out"], d["zp_out"]))
    a_gpu = host(alpha)
    xq_ref = (orc.ptf_quantize(x.astype(np.float64), s_ref, zp_ref, a_gpu) - 128).astype(np.int8)
    assert np.array_equal(host(xq), xq_ref)
    y_ref = orc.ptf_layernorm_int8(xq_ref, zp_ref - 128, a_gpu, 3, d["gamma"], d["beta"],
                                   d["s_out"], d["zp_out"])
    assert np.array_equal(y, y_ref)


REQ = [(0.02 / 32768, 0.013, 0, 8), (0.02 / 32768, 0.013, -37, 8), (3.0e-7, 0.5, 5, 8),
       (1.0, 3.0, 0, 4), (7.0, 0.001, 1, 2), (0.25, 1.0, 100, 8), (1e-12, 1.0, 0, 8),
       (5.0e4, 1e-3, -128, 8)]


@pytest.mark.parametrize("s_in,s_out,zp,bits", REQ)
def test_requant(fq, orc, s_in, s_out, zp, bits):
    say("requant", s_in, s_out, zp, bits)
    rng = np.random.default_rng(abs(zp) + bits)
    s_in32, s_out32 = float(np.float32(s_in)), float(np.float32(s_out))
    span = rng.uniform(-300, 300, size=100003) * s_out32 / s_in32
    q = np.clip(np.rint(span), -2 ** 31, 2 ** 31 - 1).astype(np.int64).astype(np.int32)
    q[:6] = [0, 1, -1, 2 ** 31 - 1, -2 ** 31, 12345]
    got = host(fq.requant_dyadic_int8(dev(q), s_in32, s_out32, zp, bits))
    assert np.array_equal(got, orc.requant_dyadic_int8(q, s_in32, s_out32, zp, bits))


def test_requant_of_attention_output(fq, orc):
    """The fused head's int32 output (scale s_V / 2^15) requantized to the
    next layer's int8 input, against the oracle head followed by the oracle
    requantization; odd sizes and an offset view take the scalar path."""
    import torch
    say("requant attention output")
    a = W.attn_inputs(6, 49, 49, 32, seed=3)
    out = fq.lis_attention_head(dev(a["logits"]), dev(a["v"]), a["s_logit"])
    out_ref = orc.lis_attention_head(a["logits"], a["v"], a["s_logit"])
    assert np.array_equal(host(out), out_ref)
    s_in = float(np.float32(0.02 / 32768))
    got = host(fq.requant_dyadic_int8(out, s_in, 0.011, -3))
    assert np.array_equal(got, orc.requant_dyadic_int8(out_ref, s_in, 0.011, -3))
    flat = out.reshape(-1)
    qb = torch.zeros(flat.numel() + 1, dtype=torch.int32, device="cuda:0")
    qb[1:] = flat
    got = host(fq.requant_dyadic_int8(qb[1:][:1001], s_in, 0.011, -3))
    assert np.array_equal(got, orc.requant_dyadic_int8(out_ref.reshape(-1)[:1001], s_in, 0.011, -3))
