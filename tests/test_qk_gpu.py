"""Parity of the integer-only attention from int8 Q and K (Q K^T on MFMA,
Log-Int-Softmax and BitShift Attn x V in one kernel) with the CPU oracle,
every output element bit for bit.  Q and K are rounded Gaussians around their
zero points; scales pick the float (s = 2^-10, 1e-3) or the integer (s = 2e-4)
Log-Int-Softmax path."""
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


def _check(fq, orc, G, Lq, Lk, dk, d, s, sigma=19.6, zp_q=0, zp_k=0, zp_v=0, heads=1,
           bias=False, seed=0):
    x = W.qk_inputs(G, Lq, Lk, dk, d, seed=seed, sigma=sigma, zp_q=zp_q, zp_k=zp_k, heads=heads,
                    bias=bias)
    b = x["bias"]
    got = host(fq.lis_attention_qk(dev(x["q"]), dev(x["k"]), dev(x["v"]), s, zp_q, zp_k,
                                   zp_v=zp_v, bias=dev(b) if b is not None else None))
    ref = orc.lis_attention_qk(x["q"], x["k"], x["v"], s, zp_q, zp_k, zp_v=zp_v, bias=b)
    assert np.array_equal(got, ref)


SHAPES = [  # G, Lq, Lk, dk, d
    (64, 197, 197, 64, 64),     # ViT / DeiT heads
    (96, 49, 49, 32, 32),       # Swin windows
    (8, 20, 20, 64, 64),        # ragged query tile
    (16, 1, 1, 32, 16),
    (16, 16, 16, 64, 64),       # one half chunk
    (16, 17, 17, 64, 40),       # chunk of 17 keys
    (8, 50, 224, 64, 64),       # longest row held in registers
    (8, 33, 100, 32, 20),
    (4, 40, 225, 64, 64),       # shortest row of the three-pass kernel
    (3, 50, 577, 64, 64),       # ViT-L/16 at 384 px
    (2, 33, 640, 32, 20),       # longest supported row
    (2, 17, 300, 64, 48),
    (8, 33, 100, 32, 30),       # d % 4 != 0: output written element by element
    (2, 20, 300, 64, 30),
]


@pytest.mark.parametrize("G,Lq,Lk,dk,d", SHAPES)
def test_qk_shapes_float_path(fq, orc, G, Lq, Lk, dk, d):
    say("qk fp", G, Lq, Lk, dk, d)
    _check(fq, orc, G, Lq, Lk, dk, d, 2.0 ** -10, seed=G + Lk)


@pytest.mark.parametrize("G,Lq,Lk,dk,d", SHAPES[:4] + SHAPES[6:])
def test_qk_shapes_integer_path(fq, orc, G, Lq, Lk, dk, d):
    say("qk int", G, Lq, Lk, dk, d)
    _check(fq, orc, G, Lq, Lk, dk, d, 2e-4, sigma=30.0, seed=G + Lk + 1)


def test_qk_zero_points_and_bias(fq, orc):
    """Asymmetric Q and K (zero points folded in exactly), a non-zero V zero
    point, and a per-head bias as for Swin's relative positions."""
    say("qk zero points + bias")
    _check(fq, orc, 12, 49, 49, 32, 32, 1e-3, sigma=25.0, zp_q=-20, zp_k=13, zp_v=3, heads=3,
           bias=True, seed=7)
    _check(fq, orc, 6, 197, 197, 64, 64, 2.0 ** -10, zp_q=101, zp_k=-97, seed=8)


def test_qk_saturated_operands(fq, orc):
    """Operands at the int8 extremes: the largest logits the kernel can see."""
    say("qk saturated")
    G, Lq, Lk, dk, d = 4, 40, 60, 64, 64
    rng = np.random.default_rng(9)
    q = rng.choice(np.array([-128, 127], dtype=np.int8), size=(G, Lq, dk))
    k = rng.choice(np.array([-128, 127], dtype=np.int8), size=(G, Lk, dk))
    v = rng.integers(-127, 128, size=(G, Lk, d)).astype(np.int8)
    s = 0.5
    got = host(fq.lis_attention_qk(dev(q), dev(k), dev(v), s, 127, -128))
    assert np.array_equal(got, orc.lis_attention_qk(q, k, v, s, 127, -128))


def test_qk_long_rows_zero_points_and_bias(fq, orc):
    """The three-pass kernel with asymmetric Q and K, a V zero point and a
    per-head bias on rows of 577 keys."""
    say("qk long zero points + bias")
    _check(fq, orc, 4, 33, 577, 64, 64, 2.0 ** -10, sigma=25.0, zp_q=-20, zp_k=13, zp_v=3,
           heads=2, bias=True, seed=17)
    _check(fq, orc, 4, 20, 400, 32, 32, 1e-3, zp_q=9, zp_k=-4, seed=18)


def test_qk_full_vit_large(fq, orc):
    """The ViT-L/16 at 384 px attention shape: 256 units of 577 x 577, dk = d = 64."""
    say("qk full vit_l")
    _check(fq, orc, 256, 577, 577, 64, 64, 2.0 ** -10, seed=3)


def test_qk_full_vit_base(fq, orc):
    """The ViT-B/16 batch-64 attention shape: 768 units of 197 x 197, dk = d = 64."""
    say("qk full vit_b")
    _check(fq, orc, 768, 197, 197, 64, 64, 2.0 ** -10, seed=2)
