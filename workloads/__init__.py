"""Seeded synthetic inputs for the PTF-LayerNorm and LIS-attention hot path.

This module only draws inputs; it holds none of the method's arithmetic (no
integer LayerNorm, no I-Exp, I-Log2 or BitShift).  Both the HIP path and the
CPU oracle consume what it returns.

The paper's activations, weights and datasets are not available, so the
shapes come from the models it evaluates (DeiT-T/S, ViT-B/16, ViT-L/16 at
384 px, Swin-S windows) and the value distributions from its statistics:
LayerNorm inputs with strong inter-channel variation (channel ranges tens of
times the median, Sec. 1 and Sec. 3.2) and attention rows concentrated near
zero with a few large values (Sec. 3.3).

LayerNorm input recipe (per config):
  * per-channel spread ``scale_c`` log-uniform on [0.05, 2.5]; on the ViT-B
    config 8 seeded channels get 40x the median spread;
  * the layer-wise integer grid of a PTF-calibrated tensor with K = 3:
    ``unit = (max X - min X) / 255 / 2^K`` over the float draw
    X = N(0,1) * scale_c, and zero point ``zp`` = nearest integer to -min X /
    (2^K unit), clipped to [0, 255];
  * per-channel factor alpha: the smallest alpha in {0..K} whose grid
    2^alpha * unit holds the channel without clipping (a stand-in for the
    calibration search, which is not part of this path), or uniform in
    {0..K} on the ViT-L config;
  * X_Q = clip(zp + rint(X / (2^alpha_c unit)), 0, 255), stored as an int8
    container (value - 128);
  * gamma = f32(1 + 0.5 N(0,1)), beta = f32(0.5 N(0,1));
  * the output scale and zero point cover the range of the float LayerNorm of
    the first rows of X (eps = 1e-6).

Attention recipe: logits = rint(N(0, sigma_h^2) / s_logit) as int32 with
s_logit = 2^-10 and sigma_h = 3 (ViT-B: sigma_h = linspace(1, 6, 12)[h]);
V uniform integers in [-127, 127] as int8 with zp_V = 0; Swin-S adds an int32
relative-position bias uniform on [-64, 64] of shape [heads, 49, 49].

Seeds: numpy PCG64, ``SeedSequence(seed).spawn(4)`` gives independent streams
for [LayerNorm data, logits, V, parameters]; config i uses seed i.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

S_LOGIT = 2.0 ** -10
EXP_N = 20
LIS_BITS = 4
LN_BITS = 8
PTF_K = 3


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    batch: int
    tokens: int          # tokens per image (LayerNorm rows per image)
    channels: int
    heads: int
    head_dim: int
    seq: int             # attention row length (Lq = Lk)
    windows: int         # attention units per image per head (Swin windows; 1 otherwise)
    seed: int
    sigma: tuple         # per-head logit sigma
    outliers: int = 0    # channels with 40x the median spread
    alpha_uniform: bool = False
    bias: bool = False

    @property
    def T(self) -> int:
        return self.batch * self.tokens

    @property
    def G(self) -> int:
        return self.batch * self.windows * self.heads

    @property
    def Lq(self) -> int:
        return self.seq

    @property
    def Lk(self) -> int:
        return self.seq

    @property
    def d(self) -> int:
        return self.head_dim


CONFIGS = [
    Config("deit_tiny_b1", 1, 197, 192, 3, 64, 197, 1, 0, (3.0,) * 3),
    Config("deit_small_b8", 8, 197, 384, 6, 64, 197, 1, 1, (3.0,) * 6),
    Config("vit_base16_224_b64", 64, 197, 768, 12, 64, 197, 1, 2,
           tuple(float(x) for x in np.linspace(1.0, 6.0, 12)), outliers=8),
    Config("vit_large16_384_b16", 16, 577, 1024, 16, 64, 577, 1, 3, (3.0,) * 16,
           alpha_uniform=True),
    Config("swin_small_win7_b32", 32, 3136, 96, 3, 32, 49, 64, 4, (3.0,) * 3, bias=True),
]
BY_NAME = {c.name: c for c in CONFIGS}


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]


# ---------------------------------------------------------------------------
# LayerNorm inputs
# ---------------------------------------------------------------------------

def ln_inputs(T: int, C: int, seed: int, outliers: int = 0, alpha_uniform: bool = False,
              K: int = PTF_K, scale_lo: float = 0.05, scale_hi: float = 2.5,
              out_rows: int = 4096) -> dict:
    """Synthetic PTF-quantized LayerNorm input of shape [T, C] (see module doc)."""
    r_ln, _, _, r_par = _streams(seed)
    scale = np.exp(r_par.uniform(np.log(scale_lo), np.log(scale_hi), size=C))
    if outliers:
        idx = r_par.choice(C, size=outliers, replace=False)
        scale[idx] = 40.0 * np.median(scale)
    gamma = (1.0 + 0.5 * r_par.standard_normal(C)).astype(np.float32)
    beta = (0.5 * r_par.standard_normal(C)).astype(np.float32)
    alpha_draw = r_par.integers(0, K + 1, size=C)

    X = r_ln.standard_normal((T, C)) * scale[None, :]
    lo, hi = float(X.min()), float(X.max())
    unit = (hi - lo) / 255.0 / 2.0 ** K
    zp = int(np.clip(np.rint(-lo / (2.0 ** K * unit)), 0, 255))

    if alpha_uniform:
        alpha = alpha_draw.astype(np.uint8)
    else:
        cmin, cmax = X.min(axis=0), X.max(axis=0)
        alpha = np.full(C, K, dtype=np.uint8)
        for a in range(K, -1, -1):
            step = 2.0 ** a * unit
            fits = (np.rint(cmin / step) + zp >= 0) & (np.rint(cmax / step) + zp <= 255)
            alpha[fits] = a
    step = (2.0 ** alpha.astype(np.float64)) * unit
    xq_u = np.clip(zp + np.rint(X / step[None, :]), 0, 255)
    x_q = (xq_u - 128).astype(np.int8)

    # Output scale: range of the float LayerNorm of the first rows.
    Xs = X[:min(T, out_rows)]
    mu = Xs.mean(axis=1, keepdims=True)
    var = Xs.var(axis=1, keepdims=True)
    Y = (Xs - mu) / np.sqrt(var + 1e-6) * gamma.astype(np.float64) + beta.astype(np.float64)
    ylo, yhi = float(Y.min()), float(Y.max())
    if yhi - ylo < 1e-3:            # e.g. C = 1: the output is beta on every row
        ylo, yhi = ylo - 0.5, yhi + 0.5
    s_out = np.float32((yhi - ylo) / 255.0)
    zp_out = int(np.clip(np.rint(-ylo / float(s_out)), 0, 255)) - 128

    return dict(x_q=x_q, zp_in=zp - 128, alpha=alpha, K=K, gamma=gamma, beta=beta,
                s_out=float(s_out), zp_out=zp_out, bits=LN_BITS, s_in=unit, x_float=X)


# ---------------------------------------------------------------------------
# Attention inputs
# ---------------------------------------------------------------------------

def attn_inputs(G: int, Lq: int, Lk: int, d: int, seed: int, heads: int = 1,
                sigma=(3.0,), s_logit: float = S_LOGIT, bias: bool = False,
                v_lo: int = -127, v_hi: int = 127) -> dict:
    """int32 logits [G, Lq, Lk], int8 V [G, Lk, d], optional bias [heads, Lq, Lk]."""
    _, r_lg, r_v, r_par = _streams(seed)
    sig = np.asarray(sigma, dtype=np.float64)
    logits = np.empty((G, Lq, Lk), dtype=np.int32)
    for g in range(G):
        h = g % heads
        logits[g] = np.rint(r_lg.standard_normal((Lq, Lk)) * (sig[h % sig.size] / s_logit))
    v = r_v.integers(v_lo, v_hi + 1, size=(G, Lk, d)).astype(np.int8)
    b = None
    if bias:
        b = r_par.integers(-64, 65, size=(heads, Lq, Lk)).astype(np.int32)
    return dict(logits=logits, v=v, zp_v=0, bias=b, Hb=heads if bias else 0,
                s_logit=s_logit, bits=LIS_BITS, exp_n=EXP_N)


def shifted_window_mask(hw: int, window: int, shift: int, masked: int) -> np.ndarray:
    """Additive mask [nW, window^2, window^2] int32 of shifted-window attention
    on an hw x hw token grid: after a cyclic shift by `shift`, the grid is cut
    into nW = (hw / window)^2 windows; tokens that came from different regions
    of the unshifted grid (three bands per axis: [0, hw - window),
    [hw - window, hw - shift), [hw - shift, hw)) get `masked`, others 0."""
    assert hw % window == 0 and 0 < shift < window
    bands = np.zeros(hw, dtype=np.int64)
    bands[hw - window:hw - shift] = 1
    bands[hw - shift:] = 2
    region = bands[:, None] * 3 + bands[None, :]          # [hw, hw]
    n = hw // window
    wins = region.reshape(n, window, n, window).transpose(0, 2, 1, 3).reshape(n * n, window * window)
    return np.where(wins[:, :, None] != wins[:, None, :], masked, 0).astype(np.int32)


def qk_inputs(G: int, Lq: int, Lk: int, dk: int, d: int, seed: int, sigma: float = 30.0,
              zp_q: int = 0, zp_k: int = 0, heads: int = 1, bias: bool = False) -> dict:
    """int8 query and key activations [G, Lq|Lk, dk] (rounded Gaussians of
    standard deviation `sigma` around their zero points, clipped to int8),
    int8 V [G, Lk, d] and an optional bias [heads, Lq, Lk]."""
    _, r_lg, r_v, r_par = _streams(seed)
    q = np.clip(np.rint(r_lg.standard_normal((G, Lq, dk)) * sigma) + zp_q, -128, 127).astype(np.int8)
    k = np.clip(np.rint(r_lg.standard_normal((G, Lk, dk)) * sigma) + zp_k, -128, 127).astype(np.int8)
    v = r_v.integers(-127, 128, size=(G, Lk, d)).astype(np.int8)
    b = r_par.integers(-64, 65, size=(heads, Lq, Lk)).astype(np.int32) if bias else None
    return dict(q=q, k=k, v=v, zp_q=zp_q, zp_k=zp_k, bias=b)


def lis_lattice(chunk: int, step: int, jitter: int = 0, seed: int = 0, rows_per_chunk_log8: int = 7):
    """Rows of 8 keys whose entries run over {0, -1, ..., -7} * step, every
    combination once (8^8 rows in 8^(8 - rows_per_chunk_log8) chunks; row r of
    the whole lattice has entry k equal to -digit_k(r) step, digit_k the k-th
    base-8 digit), optionally plus an integer jitter uniform on
    [-jitter, jitter] (seeded by seed and chunk).  Returned as int32
    [rows / 4, 4, 8]: attention units of 4 query rows and 8 keys."""
    n = 8 ** rows_per_chunk_log8
    idx = np.arange(chunk * n, (chunk + 1) * n, dtype=np.int64)
    digits = np.stack([(idx >> (3 * k)) & 7 for k in range(8)], axis=1)
    rows = -digits * step
    if jitter:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, chunk])))
        rows = rows + rng.integers(-jitter, jitter + 1, size=rows.shape)
    return rows.astype(np.int32).reshape(n // 4, 4, 8)


def config_inputs(cfg: Config, part: str = "all", G: Optional[int] = None,
                  T: Optional[int] = None) -> dict:
    """Inputs of a named config.  ``G`` truncates the attention unit count (the
    first units are the same draws as at full size); ``T`` truncates the
    LayerNorm rows (the layer-wise grid is then taken over the rows drawn)."""
    out = {}
    if part in ("all", "ln"):
        out["ln"] = ln_inputs(cfg.T if T is None else T, cfg.channels, cfg.seed,
                              outliers=cfg.outliers, alpha_uniform=cfg.alpha_uniform)
    if part in ("all", "attn"):
        out["attn"] = attn_inputs(cfg.G if G is None else G, cfg.Lq, cfg.Lk, cfg.d, cfg.seed,
                                  heads=cfg.heads, sigma=cfg.sigma, bias=cfg.bias)
    return out
