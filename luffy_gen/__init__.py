"""Seeded synthetic inputs for the token-condensation MoE layer.

This module only draws random numbers and lays them out.  It holds none of
the layer's arithmetic (no gating, no similarity, no grouping, no FFN): the
CPU oracle and the HIP path both consume exactly the arrays produced here and
nothing else is shared between them.

Workloads (stand-ins for the paper's model activations, which are not
available; the paper motivates clustered tokens in Sec. 2.2 "Token
Similarity" and biased expert activation in Sec. 2.2 / Fig. biased_exp):

  c1  T=512    d=256   E=4   top-1  FFN 256->1024->256   GELU  fp32
      64 centres, noise 0.05, h=0.95
  c2  T=8192   d=1024  E=16  top-2  FFN 1024->4096->1024 GELU  bf16
      2048 centres, noise 0.03, capacity factor 1.25, h=0.95
  c3  T=32768  d=2048  E=32  top-2  FFN 2048->8192->2048 GELU  bf16
      4096 centres, noise 0.02, gate bias calibrated so the expected
      expert load follows Zipf(1.1), h=0.90
  c4  T=16384  d=4096  E=8   top-1  FFN 4096->11008->4096 SiLU bf16
      i.i.d. N(0,1) tokens (nothing merges), h in {0.80,0.90,0.95,0.99}
  c5  T=65536  d=1024  E=64  top-1  FFN 1024->4096->1024 GELU  bf16
      8192 centres, noise 0.05, gate bias ln Zipf(1.3) with N(0,1) logit
      noise, capacity factor 1.0, h=0.95

Draw order (one numpy PCG64 generator per call, seeded with ``seed``):
  1. centres ~ N(0,1) [n_c, d]            (skipped when n_c == 0)
  2. centre ids ~ U{0..n_c-1} [T]         (skipped when n_c == 0)
  3. X = centre[id] + sigma * N(0,1) [T,d] (X ~ N(0,1) when n_c == 0)
  4. W_g = w_scale * N(0,1) [E,d]
  5. W1 = 0.02 * N(0,1) [E, d_ff, d]
  6. W2 = 0.02 * N(0,1) [E, d, d_ff]
The gate bias is not drawn; it is a function of the configuration (see
``gate_bias``).  Optional planted duplicates copy whole rows of X after the
draws (used for the "exact duplicates always merge" invariant).

For bf16 configurations X, W_g, W1 and W2 are rounded to bf16
(round-to-nearest-even) once, here, and both sides consume the rounded values
(held in float32 arrays, which represent them exactly).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

__all__ = [
    "LayerConfig", "CONFIGS", "config", "Inputs", "make_inputs",
    "round_bf16", "bf16_bits", "gate_bias", "make_stack",
]


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int
    d: int
    E: int
    k: int
    d_ff: int
    act: str                      # "gelu" (exact erf form) or "silu"
    dtype: str                    # "f32" or "bf16"
    n_centres: int                # 0: tokens are i.i.d. N(0,1)
    sigma: float                  # per-token noise around its centre
    w_scale: float                # std of the gate weights
    bias: str                     # "zero" | "zipf_calibrated" | "ln_zipf"
    zipf_s: float
    capacity_factor: float        # <= 0: no capacity limit
    thresholds: tuple             # cosine thresholds; the first is the default
    batch: int
    seq: int

    @property
    def h(self) -> float:
        return self.thresholds[0]

    def replace(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    "c1": LayerConfig("c1", 512, 256, 4, 1, 1024, "gelu", "f32", 64, 0.05,
                      0.02, "zero", 0.0, 0.0, (0.95,), 2, 256),
    "c2": LayerConfig("c2", 8192, 1024, 16, 2, 4096, "gelu", "bf16", 2048,
                      0.03, 0.02, "zero", 0.0, 1.25, (0.95,), 8, 1024),
    "c3": LayerConfig("c3", 32768, 2048, 32, 2, 8192, "gelu", "bf16", 4096,
                      0.02, 0.02, "zipf_calibrated", 1.1, 0.0, (0.90,), 16,
                      2048),
    "c4": LayerConfig("c4", 16384, 4096, 8, 1, 11008, "silu", "bf16", 0, 1.0,
                      0.02, "zero", 0.0, 0.0, (0.80, 0.90, 0.95, 0.99), 8,
                      2048),
    "c5": LayerConfig("c5", 65536, 1024, 64, 1, 4096, "gelu", "bf16", 8192,
                      0.05, -1.0, "ln_zipf", 1.3, 1.0, (0.95,), 32, 2048),
}


def config(name: str, **overrides) -> LayerConfig:
    """Named configuration, optionally resized (tests shrink T, d, d_ff)."""
    cfg = CONFIGS[name]
    if overrides:
        cfg = cfg.replace(**overrides)
    return cfg


def round_bf16(a: np.ndarray, inplace: bool = False) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), as float32.

    Finite inputs only.  ``inplace`` overwrites a C-contiguous float32 array.
    """
    if inplace and a.dtype == np.float32 and a.flags.c_contiguous:
        out = a
    else:
        out = np.array(a, dtype=np.float32, order="C", copy=True)
    flat = out.reshape(-1).view(np.uint32)
    step = 1 << 20
    buf = np.empty(min(step, flat.size), np.uint32)
    for i in range(0, flat.size, step):          # chunked, in place
        u = flat[i:i + step]
        lsb = buf[: u.size]
        np.right_shift(u, np.uint32(16), out=lsb)
        lsb &= np.uint32(1)
        u += np.uint32(0x7FFF)
        u += lsb
        u &= np.uint32(0xFFFF0000)
    return out


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-exact."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("array is not bf16-representable")
    return (u >> 16).astype(np.uint16)


def _zipf(E: int, s: float) -> np.ndarray:
    p = (np.arange(1, E + 1, dtype=np.float64)) ** (-s)
    return p / p.sum()


def _expected_topk_share(b: np.ndarray, s: float, k: int) -> np.ndarray:
    """Expected share of top-k slots per expert when expert logits are
    independent N(b_e, s^2).  Pure probability (order statistics of Gaussians,
    evaluated by quadrature); no token is routed here."""
    from scipy.special import log_ndtr
    E = b.shape[0]
    lo, hi = b.min() - 9 * s, b.max() + 9 * s
    z = np.linspace(lo, hi, 6001)
    dz = z[1] - z[0]
    u = (z[None, :] - b[:, None]) / s                       # [E, Z]
    logF = log_ndtr(u)                                      # log P(X_e <= z)
    logf = -0.5 * u * u - math.log(s * math.sqrt(2 * math.pi))
    sum_logF = logF.sum(0)                                  # log prod_e F_e
    # P(e is the maximum) = int f_e * prod_{f != e} F_f
    p1 = np.exp(logf + sum_logF[None, :] - logF).sum(1) * dz
    if k == 1:
        return p1
    # P(e is exactly second) = int f_e * sum_{g != e} (1-F_g) prod_{f != e,g} F_f
    log1mF = log_ndtr(-u)                                   # log(1 - F_e)
    ratio = np.exp(log1mF - logF)                           # (1-F)/F
    tot = ratio.sum(0)
    p2 = (np.exp(logf + sum_logF[None, :] - logF) * (tot[None, :] - ratio)).sum(1) * dz
    return (p1 + p2) / 2.0


def gate_bias(cfg: LayerConfig) -> np.ndarray:
    """Gate bias b_g [E] (float32) for a configuration.

    zero            : no bias.
    ln_zipf         : b_e = ln p_e with p_e proportional to (e+1)^-s.  With
                      W_g ~ N(0, 1/d) the token part of each logit is about
                      N(0,1), i.e. "Zipf over experts plus N(0,1) noise".
    zipf_calibrated : b chosen so that the expected share of top-k slots of
                      expert e is Zipf(s), modelling the token part of each
                      logit as independent N(0, s_l^2) with
                      s_l = w_scale * sqrt(d * (1 + sigma^2)).  Fixed-point
                      iteration on the log shares; depends on the config only.
    """
    E = cfg.E
    if cfg.bias == "zero":
        return np.zeros(E, np.float32)
    p = _zipf(E, cfg.zipf_s)
    if cfg.bias == "ln_zipf":
        return np.log(p).astype(np.float32)
    if cfg.bias == "zipf_calibrated":
        s_l = cfg.w_scale * math.sqrt(cfg.d * (1.0 + cfg.sigma ** 2))
        b = np.log(p) * s_l
        for _ in range(400):
            share = _expected_topk_share(b, s_l, cfg.k)
            step = np.log(p) - np.log(share)
            b = b + 0.5 * s_l * step
            b -= b.mean()
            if np.abs(step).max() < 1e-6:
                break
        return b.astype(np.float32)
    raise ValueError(cfg.bias)


@dataclasses.dataclass
class Inputs:
    cfg: LayerConfig
    seed: int
    x: np.ndarray                 # [T, d] float32 (bf16-exact for bf16 configs)
    w_g: np.ndarray               # [E, d]
    b_g: np.ndarray               # [E] float32 (never rounded: fp32 bias)
    w1: Optional[np.ndarray]      # [E, d_ff, d]
    w2: Optional[np.ndarray]      # [E, d, d_ff]
    centre_id: Optional[np.ndarray]   # [T] int64, or None for i.i.d. tokens
    planted: Optional[np.ndarray]     # [n, 2] (source row, copy row) or None

    @property
    def h(self) -> float:
        return self.cfg.h


def _normal(rng: np.random.Generator, shape, scale: float) -> np.ndarray:
    a = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        a *= np.float32(scale)
    return a


def make_inputs(cfg, seed: int = 0, *, weights: bool = True,
                planted_duplicates: int = 0, **overrides) -> Inputs:
    """Draw the inputs of one MoE layer.

    cfg                : a LayerConfig or a config name ("c1".."c5").
    weights            : False skips W1/W2 (route/condense-only tests); the
                         draws for X, W_g are identical either way because
                         W1/W2 are drawn last.
    planted_duplicates : copy this many randomly chosen rows over other rows
                         (after all draws, with a sub-seeded generator), so
                         that exact duplicate tokens exist.
    overrides          : resize fields of the configuration (T, d, d_ff ...).
    """
    if isinstance(cfg, str):
        cfg = config(cfg)
    if overrides:
        cfg = cfg.replace(**overrides)
    rng = np.random.default_rng(seed)
    T, d, E = cfg.T, cfg.d, cfg.E
    if cfg.n_centres > 0:
        centres = _normal(rng, (cfg.n_centres, d), 1.0)
        cid = rng.integers(0, cfg.n_centres, size=T, dtype=np.int64)
        x = centres[cid]
        x += _normal(rng, (T, d), cfg.sigma)
        del centres
    else:
        cid = None
        x = _normal(rng, (T, d), 1.0)
    w_scale = cfg.w_scale if cfg.w_scale > 0 else 1.0 / math.sqrt(d)
    w_g = _normal(rng, (E, d), w_scale)
    w1 = w2 = None
    if weights:
        w1 = _normal(rng, (E, cfg.d_ff, d), 0.02)
        w2 = _normal(rng, (E, d, cfg.d_ff), 0.02)
    planted = None
    if planted_duplicates > 0:
        prng = np.random.default_rng([seed, 0x9E3779B9])
        rows = prng.permutation(T)[: 2 * planted_duplicates].reshape(-1, 2)
        x[rows[:, 1]] = x[rows[:, 0]]
        if cid is not None:
            cid = cid.copy()
            cid[rows[:, 1]] = cid[rows[:, 0]]
        planted = rows
    if cfg.dtype == "bf16":
        x = round_bf16(x, inplace=True)
        w_g = round_bf16(w_g, inplace=True)
        if weights:
            w1 = round_bf16(w1, inplace=True)
            w2 = round_bf16(w2, inplace=True)
    return Inputs(cfg=cfg, seed=seed, x=x, w_g=w_g, b_g=gate_bias(cfg),
                  w1=w1, w2=w2, centre_id=cid, planted=planted)


def make_stack(cfg, blocks: int, seed: int = 0, *, token_drift: float = 1.0, gate_drift: float = 0.0,
               mix_fraction: float = 0.0, weights: bool = False, **overrides) -> list:
    """Inputs of a stack of MoE blocks over the same tokens (token ids are
    shared by every block), for the historical similarity of Sec. 5.1 step 2.

    The paper observes that pairs that are very similar or very dissimilar in
    one block stay so in the next; these inputs keep each token's centre for
    the whole stack and redraw what varies from block to block.

    Draw order (numpy PCG64 seeded with [seed, 7]):
      1. centres ~ N(0,1) [n_c, d], centre ids ~ U{0..n_c-1} [T]
      2. mixed tokens: each token is mixed with probability mix_fraction
         (U[0,1) [T] < mix_fraction), second centre ids ~ U{0..n_c-1} [T];
         a mixed token's base is (c_id + c_id2) / sqrt(2) (cosine about
         0.71 with a plain token of either centre), a plain token's c_id
      3. gate weights of block 0: w_scale * N(0,1) [E, d]
      4. per block b: noise N(0,1) [T, d]; x_b = base + sigma * noise for
         b = 0, x_b = x_{b-1} + token_drift * sigma * noise after it
         (token_drift = 1: a fresh draw of the same size each block);
         gate weights W_b = W_{b-1} + gate_drift * w_scale * N(0,1) [E, d]
         for b >= 1
      5. with weights: W1, W2 per block as in make_inputs
    bf16 workloads round x_b and the weights to bf16 after the draws (the
    drift is applied to the unrounded values).  The gate bias is the
    configuration's.  Returns one Inputs per block."""
    if isinstance(cfg, str):
        cfg = config(cfg)
    if overrides:
        cfg = cfg.replace(**overrides)
    if cfg.n_centres <= 0:
        raise ValueError("make_stack needs a clustered workload (n_centres > 0)")
    rng = np.random.default_rng([seed, 7])
    T, d, E = cfg.T, cfg.d, cfg.E
    centres = _normal(rng, (cfg.n_centres, d), 1.0)
    cid = rng.integers(0, cfg.n_centres, size=T, dtype=np.int64)
    mixed = rng.random(T) < mix_fraction
    cid2 = rng.integers(0, cfg.n_centres, size=T, dtype=np.int64)
    base = centres[cid]
    base[mixed] = (centres[cid[mixed]] + centres[cid2[mixed]]) * np.float32(1.0 / math.sqrt(2.0))
    del centres
    w_scale = cfg.w_scale if cfg.w_scale > 0 else 1.0 / math.sqrt(d)
    w_g = _normal(rng, (E, d), w_scale)
    bias = gate_bias(cfg)
    out = []
    x = None
    for b in range(blocks):
        noise = _normal(rng, (T, d), cfg.sigma)
        if b == 0:
            x = base + noise
        else:
            x = x + np.float32(token_drift) * noise
            w_g = w_g + _normal(rng, (E, d), gate_drift * w_scale)
        w1 = w2 = None
        if weights:
            w1 = _normal(rng, (E, cfg.d_ff, d), 0.02)
            w2 = _normal(rng, (E, d, cfg.d_ff), 0.02)
        xb, wgb = x.copy(), w_g.copy()
        if cfg.dtype == "bf16":
            xb = round_bf16(xb, inplace=True)
            wgb = round_bf16(wgb, inplace=True)
            if weights:
                w1 = round_bf16(w1, inplace=True)
                w2 = round_bf16(w2, inplace=True)
        cid_b = np.where(mixed, -1, cid)     # centre of plain tokens, -1 for mixed ones
        out.append(Inputs(cfg=cfg, seed=seed, x=xb, w_g=wgb, b_g=bias, w1=w1, w2=w2, centre_id=cid_b,
                          planted=None))
    return out
