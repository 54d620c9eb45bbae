"""Seeded synthetic workloads for the block-diffusion Gated Delta Rule.

This module only draws random inputs; it holds none of the method's arithmetic.
Both the HIP path (tests, benchmark, smoke check) and the CPU oracle are fed from
here.  The paper trains and benchmarks on Qwen3.5 GDN-layer shapes with real
data; these seeded inputs stand in for those activations.

Input recipe (per stream, drawn in this order from ``numpy.random.default_rng``):
  q, k  ~ N(0, 1), then L2-normalised over the head dimension;
  v     ~ N(0, 1);
  g     = -softplus(x), x ~ U(-6, -2)      (log-gate; alpha = exp(g) in (0.881, 0.9975));
  beta  = sigmoid(y),   y ~ U(-2, 2)       (beta in (0.119, 0.881)).
The clean stream is drawn first, then the noisy stream.  q, k, v are rounded
(round-to-nearest-even) to the workload dtype; g and beta are stored as fp32.
Draws use float32 for bf16 workloads and float64 for fp32 workloads.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class TrainWorkload:
    """Two-stream training forward: ``batch`` sequences of ``seqlen`` clean and
    ``seqlen`` noisy tokens, or (``n_docs`` > 0) one packed axis of ``seqlen``
    tokens split into documents by cu_seqlens."""
    name: str
    batch: int
    seqlen: int
    h_qk: int
    h_v: int
    d_k: int
    d_v: int
    block: int
    dtype: str
    seed: int
    n_docs: int = 0
    doc_min: int = 0
    doc_max: int = 0

    @property
    def tokens(self) -> int:
        return self.batch * self.seqlen


@dataclass(frozen=True)
class ServeWorkload:
    """Concurrent Diffusion-Trust serving: ``requests`` cached fp32 states of
    ``h_v`` heads, ``steps`` denoise calls on fresh blocks of ``block`` tokens,
    then one commit."""
    name: str
    requests: int
    h_qk: int
    h_v: int
    d_k: int
    d_v: int
    block: int
    steps: int
    dtype: str
    seed: int


@dataclass(frozen=True)
class ConvWorkload:
    """Two-stream ShortConv: ``batch`` sequences of ``seqlen`` clean and ``seqlen`` noisy
    rows of ``channels`` (the q, k, v projections side by side), a depthwise causal
    filter of ``width`` taps, diffusion blocks of ``block`` rows."""
    name: str
    batch: int
    seqlen: int
    channels: int
    width: int
    block: int
    act: int
    dtype: str
    seed: int


TINY_F32 = TrainWorkload("tiny_f32_b1_t256_h2_d64_l16", 1, 256, 2, 2, 64, 64, 16, "f32", 0)
TRAIN_4K = TrainWorkload("train_bf16_b4_t4096_h16_d128_l32", 4, 4096, 16, 16, 128, 128, 32,
                         "bf16", 1)
GVA_16K = TrainWorkload("gva_bf16_b2_t16384_hqk16_hv32_d128_l64", 2, 16384, 16, 32, 128, 128,
                        64, "bf16", 2)
SERVE_64 = ServeWorkload("serve_bf16_r64_h32_d128_l32_x8", 64, 32, 32, 128, 128, 32, 8, "bf16", 3)
# AR-Trust verify round: the anchor and 7 draft tokens per request (the verify pass keeps
# the states before the 7 draft positions)
VERIFY_64 = ServeWorkload("verify_bf16_r64_h32_d128_l8_rec7", 64, 32, 32, 128, 128, 8, 1, "bf16", 5)
VARLEN_128K = TrainWorkload("varlen_bf16_n32_t131072_h16_d128_l32", 1, 131072, 16, 16, 128, 128,
                            32, "bf16", 4, n_docs=32, doc_min=512, doc_max=8192)

# The GDN layer's ShortConv at the 16-head, d = 128 shape (channels 3 x 16 x 128): 4096
# clean + 4096 noisy rows, width 4, silu
CONV_4K = ConvWorkload("shortconv_bf16_b1_t4096_d6144_w4_l32", 1, 4096, 6144, 4, 32, 1, "bf16", 6)
CONV_TRAIN = ConvWorkload("shortconv_bf16_b4_t4096_d6144_w4_l32", 4, 4096, 6144, 4, 32, 1, "bf16", 7)

WORKLOADS = {w.name: w for w in (TINY_F32, TRAIN_4K, GVA_16K, SERVE_64, VARLEN_128K, CONV_4K, CONV_TRAIN)}

_TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}


def torch_dtype(name: str) -> torch.dtype:
    return _TORCH_DTYPE[name]


def _unit_rows(rng, shape, fdt):
    x = rng.standard_normal(shape, dtype=fdt)
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    return x


def draw_stream(rng, rows_shape, h_qk, h_v, d_k, d_v, dtype):
    """One stream (q, k, v, g, beta) as torch CPU tensors.

    rows_shape is the leading token shape, e.g. (B, T) or (R, L).
    """
    fdt = np.float32 if dtype == "bf16" else np.float64
    tdt = _TORCH_DTYPE[dtype]
    q = _unit_rows(rng, (*rows_shape, h_qk, d_k), fdt)
    k = _unit_rows(rng, (*rows_shape, h_qk, d_k), fdt)
    v = rng.standard_normal((*rows_shape, h_v, d_v), dtype=fdt)
    g_raw = rng.uniform(-6.0, -2.0, size=(*rows_shape, h_v))
    b_raw = rng.uniform(-2.0, 2.0, size=(*rows_shape, h_v))
    g = -np.log1p(np.exp(g_raw))
    beta = 1.0 / (1.0 + np.exp(-b_raw))
    out = dict(
        q=torch.from_numpy(q).to(tdt), k=torch.from_numpy(k).to(tdt),
        v=torch.from_numpy(v).to(tdt),
        g=torch.from_numpy(g.astype(np.float32)), beta=torch.from_numpy(beta.astype(np.float32)))
    return out


def varlen_lengths(rng, n_docs, total, block, lo, hi):
    """n_docs lengths ~ U(lo, hi), scaled to sum exactly to ``total``, each a
    multiple of ``block`` within [lo, hi] (largest-remainder adjustment)."""
    raw = rng.uniform(lo, hi, size=n_docs)
    scaled = raw * (total / raw.sum())
    base = np.clip(np.floor(scaled / block) * block, lo, hi).astype(np.int64)
    rem = scaled - base
    deficit = total - int(base.sum())
    assert deficit % block == 0
    order_up = np.argsort(-rem, kind="stable")
    order_dn = np.argsort(rem, kind="stable")
    while deficit != 0:
        moved = False
        for i in (order_up if deficit > 0 else order_dn):
            step = block if deficit > 0 else -block
            if lo <= base[i] + step <= hi:
                base[i] += step
                deficit -= step
                moved = True
                if deficit == 0:
                    break
        if not moved:
            raise ValueError("cannot reach the requested total within [lo, hi]")
    return base


def make_train(w: TrainWorkload, seed: int | None = None):
    """Inputs of a training workload: dict with clean (q,k,v,g,beta), noisy
    (qn,kn,vn,gn,betan) and, if packed, cu_seqlens (torch int32) and lengths."""
    rng = np.random.default_rng(w.seed if seed is None else seed)
    out = {}
    lengths = None
    if w.n_docs:
        lengths = varlen_lengths(rng, w.n_docs, w.seqlen, w.block, w.doc_min, w.doc_max)
    rows = (w.batch, w.seqlen)
    c = draw_stream(rng, rows, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype)
    n = draw_stream(rng, rows, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype)
    out.update(c)
    out.update({k + "n": val for k, val in n.items()})
    if lengths is not None:
        cu = np.zeros(len(lengths) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(lengths)
        out["cu_seqlens"] = torch.from_numpy(cu)
        out["lengths"] = lengths
    return out


def make_custom_train(batch, seqlen, h_qk, h_v, d_k, d_v, dtype, seed, lengths=None):
    """Training inputs of any shape (tests).  ``lengths`` packs documents."""
    rng = np.random.default_rng(seed)
    rows = (batch, seqlen)
    c = draw_stream(rng, rows, h_qk, h_v, d_k, d_v, dtype)
    n = draw_stream(rng, rows, h_qk, h_v, d_k, d_v, dtype)
    out = dict(c)
    out.update({k + "n": val for k, val in n.items()})
    if lengths is not None:
        cu = np.zeros(len(lengths) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(lengths)
        out["cu_seqlens"] = torch.from_numpy(cu)
    return out


def make_serve_block(w: ServeWorkload, step: int, requests: int | None = None):
    """Fresh (q,k,v,g,beta) block for serving step ``step`` (seed*1000+step)."""
    rng = np.random.default_rng(w.seed * 1000 + step)
    R = w.requests if requests is None else requests
    return draw_stream(rng, (R, w.block), w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype)


def make_state_pool(n_slots, h_v, d_k, d_v, seed, sigma=0.3):
    """A synthetic fp32 state pool [n_slots, h_v, d_k, d_v] ~ N(0, sigma^2)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n_slots, h_v, d_k, d_v), dtype=np.float32) * np.float32(sigma)
    return torch.from_numpy(x)


def draw_conv(rng, batch, seqlen, channels, width, dtype, bias=True):
    """ShortConv inputs: x, xn, dy, dyn ~ N(0, 1) of shape [batch, seqlen, channels]
    rounded to ``dtype``; w [channels, width] and bias [channels] ~ U(-1/sqrt(width),
    1/sqrt(width)) (a depthwise filter's default fan-in scaling), fp32."""
    fdt = np.float64 if dtype == "f32" else np.float32
    tdt = torch_dtype(dtype)
    out = {}
    for key in ("x", "xn", "dy", "dyn"):
        a = rng.standard_normal((batch, seqlen, channels), dtype=fdt)
        out[key] = torch.from_numpy(a).to(tdt)
    bound = 1.0 / np.sqrt(width)
    out["w"] = torch.from_numpy(rng.uniform(-bound, bound, (channels, width)).astype(np.float32))
    out["bias"] = torch.from_numpy(rng.uniform(-bound, bound, channels).astype(np.float32)) if bias else None
    return out


def make_conv(w: ConvWorkload, seed: int | None = None):
    rng = np.random.default_rng(w.seed if seed is None else seed)
    return draw_conv(rng, w.batch, w.seqlen, w.channels, w.width, w.dtype)


# Serving pools: each request's cached state is the clean state after a seeded prefix of
# SERVE_PREFIX_BLOCKS blocks of the workload's block length (256 tokens at L = 32).
SERVE_PREFIX_BLOCKS = 8


def make_serve_prefix_block(w: ServeWorkload, pool: int, block: int):
    """Prefix block ``block`` of state pool ``pool`` (seed (seed*1000 + 500 + 16*pool + block)),
    drawn with the same recipe as the serving blocks."""
    rng = np.random.default_rng(w.seed * 1000 + 500 + 16 * pool + block)
    return draw_stream(rng, (w.requests, w.block), w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype)
