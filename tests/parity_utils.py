"""Helpers shared by the GPU parity tests (host-side comparisons only)."""
import numpy as np
import torch

import oracle

# Tolerance on max |gpu - oracle| / rms(oracle), per output tensor.
TOL = {"bf16": 2e-2, "f32": 1e-4}


def rel_err(gpu, ref):
    g = gpu.detach().double().cpu().numpy() if isinstance(gpu, torch.Tensor) else np.asarray(gpu)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    assert rms > 0
    return float(np.abs(g - ref).max()) / rms


def to_dev(inp, device="cuda"):
    return {k: (v.to(device) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}


STREAM_KEYS = ("q", "k", "v", "g", "beta")


def oracle_unit(inp, b, h, hv_per_qk, block, scale, rows=None, h0=None):
    """Oracle on one (sequence, v-head) unit: slices [b, rows, head] and runs the
    fp64 oracle on that single unit.  Returns (o, on, ht) for the unit."""
    hq = h // hv_per_qk
    sl = slice(None) if rows is None else slice(*rows)
    c, n = {}, {}
    for key in STREAM_KEYS:
        head = hq if key in ("q", "k") else h
        c[key] = inp[key][b:b + 1, sl, head:head + 1].double().numpy()
        n[key] = inp[key + "n"][b:b + 1, sl, head:head + 1].double().numpy()
    h0u = None if h0 is None else h0[b:b + 1, h:h + 1].double().numpy()
    o, on, ht = oracle.fwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"],
                                 n["q"], n["k"], n["v"], n["g"], n["beta"],
                                 block=block, scale=scale, h0=h0u)
    return o[0, :, 0], on[0, :, 0], ht[0, 0]


def oracle_full(inp, block, scale, h0=None, cu=None):
    args = [inp[k] for k in STREAM_KEYS] + [inp[k + "n"] for k in STREAM_KEYS]
    return oracle.fwd_train(*args, block=block, scale=scale, h0=h0,
                            cu_seqlens=None if cu is None else cu.numpy())
