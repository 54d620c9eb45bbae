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


def unit_errors(gpu, ref, cu=None, per_token=False):
    """Per-unit parity: for every (sequence or document, head) unit, max |gpu - ref| over
    the unit divided by the RMS of ref over the unit.

    Token tensors are [B, T, H, d] ([B, T, H] with per_token=True); with ``cu`` (packed
    documents, B == 1) the units are (document, head).  State tensors [N, H, dk, dv] are
    passed with per_token=None: one unit per (n, h).  Units whose reference is all zero
    (empty documents) are skipped.  Returns (worst ratio, its unit, number of units)."""
    g = gpu.detach().cpu() if isinstance(gpu, torch.Tensor) else torch.from_numpy(np.asarray(gpu))
    r = torch.from_numpy(np.ascontiguousarray(np.asarray(ref, dtype=np.float64)))
    g = g.double()
    if per_token is None:   # states: (n, h) units
        diff = (g - r).abs().amax(dim=(2, 3))
        rms = (r * r).mean(dim=(2, 3)).sqrt()
        pieces = [((n, h), float(diff[n, h]), float(rms[n, h]))
                  for n in range(r.shape[0]) for h in range(r.shape[1])]
    else:
        red = (1,) if per_token else (1, 3)
        spans = ([(b, slice(None)) for b in range(r.shape[0])] if cu is None else
                 [(i, (0, slice(int(cu[i]), int(cu[i + 1])))) for i in range(len(cu) - 1)])
        pieces = []
        for idx, sl in spans:
            if cu is None:
                gs, rs = g[idx:idx + 1], r[idx:idx + 1]
            else:
                gs, rs = g[sl[0]:sl[0] + 1, sl[1]], r[sl[0]:sl[0] + 1, sl[1]]
            if rs.shape[1] == 0:
                continue
            diff = (gs - rs).abs().amax(dim=red).reshape(-1)
            rms = (rs * rs).mean(dim=red).sqrt().reshape(-1)
            pieces += [((idx, h), float(diff[h]), float(rms[h])) for h in range(diff.shape[0])]
    worst, where, n = 0.0, None, 0
    for unit, dmax, rms in pieces:
        if rms == 0.0:
            assert dmax == 0.0, (unit, dmax)
            continue
        n += 1
        e = dmax / rms
        if e > worst:
            worst, where = e, unit
    return worst, where, n
