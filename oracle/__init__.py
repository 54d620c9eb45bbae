"""Sequential fp64 CPU oracle of the block-diffusion Gated Delta Rule.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import this package; the product library never does.

The arithmetic lives in ``bdgdn_oracle.c`` (plain C, fp64, OpenMP over
independent (sequence, v-head) units).  This module only marshals numpy arrays
to it.  Each entry point follows the paper (FLARE, arXiv 2606.01774):

* ``fwd_train``  -- two-stream training forward: clean causal recurrence
  (eq. gdn-recurrence in its per-step form, eq. per-step-fwd) and noisy blocks
  seeded from the clean boundary state with block-end readout (eq.
  flare-gdn-schedule, eq. noisy-block-fwd); document packing per the
  "Document-packed training" appendix.
* ``denoise``    -- Diffusion-Trust denoise pass: reads the cached state, never
  writes it (appendix "Differences between the denoise pass and the
  state-update pass").
* ``commit``     -- token-causal state-update pass that writes the state back.
* ``bwd_train``  -- gradients of the two-stream training forward (appendix
  "Backward primitives": the per-step backward, eq. per-step-bwd; the noisy
  block-end readout backward, eq. noisy-readout-bwd; the block-level chain rule,
  eq. dh-block-recursion).
* ``bwd_train_views`` -- gradients of the complementary-view objective (Sec. 3.3 "Training
  Objective and Mask Design": several noisy views, each block seeded from the same clean
  state), composed from ``bwd_train`` by linearity.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bdgdn_oracle.c")
_LIB = os.path.join(_HERE, "libbdgdn_oracle.so")
# The mutation tests point this at a deliberately broken copy of the oracle to show
# that the pins catch it; nothing else sets it.
_LIB_OVERRIDE = os.environ.get("BDGDN_ORACLE_LIB")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE fp64, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-Wall",
                        "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        path = _LIB_OVERRIDE or _LIB
        if not _LIB_OVERRIDE and not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        I = ctypes.c_int
        D = ctypes.c_double
        lib.oracle_fwd_train.argtypes = [I, I, I, P, I, I, I, I, I, D] + [P] * 14
        lib.oracle_fwd_train.restype = I
        lib.oracle_bwd_train.argtypes = [I, I, I, P, I, I, I, I, I, D] + [P] * 25
        lib.oracle_bwd_train.restype = I
        lib.oracle_denoise.argtypes = [I, I, I, I, I, I, D, P, P] + [P] * 6
        lib.oracle_denoise.restype = I
        lib.oracle_commit.argtypes = [I, I, I, I, I, I, D, P, P] + [P] * 6
        lib.oracle_commit.restype = I
        lib.oracle_commit_record.argtypes = [I, I, I, I, I, I, I, D, P, P] + [P] * 7
        lib.oracle_commit_record.restype = I
        lib.oracle_accept_states.argtypes = [I, I, I, I, I, P, P, P, P]
        lib.oracle_accept_states.restype = I
        lib.oracle_shortconv_fwd.argtypes = [I, P, I, I, I, I] + [P] * 6
        lib.oracle_shortconv_fwd.restype = I
        lib.oracle_shortconv_bwd.argtypes = [I, P, I, I, I, I] + [P] * 10
        lib.oracle_shortconv_bwd.restype = I
        lib.oracle_set_threads.argtypes = [I]
        lib.oracle_max_threads.restype = I
        _lib = lib
    return _lib


def set_threads(n: int) -> None:
    _load().oracle_set_threads(int(n))


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def _f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().cpu().double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def fwd_train(q, k, v, g, beta, qn, kn, vn, gn, betan, *, block, scale,
              cu_seqlens=None, h0=None, want_ht=True):
    """Two-stream forward.

    Shapes (non-packed): q,k [B,T,Hqk,dk]; v [B,T,Hv,dv]; g,beta [B,T,Hv].
    Packed: the same with B == 1 and ``cu_seqlens`` [N+1] int offsets.
    Returns (o, on, ht) as fp64 arrays; ht is [B or N, Hv, dk, dv] or None.
    """
    q, k, v, g, beta = map(_f64, (q, k, v, g, beta))
    qn, kn, vn, gn, betan = map(_f64, (qn, kn, vn, gn, betan))
    B, T, Hqk, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    cu = None
    nseq = B
    if cu_seqlens is not None:
        cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        nseq = cu.shape[0] - 1
        assert B == 1 and int(cu[-1]) <= T
    h0a = _f64(h0)
    o = np.zeros((B, T, Hv, dv))
    on = np.zeros((B, T, Hv, dv))
    ht = np.zeros((nseq, Hv, dk, dv)) if want_ht else None
    rc = _load().oracle_fwd_train(
        B, T, nseq, _ptr(cu), Hqk, Hv, dk, dv, int(block), float(scale),
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
        _ptr(qn), _ptr(kn), _ptr(vn), _ptr(gn), _ptr(betan),
        _ptr(h0a), _ptr(o), _ptr(on), _ptr(ht))
    if rc != 0:
        raise RuntimeError(f"oracle_fwd_train failed: {rc}")
    return o, on, ht


def bwd_train(q, k, v, g, beta, qn, kn, vn, gn, betan, do, don, *, block, scale,
              cu_seqlens=None, h0=None, dht=None, want_dh0=True):
    """Gradients of  sum(do * o) + sum(don * on) + sum(dht * ht)  for fwd_train's inputs.

    Same shapes as fwd_train; do, don like v; dht like ht (or None for zero).  Returns a
    dict with dq, dk, dv, dg, dbeta (clean), dqn, dkn, dvn, dgn, dbetan (noisy) and dh0
    ([B or N, Hv, dk, dv], or None), all fp64.  dq, dk of a q/k head sum over its v-heads.
    """
    q, k, v, g, beta = map(_f64, (q, k, v, g, beta))
    qn, kn, vn, gn, betan = map(_f64, (qn, kn, vn, gn, betan))
    do, don = _f64(do), _f64(don)
    B, T, Hqk, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    cu = None
    nseq = B
    if cu_seqlens is not None:
        cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        nseq = cu.shape[0] - 1
        assert B == 1 and int(cu[-1]) <= T
    h0a, dhta = _f64(h0), _f64(dht)
    out = {name: np.zeros(ref.shape) for name, ref in
           (("dq", q), ("dk", k), ("dv", v), ("dg", g), ("dbeta", beta),
            ("dqn", qn), ("dkn", kn), ("dvn", vn), ("dgn", gn), ("dbetan", betan))}
    out["dh0"] = np.zeros((nseq, Hv, dk, dv)) if want_dh0 else None
    rc = _load().oracle_bwd_train(
        B, T, nseq, _ptr(cu), Hqk, Hv, dk, dv, int(block), float(scale),
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
        _ptr(qn), _ptr(kn), _ptr(vn), _ptr(gn), _ptr(betan),
        _ptr(h0a), _ptr(do), _ptr(don), _ptr(dhta),
        *[_ptr(out[n]) for n in ("dq", "dk", "dv", "dg", "dbeta", "dqn", "dkn", "dvn", "dgn", "dbetan")],
        _ptr(out["dh0"]))
    if rc != 0:
        raise RuntimeError(f"oracle_bwd_train failed: {rc}")
    return out


def bwd_train_views(q, k, v, g, beta, views, do, *, block, scale, cu_seqlens=None, h0=None, dht=None):
    """Gradients of  sum(do * o) + sum_i sum(views[i]["do"] * o_i) + sum(dht * ht)  where o_i
    is the block-end readout of noisy view i (each view a noisy stream seeded from the same
    clean states; o and ht are the clean stream's, shared by every view).

    The loss is linear in its upstream gradients, so it is the sum over views of two-stream
    losses: view 0 carries do and dht, every other view only its own readout term (clean
    upstream gradient zero).  bwd_train of each gives that view's gradients and its share of
    the clean gradients; the clean ones add up.  Returns (clean, per_view): ``clean`` a dict
    dq, dk, dv, dg, dbeta, dh0, ``per_view`` one dict dq, dk, dv, dg, dbeta per view (fp64).
    """
    clean, per_view = None, []
    zero_do = np.zeros(np.shape(do))
    for i, w in enumerate(views):
        r = bwd_train(q, k, v, g, beta, w["q"], w["k"], w["v"], w["g"], w["beta"],
                      do if i == 0 else zero_do, w["do"], block=block, scale=scale,
                      cu_seqlens=cu_seqlens, h0=h0, dht=dht if i == 0 else None)
        per_view.append({name: r[name + "n"] for name in ("dq", "dk", "dv", "dg", "dbeta")})
        part = {name: r[name] for name in ("dq", "dk", "dv", "dg", "dbeta", "dh0")}
        clean = part if clean is None else {name: clean[name] + part[name] for name in part}
    return clean, per_view


def denoise(pool, q, k, v, g, beta, *, scale, slot=None):
    """Block-end readout of R blocks seeded from pool[slot[r]].

    pool [n_slots,Hv,dk,dv]; q,k [R,L,Hqk,dk]; v [R,L,Hv,dv]; g,beta [R,L,Hv].
    Returns o [R,L,Hv,dv] (fp64).  The pool is not modified.
    """
    pool = _f64(pool)
    q, k, v, g, beta = map(_f64, (q, k, v, g, beta))
    R, L, Hqk, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    sl = None if slot is None else np.ascontiguousarray(np.asarray(slot, dtype=np.int32))
    o = np.zeros((R, L, Hv, dv))
    rc = _load().oracle_denoise(R, Hqk, Hv, dk, dv, L, float(scale), _ptr(pool), _ptr(sl),
                                _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(o))
    if rc != 0:
        raise RuntimeError(f"oracle_denoise failed: {rc}")
    return o


def commit(pool, q, k, v, g, beta, *, scale, slot=None, want_o=True):
    """Token-causal pass over R blocks; returns (new_pool, o or None) in fp64.

    The input pool is copied; the returned pool holds the advanced states.
    """
    pool = _f64(pool).copy()
    q, k, v, g, beta = map(_f64, (q, k, v, g, beta))
    R, L, Hqk, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    sl = None if slot is None else np.ascontiguousarray(np.asarray(slot, dtype=np.int32))
    o = np.zeros((R, L, Hv, dv)) if want_o else None
    rc = _load().oracle_commit(R, Hqk, Hv, dk, dv, L, float(scale), _ptr(pool), _ptr(sl),
                               _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(o))
    if rc != 0:
        raise RuntimeError(f"oracle_commit failed: {rc}")
    return pool, o


def commit_record(pool, q, k, v, g, beta, *, scale, n_record, slot=None, want_o=True):
    """The commit pass that also keeps the verify-position states: states[r, i] is the
    state before block position L - n_record + i.  Returns (new_pool, o or None,
    states [R, n_record, Hv, dk, dv]) in fp64; the input pool is copied."""
    pool = _f64(pool).copy()
    q, k, v, g, beta = map(_f64, (q, k, v, g, beta))
    R, L, Hqk, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    sl = None if slot is None else np.ascontiguousarray(np.asarray(slot, dtype=np.int32))
    o = np.zeros((R, L, Hv, dv)) if want_o else None
    states = np.zeros((R, n_record, Hv, dk, dv))
    rc = _load().oracle_commit_record(R, Hqk, Hv, dk, dv, L, int(n_record), float(scale), _ptr(pool),
                                      _ptr(sl), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(o),
                                      _ptr(states))
    if rc != 0:
        raise RuntimeError(f"oracle_commit_record failed: {rc}")
    return pool, o, states


def accept_states(pool, states, accept, *, slot=None):
    """Pool after the verify decision: request r keeps states[r, accept[r]] (or the pool's
    state when accept[r] == n_record).  Returns the new pool (fp64 copy)."""
    pool = _f64(pool).copy()
    states = _f64(states)
    R, n_rec, Hv, dk, dv = states.shape
    acc = np.ascontiguousarray(np.asarray(accept, dtype=np.int32))
    sl = None if slot is None else np.ascontiguousarray(np.asarray(slot, dtype=np.int32))
    rc = _load().oracle_accept_states(R, Hv, dk, dv, n_rec, _ptr(pool), _ptr(sl), _ptr(states), _ptr(acc))
    if rc != 0:
        raise RuntimeError(f"oracle_accept_states failed: {rc}")
    return pool


def _conv_cu(rows, cu_seqlens):
    cu = np.array([0, rows], np.int32) if cu_seqlens is None else np.asarray(cu_seqlens, np.int32)
    return np.ascontiguousarray(cu), len(cu) - 1


def shortconv_fwd(x, xn, w, bias=None, *, block, act=1, cu_seqlens=None):
    """Two-stream ShortConv forward on one packed axis: x, xn [rows, D], w [D, W] (lag-i
    weight in column i), bias [D] or None.  Returns (y, yn) in fp64."""
    x, xn, w = _f64(x), _f64(xn), _f64(w)
    b = None if bias is None else _f64(bias)
    rows, D = x.shape
    W = w.shape[1]
    cu, n = _conv_cu(rows, cu_seqlens)
    y, yn = np.zeros((rows, D)), np.zeros((rows, D))
    rc = _load().oracle_shortconv_fwd(n, _ptr(cu), D, W, int(block), int(act), _ptr(x), _ptr(xn), _ptr(w),
                                      _ptr(b), _ptr(y), _ptr(yn))
    if rc != 0:
        raise RuntimeError(f"oracle_shortconv_fwd failed: {rc}")
    return y, yn


def shortconv_bwd(x, xn, w, bias, dy, dyn, *, block, act=1, cu_seqlens=None):
    """Backward of shortconv_fwd: returns (dx, dxn, dw, dbias or None) in fp64."""
    x, xn, w, dy, dyn = map(_f64, (x, xn, w, dy, dyn))
    b = None if bias is None else _f64(bias)
    rows, D = x.shape
    W = w.shape[1]
    cu, n = _conv_cu(rows, cu_seqlens)
    dx, dxn, dw = np.zeros((rows, D)), np.zeros((rows, D)), np.zeros((D, W))
    db = None if bias is None else np.zeros(D)
    rc = _load().oracle_shortconv_bwd(n, _ptr(cu), D, W, int(block), int(act), _ptr(x), _ptr(xn), _ptr(w),
                                      _ptr(b), _ptr(dy), _ptr(dyn), _ptr(dx), _ptr(dxn), _ptr(dw), _ptr(db))
    if rc != 0:
        raise RuntimeError(f"oracle_shortconv_bwd failed: {rc}")
    return dx, dxn, dw, db
