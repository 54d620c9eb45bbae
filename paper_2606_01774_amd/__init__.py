"""Block-diffusion Gated DeltaNet for AMD MI355X (gfx950): Python binding.

A thin ctypes layer over ``libbdgdn.so`` (C ABI in ``include/bdgdn.h``).  The
functions carry the C names and only marshal arguments: PyTorch supplies device
memory and the current HIP stream; every step of the computation runs in the HIP
kernels.  There is no CPU fallback: without the built library (or without a GPU)
these functions raise.

Layouts (token-major, contiguous): q, k ``[rows, h_qk, d_k]`` (or any leading
shape that flattens to rows), v, o ``[rows, h_v, d_v]``, g (log-gate), beta
``[rows, h_v]`` fp32; states ``[units, h_v, d_k, d_v]`` fp32.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

__all__ = [
    "BdgdnError", "BDGDN_BF16", "BDGDN_F32", "BDGDN_ROUTE_FUSED", "BDGDN_ROUTE_SPLIT",
    "BDGDN_ROUTE_ONEPASS", "BDGDN_ROUTE_RECORDS", "BDGDN_ROUTE_CHUNKED",
    "bdgdn_version", "bdgdn_status_string", "bdgdn_fwd_train_workspace", "bdgdn_fwd_train",
    "bdgdn_commit_record", "bdgdn_accept_states", "BDGDN_ACT_NONE", "BDGDN_ACT_SILU",
    "bdgdn_shortconv_fwd", "bdgdn_shortconv_bwd_workspace", "bdgdn_shortconv_bwd",
    "bdgdn_bwd_train_workspace", "bdgdn_bwd_train_workspace_segmented", "bdgdn_bwd_train",
    "bdgdn_fwd_train_views_workspace", "bdgdn_fwd_train_views",
    "bdgdn_bwd_train_views_workspace", "bdgdn_bwd_train_views", "bdgdn_denoise_step", "bdgdn_commit", "library_path", "load_library", "EXPORTED_SYMBOLS",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libbdgdn.so")

BDGDN_OK = 0
BDGDN_ERR_INVALID_ARG = -1
BDGDN_ERR_UNSUPPORTED = -2
BDGDN_ERR_UNALIGNED = -3
BDGDN_ERR_WORKSPACE = -4
BDGDN_ERR_LAUNCH = -5
BDGDN_ERR_SCRATCH = -6
BDGDN_NOALLOC_SCRATCH_BYTES = 32 << 20
BDGDN_BF16 = 0
BDGDN_F32 = 1
BDGDN_ROUTE_FUSED = 0
BDGDN_ROUTE_SPLIT = 1
BDGDN_ROUTE_ONEPASS = 2
BDGDN_ROUTE_RECORDS = 3
BDGDN_ROUTE_CHUNKED = 4
BDGDN_ACT_NONE = 0
BDGDN_ACT_SILU = 1

EXPORTED_SYMBOLS = ("bdgdn_version", "bdgdn_status_string", "bdgdn_fwd_train_workspace",
                    "bdgdn_fwd_train", "bdgdn_denoise_step", "bdgdn_commit", "bdgdn_commit_record",
                    "bdgdn_accept_states", "bdgdn_shortconv_fwd", "bdgdn_shortconv_bwd_workspace",
                    "bdgdn_shortconv_bwd", "bdgdn_bwd_train_workspace", "bdgdn_bwd_train",
                    "bdgdn_fwd_train_views_workspace", "bdgdn_fwd_train_views",
                    "bdgdn_bwd_train_views_workspace", "bdgdn_bwd_train_views",
                    "bdgdn_shortconv_bwd_noalloc", "bdgdn_bwd_train_workspace_segmented")


class FwdDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seqlen", ctypes.c_int32),
                ("num_seqs", ctypes.c_int32), ("h_qk", ctypes.c_int32),
                ("h_v", ctypes.c_int32), ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("block", ctypes.c_int32), ("scale", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("route", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32)]


class ServeDesc(ctypes.Structure):
    _fields_ = [("num_req", ctypes.c_int32), ("h_qk", ctypes.c_int32),
                ("h_v", ctypes.c_int32), ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("block", ctypes.c_int32), ("scale", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class NoisyView(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("beta", ctypes.c_void_p), ("o", ctypes.c_void_p)]


class NoisyViewGrad(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("beta", ctypes.c_void_p), ("do_", ctypes.c_void_p),
                ("dq", ctypes.c_void_p), ("dk", ctypes.c_void_p), ("dv", ctypes.c_void_p),
                ("dg", ctypes.c_void_p), ("dbeta", ctypes.c_void_p)]


class ConvDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seqlen", ctypes.c_int32),
                ("num_seqs", ctypes.c_int32), ("channels", ctypes.c_int32),
                ("width", ctypes.c_int32), ("block", ctypes.c_int32),
                ("activation", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class BdgdnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {bdgdn_status_string(status)} ({status})")


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libbdgdn.so (built in-tree by ``build.py``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run paper_2606_01774_amd/build.py")
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    lib.bdgdn_version.restype = ctypes.c_int32
    lib.bdgdn_status_string.argtypes = [ctypes.c_int]
    lib.bdgdn_status_string.restype = ctypes.c_char_p
    lib.bdgdn_fwd_train_workspace.argtypes = [ctypes.POINTER(FwdDesc)]
    lib.bdgdn_fwd_train_workspace.restype = ctypes.c_size_t
    lib.bdgdn_fwd_train.argtypes = [ctypes.POINTER(FwdDesc)] + [P] * 17 + [ctypes.c_size_t, P]
    lib.bdgdn_fwd_train.restype = ctypes.c_int
    lib.bdgdn_denoise_step.argtypes = [ctypes.POINTER(ServeDesc)] + [P] * 9
    lib.bdgdn_denoise_step.restype = ctypes.c_int
    lib.bdgdn_commit.argtypes = [ctypes.POINTER(ServeDesc)] + [P] * 9
    lib.bdgdn_commit.restype = ctypes.c_int
    lib.bdgdn_commit_record.argtypes = [ctypes.POINTER(ServeDesc)] + [P] * 8 + [ctypes.c_int32, P, P]
    lib.bdgdn_commit_record.restype = ctypes.c_int
    lib.bdgdn_accept_states.argtypes = [ctypes.POINTER(ServeDesc), P, P, P, ctypes.c_int32, P, P]
    lib.bdgdn_accept_states.restype = ctypes.c_int
    lib.bdgdn_fwd_train_views_workspace.argtypes = [ctypes.POINTER(FwdDesc)]
    lib.bdgdn_fwd_train_views_workspace.restype = ctypes.c_size_t
    lib.bdgdn_fwd_train_views.argtypes = ([ctypes.POINTER(FwdDesc)] + [P] * 5 + [ctypes.POINTER(NoisyView), ctypes.c_int32]
                                          + [P] * 6 + [ctypes.c_size_t, P])
    lib.bdgdn_fwd_train_views.restype = ctypes.c_int
    lib.bdgdn_bwd_train_workspace.argtypes = [ctypes.POINTER(FwdDesc)]
    lib.bdgdn_bwd_train_workspace.restype = ctypes.c_size_t
    lib.bdgdn_bwd_train_workspace_segmented.argtypes = [ctypes.POINTER(FwdDesc), P, ctypes.c_int32]
    lib.bdgdn_bwd_train_workspace_segmented.restype = ctypes.c_size_t
    lib.bdgdn_bwd_train.argtypes = [ctypes.POINTER(FwdDesc)] + [P] * 28 + [ctypes.c_size_t, P]
    lib.bdgdn_bwd_train.restype = ctypes.c_int
    lib.bdgdn_bwd_train_views_workspace.argtypes = [ctypes.POINTER(FwdDesc)]
    lib.bdgdn_bwd_train_views_workspace.restype = ctypes.c_size_t
    lib.bdgdn_bwd_train_views.argtypes = ([ctypes.POINTER(FwdDesc)] + [P] * 5
                                          + [ctypes.POINTER(NoisyViewGrad), ctypes.c_int32] + [P] * 12
                                          + [ctypes.c_size_t, P])
    lib.bdgdn_bwd_train_views.restype = ctypes.c_int
    lib.bdgdn_shortconv_fwd.argtypes = [ctypes.POINTER(ConvDesc)] + [P] * 9
    lib.bdgdn_shortconv_fwd.restype = ctypes.c_int
    lib.bdgdn_shortconv_bwd_workspace.argtypes = [ctypes.POINTER(ConvDesc)]
    lib.bdgdn_shortconv_bwd_workspace.restype = ctypes.c_size_t
    lib.bdgdn_shortconv_bwd.argtypes = [ctypes.POINTER(ConvDesc)] + [P] * 13 + [ctypes.c_size_t, P]
    lib.bdgdn_shortconv_bwd.restype = ctypes.c_int
    lib.bdgdn_shortconv_bwd_noalloc.argtypes = [ctypes.POINTER(ConvDesc)] + [P] * 13
    lib.bdgdn_shortconv_bwd_noalloc.restype = ctypes.c_int
    _lib = lib
    return lib


def bdgdn_version() -> int:
    return int(load_library().bdgdn_version())


def bdgdn_status_string(status: int) -> str:
    return load_library().bdgdn_status_string(int(status)).decode()


# ------------------------------------------------------------------ marshalling
_DT = {torch.bfloat16: BDGDN_BF16, torch.float32: BDGDN_F32}


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _dev(t, name, dtype=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status, where):
    if status != BDGDN_OK:
        raise BdgdnError(status, where)


def make_fwd_desc(q, v, *, block, scale=None, batch=None, num_seqs=0, route=BDGDN_ROUTE_FUSED,
                  out_dtype=torch.float32):
    """Descriptor from 4-D tensors q [B,T,h_qk,d_k], v [B,T,h_v,d_v]."""
    B, T, h_qk, d_k = q.shape
    h_v, d_v = v.shape[2], v.shape[3]
    if scale is None:
        scale = 1.0 / math.sqrt(d_k)
    return FwdDesc(B if batch is None else batch, T, num_seqs, h_qk, h_v, d_k, d_v, int(block),
                   float(scale), _DT.get(q.dtype, -1), int(route), _DT.get(out_dtype, -1))


def bdgdn_fwd_train_workspace(desc: FwdDesc) -> int:
    return int(load_library().bdgdn_fwd_train_workspace(ctypes.byref(desc)))


def bdgdn_fwd_train(q, k, v, g, beta, qn, kn, vn, gn, betan, *, block, scale=None,
                    cu_seqlens=None, cu_seqlens_host=None, h0=None, o=None, on=None,
                    ht=None, want_ht=False, route=BDGDN_ROUTE_FUSED, workspace=None,
                    out_dtype=torch.float32, stream=None):
    """Two-stream training forward.  Tensors are [B,T,h,d] (packed: B == 1 and
    cu_seqlens [N+1] int32 on the device; cu_seqlens_host may be given to avoid a
    device-to-host copy).  Outputs are ``out_dtype`` (fp32 by default; bf16 is
    offered for bf16 inputs).  Returns (o, on, ht)."""
    lib = load_library()
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v), ("qn", qn), ("kn", kn), ("vn", vn)):
        _dev(t, name, dt)
    for name, t in (("g", g), ("beta", beta), ("gn", gn), ("betan", betan)):
        _dev(t, name, torch.float32)
    if q.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v must be [B, T, heads, dim]")
    num_seqs = 0
    cu_h = None
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        num_seqs = cu_seqlens.numel() - 1
        if cu_seqlens_host is None:
            cu_seqlens_host = cu_seqlens.cpu()
        cu_h = torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
        if cu_h.numel() != num_seqs + 1:
            raise ValueError("cu_seqlens_host and cu_seqlens differ in length")
    if o is not None:
        out_dtype = o.dtype
    desc = make_fwd_desc(q, v, block=block, scale=scale, num_seqs=num_seqs, route=route,
                         out_dtype=out_dtype)
    if o is None:
        o = torch.empty(v.shape, dtype=out_dtype, device=v.device)
    if on is None:
        on = torch.empty(vn.shape, dtype=out_dtype, device=vn.device)
    _dev(o, "o", out_dtype)
    _dev(on, "on", out_dtype)
    units = num_seqs if num_seqs else q.shape[0]
    if ht is None and want_ht:
        ht = torch.empty(units, v.shape[2], q.shape[3], v.shape[3], device=q.device,
                         dtype=torch.float32)
    _dev(ht, "ht", torch.float32)
    _dev(h0, "h0", torch.float32)
    ws_bytes = bdgdn_fwd_train_workspace(desc)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_size = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.bdgdn_fwd_train(
        ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
        _ptr(qn), _ptr(kn), _ptr(vn), _ptr(gn), _ptr(betan),
        _ptr(cu_seqlens), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
        _ptr(h0), _ptr(o), _ptr(on), _ptr(ht), _ptr(workspace), ws_size, _stream(stream))
    _check(st, "bdgdn_fwd_train")
    return o, on, ht


def bdgdn_fwd_train_views_workspace(desc: FwdDesc) -> int:
    return int(load_library().bdgdn_fwd_train_views_workspace(ctypes.byref(desc)))


def bdgdn_fwd_train_views(q, k, v, g, beta, views, *, block, scale=None, cu_seqlens=None, cu_seqlens_host=None,
                          h0=None, o=None, ht=None, want_ht=False, out_dtype=torch.float32,
                          route=BDGDN_ROUTE_FUSED, workspace=None, stream=None):
    """Complementary-view forward: one clean stream (q, k, v, g, beta, [B,T,h,d]) and
    ``views``, a list of noisy streams, each a dict with q, k, v, g, beta (and optionally o).
    route FUSED (a one-kernel pass per view) or SPLIT (one clean pass writing the seeds, then
    a noisy pass per further view).  Returns (o, [view outputs], ht)."""
    lib = load_library()
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, dt)
    for name, t in (("g", g), ("beta", beta)):
        _dev(t, name, torch.float32)
    if o is not None:
        out_dtype = o.dtype
    num_seqs = 0
    cu_h = None
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        num_seqs = cu_seqlens.numel() - 1
        if cu_seqlens_host is None:
            cu_seqlens_host = cu_seqlens.cpu()
        cu_h = torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
    desc = make_fwd_desc(q, v, block=block, scale=scale, num_seqs=num_seqs, route=route, out_dtype=out_dtype)
    if o is None:
        o = torch.empty(v.shape, dtype=out_dtype, device=v.device)
    _dev(o, "o", out_dtype)
    outs = []
    arr = (NoisyView * max(1, len(views)))()
    for i, w in enumerate(views):
        for name in ("q", "k", "v"):
            _dev(w[name], f"views[{i}].{name}", dt)
        for name in ("g", "beta"):
            _dev(w[name], f"views[{i}].{name}", torch.float32)
        ov = w.get("o")
        if ov is None:
            ov = torch.empty(w["v"].shape, dtype=out_dtype, device=v.device)
        _dev(ov, f"views[{i}].o", out_dtype)
        outs.append(ov)
        arr[i] = NoisyView(w["q"].data_ptr(), w["k"].data_ptr(), w["v"].data_ptr(), w["g"].data_ptr(),
                           w["beta"].data_ptr(), ov.data_ptr())
    units = num_seqs if num_seqs else q.shape[0]
    if ht is None and want_ht:
        ht = torch.empty(units, v.shape[2], q.shape[3], v.shape[3], device=q.device, dtype=torch.float32)
    _dev(ht, "ht", torch.float32)
    _dev(h0, "h0", torch.float32)
    ws_bytes = bdgdn_fwd_train_views_workspace(desc)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_size = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.bdgdn_fwd_train_views(
        ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), arr, len(views),
        _ptr(cu_seqlens), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
        _ptr(h0), _ptr(o), _ptr(ht), _ptr(workspace), ws_size, _stream(stream))
    _check(st, "bdgdn_fwd_train_views")
    return o, outs, ht


def bdgdn_bwd_train_workspace(desc: FwdDesc) -> int:
    return int(load_library().bdgdn_bwd_train_workspace(ctypes.byref(desc)))


def bdgdn_bwd_train_workspace_segmented(desc: FwdDesc, cu_seqlens_host, segments: int) -> int:
    """Workspace of the backward run in ``segments`` time segments (cu_seqlens_host: the
    packing as an int32 CPU tensor, or None)."""
    cu_h = None if cu_seqlens_host is None else torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
    return int(load_library().bdgdn_bwd_train_workspace_segmented(
        ctypes.byref(desc), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()), int(segments)))


def _bwd_workspace(desc, cu_h, segments, full, device):
    """The backward's workspace: the full size, or that of ``segments`` time segments."""
    ws_bytes = full if segments is None else bdgdn_bwd_train_workspace_segmented(desc, cu_h, segments)
    return torch.empty(ws_bytes, dtype=torch.uint8, device=device) if ws_bytes else None


_BWD_NAMES = ("dq", "dk", "dv", "dg", "dbeta", "dqn", "dkn", "dvn", "dgn", "dbetan")


def bdgdn_bwd_train(q, k, v, g, beta, qn, kn, vn, gn, betan, do, don, *, block, scale=None,
                    cu_seqlens=None, cu_seqlens_host=None, h0=None, dht=None, want_dh0=False,
                    grads=None, workspace=None, segments=None, stream=None):
    """Backward of bdgdn_fwd_train: gradients of sum(do*o) + sum(don*on) + sum(dht*ht).
    Inputs as for bdgdn_fwd_train; do, don [B,T,h_v,d_v] in the forward's output dtype
    (fp32 or bf16); dht like ht or None.  Returns a dict of fp32 tensors (dq, dk, dv, dg,
    dbeta and the noisy dqn, ..., dbetan; dh0 when want_dh0).  ``grads`` may supply the
    output tensors (same names).  Without ``workspace``, one of the full size is allocated,
    or with ``segments`` that of that many time segments (the library then runs the
    segmented schedule)."""
    lib = load_library()
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v), ("qn", qn), ("kn", kn), ("vn", vn)):
        _dev(t, name, dt)
    for name, t in (("g", g), ("beta", beta), ("gn", gn), ("betan", betan)):
        _dev(t, name, torch.float32)
    _dev(do, "do")
    _dev(don, "don", do.dtype)
    num_seqs = 0
    cu_h = None
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        num_seqs = cu_seqlens.numel() - 1
        if cu_seqlens_host is None:
            cu_seqlens_host = cu_seqlens.cpu()
        cu_h = torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
    desc = make_fwd_desc(q, v, block=block, scale=scale, num_seqs=num_seqs, out_dtype=do.dtype)
    out = {} if grads is None else dict(grads)
    like = {"dq": q, "dk": k, "dv": v, "dg": g, "dbeta": beta, "dqn": qn, "dkn": kn, "dvn": vn, "dgn": gn,
            "dbetan": betan}
    for name in _BWD_NAMES:
        if name not in out:
            out[name] = torch.empty(like[name].shape, dtype=torch.float32, device=q.device)
        _dev(out[name], name, torch.float32)
    units = num_seqs if num_seqs else q.shape[0]
    if want_dh0 and "dh0" not in out:
        out["dh0"] = torch.empty(units, v.shape[2], q.shape[3], v.shape[3], dtype=torch.float32, device=q.device)
    _dev(h0, "h0", torch.float32)
    _dev(dht, "dht", torch.float32)
    if workspace is None:
        workspace = _bwd_workspace(desc, cu_h, segments, bdgdn_bwd_train_workspace(desc), q.device)
    ws_size = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.bdgdn_bwd_train(
        ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
        _ptr(qn), _ptr(kn), _ptr(vn), _ptr(gn), _ptr(betan),
        _ptr(cu_seqlens), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
        _ptr(h0), _ptr(do), _ptr(don), _ptr(dht),
        *[_ptr(out[n]) for n in _BWD_NAMES], _ptr(out.get("dh0")),
        _ptr(workspace), ws_size, _stream(stream))
    _check(st, "bdgdn_bwd_train")
    return out


def bdgdn_bwd_train_views_workspace(desc: FwdDesc) -> int:
    return int(load_library().bdgdn_bwd_train_views_workspace(ctypes.byref(desc)))


_VIEW_GRAD_NAMES = ("dq", "dk", "dv", "dg", "dbeta")


def bdgdn_bwd_train_views(q, k, v, g, beta, views, do, *, block, scale=None, cu_seqlens=None,
                          cu_seqlens_host=None, h0=None, dht=None, want_dh0=False, grads=None, workspace=None,
                          segments=None, stream=None):
    """Backward of bdgdn_fwd_train_views: gradients of sum(do*o) + sum_i sum(views[i]["do"]*o_i)
    + sum(dht*ht).  ``views`` is a list of dicts with the view's q, k, v, g, beta and the
    upstream gradient "do" of its readout.  Returns (clean, per_view): ``clean`` a dict of
    fp32 tensors dq, dk, dv, dg, dbeta (and dh0 when want_dh0), ``per_view`` one such dict per
    view.  ``grads`` may supply them (a previous call's result).  ``workspace`` and
    ``segments`` as for bdgdn_bwd_train."""
    lib = load_library()
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, dt)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    _dev(do, "do")
    n = len(views)
    arr = (NoisyViewGrad * max(n, 1))()
    per_view = []
    like = {"dq": q, "dk": k, "dv": v, "dg": g, "dbeta": beta}
    for i, w in enumerate(views):
        for name in ("q", "k", "v"):
            _dev(w[name], f"views[{i}].{name}", dt)
        for name in ("g", "beta"):
            _dev(w[name], f"views[{i}].{name}", torch.float32)
        _dev(w["do"], f"views[{i}].do", do.dtype)
        gr = grads[1][i] if grads is not None else {
            name: torch.empty(like[name].shape, dtype=torch.float32, device=q.device) for name in _VIEW_GRAD_NAMES}
        for name in _VIEW_GRAD_NAMES:
            _dev(gr[name], f"views[{i}] {name}", torch.float32)
        per_view.append(gr)
        arr[i] = NoisyViewGrad(*[_ptr(w[name]) for name in ("q", "k", "v", "g", "beta", "do")],
                               *[_ptr(gr[name]) for name in _VIEW_GRAD_NAMES])
    num_seqs = 0
    cu_h = None
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        num_seqs = cu_seqlens.numel() - 1
        if cu_seqlens_host is None:
            cu_seqlens_host = cu_seqlens.cpu()
        cu_h = torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
    desc = make_fwd_desc(q, v, block=block, scale=scale, num_seqs=num_seqs, out_dtype=do.dtype)
    clean = dict(grads[0]) if grads is not None else {
        name: torch.empty(like[name].shape, dtype=torch.float32, device=q.device) for name in _VIEW_GRAD_NAMES}
    for name in _VIEW_GRAD_NAMES:
        _dev(clean[name], name, torch.float32)
    units = num_seqs if num_seqs else q.shape[0]
    if want_dh0 and "dh0" not in clean:
        clean["dh0"] = torch.empty(units, v.shape[2], q.shape[3], v.shape[3], dtype=torch.float32, device=q.device)
    _dev(h0, "h0", torch.float32)
    _dev(dht, "dht", torch.float32)
    if workspace is None:
        workspace = _bwd_workspace(desc, cu_h, segments, bdgdn_bwd_train_views_workspace(desc), q.device)
    ws_size = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.bdgdn_bwd_train_views(
        ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), arr, n,
        _ptr(cu_seqlens), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
        _ptr(h0), _ptr(do), _ptr(dht), *[_ptr(clean[name]) for name in _VIEW_GRAD_NAMES], _ptr(clean.get("dh0")),
        _ptr(workspace), ws_size, _stream(stream))
    _check(st, "bdgdn_bwd_train_views")
    return clean, per_view


def _serve_desc(q, v, scale, out_dtype):
    R, L, h_qk, d_k = q.shape
    h_v, d_v = v.shape[2], v.shape[3]
    if scale is None:
        scale = 1.0 / math.sqrt(d_k)
    return ServeDesc(R, h_qk, h_v, d_k, d_v, L, float(scale), _DT.get(q.dtype, -1),
                     _DT.get(out_dtype, -1))


def bdgdn_denoise_step(state_pool, q, k, v, g, beta, *, scale=None, slot=None, o=None,
                       out_dtype=torch.float32, stream=None):
    """Block-end readout of R blocks ([R, L, h, d] tensors) seeded from
    state_pool[slot[r]]; the pool is only read.  Returns o."""
    lib = load_library()
    dt = q.dtype
    _dev(state_pool, "state_pool", torch.float32)
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, dt)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    _dev(slot, "slot", torch.int32)
    if o is not None:
        out_dtype = o.dtype
    if o is None:
        o = torch.empty(v.shape, dtype=out_dtype, device=v.device)
    _dev(o, "o", out_dtype)
    desc = _serve_desc(q, v, scale, out_dtype)
    st = lib.bdgdn_denoise_step(ctypes.byref(desc), _ptr(state_pool), _ptr(slot), _ptr(q),
                                _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(o), _stream(stream))
    _check(st, "bdgdn_denoise_step")
    return o


def bdgdn_commit(state_pool, q, k, v, g, beta, *, scale=None, slot=None, o_causal=None,
                 want_o=False, out_dtype=torch.float32, stream=None):
    """Token-causal pass over R blocks; advances state_pool[slot[r]] in place.
    Returns o_causal (or None)."""
    lib = load_library()
    dt = q.dtype
    _dev(state_pool, "state_pool", torch.float32)
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, dt)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    _dev(slot, "slot", torch.int32)
    if o_causal is not None:
        out_dtype = o_causal.dtype
    if o_causal is None and want_o:
        o_causal = torch.empty(v.shape, dtype=out_dtype, device=v.device)
    _dev(o_causal, "o_causal", out_dtype)
    desc = _serve_desc(q, v, scale, out_dtype)
    st = lib.bdgdn_commit(ctypes.byref(desc), _ptr(state_pool), _ptr(slot), _ptr(q), _ptr(k),
                          _ptr(v), _ptr(g), _ptr(beta), _ptr(o_causal), _stream(stream))
    _check(st, "bdgdn_commit")
    return o_causal


def bdgdn_commit_record(state_pool, q, k, v, g, beta, *, n_record, scale=None, slot=None, states=None,
                        o_causal=None, want_o=False, out_dtype=torch.float32, stream=None):
    """The AR-Trust verify pass: bdgdn_commit over R blocks of L positions that also writes
    states[r, i] = the state before block position L - n_record + i.
    Returns (states [R, n_record, Hv, dk, dv] fp32, o_causal or None)."""
    lib = load_library()
    dt = q.dtype
    _dev(state_pool, "state_pool", torch.float32)
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, dt)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    _dev(slot, "slot", torch.int32)
    R, L, _, dk = q.shape
    Hv, dv = v.shape[2], v.shape[3]
    if states is None:
        states = torch.empty(R, int(n_record), Hv, dk, dv, dtype=torch.float32, device=q.device)
    _dev(states, "states", torch.float32)
    if o_causal is not None:
        out_dtype = o_causal.dtype
    if o_causal is None and want_o:
        o_causal = torch.empty(v.shape, dtype=out_dtype, device=v.device)
    _dev(o_causal, "o_causal", out_dtype)
    desc = _serve_desc(q, v, scale, out_dtype)
    st = lib.bdgdn_commit_record(ctypes.byref(desc), _ptr(state_pool), _ptr(slot), _ptr(q), _ptr(k),
                                 _ptr(v), _ptr(g), _ptr(beta), _ptr(o_causal), int(n_record), _ptr(states),
                                 _stream(stream))
    _check(st, "bdgdn_commit_record")
    return states, o_causal


def bdgdn_accept_states(state_pool, states, accept, *, block, h_qk=None, slot=None, stream=None):
    """The accept step: state_pool[slot[r]] <- states[r, accept[r]] where accept[r] <
    n_record (states [R, n_record, Hv, dk, dv] from bdgdn_commit_record; block = its L)."""
    lib = load_library()
    _dev(state_pool, "state_pool", torch.float32)
    _dev(states, "states", torch.float32)
    _dev(accept, "accept", torch.int32)
    _dev(slot, "slot", torch.int32)
    R, n_record, Hv, dk, dv = states.shape
    desc = ServeDesc(R, Hv if h_qk is None else int(h_qk), Hv, dk, dv, int(block), 1.0, BDGDN_BF16,
                     _DT[torch.float32])
    st = lib.bdgdn_accept_states(ctypes.byref(desc), _ptr(state_pool), _ptr(slot), _ptr(states),
                                 int(n_record), _ptr(accept), _stream(stream))
    _check(st, "bdgdn_accept_states")


# ------------------------------------------------------------------ ShortConv
def _conv_packing(x, cu_seqlens, cu_seqlens_host):
    if x.dim() != 3:
        raise ValueError("x must be [B, T, channels]")
    if cu_seqlens is None:
        return 0, None
    _dev(cu_seqlens, "cu_seqlens", torch.int32)
    n = cu_seqlens.numel() - 1
    if cu_seqlens_host is None:
        cu_seqlens_host = cu_seqlens.cpu()
    cu_h = torch.as_tensor(cu_seqlens_host, dtype=torch.int32).contiguous()
    if cu_h.numel() != n + 1:
        raise ValueError("cu_seqlens_host and cu_seqlens differ in length")
    return n, cu_h


def make_conv_desc(x, w, *, block, activation=BDGDN_ACT_SILU, num_seqs=0):
    """Descriptor from x [B, T, channels] and w [channels, width]."""
    B, T, D = x.shape
    return ConvDesc(B, T, num_seqs, D, int(w.shape[1]), int(block), int(activation), _DT.get(x.dtype, -1))


def bdgdn_shortconv_fwd(x, xn, w, bias=None, *, block, activation=BDGDN_ACT_SILU, cu_seqlens=None,
                        cu_seqlens_host=None, y=None, yn=None, stream=None):
    """Two-stream ShortConv forward.  x, xn [B, T, channels] (bf16 or fp32; packed: B == 1
    and cu_seqlens [N+1] int32 on the device), w [channels, width] fp32 (lag-i weight in
    column i), bias [channels] fp32 or None.  Returns (y, yn) of x's dtype."""
    lib = load_library()
    _dev(x, "x")
    _dev(xn, "xn", x.dtype)
    _dev(w, "w", torch.float32)
    _dev(bias, "bias", torch.float32)
    n, cu_h = _conv_packing(x, cu_seqlens, cu_seqlens_host)
    if xn.shape != x.shape or w.dim() != 2 or w.shape[0] != x.shape[2]:
        raise ValueError("xn must match x and w must be [channels, width]")
    desc = make_conv_desc(x, w, block=block, activation=activation, num_seqs=n)
    if y is None:
        y = torch.empty_like(x)
    if yn is None:
        yn = torch.empty_like(x)
    _dev(y, "y", x.dtype)
    _dev(yn, "yn", x.dtype)
    st = lib.bdgdn_shortconv_fwd(ctypes.byref(desc), _ptr(x), _ptr(xn), _ptr(w), _ptr(bias), _ptr(cu_seqlens),
                                 None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()), _ptr(y), _ptr(yn),
                                 _stream(stream))
    _check(st, "bdgdn_shortconv_fwd")
    return y, yn


def bdgdn_shortconv_bwd_workspace(desc: ConvDesc) -> int:
    return int(load_library().bdgdn_shortconv_bwd_workspace(ctypes.byref(desc)))


def bdgdn_shortconv_bwd(x, xn, w, bias, dy, dyn, *, block, activation=BDGDN_ACT_SILU, cu_seqlens=None,
                        cu_seqlens_host=None, dx=None, dxn=None, dw=None, dbias=None, workspace=None,
                        stream=None):
    """Backward of bdgdn_shortconv_fwd for upstream gradients dy, dyn (x's shape and dtype).
    Returns (dx, dxn, dw, dbias); dbias is None when bias is None."""
    lib = load_library()
    _dev(x, "x")
    for name, t in (("xn", xn), ("dy", dy), ("dyn", dyn)):
        _dev(t, name, x.dtype)
        if t.shape != x.shape:
            raise ValueError(f"{name} must match x")
    _dev(w, "w", torch.float32)
    _dev(bias, "bias", torch.float32)
    n, cu_h = _conv_packing(x, cu_seqlens, cu_seqlens_host)
    desc = make_conv_desc(x, w, block=block, activation=activation, num_seqs=n)
    dx = torch.empty_like(x) if dx is None else dx
    dxn = torch.empty_like(x) if dxn is None else dxn
    dw = torch.empty_like(w) if dw is None else dw
    if dbias is None and bias is not None:
        dbias = torch.empty_like(bias)
    for name, t, dt in (("dx", dx, x.dtype), ("dxn", dxn, x.dtype), ("dw", dw, torch.float32),
                        ("dbias", dbias, torch.float32)):
        _dev(t, name, dt)
    ws_bytes = bdgdn_shortconv_bwd_workspace(desc)
    if workspace is None and ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    ws_size = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.bdgdn_shortconv_bwd(ctypes.byref(desc), _ptr(x), _ptr(xn), _ptr(w), _ptr(bias), _ptr(dy), _ptr(dyn),
                                 _ptr(cu_seqlens), None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
                                 _ptr(dx), _ptr(dxn), _ptr(dw), _ptr(dbias), _ptr(workspace), ws_size,
                                 _stream(stream))
    _check(st, "bdgdn_shortconv_bwd")
    return dx, dxn, dw, dbias


def bdgdn_shortconv_bwd_noalloc(x, xn, w, bias, dy, dyn, *, block, activation=BDGDN_ACT_SILU, cu_seqlens=None,
                                cu_seqlens_host=None, dx=None, dxn=None, dw=None, dbias=None, stream=None):
    """bdgdn_shortconv_bwd through the entry point that allocates nothing: its partial sums
    live in the library's fixed per-GPU scratch (BDGDN_NOALLOC_SCRATCH_BYTES).  Pass every
    output to keep the call free of allocation here too.  Returns (dx, dxn, dw, dbias)."""
    lib = load_library()
    _dev(x, "x")
    for name, t in (("xn", xn), ("dy", dy), ("dyn", dyn)):
        _dev(t, name, x.dtype)
        if t.shape != x.shape:
            raise ValueError(f"{name} must match x")
    _dev(w, "w", torch.float32)
    _dev(bias, "bias", torch.float32)
    n, cu_h = _conv_packing(x, cu_seqlens, cu_seqlens_host)
    desc = make_conv_desc(x, w, block=block, activation=activation, num_seqs=n)
    dx = torch.empty_like(x) if dx is None else dx
    dxn = torch.empty_like(x) if dxn is None else dxn
    dw = torch.empty_like(w) if dw is None else dw
    if dbias is None and bias is not None:
        dbias = torch.empty_like(bias)
    for name, t, dt in (("dx", dx, x.dtype), ("dxn", dxn, x.dtype), ("dw", dw, torch.float32),
                        ("dbias", dbias, torch.float32)):
        _dev(t, name, dt)
    st = lib.bdgdn_shortconv_bwd_noalloc(ctypes.byref(desc), _ptr(x), _ptr(xn), _ptr(w), _ptr(bias), _ptr(dy),
                                         _ptr(dyn), _ptr(cu_seqlens),
                                         None if cu_h is None else ctypes.c_void_p(cu_h.data_ptr()),
                                         _ptr(dx), _ptr(dxn), _ptr(dw), _ptr(dbias), _stream(stream))
    _check(st, "bdgdn_shortconv_bwd_noalloc")
    return dx, dxn, dw, dbias
