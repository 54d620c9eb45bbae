"""GPU parity of the two-stream ShortConv (bdgdn_shortconv_fwd / _bwd) against the fp64
oracle, through the C ABI: ragged row and channel tails, every supported width, blocks
of one row and blocks longer than the sequence, packed documents (empty ones and ones
shorter than the filter), the full 4096 x 6144 layer shape, and bit-for-bit repeatable
filter gradients."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W
from parity_utils import TOL, rel_err

pytestmark = pytest.mark.gpu


def _run(inp, block, act, cu=None):
    dev = {k: (None if v is None else v.cuda()) for k, v in inp.items()}
    cu_dev = None if cu is None else torch.tensor(cu, dtype=torch.int32, device="cuda")
    y, yn = bd.bdgdn_shortconv_fwd(dev["x"], dev["xn"], dev["w"], dev["bias"], block=block, activation=act,
                                   cu_seqlens=cu_dev)
    dx, dxn, dw, db = bd.bdgdn_shortconv_bwd(dev["x"], dev["xn"], dev["w"], dev["bias"], dev["dy"], dev["dyn"],
                                             block=block, activation=act, cu_seqlens=cu_dev)
    torch.cuda.synchronize()
    return y, yn, dx, dxn, dw, db


def _oracle(inp, block, act, cu):
    B, T, D = inp["x"].shape
    flat = {k: (None if v is None else (v.reshape(B * T, D) if v.dim() == 3 else v).double().numpy())
            for k, v in inp.items()}
    y, yn = oracle.shortconv_fwd(flat["x"], flat["xn"], flat["w"], flat["bias"], block=block, act=act,
                                 cu_seqlens=cu)
    dx, dxn, dw, db = oracle.shortconv_bwd(flat["x"], flat["xn"], flat["w"], flat["bias"], flat["dy"],
                                           flat["dyn"], block=block, act=act, cu_seqlens=cu)
    return y, yn, dx, dxn, dw, db


def _budget(ref, stored):
    """The stated tolerance, plus for a tensor stored in bf16 its own rounding: the
    kernels compute in fp32 and round once on the store, the same rule as the bf16
    outputs of the GDR passes."""
    if stored != "bf16":
        return TOL[stored]
    rnd = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).double().numpy()
    return TOL["bf16"] + np.abs(rnd - ref).max() / np.sqrt((ref ** 2).mean())


def _check(got, ref, dtype):
    names = ("y", "yn", "dx", "dxn", "dw", "dbias")
    for name, g, r in zip(names, got, ref):
        if r is None:
            assert g is None, name
            continue
        g = g.reshape(r.shape)
        err = rel_err(g, r)
        # dw, dbias are fp32 sums of products of the stored inputs: the plain tolerance
        budget = _budget(r, dtype) if name in ("y", "yn", "dx", "dxn") else TOL[dtype]
        print(f"  {name}: {err:.3e} (budget {budget:.3e})")
        assert err <= budget, f"{name}: {err:.3e} > {budget:.3e}"


@pytest.mark.parametrize("B,T,D,width,block,act,dtype,bias,lengths", [
    (2, 100, 280, 4, 8, 1, "bf16", True, None),          # ragged rows and channel groups
    (1, 77, 64, 3, 1, 0, "f32", False, None),            # one-row blocks: noisy lags read clean
    (3, 64, 128, 1, 32, 1, "bf16", True, None),          # width 1
    (2, 40, 64, 4, 64, 1, "bf16", True, None),           # block longer than the sequence
    (1, 300, 136, 4, 32, 1, "f32", True, [0, 5, 1, 130, 0, 3, 161]),   # empty and short docs
    (1, 200, 256, 2, 7, 1, "bf16", False, [64, 64, 72]),
    (1, 129, 8, 4, 16, 0, "bf16", True, [129]),
])
def test_shortconv_small(B, T, D, width, block, act, dtype, bias, lengths):
    print(f"shortconv B={B} T={T} D={D} W={width} L={block} act={act} {dtype} lengths={lengths}", flush=True)
    rng = np.random.default_rng(1000 + T + D + width)
    inp = W.draw_conv(rng, B, T, D, width, dtype, bias=bias)
    if lengths is not None:
        cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
        assert cu[-1] == T
    else:
        cu = (np.arange(B + 1) * T).astype(np.int32)
    got = _run(inp, block, act, None if lengths is None else cu)
    ref = _oracle(inp, block, act, cu)
    _check(got, ref, dtype)


def test_shortconv_layer_shape():
    """4096 clean + 4096 noisy rows of 6144 channels, width 4, silu, blocks of 32."""
    w = W.CONV_4K
    print(f"shortconv {w.name}", flush=True)
    inp = W.make_conv(w)
    got = _run(inp, w.block, w.act)
    ref = _oracle(inp, w.block, w.act, np.array([0, w.seqlen], np.int32))
    _check(got, ref, w.dtype)


def test_shortconv_packed_batch_equivalence_and_determinism():
    """B sequences equal B packed documents of the same lengths, and two backward calls
    give the same filter gradients bit for bit."""
    rng = np.random.default_rng(77)
    inp = W.draw_conv(rng, 3, 96, 192, 4, "bf16")
    a = _run(inp, 16, 1)
    packed = {k: (None if v is None else (v.reshape(1, 288, 192) if v.dim() == 3 else v)) for k, v in inp.items()}
    b = _run(packed, 16, 1, [0, 96, 192, 288])
    for x, y in zip(a, b):
        assert torch.equal(x.reshape(y.shape), y)
    c = _run(inp, 16, 1)
    assert torch.equal(a[4], c[4]) and torch.equal(a[5], c[5])


def test_shortconv_zero_rows():
    """An empty batch writes zero filter gradients."""
    x = torch.empty(1, 0, 64, dtype=torch.bfloat16, device="cuda")
    w = torch.ones(64, 4, device="cuda")
    bias = torch.ones(64, device="cuda")
    y, yn = bd.bdgdn_shortconv_fwd(x, x, w, bias, block=8)
    dx, dxn, dw, db = bd.bdgdn_shortconv_bwd(x, x, w, bias, x, x, block=8,
                                             dw=torch.full((64, 4), 7.0, device="cuda"),
                                             dbias=torch.full((64,), 7.0, device="cuda"))
    torch.cuda.synchronize()
    assert y.numel() == 0 and dx.numel() == 0
    assert torch.count_nonzero(dw).item() == 0 and torch.count_nonzero(db).item() == 0
