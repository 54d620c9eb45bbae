"""GPU check of bdgdn_shortconv_bwd_noalloc, the ShortConv backward that allocates nothing
(its partial sums live in the library's fixed per-GPU scratch): called through the C ABI,
its outputs equal bdgdn_shortconv_bwd's bit for bit on two calls in a row, the second on a
smaller input (the scratch keeps the first call's partials, which must not leak into the
second), and an input beyond the scratch is rejected before anything runs."""
import numpy as np
import pytest
import torch

import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W

pytestmark = pytest.mark.gpu


def _inputs(batch, seqlen, channels, width, seed, lengths=None):
    rng = np.random.default_rng(seed)
    c = W.draw_conv(rng, batch, seqlen, channels, width, "bf16")
    d = {k: (None if v is None else v.cuda()) for k, v in c.items()}
    if lengths is not None:
        cu = torch.tensor(np.concatenate([[0], np.cumsum(lengths)]), dtype=torch.int32)
        for k in ("x", "xn", "dy", "dyn"):
            d[k] = d[k].reshape(1, batch * seqlen, channels)
        d["cu"], d["cu_host"] = cu.cuda(), cu
    return d


def _both(d, block):
    kw = dict(block=block, activation=bd.BDGDN_ACT_SILU, cu_seqlens=d.get("cu"), cu_seqlens_host=d.get("cu_host"))
    ref = bd.bdgdn_shortconv_bwd(d["x"], d["xn"], d["w"], d["bias"], d["dy"], d["dyn"], **kw)
    out = [torch.full_like(t, float("nan")) for t in ref]
    got = bd.bdgdn_shortconv_bwd_noalloc(d["x"], d["xn"], d["w"], d["bias"], d["dy"], d["dyn"], dx=out[0],
                                         dxn=out[1], dw=out[2], dbias=out[3], **kw)
    torch.cuda.synchronize()
    return ref, got


def test_noalloc_matches_workspace_entry_point_twice():
    print("noalloc: 4 x 4096 rows x 6144 channels, width 4", flush=True)
    big = _inputs(4, 4096, 6144, 4, seed=11)
    ref, got = _both(big, 32)
    for name, r, g in zip(("dx", "dxn", "dw", "dbias"), ref, got):
        assert torch.equal(r, g), name
    del big
    print("noalloc: 3 packed documents, 1000 rows x 512 channels, width 3", flush=True)
    small = _inputs(1, 1000, 512, 3, seed=12, lengths=[300, 0, 700])
    ref, got = _both(small, 16)
    for name, r, g in zip(("dx", "dxn", "dw", "dbias"), ref, got):
        assert torch.equal(r, g), name


def test_noalloc_rejects_inputs_beyond_the_scratch():
    per_group = 5 * 6144 * 4
    rows = 1024 * (bd.BDGDN_NOALLOC_SCRATCH_BYTES // per_group) + 1
    print(f"noalloc: {rows} rows x 6144 channels (beyond the scratch)", flush=True)
    x = torch.zeros(1, rows, 6144, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(6144, 4, device="cuda")
    dx, dxn, dw = torch.zeros_like(x), torch.zeros_like(x), torch.zeros_like(w)
    with pytest.raises(bd.BdgdnError) as err:
        bd.bdgdn_shortconv_bwd_noalloc(x, x, w, None, x, x, block=32, dx=dx, dxn=dxn, dw=dw)
    assert err.value.status == bd.BDGDN_ERR_SCRATCH
    torch.cuda.synchronize()
    assert not dw.any()
