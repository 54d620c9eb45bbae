"""GPU parity of the complementary-view forward (bdgdn_fwd_train_views): one clean scan
seeding several noisy views.  Each view's readout must match the fp64 oracle's two-stream
forward with that view as the noisy stream, the clean outputs must match too, and one view
equals the split route of bdgdn_fwd_train bit for bit."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W
from parity_utils import TOL, rel_err

pytestmark = pytest.mark.gpu

KEYS = ("q", "k", "v", "g", "beta")


def _view(B, T, hqk, hv, seed, lengths=None):
    inp = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=seed, lengths=lengths)
    return {k: inp[k + "n"] for k in KEYS}


@pytest.mark.parametrize("route", [bd.BDGDN_ROUTE_FUSED, bd.BDGDN_ROUTE_SPLIT])
@pytest.mark.parametrize("B,T,hqk,hv,L,lengths,n_views", [
    (2, 96, 2, 2, 32, None, 2),
    (1, 130, 1, 2, 16, None, 3),                 # grouped heads, ragged tail
    (1, 160, 2, 2, 32, [64, 32, 64], 2),         # packed documents
    (1, 150, 1, 2, 4, None, 3),                  # small blocks: the first pass on 32-position chunks
])
def test_views_match_oracle(B, T, hqk, hv, L, lengths, n_views, route):
    print(f"views B={B} T={T} hqk={hqk} hv={hv} L={L} n={n_views} lengths={lengths} route={route}", flush=True)
    base = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=700 + T, lengths=lengths)
    clean = {k: base[k] for k in KEYS}
    views = [{k: base[k + "n"] for k in KEYS}] + [_view(B, T, hqk, hv, 800 + 7 * i + T, lengths)
                                                  for i in range(n_views - 1)]
    cu = None if lengths is None else np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    scale = 1.0 / math.sqrt(128)
    dc = {k: v.cuda() for k, v in clean.items()}
    dv = [{k: v.cuda() for k, v in w.items()} for w in views]
    o, outs, ht = bd.bdgdn_fwd_train_views(dc["q"], dc["k"], dc["v"], dc["g"], dc["beta"], dv, block=L, scale=scale,
                                           cu_seqlens=None if cu is None else torch.from_numpy(cu).cuda(),
                                           cu_seqlens_host=None if cu is None else torch.from_numpy(cu),
                                           want_ht=True, route=route)
    torch.cuda.synchronize()
    for i, w in enumerate(views):
        ro, ron, rht = oracle.fwd_train(*[clean[k] for k in KEYS], *[w[k] for k in KEYS], block=L, scale=scale,
                                        cu_seqlens=cu)
        e_on = rel_err(outs[i], ron)
        print(f"  view {i}: on {e_on:.2e}", flush=True)
        assert e_on <= TOL["bf16"]
        if i == 0:
            assert rel_err(o, ro) <= TOL["bf16"]
            assert rel_err(ht, rht) <= TOL["bf16"]


@pytest.mark.parametrize("B,T,hqk,hv,L,lengths,n_views", [
    (1, 200, 1, 2, 64, None, 2),                 # blocks of 64 (two halves), ragged tail
    (1, 256, 2, 2, 64, [128, 64, 64], 3),        # packed documents
])
def test_views_pair_blocks_match_oracle(B, T, hqk, hv, L, lengths, n_views):
    """Blocks of more than 32 positions: the fused route runs the one-kernel forward on
    half-block sub-blocks once per view."""
    test_views_match_oracle(B, T, hqk, hv, L, lengths, n_views, bd.BDGDN_ROUTE_FUSED)


def test_one_view_equals_fused_forward_and_views_equal_split_route():
    """One view is the one-kernel forward; a second view's readout is the split route's noisy
    pass from the same seeds (bit for bit)."""
    base = W.make_custom_train(2, 100, 2, 2, 128, 128, "bf16", seed=5)
    v2 = W.make_custom_train(2, 100, 2, 2, 128, 128, "bf16", seed=6)
    d = {k: v.cuda() for k, v in base.items()}
    d2 = {k: v.cuda() for k, v in v2.items()}
    scale = 1.0 / math.sqrt(128)
    of, onf, htf = bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"],
                                      d["gn"], d["betan"], block=32, scale=scale, want_ht=True)
    _, ons, _ = bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d2["qn"], d2["kn"], d2["vn"],
                                   d2["gn"], d2["betan"], block=32, scale=scale, route=bd.BDGDN_ROUTE_SPLIT)
    o1, outs1, ht1 = bd.bdgdn_fwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                              [{k: d[k + "n"] for k in KEYS}], block=32, scale=scale, want_ht=True)
    o2, outs2, ht2 = bd.bdgdn_fwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                              [{k: d[k + "n"] for k in KEYS}, {k: d2[k + "n"] for k in KEYS}],
                                              block=32, scale=scale, want_ht=True, route=bd.BDGDN_ROUTE_SPLIT)
    torch.cuda.synchronize()
    for a_, b_ in ((of, o1), (onf, outs1[0]), (htf, ht1), (of, o2), (onf, outs2[0]), (htf, ht2), (ons, outs2[1])):
        assert torch.equal(a_, b_)
