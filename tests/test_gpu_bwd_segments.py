"""GPU checks of the time-segmented training backward (strided clean-state checkpoints):
given a workspace below the full size, bdgdn_bwd_train and bdgdn_bwd_train_views run the
fewest time segments that fit, and every gradient (and dh0) equals the one-pass call's bit
for bit, over ragged tails, packed documents (an empty one among them), grouped value
heads, blocks of 16, 20, 32 and 64 (noisy blocks of two sub-blocks), an initial state with
a final-state gradient, bf16 upstream gradients and two noisy views; then the 4 x 4096
training shape in four segments, under 256 MiB of workspace, and the grouped-value and packed
128k workloads in eight, whole."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W
from parity_utils import TOL, rel_err

pytestmark = pytest.mark.gpu

NAMES = ("dq", "dk", "dv", "dg", "dbeta", "dqn", "dkn", "dvn", "dgn", "dbetan", "dh0")


def _desc(q, v, L, cu, do_dtype):
    return bd.make_fwd_desc(q, v, block=L, scale=1.0 / math.sqrt(q.shape[-1]),
                            num_seqs=0 if cu is None else cu.numel() - 1, out_dtype=do_dtype)


def _segments_run(desc, cu, budget):
    """The segment count the library runs with `budget` bytes: the fewest that fit."""
    for k in range(2, 1 << 16):
        need = bd.bdgdn_bwd_train_workspace_segmented(desc, cu, k)
        if need and need <= budget:
            return k
    raise AssertionError("no segment count fits")


def _case(B, T, hqk, hv, L, seed, lengths=None, do_dtype=torch.float32):
    inp = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=seed, lengths=lengths)
    rng = np.random.default_rng(seed + 1)
    nseq = B if lengths is None else len(lengths)
    do = torch.from_numpy(rng.standard_normal((B, T, hv, 128)).astype(np.float32)).to(do_dtype)
    don = torch.from_numpy(rng.standard_normal((B, T, hv, 128)).astype(np.float32)).to(do_dtype)
    h0 = torch.from_numpy((0.3 * rng.standard_normal((nseq, hv, 128, 128))).astype(np.float32))
    dht = torch.from_numpy(rng.standard_normal((nseq, hv, 128, 128)).astype(np.float32))
    cu = None if lengths is None else torch.tensor(np.concatenate([[0], np.cumsum(lengths)]), dtype=torch.int32)
    return inp, do, don, h0, dht, cu


def _bwd(d, do, don, L, cu, h0, dht, workspace=None):
    return bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                              d["betan"], do, don, block=L, cu_seqlens=None if cu is None else cu.cuda(),
                              cu_seqlens_host=cu, h0=h0, dht=dht, want_dh0=True, workspace=workspace)


@pytest.mark.parametrize("B,T,hqk,hv,L,lengths,segments,do_dtype", [
    (1, 2000, 1, 1, 32, None, 3, torch.float32),                      # ragged tail, segments of 22 blocks
    (1, 2048, 1, 1, 32, None, 8, torch.float32),                      # eight segments of 8
    (2, 1000, 1, 2, 16, None, 5, torch.float32),                      # grouped heads, blocks of 16
    (1, 3000, 2, 2, 20, None, 6, torch.bfloat16),                     # blocks of 20, bf16 upstream gradients
    (1, 2999, 1, 2, 32, [1024, 0, 544, 1431], 4, torch.float32),      # packed, an empty document
    (1, 2048, 1, 1, 64, None, 4, torch.float32),                      # noisy blocks of two sub-blocks
    (2, 1500, 1, 2, 48, None, 3, torch.float32),                      # blocks of 48, ragged
    (1, 2262, 1, 1, 64, [64, 0, 1408, 790], 3, torch.float32),        # packed, blocks of 64
])
def test_segmented_equals_one_pass_bitwise(B, T, hqk, hv, L, lengths, segments, do_dtype):
    inp, do, don, h0, dht, cu = _case(B, T, hqk, hv, L, 3000 + T + L, lengths, do_dtype)
    d = {k: v.cuda() for k, v in inp.items() if isinstance(v, torch.Tensor)}
    desc = _desc(d["q"], d["v"], L, cu, do_dtype)
    full = bd.bdgdn_bwd_train_workspace(desc)
    budget = bd.bdgdn_bwd_train_workspace_segmented(desc, cu, segments)
    ran = _segments_run(desc, cu, budget)
    print(f"segmented bwd B={B} T={T} hqk={hqk} hv={hv} L={L} lengths={lengths}: workspace {budget} of {full} "
          f"bytes, {ran} segments", flush=True)
    assert 0 < budget < full
    ref = _bwd(d, do.cuda(), don.cuda(), L, cu, h0.cuda(), dht.cuda())
    ws = torch.empty(budget, dtype=torch.uint8, device="cuda")
    got = _bwd(d, do.cuda(), don.cuda(), L, cu, h0.cuda(), dht.cuda(), workspace=ws)
    torch.cuda.synchronize()
    for name in NAMES:
        assert torch.equal(got[name], ref[name]), name


def test_segmented_matches_oracle():
    """One segmented call against the fp64 oracle directly (ragged tail, grouped heads)."""
    B, T, hqk, hv, L = 1, 700, 1, 2, 32
    inp, do, don, h0, dht, cu = _case(B, T, hqk, hv, L, 77)
    d = {k: v.cuda() for k, v in inp.items() if isinstance(v, torch.Tensor)}
    desc = _desc(d["q"], d["v"], L, None, torch.float32)
    budget = bd.bdgdn_bwd_train_workspace_segmented(desc, None, 3)
    print(f"segmented bwd vs oracle: {_segments_run(desc, None, budget)} segments", flush=True)
    got = _bwd(d, do.cuda(), don.cuda(), L, None, h0.cuda(), dht.cuda(),
               workspace=torch.empty(budget, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    ref = oracle.bwd_train(inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], inp["qn"], inp["kn"], inp["vn"],
                           inp["gn"], inp["betan"], do, don, block=L, scale=1.0 / math.sqrt(128), h0=h0, dht=dht)
    for name in NAMES:
        e = rel_err(got[name], ref[name])
        assert e <= TOL["bf16"], f"{name}: {e:.3e}"


@pytest.mark.parametrize("L,lengths", [(32, None), (64, [512, 640, 384])])
def test_segmented_views_equal_one_pass_bitwise(L, lengths):
    """The complementary-view backward with two views, segmented and not: the same bits."""
    B, T, hqk, hv = 1, 1536, 1, 2
    keys = ("q", "k", "v", "g", "beta")
    base = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=41, lengths=lengths)
    other = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=43, lengths=lengths)
    rng = np.random.default_rng(45)
    cu = None if lengths is None else torch.tensor(np.concatenate([[0], np.cumsum(lengths)]), dtype=torch.int32)
    views = []
    for src in (base, other):
        w = {k: src[k + "n"].cuda() for k in keys}
        w["do"] = torch.from_numpy(rng.standard_normal((B, T, hv, 128)).astype(np.float32)).cuda()
        views.append(w)
    dc = {k: base[k].cuda() for k in keys}
    do = torch.from_numpy(rng.standard_normal((B, T, hv, 128)).astype(np.float32)).cuda()
    nseq = B if lengths is None else len(lengths)
    h0 = torch.from_numpy((0.3 * rng.standard_normal((nseq, hv, 128, 128))).astype(np.float32)).cuda()
    desc = _desc(dc["q"], dc["v"], L, cu, torch.float32)
    budget = bd.bdgdn_bwd_train_workspace_segmented(desc, cu, 4)
    print(f"segmented views bwd L={L} lengths={lengths}: {_segments_run(desc, cu, budget)} segments", flush=True)

    def run(ws):
        return bd.bdgdn_bwd_train_views(dc["q"], dc["k"], dc["v"], dc["g"], dc["beta"], views, do, block=L,
                                        cu_seqlens=None if cu is None else cu.cuda(), cu_seqlens_host=cu, h0=h0,
                                        want_dh0=True, workspace=ws)
    ref_c, ref_v = run(None)
    got_c, got_v = run(torch.empty(budget, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    for n in ("dq", "dk", "dv", "dg", "dbeta", "dh0"):
        assert torch.equal(got_c[n], ref_c[n]), n
    for i in range(2):
        for n in ("dq", "dk", "dv", "dg", "dbeta"):
            assert torch.equal(got_v[i][n], ref_v[i][n]), (i, n)


def test_segmented_training_workload_under_256_mib():
    """The 4 x 4096 training shape (16 heads, blocks of 32) in four segments: its workspace
    under 256 MiB (against 604 MB in one pass), every gradient equal to the one-pass call's."""
    w = W.TRAIN_4K
    inp = W.make_train(w)
    d = {k: v.cuda() for k, v in inp.items() if isinstance(v, torch.Tensor)}
    rng = np.random.default_rng(5)
    shape = (w.batch, w.seqlen, w.h_v, 128)
    do = torch.from_numpy(rng.standard_normal(shape, dtype=np.float32)).cuda()
    don = torch.from_numpy(rng.standard_normal(shape, dtype=np.float32)).cuda()
    desc = _desc(d["q"], d["v"], w.block, None, torch.float32)
    budget = bd.bdgdn_bwd_train_workspace_segmented(desc, None, 4)
    print(f"segmented 4 x 4096: {budget} bytes, {_segments_run(desc, None, budget)} segments", flush=True)
    assert budget <= 256 << 20
    ref = _bwd(d, do, don, w.block, None, None, None)
    ref = {k: v.cpu() for k, v in ref.items()}
    got = _bwd(d, do, don, w.block, None, None, None, workspace=torch.empty(budget, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    for name in NAMES:
        assert torch.equal(got[name].cpu(), ref[name]), name


@pytest.mark.parametrize("name", ["GVA_16K", "VARLEN_128K"])
def test_segmented_full_workloads_equal_one_pass(name):
    """The grouped-value workload (blocks of 64: the pair kernel) and the packed 128k workload
    (32 documents) in eight segments, whole: every gradient equal to the one-pass call's."""
    w = getattr(W, name)
    raw = W.make_train(w)
    d = {k: v.cuda() for k, v in raw.items() if isinstance(v, torch.Tensor)}
    cu = raw.get("cu_seqlens")
    rng = np.random.default_rng(7)
    shape = (w.batch, w.seqlen, w.h_v, w.d_v)
    do = torch.from_numpy(rng.standard_normal(shape, dtype=np.float32)).cuda()
    don = torch.from_numpy(rng.standard_normal(shape, dtype=np.float32)).cuda()
    desc = _desc(d["q"], d["v"], w.block, cu, torch.float32)
    budget = bd.bdgdn_bwd_train_workspace_segmented(desc, cu, 8)
    print(f"segmented {w.name}: {budget} of {bd.bdgdn_bwd_train_workspace(desc)} bytes, "
          f"{_segments_run(desc, cu, budget)} segments", flush=True)
    ref = _bwd(d, do, don, w.block, cu, None, None)
    ref = {k: v.cpu() for k, v in ref.items()}
    torch.cuda.empty_cache()
    got = _bwd(d, do, don, w.block, cu, None, None, workspace=torch.empty(budget, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    for n in NAMES:
        assert torch.equal(got[n].cpu(), ref[n]), n
