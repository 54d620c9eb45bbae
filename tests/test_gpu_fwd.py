"""GPU parity of the two-stream training forward (bdgdn_fwd_train) against the
fp64 oracle, called through the C ABI.  Tolerance: max |gpu - oracle| divided by
the oracle output RMS, <= 2e-2 for bf16 inputs and <= 1e-4 for fp32, per tensor."""
import math

import numpy as np
import pytest
import torch

import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W
from parity_utils import TOL, oracle_full, rel_err, to_dev, unit_errors

pytestmark = pytest.mark.gpu


def _run_gpu(d, block, scale, h0=None, want_ht=True, route=bd.BDGDN_ROUTE_FUSED):
    o, on, ht = bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                   d["qn"], d["kn"], d["vn"], d["gn"], d["betan"],
                                   block=block, scale=scale, h0=h0,
                                   cu_seqlens=d.get("cu_seqlens"),
                                   cu_seqlens_host=d.get("cu_host"),
                                   want_ht=want_ht, route=route)
    torch.cuda.synchronize()
    return o, on, ht


def _check_full(inp, block, dtype, h0=None, route=bd.BDGDN_ROUTE_FUSED):
    scale = 1.0 / math.sqrt(inp["q"].shape[-1])
    d = to_dev(inp)
    if "cu_seqlens" in inp:
        d["cu_host"] = inp["cu_seqlens"]
    o, on, ht = _run_gpu(d, block, scale, h0=None if h0 is None else h0.cuda(), route=route)
    ro, ron, rht = oracle_full(inp, block, scale, h0=h0, cu=inp.get("cu_seqlens"))
    tol = TOL[dtype]
    eo, eon, eht = rel_err(o, ro), rel_err(on, ron), rel_err(ht, rht)
    print(f"err o={eo:.3e} on={eon:.3e} ht={eht:.3e}")
    assert eo <= tol and eon <= tol and eht <= tol, (eo, eon, eht)
    return o, on, ht


def test_tiny_f32_full_config():
    w = W.TINY_F32
    _check_full(W.make_train(w), w.block, "f32")


ROUTES = [bd.BDGDN_ROUTE_FUSED, bd.BDGDN_ROUTE_ONEPASS, bd.BDGDN_ROUTE_RECORDS]


@pytest.mark.parametrize("route", ROUTES)
@pytest.mark.parametrize("B,T,hqk,hv,d,L,dtype", [
    (2, 200, 2, 2, 128, 32, "bf16"),     # ragged tail (200 = 6*32 + 8)
    (1, 256, 2, 4, 128, 64, "bf16"),     # grouped value heads, L = 64
    (1, 160, 1, 2, 128, 16, "bf16"),
    (1, 120, 2, 2, 64, 24, "bf16"),      # block padded inside the tile, d = 64
    (1, 70, 1, 1, 128, 5, "bf16"),       # small block
    (1, 33, 1, 1, 64, 1, "bf16"),        # L = 1: each noisy block is one step
    (2, 100, 1, 2, 128, 32, "f32"),
    (1, 96, 2, 2, 64, 16, "f32"),
])
def test_small_shapes(B, T, hqk, hv, d, L, dtype, route):
    inp = W.make_custom_train(B, T, hqk, hv, d, d, dtype, seed=1000 + T + L)
    h0 = torch.randn(B, hv, d, d, generator=torch.Generator().manual_seed(T)) * 0.3
    _check_full(inp, L, dtype, h0=h0, route=route)


@pytest.mark.parametrize("B,T,hqk,hv,d,L,lengths", [
    (2, 64 * 3 + 20, 2, 4, 128, 64, None),    # last block: a partial first half, no second half
    (1, 64 * 2 + 45, 1, 2, 128, 64, None),    # last block: a full first half, a partial second half
    (1, 64 * 2 + 32, 1, 1, 128, 64, None),    # last block: exactly its first half
    (1, 200, 2, 2, 64, 64, None),             # d = 64
    (1, 150, 1, 1, 128, 48, None),            # halves of 24 positions
    (1, 136, 1, 1, 128, 34, None),            # halves of 17
    (1, 64 + 128 + 0 + 50, 2, 2, 128, 64, [64, 128, 0, 50]),   # packed: an empty and a partial document
])
def test_pair_blocks(B, T, hqk, hv, d, L, lengths):
    """Blocks of 34 to 64 positions in the one-kernel forward: each noisy block spans two
    sub-blocks of half the block, its state carried across them, and the first half's rows
    read the state at the block's end."""
    inp = W.make_custom_train(B, T, hqk, hv, d, d, "bf16", seed=2000 + T + L, lengths=lengths)
    h0 = None if lengths else torch.randn(B, hv, d, d, generator=torch.Generator().manual_seed(T + 1)) * 0.3
    _check_full(inp, L, "bf16", h0=h0)


@pytest.mark.parametrize("B,T,hqk,hv,d,L,lengths", [
    (2, 200, 2, 2, 128, 8, None),        # 200 = 6 * 32 + 8: the last chunk holds one noisy block
    (1, 150, 1, 2, 128, 4, None),        # 150 = 4 * 32 + 22: the last chunk ends inside a noisy block
    (1, 97, 2, 2, 64, 2, None),          # d = 64
    (1, 70, 1, 1, 128, 1, None),         # every noisy block one step
    (1, 256, 2, 4, 128, 8, None),        # grouped value heads
    (1, 8 + 40 + 0 + 96 + 23, 2, 2, 128, 8, [8, 40, 0, 96, 23]),   # packed: documents starting inside a chunk
])
def test_small_blocks(B, T, hqk, hv, d, L, lengths):
    """Noisy blocks of 1, 2, 4 or 8 positions in the one-kernel forward: the chain runs on
    32-position clean chunks and each chunk's noisy blocks are seeded with the clean state at
    their own start, formed on chip.  Against the oracle, and against the records route
    (one padded block per step)."""
    inp = W.make_custom_train(B, T, hqk, hv, d, d, "bf16", seed=7000 + T + L, lengths=lengths)
    h0 = None if lengths else torch.randn(B, hv, d, d, generator=torch.Generator().manual_seed(T + 3)) * 0.3
    o, on, ht = _check_full(inp, L, "bf16", h0=h0)
    d_ = to_dev(inp)
    if lengths:
        d_["cu_host"] = inp["cu_seqlens"]
    b = _run_gpu(d_, L, 1.0 / math.sqrt(d), h0=None if h0 is None else h0.cuda(), route=bd.BDGDN_ROUTE_RECORDS)
    for x, y in zip((o, on, ht), b):
        e = rel_err(x, y.double().cpu().numpy())
        print(f"small-block kernel vs records route {e:.3e}")
        assert e <= TOL["bf16"]


def test_small_blocks_bf16_outputs():
    """The small-block kernel with bf16 outputs: the fp32-output kernel's results rounded, bit
    for bit, and the same final state."""
    inp = W.make_custom_train(2, 150, 2, 2, 128, 128, "bf16", seed=23)
    d = to_dev(inp)
    o16, on16, ht16 = bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                         d["qn"], d["kn"], d["vn"], d["gn"], d["betan"],
                                         block=4, scale=0.0884, want_ht=True, out_dtype=torch.bfloat16)
    o32, on32, ht32 = _run_gpu(d, 4, 0.0884)
    assert o16.dtype == torch.bfloat16 and on16.dtype == torch.bfloat16
    assert torch.equal(o32.to(torch.bfloat16), o16) and torch.equal(on32.to(torch.bfloat16), on16)
    assert torch.equal(ht32, ht16)


@pytest.mark.parametrize("L", [1, 8])
def test_full_small_blocks_all_units(L):
    """The block-size sweep's shape (1 x 4096 clean + 4096 noisy tokens, 16 heads, d = 128)
    at noisy blocks of 1 and 8 positions: every (sequence, head) unit against the oracle."""
    inp = W.make_custom_train(1, 4096, 16, 16, 128, 128, "bf16", seed=8000 + L)
    d = to_dev(inp)
    scale = 1.0 / math.sqrt(128)
    print(f"small blocks L={L}: GPU", flush=True)
    o, on, ht = _run_gpu(d, L, scale)
    o, on, ht = o.cpu(), on.cpu(), ht.cpu()
    print(f"small blocks L={L}: oracle", flush=True)
    ro, ron, rht = oracle_full(inp, L, scale)
    worst = {}
    for name, gpu, ref, kind in (("o", o, ro, False), ("on", on, ron, False), ("ht", ht, rht, None)):
        e, where, n = unit_errors(gpu, ref, per_token=kind)
        print(f"  {name}: worst unit {where} max|err|/rms = {e:.3e} over {n} units", flush=True)
        worst[name] = e
        assert n == 16
    assert max(worst.values()) <= TOL["bf16"], worst


@pytest.mark.parametrize("route", ROUTES)
def test_packed_documents_small(route):
    lengths = [64, 96, 32, 0, 64, 128, 17]   # an empty doc and a ragged last doc
    inp = W.make_custom_train(1, sum(lengths), 2, 2, 128, 128, "bf16", seed=77, lengths=lengths)
    _check_full(inp, 32, "bf16", route=route)


@pytest.mark.parametrize("L", [16, 32, 64])
def test_routes_agree(L):
    """The schedules compute the same function: the fused route (one kernel up to
    32-position blocks), the records route and the one-pass route agree to rounding."""
    inp = W.make_custom_train(2, 4 * L + 5, 2, 4, 128, 128, "bf16", seed=L)
    d = to_dev(inp)
    a = _run_gpu(d, L, 0.1, route=bd.BDGDN_ROUTE_FUSED)
    for other in (bd.BDGDN_ROUTE_ONEPASS, bd.BDGDN_ROUTE_RECORDS):
        b = _run_gpu(d, L, 0.1, route=other)
        for x, y in zip(a, b):
            e = rel_err(x, y.double().cpu().numpy())
            print(f"route {other} difference {e:.3e}")
            assert e <= TOL["bf16"]


@pytest.mark.parametrize("B,T,hqk,hv,L,lengths", [
    (2, 200, 2, 2, 32, None),           # ragged tail
    (1, 256, 2, 4, 32, None),           # grouped value heads
    (1, 150, 1, 2, 16, None),
    (1, 70, 1, 1, 5, None),             # small block, padded to 16
    (1, 401, 2, 2, 32, [64, 96, 0, 32, 192, 17]),   # packed, an empty and a ragged doc
])
def test_split_route(B, T, hqk, hv, L, lengths):
    """The split schedule (clean scan writing the seed states, then the noisy-block kernel)
    against the oracle, and against the fused schedule: the same clean arithmetic, and
    noisy outputs within rounding of each other."""
    inp = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=500 + T + L, lengths=lengths)
    h0 = None if lengths else torch.randn(B, hv, 128, 128, generator=torch.Generator().manual_seed(L)) * 0.3
    o, on, ht = _check_full(inp, L, "bf16", h0=h0, route=bd.BDGDN_ROUTE_SPLIT)
    d = to_dev(inp)
    if lengths:
        d["cu_host"] = inp["cu_seqlens"]
    fo, fon, fht = _run_gpu(d, L, 1.0 / math.sqrt(128), h0=None if h0 is None else h0.cuda())
    assert torch.equal(o, fo) and torch.equal(ht, fht)
    e = rel_err(on, fon.double().cpu().numpy())
    print(f"split vs fused noisy difference {e:.3e}")
    assert e <= TOL["bf16"]


@pytest.mark.parametrize("B,T,hqk,hv,d,L,lengths", [
    (2, 1100, 2, 2, 128, 32, None),     # 35 blocks: three segments of 16, a ragged tail
    (1, 600, 2, 4, 128, 16, None),      # grouped value heads, L = 16: 38 blocks
    (1, 300, 1, 2, 64, 5, None),        # d = 64, L = 5 (padded to 16): 60 blocks, 4 segments
    (1, 520, 1, 1, 128, 32, None),      # 17 blocks: a last segment of one partial block
    (1, 1024 + 64 + 544 + 640 + 17, 2, 2, 128, 32, [1024, 64, 0, 544, 640, 17]),   # packed
])
def test_chunked_route(B, T, hqk, hv, d, L, lengths):
    """The chunk-parallel schedule (state pass over the segment starts, then one workgroup
    per (chain, segment)) against the oracle, and against the fused schedule within the
    same tolerance."""
    inp = W.make_custom_train(B, T, hqk, hv, d, d, "bf16", seed=3000 + T + L, lengths=lengths)
    h0 = None if lengths else torch.randn(B, hv, d, d, generator=torch.Generator().manual_seed(T + 7)) * 0.3
    o, on, ht = _check_full(inp, L, "bf16", h0=h0, route=bd.BDGDN_ROUTE_CHUNKED)
    dd = to_dev(inp)
    if lengths:
        dd["cu_host"] = inp["cu_seqlens"]
    fused = _run_gpu(dd, L, 1.0 / math.sqrt(d), h0=None if h0 is None else h0.cuda())
    for x, y in zip((o, on, ht), fused):
        e = rel_err(x, y.double().cpu().numpy())
        print(f"chunked vs fused difference {e:.3e}")
        assert e <= TOL["bf16"]


@pytest.mark.parametrize("B,T,hqk,hv,d,L,lengths", [
    (2, 500, 2, 2, 128, 32, None),      # 16 blocks: one segment per chain, a ragged tail
    (1, 256, 1, 2, 64, 16, None),
    (1, 64 + 96 + 17, 1, 1, 128, 32, [64, 96, 17]),
])
def test_chunked_one_segment_equals_fused_bitwise(B, T, hqk, hv, d, L, lengths):
    """With one segment per chain the chunk-parallel schedule has no state pass, and its
    workgroup carries out the fused schedule's block arithmetic operation for operation:
    the results are equal bit for bit."""
    inp = W.make_custom_train(B, T, hqk, hv, d, d, "bf16", seed=4000 + T, lengths=lengths)
    dd = to_dev(inp)
    if lengths:
        dd["cu_host"] = inp["cu_seqlens"]
    h0 = None if lengths else (torch.randn(B, hv, d, d, generator=torch.Generator().manual_seed(T)) * 0.3).cuda()
    a = _run_gpu(dd, L, 0.1, h0=h0, route=bd.BDGDN_ROUTE_CHUNKED)
    b = _run_gpu(dd, L, 0.1, h0=h0)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


@pytest.mark.parametrize("B,T,hqk,hv,L,lengths", [
    (16, 150, 4, 16, 32, None),    # 256 chains, a ragged tail
    (1, 17 * 64 + 5 * 96 + 33, 8, 16, 32, [64] * 9 + [0] + [96] * 5 + [64] * 8 + [33]),   # 24 documents
])
def test_fused_wide_pass_many_chains(B, T, hqk, hv, L, lengths):
    """With (sequences or documents) x v-heads >= 256 the fused route runs one workgroup
    per chain over all d_v columns (the chunk-parallel output pass, one segment per chain)."""
    inp = W.make_custom_train(B, T, hqk, hv, 128, 128, "bf16", seed=6000 + T, lengths=lengths)
    h0 = None if lengths else torch.randn(B, hv, 128, 128, generator=torch.Generator().manual_seed(T)) * 0.3
    o, on, ht = _check_full(inp, L, "bf16", h0=h0)
    d = to_dev(inp)
    if lengths:
        d["cu_host"] = inp["cu_seqlens"]
    b = _run_gpu(d, L, 1.0 / math.sqrt(128), h0=None if h0 is None else h0.cuda(), route=bd.BDGDN_ROUTE_ONEPASS)
    for x, y in zip((o, on, ht), b):
        e = rel_err(x, y.double().cpu().numpy())
        print(f"wide pass vs one-pass route {e:.3e}")
        assert e <= TOL["bf16"]


def test_packed_equals_separate_bitwise():
    """Packing reproduces per-document results exactly (Appendix, packing contract)."""
    lengths = [96, 64, 40]
    inp = W.make_custom_train(1, sum(lengths), 1, 2, 128, 128, "bf16", seed=5, lengths=lengths)
    d = to_dev(inp)
    d["cu_host"] = inp["cu_seqlens"]
    o, on, ht = _run_gpu(d, 32, 0.1)
    cu = inp["cu_seqlens"].tolist()
    for i in range(len(lengths)):
        sub = {k: v[:, cu[i]:cu[i + 1]].contiguous().cuda() for k, v in inp.items()
               if k not in ("cu_seqlens",)}
        so, son, sht = _run_gpu(sub, 32, 0.1)
        assert torch.equal(so, o[:, cu[i]:cu[i + 1]])
        assert torch.equal(son, on[:, cu[i]:cu[i + 1]])
        assert torch.equal(sht[0], ht[i])


def test_determinism_and_isolation():
    """Run-to-run bitwise determinism; perturbing one noisy block changes only that
    block's noisy outputs (clean outputs and other blocks bitwise unchanged)."""
    inp = W.make_custom_train(1, 256, 2, 2, 128, 128, "bf16", seed=9)
    d = to_dev(inp)
    o1, on1, ht1 = _run_gpu(d, 32, 0.1)
    o2, on2, ht2 = _run_gpu(d, 32, 0.1)
    assert torch.equal(o1, o2) and torch.equal(on1, on2) and torch.equal(ht1, ht2)
    blk = slice(64, 96)
    d2 = dict(d)
    for key in ("qn", "kn", "vn"):
        t = d[key].clone()
        t[:, blk] = torch.flip(t[:, blk], dims=[1])
        d2[key] = t
    o3, on3, ht3 = _run_gpu(d2, 32, 0.1)
    assert torch.equal(o3, o1) and torch.equal(ht3, ht1)
    mask = torch.zeros(256, dtype=torch.bool)
    mask[blk] = True
    assert torch.equal(on3[:, ~mask], on1[:, ~mask])
    assert not torch.equal(on3[:, mask], on1[:, mask])


def _full_size(w, route=bd.BDGDN_ROUTE_FUSED):
    """The whole workload on the GPU in the benchmark's launch configuration, every
    (sequence or document, v-head) unit compared with one multi-threaded oracle call:
    the worst per-unit max |err| / RMS of o, on and ht must meet the tolerance."""
    inp = W.make_train(w)
    d = to_dev(inp)
    cu = inp.get("cu_seqlens")
    if cu is not None:
        d["cu_host"] = cu
    scale = 1.0 / math.sqrt(w.d_k)
    print(f"{w.name}: GPU (route {route})", flush=True)
    o, on, ht = _run_gpu(d, w.block, scale, route=route)
    assert torch.isfinite(o.float()).all() and torch.isfinite(on.float()).all()
    o, on, ht = o.cpu(), on.cpu(), ht.cpu()
    del d
    print(f"{w.name}: oracle", flush=True)
    ro, ron, rht = oracle_full(inp, w.block, scale, cu=cu)
    tol = TOL[w.dtype]
    worst = {}
    for name, gpu, ref, kind in (("o", o, ro, False), ("on", on, ron, False), ("ht", ht, rht, None)):
        e, where, n = unit_errors(gpu, ref, cu=None if cu is None else cu.numpy(), per_token=kind)
        print(f"  {name}: worst unit {where} max|err|/rms = {e:.3e} over {n} units; "
              f"whole tensor {rel_err(gpu, ref):.3e}", flush=True)
        worst[name] = e
    expected = (len(cu) - 1 if cu is not None else w.batch) * w.h_v
    assert n == expected - (0 if cu is None else int((np.diff(cu.numpy()) == 0).sum()) * w.h_v)
    assert max(worst.values()) <= tol, worst


def test_full_train_4k_all_units():
    _full_size(W.TRAIN_4K)


def test_full_train_4k_all_units_chunked():
    _full_size(W.TRAIN_4K, route=bd.BDGDN_ROUTE_CHUNKED)


def test_full_varlen_128k_all_units_chunked():
    _full_size(W.VARLEN_128K, route=bd.BDGDN_ROUTE_CHUNKED)


def test_full_gva_16k_all_units():
    _full_size(W.GVA_16K)


def test_full_varlen_128k_all_units():
    _full_size(W.VARLEN_128K)


def test_bf16_outputs():
    """bf16 outputs (the production-training format): the error budget is the
    stated tolerance plus the output's own rounding (|bf16(x) - x| of the oracle)."""
    inp = W.make_custom_train(2, 192, 2, 2, 128, 128, "bf16", seed=21)
    d = to_dev(inp)
    o, on, ht = bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                   d["qn"], d["kn"], d["vn"], d["gn"], d["betan"],
                                   block=32, scale=0.0884, want_ht=True,
                                   out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert o.dtype == torch.bfloat16 and on.dtype == torch.bfloat16
    ro, ron, rht = oracle_full(inp, 32, 0.0884)
    for name, gpu, ref in (("o", o, ro), ("on", on, ron)):
        rnd = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).double().numpy()
        budget = TOL["bf16"] + np.abs(rnd - ref).max() / np.sqrt((ref ** 2).mean())
        e = rel_err(gpu, ref)
        print(f"{name}: err {e:.3e} budget {budget:.3e}")
        assert e <= budget
    assert rel_err(ht, rht) <= TOL["bf16"]
    # same arithmetic as the fp32-output kernel up to the final rounding
    o32, on32, _ = _run_gpu(d, 32, 0.0884)
    assert torch.equal(o32.to(torch.bfloat16), o) and torch.equal(on32.to(torch.bfloat16), on)
