"""GPU parity of the serving passes (bdgdn_denoise_step, bdgdn_commit) against the
fp64 oracle, through the C ABI, plus the state-pool contracts: denoise never
writes the pool; commit writes exactly the named slots."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01774_amd as bd
from paper_2606_01774_amd import workloads as W
from parity_utils import TOL, rel_err

pytestmark = pytest.mark.gpu


def _block(R, L, hqk, hv, d, dtype, seed):
    rng = np.random.default_rng(seed)
    return W.draw_stream(rng, (R, L), hqk, hv, d, d, dtype)


def _realistic_pool(n, hv, d, seed, prefix=64):
    """Prefix states made by the oracle's causal pass over seeded prefix tokens."""
    blk = _block(n, prefix, hv, hv, d, "f32", seed)
    zero = np.zeros((n, hv, d, d))
    pool, _ = oracle.commit(zero, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                            scale=1.0, want_o=False)
    return torch.from_numpy(pool.astype(np.float32))


@pytest.mark.parametrize("R,L,hqk,hv,d,dtype", [
    (3, 32, 2, 4, 128, "bf16"), (2, 64, 1, 1, 128, "bf16"), (4, 16, 2, 2, 64, "bf16"),
    (2, 7, 1, 1, 128, "bf16"), (3, 16, 1, 2, 64, "f32"), (2, 32, 1, 1, 128, "f32"),
])
def test_denoise_and_commit_small(R, L, hqk, hv, d, dtype):
    pool = _realistic_pool(R + 1, hv, d, seed=R * 100 + L)
    slot = torch.tensor(list(range(R, 0, -1)), dtype=torch.int32)   # permuted, slot 0 unused
    blk = _block(R, L, hqk, hv, d, dtype, seed=L)
    scale = 1.0 / math.sqrt(d)
    dp = pool.cuda()
    db = {k: v.cuda() for k, v in blk.items()}
    before = dp.clone()
    o = bd.bdgdn_denoise_step(dp, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale,
                              slot=slot.cuda())
    torch.cuda.synchronize()
    assert torch.equal(dp, before), "denoise wrote the state pool"
    ref = oracle.denoise(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], scale=scale,
                         slot=slot.numpy())
    e = rel_err(o, ref)
    print(f"denoise err={e:.3e}")
    assert e <= TOL[dtype]
    oc = bd.bdgdn_commit(dp, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale,
                         slot=slot.cuda(), want_o=True)
    torch.cuda.synchronize()
    rpool, ro = oracle.commit(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                              scale=scale, slot=slot.numpy())
    eo, es = rel_err(oc, ro), rel_err(dp[1:], rpool[1:])
    print(f"commit err o={eo:.3e} state={es:.3e}")
    assert eo <= TOL[dtype] and es <= TOL[dtype]
    assert torch.equal(dp[0], before[0]), "commit wrote an unnamed slot"
    # commit without the causal output writes the same state
    dp2 = before.clone()
    bd.bdgdn_commit(dp2, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale,
                    slot=slot.cuda())
    torch.cuda.synchronize()
    assert torch.equal(dp2, dp)


def test_denoise_matches_training_noisy_block():
    """The denoise pass from a cached state equals the training forward's noisy
    block that follows the same prefix (h0 = the cached state)."""
    R, L, hv, d = 2, 32, 2, 128
    pool = _realistic_pool(R, hv, d, seed=3)
    blk = _block(R, L, hv, hv, d, "bf16", seed=4)
    db = {k: v.cuda() for k, v in blk.items()}
    o = bd.bdgdn_denoise_step(pool.cuda(), db["q"], db["k"], db["v"], db["g"], db["beta"], scale=0.2)
    _, on, _ = bd.bdgdn_fwd_train(db["q"], db["k"], db["v"], db["g"], db["beta"],
                                  db["q"], db["k"], db["v"], db["g"], db["beta"],
                                  block=L, scale=0.2, h0=pool.cuda())
    torch.cuda.synchronize()
    e = rel_err(o, on.double().cpu().numpy())
    print(f"denoise vs training noisy block: {e:.3e} (bitwise {torch.equal(o, on)})")
    assert e <= 1e-2


def test_full_serving_workload():
    """64 requests x 32 heads x 128x128 states, 8 denoise steps then one commit."""
    w = W.SERVE_64
    pool = _realistic_pool(w.requests, w.h_v, w.d_k, seed=w.seed)
    dp = pool.cuda()
    before = dp.clone()
    scale = 1.0 / math.sqrt(w.d_k)
    for step in range(w.steps):
        blk = W.make_serve_block(w, step)
        db = {k: v.cuda() for k, v in blk.items()}
        o = bd.bdgdn_denoise_step(dp, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale)
        if step in (0, w.steps - 1):
            ref = oracle.denoise(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], scale=scale)
            e = rel_err(o, ref)
            print(f"step {step}: denoise err={e:.3e}")
            assert e <= TOL[w.dtype]
    torch.cuda.synchronize()
    assert torch.equal(dp, before), "denoise steps changed the pool"
    blk = W.make_serve_block(w, w.steps)
    db = {k: v.cuda() for k, v in blk.items()}
    oc = bd.bdgdn_commit(dp, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale, want_o=True)
    torch.cuda.synchronize()
    rpool, ro = oracle.commit(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], scale=scale)
    eo, es = rel_err(oc, ro), rel_err(dp, rpool)
    print(f"commit err o={eo:.3e} state={es:.3e}")
    assert eo <= TOL[w.dtype] and es <= TOL[w.dtype]


@pytest.mark.parametrize("R,L,hqk,hv", [(3, 20, 1, 4), (2, 1, 2, 2), (1, 32, 1, 1), (5, 16, 2, 4)])
def test_streaming_kernels_ragged_blocks(R, L, hqk, hv):
    """The streaming denoise/commit kernels (bf16, d = 128) on blocks that pad to 16 or 32
    positions, grouped value heads up to 4 per q/k head, and two commits in a row (the
    second starting from the state the first wrote)."""
    d = 128
    pool = _realistic_pool(R, hv, d, seed=7 * R + L)
    b1 = _block(R, L, hqk, hv, d, "bf16", seed=100 + L)
    b2 = _block(R, L, hqk, hv, d, "bf16", seed=200 + L)
    scale = 1.0 / math.sqrt(d)
    dp = pool.cuda()
    d1 = {k: v.cuda() for k, v in b1.items()}
    d2 = {k: v.cuda() for k, v in b2.items()}
    o = bd.bdgdn_denoise_step(dp, d1["q"], d1["k"], d1["v"], d1["g"], d1["beta"], scale=scale)
    oc1 = bd.bdgdn_commit(dp, d1["q"], d1["k"], d1["v"], d1["g"], d1["beta"], scale=scale, want_o=True)
    oc2 = bd.bdgdn_commit(dp, d2["q"], d2["k"], d2["v"], d2["g"], d2["beta"], scale=scale, want_o=True)
    torch.cuda.synchronize()
    ref = oracle.denoise(pool, b1["q"], b1["k"], b1["v"], b1["g"], b1["beta"], scale=scale)
    p1, r1 = oracle.commit(pool, b1["q"], b1["k"], b1["v"], b1["g"], b1["beta"], scale=scale)
    p2, r2 = oracle.commit(p1, b2["q"], b2["k"], b2["v"], b2["g"], b2["beta"], scale=scale)
    errs = (rel_err(o, ref), rel_err(oc1, r1), rel_err(oc2, r2), rel_err(dp, p2))
    print("denoise, commit 1, commit 2, state:", ["%.3e" % e for e in errs])
    assert max(errs) <= TOL["bf16"]


def test_streaming_kernels_bf16_outputs():
    """bf16 outputs: the same arithmetic as the fp32-output kernels up to the final rounding,
    and within the tolerance plus the output's own rounding of the oracle."""
    R, L, h, d = 4, 32, 4, 128
    pool = _realistic_pool(R, h, d, seed=11)
    blk = _block(R, L, h, h, d, "bf16", seed=12)
    db = {k: v.cuda() for k, v in blk.items()}
    scale = 1.0 / math.sqrt(d)
    o32 = bd.bdgdn_denoise_step(pool.cuda(), db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale)
    o16 = bd.bdgdn_denoise_step(pool.cuda(), db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale,
                                out_dtype=torch.bfloat16)
    pa, pb = pool.cuda(), pool.cuda()
    c32 = bd.bdgdn_commit(pa, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale, want_o=True)
    c16 = bd.bdgdn_commit(pb, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale, want_o=True,
                          out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert o16.dtype == torch.bfloat16 and c16.dtype == torch.bfloat16
    assert torch.equal(o32.to(torch.bfloat16), o16) and torch.equal(c32.to(torch.bfloat16), c16)
    assert torch.equal(pa, pb)
    ref = oracle.denoise(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], scale=scale)
    rnd = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).double().numpy()
    budget = TOL["bf16"] + np.abs(rnd - ref).max() / np.sqrt((ref ** 2).mean())
    e = rel_err(o16, ref)
    print(f"bf16 denoise err {e:.3e} budget {budget:.3e}")
    assert e <= budget


@pytest.mark.parametrize("R,K,hqk,hv,dtype_out", [(3, 4, 1, 2, torch.float32), (2, 15, 2, 2, torch.float32),
                                                   (4, 31, 1, 1, torch.bfloat16), (2, 1, 1, 1, torch.float32)])
def test_verify_state_cache(R, K, hqk, hv, dtype_out):
    """The AR-Trust verify pass over [anchor, d_0 .. d_(K-1)] (L = K + 1 positions) keeps
    the states before the K draft positions; the accept step rewinds each request to its
    accepted offset (all offsets 0 .. K exercised), against the oracle."""
    d, L = 128, K + 1
    pool = _realistic_pool(R + 1, hv, d, seed=K + 31)
    slot = torch.tensor(list(range(R, 0, -1)), dtype=torch.int32)
    blk = _block(R, L, hqk, hv, d, "bf16", seed=K + 7)
    scale = 1.0 / math.sqrt(d)
    db = {k: v.cuda() for k, v in blk.items()}
    dp = pool.cuda()
    states, o = bd.bdgdn_commit_record(dp, db["q"], db["k"], db["v"], db["g"], db["beta"], n_record=K,
                                       scale=scale, slot=slot.cuda(), want_o=True, out_dtype=dtype_out)
    torch.cuda.synchronize()
    rpool, ro, rstates = oracle.commit_record(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                                              scale=scale, n_record=K, slot=slot.numpy())
    tol = TOL["bf16"]
    if dtype_out == torch.bfloat16:
        rnd = torch.from_numpy(ro.astype(np.float32)).to(torch.bfloat16).double().numpy()
        tol += np.abs(rnd - ro).max() / np.sqrt((ro ** 2).mean())
    es, eo, ep = rel_err(states, rstates), rel_err(o, ro), rel_err(dp[1:], rpool[1:])
    print(f"states err={es:.3e} o err={eo:.3e} pool err={ep:.3e}")
    assert es <= TOL["bf16"] and eo <= tol and ep <= TOL["bf16"]
    # the same pool as the plain commit pass, bit for bit
    dp2 = pool.cuda()
    bd.bdgdn_commit(dp2, db["q"], db["k"], db["v"], db["g"], db["beta"], scale=scale, slot=slot.cuda())
    torch.cuda.synchronize()
    assert torch.equal(dp2, dp)
    # accept: every offset 0 .. K once across the requests (cycled)
    accept = torch.tensor([(r * 7) % (K + 1) for r in range(R)], dtype=torch.int32)
    before = dp.clone()
    bd.bdgdn_accept_states(dp, states, accept.cuda(), block=L, slot=slot.cuda())
    torch.cuda.synchronize()
    want = oracle.accept_states(rpool, rstates, accept.numpy(), slot=slot.numpy())
    assert rel_err(dp[1:], want[1:]) <= TOL["bf16"]
    assert torch.equal(dp[0], before[0])
    for r in range(R):
        s = int(slot[r])
        if int(accept[r]) == K:
            assert torch.equal(dp[s], before[s])
        else:
            assert torch.equal(dp[s], states[r, int(accept[r])])
