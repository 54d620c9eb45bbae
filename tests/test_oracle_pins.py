"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check is a closed form, an
invariant stated by the paper, a special case that reduces to a textbook
formula, or a brute-force evaluation in a different formulation (the unrolled
product of transition matrices, in floating point and in exact rationals).

Paper references (FLARE, arXiv 2606.01774): eq. gdn-recurrence (Sec. 3.1), the
per-step expanded form eq. per-step-fwd, the two-stream schedule eq.
flare-gdn-schedule (Sec. 3.2), eq. noisy-block-fwd and the block-end readout,
the document-packing appendix, and the serving passes (Diffusion-Trust appendix).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _unit(rng, shape):
    x = rng.standard_normal(shape)
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _stream(rng, B, T, hqk, hv, dk, dv):
    return dict(
        q=_unit(rng, (B, T, hqk, dk)), k=_unit(rng, (B, T, hqk, dk)),
        v=rng.standard_normal((B, T, hv, dv)),
        g=-np.log1p(np.exp(rng.uniform(-6, -2, (B, T, hv)))),
        beta=1.0 / (1.0 + np.exp(-rng.uniform(-2, 2, (B, T, hv)))))


def _two(rng, B, T, hqk, hv, dk, dv):
    c = _stream(rng, B, T, hqk, hv, dk, dv)
    n = _stream(rng, B, T, hqk, hv, dk, dv)
    return c, n


def _run(c, n, L, scale=1.0, **kw):
    return oracle.fwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"],
                            n["q"], n["k"], n["v"], n["g"], n["beta"],
                            block=L, scale=scale, **kw)


# ---------------------------------------------------------------------------
# Brute force: the unrolled product of eq. gdn-recurrence,
#   S_t = (M_t ... M_1) S_0 + sum_i (M_t ... M_{i+1}) beta_i k_i v_i^T,
#   M_t = alpha_t (I - beta_t k_t k_t^T).
# ---------------------------------------------------------------------------
def _unrolled_states(k, v, alpha, beta, S0):
    T, dk = k.shape
    M = [alpha[t] * (np.eye(dk) - beta[t] * np.outer(k[t], k[t])) for t in range(T)]
    states = []
    for t in range(T):
        P = np.eye(dk)
        for j in range(t, -1, -1):
            P = P @ M[j]
        acc = P @ S0
        for i in range(t + 1):
            Q = np.eye(dk)
            for j in range(t, i, -1):
                Q = Q @ M[j]
            acc = acc + Q @ np.outer(beta[i] * k[i], v[i])
        states.append(acc)
    return states


def _brute_two_stream(c, n, L, scale, b, h, S0, hv_per_qk=1):
    """Brute-force clean and noisy outputs of sequence b, v-head h."""
    hq = h // hv_per_qk
    k, q, v = c["k"][b, :, hq], c["q"][b, :, hq], c["v"][b, :, h]
    al, be = np.exp(c["g"][b, :, h]), c["beta"][b, :, h]
    kn, qn, vn = n["k"][b, :, hq], n["q"][b, :, hq], n["v"][b, :, h]
    aln, ben = np.exp(n["g"][b, :, h]), n["beta"][b, :, h]
    T = k.shape[0]
    Sc = _unrolled_states(k, v, al, be, S0)
    o = np.stack([scale * Sc[t].T @ q[t] for t in range(T)])
    on = np.zeros_like(o)
    for p0 in range(0, T, L):
        p1 = min(p0 + L, T)
        seed = S0 if p0 == 0 else Sc[p0 - 1]
        Sn = _unrolled_states(kn[p0:p1], vn[p0:p1], aln[p0:p1], ben[p0:p1], seed)[-1]
        for l in range(p0, p1):
            on[l] = scale * Sn.T @ qn[l]
    return o, on, Sc[-1]


@pytest.mark.parametrize("L", [1, 2, 3, 4])
def test_pin_bruteforce_unrolled_product(L):
    rng = np.random.default_rng(100 + L)
    B, T, hqk, hv, dk, dv = 2, 7, 1, 2, 4, 3
    c, n = _two(rng, B, T, hqk, hv, dk, dv)
    h0 = rng.standard_normal((B, hv, dk, dv)) * 0.5
    o, on, ht = _run(c, n, L, scale=0.7, h0=h0)
    for b in range(B):
        for h in range(hv):
            bo, bon, bS = _brute_two_stream(c, n, L, 0.7, b, h, h0[b, h], hv_per_qk=hv // hqk)
            np.testing.assert_allclose(o[b, :, h], bo, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(on[b, :, h], bon, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ht[b, h], bS, rtol=1e-12, atol=1e-12)


def test_pin_exact_rational_unrolled_product():
    """Exact rational arithmetic (fractions) of the unrolled product; the oracle
    receives g = log(alpha) and must agree to fp64 rounding."""
    rng = np.random.default_rng(7)
    T, dk, dv, L = 6, 3, 2, 2
    fr = lambda x: Fraction(int(round(x * 16)), 16)
    k = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dk))]
    v = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dv))]
    q = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dk))]
    kn = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dk))]
    vn = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dv))]
    qn = [[fr(x) for x in row] for row in rng.uniform(-1, 1, (T, dk))]
    al = [Fraction(int(n), 16) for n in rng.integers(12, 16, T)]
    aln = [Fraction(int(n), 16) for n in rng.integers(12, 16, T)]
    be = [Fraction(int(n), 8) for n in rng.integers(1, 8, T)]
    ben = [Fraction(int(n), 8) for n in rng.integers(1, 8, T)]

    def step(S, kk, vv, a, b):
        # S = a (I - b k k^T) S + b k v^T, exactly
        kS = [sum(kk[i] * S[i][j] for i in range(dk)) for j in range(dv)]
        return [[a * (S[i][j] - b * kk[i] * kS[j]) + b * kk[i] * vv[j] for j in range(dv)]
                for i in range(dk)]

    def read(S, qq):
        return [sum(S[i][j] * qq[i] for i in range(dk)) for j in range(dv)]

    S = [[Fraction(0)] * dv for _ in range(dk)]
    o_ex, on_ex = [], [None] * T
    for p0 in range(0, T, L):
        Sn = [row[:] for row in S]
        for l in range(p0, p0 + L):
            Sn = step(Sn, kn[l], vn[l], aln[l], ben[l])
        for l in range(p0, p0 + L):
            on_ex[l] = read(Sn, qn[l])
        for t in range(p0, p0 + L):
            S = step(S, k[t], v[t], al[t], be[t])
            o_ex.append(read(S, q[t]))
    arr = lambda x: np.array([[float(e) for e in r] for r in x])[None, :, None, :]
    garr = lambda x: np.log(np.array([float(e) for e in x]))[None, :, None]
    barr = lambda x: np.array([float(e) for e in x])[None, :, None]
    c = dict(q=arr(q), k=arr(k), v=arr(v), g=garr(al), beta=barr(be))
    n = dict(q=arr(qn), k=arr(kn), v=arr(vn), g=garr(aln), beta=barr(ben))
    o, on, ht = _run(c, n, L)
    np.testing.assert_allclose(o[0, :, 0], np.array([[float(e) for e in r] for r in o_ex]),
                               rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(on[0, :, 0], np.array([[float(e) for e in r] for r in on_ex]),
                               rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(ht[0, 0], np.array([[float(e) for e in r] for r in S]),
                               rtol=1e-12, atol=1e-13)


def test_pin_exact_overwrite():
    """beta = 1 and ||k|| = 1 make the write an exact overwrite: S_t^T k_t = v_t.
    With q_t = k_t the clean readout is s v_t; with q~ = k~ the last position of
    each noisy block reads s v~ of that position (the block-end state holds it)."""
    rng = np.random.default_rng(1)
    B, T, dk, dv, L = 2, 12, 8, 5, 4
    c, n = _two(rng, B, T, 1, 1, dk, dv)
    for s in (c, n):
        s["q"] = s["k"].copy()
        s["beta"] = np.ones_like(s["beta"])
    h0 = rng.standard_normal((B, 1, dk, dv))
    o, on, _ = _run(c, n, L, scale=0.5, h0=h0)
    np.testing.assert_allclose(o, 0.5 * c["v"], atol=1e-13)
    np.testing.assert_allclose(on[:, L - 1::L], 0.5 * n["v"][:, L - 1::L], atol=1e-13)
    o1, on1, _ = _run(c, n, 1, scale=0.5, h0=h0)
    np.testing.assert_allclose(on1, 0.5 * n["v"], atol=1e-13)


def test_pin_frozen_state():
    """beta = 0 never writes: S_t = exp(sum g) h0, so o_t = s exp(G_t) h0^T q_t,
    and a noisy block read decays by the clean prefix and its own gates."""
    rng = np.random.default_rng(2)
    B, T, hqk, hv, dk, dv, L = 1, 10, 1, 2, 6, 4, 4
    c, n = _two(rng, B, T, hqk, hv, dk, dv)
    c["beta"][:] = 0.0
    n["beta"][:] = 0.0
    h0 = rng.standard_normal((B, hv, dk, dv))
    o, on, ht = _run(c, n, L, scale=0.3, h0=h0)
    for h in range(hv):
        G = np.cumsum(c["g"][0, :, h])
        for t in range(T):
            np.testing.assert_allclose(o[0, t, h], 0.3 * np.exp(G[t]) * h0[0, h].T @ c["q"][0, t, 0],
                                       rtol=1e-12, atol=1e-14)
        for p0 in range(0, T, L):
            p1 = min(p0 + L, T)
            dec = (G[p0 - 1] if p0 else 0.0) + n["g"][0, p0:p1, h].sum()
            for l in range(p0, p1):
                np.testing.assert_allclose(on[0, l, h], 0.3 * np.exp(dec) * h0[0, h].T @ n["q"][0, l, 0],
                                           rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(ht[0, h], np.exp(G[-1]) * h0[0, h], rtol=1e-12)
    # g = 0 as well: the state is exactly h0
    c["g"][:] = 0.0
    o, _, ht = _run(c, n, L, scale=1.0, h0=h0)
    np.testing.assert_array_equal(ht, h0)


def test_pin_orthonormal_keys_is_linear_attention():
    """With alpha = 1, h0 = 0 and mutually orthonormal keys across both streams the
    prediction error is u = v, so the GDR reduces to linear attention:
    o_t = s sum_{i<=t} beta_i (q_t.k_i) v_i, and a noisy block reads the clean
    prefix plus its own writes."""
    rng = np.random.default_rng(3)
    T, dk, dv, L = 6, 16, 5, 3
    Qm, _ = np.linalg.qr(rng.standard_normal((dk, dk)))
    c, n = _two(rng, 1, T, 1, 1, dk, dv)
    c["k"][0, :, 0] = Qm[:T]
    n["k"][0, :, 0] = Qm[T:2 * T]
    for s in (c, n):
        s["g"][:] = 0.0
    o, on, _ = _run(c, n, L, scale=0.9)
    q, k, v, be = c["q"][0, :, 0], c["k"][0, :, 0], c["v"][0, :, 0], c["beta"][0, :, 0]
    qn, kn, vn, ben = n["q"][0, :, 0], n["k"][0, :, 0], n["v"][0, :, 0], n["beta"][0, :, 0]
    for t in range(T):
        ref = sum(be[i] * (q[t] @ k[i]) * v[i] for i in range(t + 1))
        np.testing.assert_allclose(o[0, t, 0], 0.9 * ref, atol=1e-13)
    for p0 in range(0, T, L):
        for l in range(p0, p0 + L):
            ref = sum(be[i] * (qn[l] @ k[i]) * v[i] for i in range(p0))
            ref = ref + sum(ben[j] * (qn[l] @ kn[j]) * vn[j] for j in range(p0, p0 + L))
            np.testing.assert_allclose(on[0, l, 0], 0.9 * ref, atol=1e-13)


def test_pin_single_token_from_zero():
    rng = np.random.default_rng(4)
    c, n = _two(rng, 1, 1, 1, 1, 7, 3)
    o, on, ht = _run(c, n, 1, scale=0.25)
    q, k, v, be = c["q"][0, 0, 0], c["k"][0, 0, 0], c["v"][0, 0, 0], c["beta"][0, 0, 0]
    np.testing.assert_allclose(o[0, 0, 0], 0.25 * be * (q @ k) * v, rtol=1e-13)
    np.testing.assert_allclose(ht[0, 0], be * np.outer(k, v), rtol=1e-13)


def test_pin_block_one_reduces_to_causal_recurrence():
    """L = 1 and identical noisy/clean inputs: each noisy block is one causal step
    from the clean prefix, so the noisy output equals the clean output exactly."""
    rng = np.random.default_rng(5)
    c, _ = _two(rng, 2, 9, 1, 2, 5, 4)
    n = {key: val.copy() for key, val in c.items()}
    o, on, _ = _run(c, n, 1, scale=0.4)
    np.testing.assert_array_equal(on, o)


@pytest.mark.parametrize("L", [2, 3, 5])
def test_pin_identical_streams_read_block_end_clean_state(L):
    """Identical streams: the noisy block ending at p1 reads the clean state S_{p1},
    so each position reads s S_{p1}^T q_l and the last position equals o there."""
    rng = np.random.default_rng(6 + L)
    T = 11
    c, _ = _two(rng, 1, T, 1, 1, 4, 3)
    n = {key: val.copy() for key, val in c.items()}
    o, on, _ = _run(c, n, L)
    for p0 in range(0, T, L):
        p1 = min(p0 + L, T)
        np.testing.assert_array_equal(on[0, p1 - 1], o[0, p1 - 1])
        trunc = {key: val[:, :p1].copy() for key, val in c.items()}
        _, _, ht = _run(trunc, trunc, L)
        for l in range(p0, p1):
            np.testing.assert_allclose(on[0, l, 0], ht[0, 0].T @ c["q"][0, l, 0], rtol=1e-12,
                                       atol=1e-14)


def test_pin_block_independence_and_clean_isolation():
    """Perturbing the noisy inputs of one block changes only that block's noisy
    outputs; the clean outputs and final state are untouched (Sec. 3.2: all
    block-to-block flow passes through the clean stream)."""
    rng = np.random.default_rng(8)
    B, T, L = 1, 16, 4
    c, n = _two(rng, B, T, 1, 1, 6, 4)
    o, on, ht = _run(c, n, L)
    n2 = {key: val.copy() for key, val in n.items()}
    blk = slice(4, 8)
    for key in ("q", "k", "v"):
        n2[key][:, blk] += rng.standard_normal(n2[key][:, blk].shape)
    n2["g"][:, blk] *= 0.5
    n2["beta"][:, blk] *= 0.9
    o2, on2, ht2 = _run(c, n2, L)
    np.testing.assert_array_equal(o2, o)
    np.testing.assert_array_equal(ht2, ht)
    mask = np.zeros(T, bool)
    mask[blk] = True
    np.testing.assert_array_equal(on2[:, ~mask], on[:, ~mask])
    assert np.abs(on2[:, mask] - on[:, mask]).min() > 0


def test_pin_packed_equals_separate_documents():
    """Packing: each document behaves as an independent sequence whose clean and
    noisy states start from zero; the last document ends with a partial block."""
    rng = np.random.default_rng(9)
    L = 4
    lengths = [8, 12, 4, 7]
    Ttot = sum(lengths)
    c, n = _two(rng, 1, Ttot, 1, 2, 5, 3)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    o, on, ht = _run(c, n, L, scale=0.6, cu_seqlens=cu)
    assert ht.shape[0] == len(lengths)
    for d, (a, b) in enumerate(zip(cu[:-1], cu[1:])):
        cs = {key: val[:, a:b].copy() for key, val in c.items()}
        ns = {key: val[:, a:b].copy() for key, val in n.items()}
        od, ond, htd = _run(cs, ns, L, scale=0.6)
        np.testing.assert_array_equal(o[:, a:b], od)
        np.testing.assert_array_equal(on[:, a:b], ond)
        np.testing.assert_array_equal(ht[d], htd[0])


def test_pin_partial_tail_equals_identity_padding():
    """A partial last block behaves as if zero-padded with identity tokens
    (k = 0, g = 0, beta = 0), the reading of the packed-tail rule."""
    rng = np.random.default_rng(10)
    T, L = 10, 4
    c, n = _two(rng, 1, T, 1, 1, 5, 3)
    o, on, ht = _run(c, n, L)
    pad = 12 - T

    def padded(s):
        out = {}
        for key, val in s.items():
            z = np.zeros((1, pad) + val.shape[2:])
            out[key] = np.concatenate([val, z], axis=1)
        return out
    o2, on2, ht2 = _run(padded(c), padded(n), L)
    np.testing.assert_allclose(o2[:, :T], o, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(on2[:, :T], on, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(ht2, ht, rtol=1e-14, atol=1e-15)


def test_pin_grouped_value_heads_map_consecutively():
    """h_v = 2 h_qk: v-head h uses q/k head h // 2, i.e. the same result as
    repeating each q/k head twice."""
    rng = np.random.default_rng(11)
    c, n = _two(rng, 1, 8, 2, 4, 4, 3)
    o, on, ht = _run(c, n, 4)
    rep = lambda s: {**s, "q": np.repeat(s["q"], 2, axis=2), "k": np.repeat(s["k"], 2, axis=2)}
    o2, on2, ht2 = _run(rep(c), rep(n), 4)
    np.testing.assert_array_equal(o, o2)
    np.testing.assert_array_equal(on, on2)
    np.testing.assert_array_equal(ht, ht2)


# ----------------------------- serving passes -----------------------------
def _serve_block(rng, R, L, hqk, hv, dk, dv):
    s = _stream(rng, R, L, hqk, hv, dk, dv)
    return s["q"], s["k"], s["v"], s["g"], s["beta"]


def test_pin_denoise_is_noisy_block_of_training_schedule():
    """A denoise pass from a cached prefix state equals the training schedule's
    noisy output for the block that follows that prefix."""
    rng = np.random.default_rng(12)
    R, L, hv, dk, dv = 3, 4, 2, 5, 3
    pool = rng.standard_normal((R, hv, dk, dv))
    q, k, v, g, b = _serve_block(rng, R, L, 1, hv, dk, dv)
    pool0 = pool.copy()
    o = oracle.denoise(pool, q, k, v, g, b, scale=0.5)
    np.testing.assert_array_equal(pool, pool0)
    for r in range(R):
        # the same block as the first block of a training sequence seeded by h0
        n = dict(q=q[r:r + 1], k=k[r:r + 1], v=v[r:r + 1], g=g[r:r + 1], beta=b[r:r + 1])
        _, on, _ = _run(n, n, L, scale=0.5, h0=pool[r:r + 1])
        np.testing.assert_array_equal(o[r:r + 1], on)
        # and the brute-force block-end state
        for h in range(hv):
            Sn = _unrolled_states(k[r, :, 0], v[r, :, h], np.exp(g[r, :, h]), b[r, :, h], pool[r, h])[-1]
            np.testing.assert_allclose(o[r, :, h], 0.5 * (q[r, :, 0] @ Sn), rtol=1e-12, atol=1e-13)


def test_pin_commit_is_causal_pass_and_writes_state():
    rng = np.random.default_rng(13)
    R, L, hv, dk, dv = 2, 5, 2, 4, 4
    pool = rng.standard_normal((R + 1, hv, dk, dv))
    slot = np.array([2, 0], np.int32)
    q, k, v, g, b = _serve_block(rng, R, L, 1, hv, dk, dv)
    newpool, o = oracle.commit(pool, q, k, v, g, b, scale=0.8, slot=slot)
    np.testing.assert_array_equal(newpool[1], pool[1])        # untouched slot
    for r, s in enumerate(slot):
        for h in range(hv):
            st = _unrolled_states(k[r, :, 0], v[r, :, h], np.exp(g[r, :, h]), b[r, :, h], pool[s, h])
            np.testing.assert_allclose(newpool[s, h], st[-1], rtol=1e-12, atol=1e-13)
            for t in range(L):
                np.testing.assert_allclose(o[r, t, h], 0.8 * st[t].T @ q[r, t, 0], rtol=1e-12, atol=1e-13)


def test_pin_denoise_after_commit_equals_training_schedule():
    """denoise(commit(S, blk1), blk2) equals the training schedule's noisy output of
    blk2 for the clean sequence [blk1] seeded with S."""
    rng = np.random.default_rng(14)
    L, hv, dk, dv = 4, 1, 4, 3
    S = rng.standard_normal((1, hv, dk, dv))
    b1 = _serve_block(rng, 1, L, 1, hv, dk, dv)
    b2 = _serve_block(rng, 1, L, 1, hv, dk, dv)
    S1, _ = oracle.commit(S, *b1, scale=1.0)
    o2 = oracle.denoise(S1, *b2, scale=1.0)
    # the clean stream is [blk1, anything]; the noisy stream's second block is blk2
    junk = _serve_block(rng, 1, L, 1, hv, dk, dv)
    cat = lambda a, b, i: np.concatenate([a[i], b[i]], axis=1)
    keys = ("q", "k", "v", "g", "beta")
    c = {key: cat(b1, junk, i) for i, key in enumerate(keys)}
    n = {key: cat(junk, b2, i) for i, key in enumerate(keys)}
    _, on, _ = _run(c, n, L, scale=1.0, h0=S)
    np.testing.assert_array_equal(on[:, L:], o2)


# ------------------- AR-Trust verify-position states (cache-and-scatter) -------------------
def test_pin_commit_record_keeps_prefix_states():
    """The verify pass keeps, for the last n_record positions p of the block, the state
    before position p: the brute-force unrolled state after the first p tokens (the
    cached state itself for p = 0).  Its pool and outputs are those of the commit pass."""
    rng = np.random.default_rng(15)
    R, L, hv, dk, dv = 2, 5, 2, 4, 3
    pool = rng.standard_normal((R + 1, hv, dk, dv))
    slot = np.array([1, 2], np.int32)
    q, k, v, g, b = _serve_block(rng, R, L, 1, hv, dk, dv)
    for n_rec in (1, 3, L):
        newpool, o, states = oracle.commit_record(pool, q, k, v, g, b, scale=0.7, n_record=n_rec, slot=slot)
        cpool, co = oracle.commit(pool, q, k, v, g, b, scale=0.7, slot=slot)
        np.testing.assert_array_equal(newpool, cpool)
        np.testing.assert_array_equal(o, co)
        assert states.shape == (R, n_rec, hv, dk, dv)
        for r, s in enumerate(slot):
            for h in range(hv):
                st = _unrolled_states(k[r, :, 0], v[r, :, h], np.exp(g[r, :, h]), b[r, :, h], pool[s, h])
                for i in range(n_rec):
                    p = L - n_rec + i
                    want = pool[s, h] if p == 0 else st[p - 1]
                    np.testing.assert_allclose(states[r, i, h], want, rtol=1e-12, atol=1e-13)


def test_pin_accept_states_rewinds_to_accepted_offset():
    """After a verify pass over [anchor, d_0 .. d_(K-1)] (L = K + 1 positions, K recorded),
    accepting a drafts leaves the state after the anchor and a drafts: the commit pass over
    the first 1 + a tokens; accepting all K keeps the verify pass's final state."""
    rng = np.random.default_rng(16)
    R, K, hv, dk, dv = 4, 3, 2, 4, 4
    L = K + 1
    pool = rng.standard_normal((R, hv, dk, dv))
    q, k, v, g, b = _serve_block(rng, R, L, 1, hv, dk, dv)
    vpool, _, states = oracle.commit_record(pool, q, k, v, g, b, scale=1.0, n_record=K)
    accept = np.array([0, 1, K - 1, K], np.int32)
    out = oracle.accept_states(vpool, states, accept)
    for r in range(R):
        a = int(accept[r])
        blk = [x[r:r + 1, :1 + a] for x in (q, k, v, g, b)]
        want, _ = oracle.commit(pool[r:r + 1], *blk, scale=1.0)
        np.testing.assert_array_equal(out[r], want[0])
    with pytest.raises(RuntimeError):
        oracle.accept_states(vpool, states, np.array([0, 1, K + 1, 0], np.int32))


# ------------------------- two-stream 1D causal ShortConv -------------------------
def _silu(p):
    return p / (1.0 + np.exp(-p))


def _conv_inputs(rng, rows, D, W):
    x = rng.standard_normal((rows, D))
    xn = rng.standard_normal((rows, D))
    w = rng.standard_normal((D, W)) * 0.5
    b = rng.standard_normal(D) * 0.1
    return x, xn, w, b


@pytest.mark.parametrize("act", [0, 1])
def test_pin_shortconv_clean_is_causal_convolution(act):
    """The clean output is the standard causal depthwise convolution of each document
    (numpy's full convolution, first T terms), plus bias, through the activation."""
    rng = np.random.default_rng(40)
    cu = np.array([0, 7, 7, 19, 24], np.int32)   # an empty document
    x, xn, w, b = _conv_inputs(rng, 24, 3, 4)
    y, _ = oracle.shortconv_fwd(x, xn, w, b, block=3, act=act, cu_seqlens=cu)
    f = _silu if act else (lambda p: p)
    for d in range(len(cu) - 1):
        a, e = cu[d], cu[d + 1]
        if e == a:
            continue
        for c in range(3):
            ref = np.convolve(x[a:e, c], w[c])[: e - a] + b[c]
            np.testing.assert_allclose(y[a:e, c], f(ref), rtol=1e-13, atol=1e-14)


def test_pin_shortconv_noisy_block_rules():
    """Noisy outputs: one block covering the document is the convolution of the noisy
    stream alone; identical streams give the clean output for any block; blocks of one
    position read the noisy input at lag 0 and the clean inputs at every other lag."""
    rng = np.random.default_rng(41)
    rows, D, W = 11, 2, 4
    x, xn, w, b = _conv_inputs(rng, rows, D, W)
    _, yn = oracle.shortconv_fwd(x, xn, w, b, block=64, act=0)
    for c in range(D):
        np.testing.assert_allclose(yn[:, c], np.convolve(xn[:, c], w[c])[:rows] + b[c], rtol=1e-13, atol=1e-14)
    for L in (1, 2, 3, 5):
        y, yn = oracle.shortconv_fwd(x, x, w, b, block=L, act=1)
        np.testing.assert_array_equal(y, yn)
    _, yn = oracle.shortconv_fwd(x, xn, w, b, block=1, act=0)
    for t in range(rows):
        want = b + w[:, 0] * xn[t] + sum(w[:, i] * x[t - i] for i in range(1, W) if t - i >= 0)
        np.testing.assert_allclose(yn[t], want, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("act", [0, 1])
def test_pin_shortconv_backward_is_gradient(act):
    """The backward equals central finite differences of the (pinned) forward for a
    random linear functional of both outputs, with documents and several blocks."""
    rng = np.random.default_rng(42 + act)
    cu = np.array([0, 5, 12], np.int32)
    rows, D, W, L = 12, 2, 4, 3
    x, xn, w, b = _conv_inputs(rng, rows, D, W)
    gy, gyn = rng.standard_normal((rows, D)), rng.standard_normal((rows, D))
    loss = lambda x_, xn_, w_, b_: float(np.sum(gy * oracle.shortconv_fwd(x_, xn_, w_, b_, block=L, act=act,
                                                                           cu_seqlens=cu)[0])
                                         + np.sum(gyn * oracle.shortconv_fwd(x_, xn_, w_, b_, block=L, act=act,
                                                                              cu_seqlens=cu)[1]))
    dx, dxn, dw, db = oracle.shortconv_bwd(x, xn, w, b, gy, gyn, block=L, act=act, cu_seqlens=cu)
    h = 1e-6
    for name, arr, grad in (("x", x, dx), ("xn", xn, dxn), ("w", w, dw), ("b", b, db)):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args = {"x": x, "xn": xn, "w": w, "b": b}
            hi = {k: v.copy() for k, v in args.items()}
            lo = {k: v.copy() for k, v in args.items()}
            hi[name][idx] += h
            lo[name][idx] -= h
            fd[idx] = (loss(hi["x"], hi["xn"], hi["w"], hi["b"]) - loss(lo["x"], lo["xn"], lo["w"], lo["b"])) / (2 * h)
        np.testing.assert_allclose(grad, fd, rtol=1e-6, atol=1e-7, err_msg=name)


# ---------------------------------------------------------------------------
# Backward of the two-stream forward (appendix "Backward primitives"): the gradient is
# pinned to central finite differences of the forward oracle (itself pinned above), and
# to closed forms where the recurrence degenerates.
# ---------------------------------------------------------------------------
_BWD_KEYS = ("q", "k", "v", "g", "beta")


def _bwd_setup(rng, B, T, hqk, hv, d, L, lengths=None):
    c, n = _two(rng, B, T, hqk, hv, d, d)
    for s in (c, n):   # milder gates so that finite differences see every term
        s["g"] = -np.log1p(np.exp(rng.uniform(-3, 0, s["g"].shape)))
    nseq = B if lengths is None else len(lengths)
    h0 = 0.3 * rng.standard_normal((nseq, hv, d, d))
    do = rng.standard_normal((B, T, hv, d))
    don = rng.standard_normal((B, T, hv, d))
    dht = rng.standard_normal((nseq, hv, d, d))
    cu = None if lengths is None else np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    return c, n, h0, do, don, dht, cu


def _bwd_loss(c, n, L, scale, h0, do, don, dht, cu):
    o, on, ht = _run(c, n, L, scale, h0=h0, cu_seqlens=cu)
    return float((o * do).sum() + (on * don).sum() + (ht * dht).sum())


@pytest.mark.parametrize("B,T,hqk,hv,d,L,lengths", [
    (2, 11, 1, 2, 3, 4, None),        # grouped value heads, ragged tail block
    (1, 13, 2, 2, 3, 4, [8, 5]),      # two packed documents, a partial last block
    (1, 7, 1, 1, 4, 1, None),         # one-position blocks
])
def test_pin_bwd_matches_finite_differences(B, T, hqk, hv, d, L, lengths):
    rng = np.random.default_rng(40 + T + L)
    c, n, h0, do, don, dht, cu = _bwd_setup(rng, B, T, hqk, hv, d, L, lengths)
    scale = 0.7
    gr = oracle.bwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"], n["q"], n["k"], n["v"], n["g"], n["beta"],
                          do, don, block=L, scale=scale, h0=h0, dht=dht, cu_seqlens=cu)
    eps = 1e-6
    targets = [(c[k_], "d" + k_) for k_ in _BWD_KEYS] + [(n[k_], "d" + k_ + "n") for k_ in _BWD_KEYS]
    targets.append((h0, "dh0"))
    for arr, name in targets:
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + eps
            lp = _bwd_loss(c, n, L, scale, h0, do, don, dht, cu)
            arr[idx] = a0 - eps
            lm = _bwd_loss(c, n, L, scale, h0, do, don, dht, cu)
            arr[idx] = a0
            fd[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(gr[name], fd, rtol=1e-6, atol=1e-7, err_msg=name)


def test_pin_bwd_views_matches_finite_differences():
    """The complementary-view backward (several noisy views seeded from the same clean
    states) equals central finite differences of its loss  <do, o> + sum_i <do_i, o_i> +
    <dht, ht>, each view's readout o_i taken from the (pinned) two-stream forward with that
    view as the noisy stream; clean inputs, every view's inputs and h0 are perturbed."""
    rng = np.random.default_rng(77)
    B, T, hqk, hv, d, L, nv = 1, 9, 1, 2, 3, 4, 3
    c, _, h0, do, _, dht, cu = _bwd_setup(rng, B, T, hqk, hv, d, L)
    views = []
    for _ in range(nv):
        _, w, _, _, dw, _, _ = _bwd_setup(rng, B, T, hqk, hv, d, L)
        w["do"] = dw
        views.append(w)
    scale = 0.6

    def loss():
        tot = float((dht * _run(c, views[0], L, scale, h0=h0)[2]).sum())
        for i, w in enumerate(views):
            o, on, _ = _run(c, w, L, scale, h0=h0)
            tot += float((on * w["do"]).sum()) + (float((o * do).sum()) if i == 0 else 0.0)
        return tot

    clean, per_view = oracle.bwd_train_views(c["q"], c["k"], c["v"], c["g"], c["beta"], views, do, block=L,
                                             scale=scale, h0=h0, dht=dht)
    eps = 1e-6
    targets = [(c[k_], clean["d" + k_], "clean d" + k_) for k_ in _BWD_KEYS] + [(h0, clean["dh0"], "dh0")]
    for i, w in enumerate(views):
        targets += [(w[k_], per_view[i]["d" + k_], f"view {i} d{k_}") for k_ in _BWD_KEYS]
    for arr, grad, name in targets:
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a0 = arr[idx]
            arr[idx] = a0 + eps
            lp = loss()
            arr[idx] = a0 - eps
            lm = loss()
            arr[idx] = a0
            fd[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(grad, fd, rtol=1e-6, atol=1e-7, err_msg=name)


def test_pin_bwd_views_one_view_is_two_stream_backward():
    """With one view the complementary-view backward is the two-stream backward."""
    rng = np.random.default_rng(78)
    c, n, h0, do, don, dht, cu = _bwd_setup(rng, 1, 10, 1, 1, 3, 4, [6, 4])
    ref = oracle.bwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"], n["q"], n["k"], n["v"], n["g"], n["beta"],
                           do, don, block=4, scale=0.5, h0=h0, dht=dht, cu_seqlens=cu)
    clean, per_view = oracle.bwd_train_views(c["q"], c["k"], c["v"], c["g"], c["beta"], [dict(n, do=don)], do,
                                             block=4, scale=0.5, h0=h0, dht=dht, cu_seqlens=cu)
    for k_ in _BWD_KEYS:
        assert np.array_equal(clean["d" + k_], ref["d" + k_])
        assert np.array_equal(per_view[0]["d" + k_], ref["d" + k_ + "n"])
    assert np.array_equal(clean["dh0"], ref["dh0"])


def test_pin_bwd_frozen_state_closed_form():
    """beta = 0 in both streams: nothing is written, every state is the decayed h0, so
    o_t = s e^(G_t) h0^T q_t with G_t the cumulative clean log-gate, and a noisy position of
    block b reads s e^(G_(b-1) + G~_b) h0^T q~ (G~_b = the noisy block's total log-gate).
    Then dq_t = s e^(G_t) h0 do_t, dk = dv = 0, and dh0 is the sum of the outer products."""
    rng = np.random.default_rng(7)
    B, T, hqk, hv, d, L = 1, 10, 1, 1, 3, 4
    c, n, h0, do, don, dht, _ = _bwd_setup(rng, B, T, hqk, hv, d, L)
    c["beta"][:] = 0.0
    n["beta"][:] = 0.0
    s = 0.5
    gr = oracle.bwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"], n["q"], n["k"], n["v"], n["g"], n["beta"],
                          do, don, block=L, scale=s, h0=h0, dht=None)
    G = np.cumsum(c["g"][0, :, 0])
    H = h0[0, 0]
    dq = np.zeros((T, d))
    dqn = np.zeros((T, d))
    dh0 = np.zeros((d, d))
    for t in range(T):
        dq[t] = s * np.exp(G[t]) * H @ do[0, t, 0]
        dh0 += s * np.exp(G[t]) * np.outer(c["q"][0, t, 0], do[0, t, 0])
    for p0 in range(0, T, L):
        p1 = min(p0 + L, T)
        gseed = G[p0 - 1] if p0 > 0 else 0.0
        gend = gseed + n["g"][0, p0:p1, 0].sum()
        for l in range(p0, p1):
            dqn[l] = s * np.exp(gend) * H @ don[0, l, 0]
            dh0 += s * np.exp(gend) * np.outer(n["q"][0, l, 0], don[0, l, 0])
    np.testing.assert_allclose(gr["dq"][0, :, 0], dq, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gr["dqn"][0, :, 0], dqn, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gr["dh0"][0, 0], dh0, rtol=1e-12, atol=1e-14)
    for key in ("dk", "dv", "dkn", "dvn"):
        assert np.abs(gr[key]).max() == 0.0, key


def test_pin_bwd_packed_equals_separate_documents():
    """Packed documents back-propagate exactly as separate sequences (states and their
    gradients reset at every document start)."""
    rng = np.random.default_rng(11)
    L, d = 4, 3
    lengths = [8, 5]
    c, n, h0, do, don, dht, cu = _bwd_setup(rng, 1, 13, 1, 1, d, L, lengths)
    gp = oracle.bwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"], n["q"], n["k"], n["v"], n["g"], n["beta"],
                          do, don, block=L, scale=1.0, h0=h0, dht=dht, cu_seqlens=cu)
    for j, (a, e) in enumerate(zip(cu[:-1], cu[1:])):
        sl = lambda x: x[:, a:e]
        cs = {k_: sl(v_) for k_, v_ in c.items()}
        ns = {k_: sl(v_) for k_, v_ in n.items()}
        gs = oracle.bwd_train(cs["q"], cs["k"], cs["v"], cs["g"], cs["beta"], ns["q"], ns["k"], ns["v"], ns["g"],
                              ns["beta"], sl(do), sl(don), block=L, scale=1.0, h0=h0[j:j + 1], dht=dht[j:j + 1])
        for key in ("dq", "dk", "dv", "dg", "dbeta", "dqn", "dkn", "dvn", "dgn", "dbetan"):
            np.testing.assert_array_equal(gp[key][:, a:e], gs[key], err_msg=key)
        np.testing.assert_array_equal(gp["dh0"][j], gs["dh0"][0])


# ---------------------------------------------------------------------------
# Property tests on random tiny shapes: block sizes 1..4 and one larger than the
# sequence, ragged tails, grouped value heads, packed documents (empty ones
# included), with and without an initial state.
# ---------------------------------------------------------------------------
from hypothesis import HealthCheck, given, settings, strategies as st

_tiny = st.fixed_dictionaries(dict(
    seed=st.integers(0, 2**31 - 1),
    L=st.sampled_from([1, 2, 3, 4, 16]),
    hqk=st.sampled_from([1, 2]), ratio=st.sampled_from([1, 2]),
    dk=st.integers(1, 4), dv=st.integers(1, 4),
    lengths=st.one_of(st.none(), st.lists(st.integers(0, 9), min_size=1, max_size=3)),
    T=st.integers(1, 11), B=st.integers(1, 2),
    with_h0=st.booleans(), scale=st.floats(0.25, 1.5)))
_prop = settings(max_examples=80, deadline=None, derandomize=True,
                 suppress_health_check=[HealthCheck.too_slow])


def _tiny_case(p):
    rng = np.random.default_rng(p["seed"])
    hv = p["hqk"] * p["ratio"]
    if p["lengths"] is None:
        B, T, cu, nseq = p["B"], p["T"], None, p["B"]
    else:
        B, T = 1, max(1, sum(p["lengths"]))
        cu = np.concatenate([[0], np.cumsum(p["lengths"])]).astype(np.int32)
        nseq = len(p["lengths"])
    c, n = _two(rng, B, T, p["hqk"], hv, p["dk"], p["dv"])
    h0 = 0.5 * rng.standard_normal((nseq, hv, p["dk"], p["dv"])) if p["with_h0"] else None
    return rng, c, n, h0, cu, nseq, hv


@given(_tiny)
@_prop
def test_property_fwd_matches_unrolled_product(p):
    """Every document of every shape drawn equals the brute-force unrolled product of
    eq. gdn-recurrence, with the noisy blocks of eq. noisy-block-fwd aligned to the
    document's start; positions past the last document stay zero."""
    rng, c, n, h0, cu, nseq, hv = _tiny_case(p)
    L, s = p["L"], p["scale"]
    o, on, ht = _run(c, n, L, scale=s, h0=h0, cu_seqlens=cu)
    docs = [(b, 0, c["q"].shape[1]) for b in range(nseq)] if cu is None else \
        [(0, int(a), int(e)) for a, e in zip(cu[:-1], cu[1:])]
    for d, (b, a, e) in enumerate(docs):
        for h in range(hv):
            S0 = np.zeros((p["dk"], p["dv"])) if h0 is None else h0[d, h]
            if e == a:
                np.testing.assert_allclose(ht[d, h], S0, rtol=0, atol=0)
                continue
            cs = {key: val[b:b + 1, a:e] for key, val in c.items()}
            ns = {key: val[b:b + 1, a:e] for key, val in n.items()}
            bo, bon, bS = _brute_two_stream(cs, ns, L, s, 0, h, S0, hv_per_qk=p["ratio"])
            np.testing.assert_allclose(o[b, a:e, h], bo, rtol=1e-10, atol=1e-11)
            np.testing.assert_allclose(on[b, a:e, h], bon, rtol=1e-10, atol=1e-11)
            np.testing.assert_allclose(ht[d, h], bS, rtol=1e-10, atol=1e-11)
    if cu is not None and int(cu[-1]) < o.shape[1]:
        assert not o[:, int(cu[-1]):].any() and not on[:, int(cu[-1]):].any()


@given(_tiny)
@_prop
def test_property_bwd_euler_identities(p):
    """The loss <do,o> + <don,on> + <dht,ht> is homogeneous of degree one jointly in
    (v, v~, h0), since every state is linear in them, and jointly in (q, q~), which
    enter only the readouts; Euler's theorem then ties the gradients of each group to
    the forward values, with no finite differences."""
    rng, c, n, h0, cu, nseq, hv = _tiny_case(p)
    L, s = p["L"], p["scale"]
    if h0 is None:
        h0 = np.zeros((nseq, hv, p["dk"], p["dv"]))
    do = rng.standard_normal(c["v"].shape)
    don = rng.standard_normal(c["v"].shape)
    dht = rng.standard_normal(h0.shape)
    o, on, ht = _run(c, n, L, scale=s, h0=h0, cu_seqlens=cu)
    r = oracle.bwd_train(c["q"], c["k"], c["v"], c["g"], c["beta"],
                         n["q"], n["k"], n["v"], n["g"], n["beta"],
                         do, don, block=L, scale=s, h0=h0, dht=dht, cu_seqlens=cu)
    readout = float((o * do).sum() + (on * don).sum())
    loss = readout + float((ht * dht).sum())
    lin_v = float((r["dv"] * c["v"]).sum() + (r["dvn"] * n["v"]).sum() + (r["dh0"] * h0).sum())
    lin_q = float((r["dq"] * c["q"]).sum() + (r["dqn"] * n["q"]).sum())
    tol = 1e-9 * (1.0 + np.abs(o).sum() + np.abs(on).sum() + np.abs(ht).sum()) * 4
    assert abs(lin_v - loss) <= tol, (lin_v, loss)
    assert abs(lin_q - readout) <= tol, (lin_q, readout)
