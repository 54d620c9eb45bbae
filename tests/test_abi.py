"""CPU-side checks of the C ABI: the library loads and exports every function
declared in include/bdgdn.h, and host-side validation rejects bad arguments
before anything is launched (no GPU is touched: every call here fails
validation, which runs before any HIP call)."""
import ctypes
import os
import re

import pytest

import paper_2606_01774_amd as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bdgdn.h")
FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bdgdn_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = bd.load_library()
    declared = _declared_functions()
    assert set(declared) == set(bd.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_status_strings():
    assert bd.bdgdn_version() >= 1
    for st in (0, -1, -2, -3, -4, -5, -6):
        assert bd.bdgdn_status_string(st)
    assert bd.bdgdn_status_string(-99) == "unknown status"


def _desc(**kw):
    d = dict(batch=1, seqlen=64, num_seqs=0, h_qk=2, h_v=4, d_k=128, d_v=128, block=32,
             scale=0.1, dtype=bd.BDGDN_BF16, route=bd.BDGDN_ROUTE_FUSED, out_dtype=bd.BDGDN_F32)
    d.update(kw)
    return bd.FwdDesc(**d)


def _fwd(desc, cu_dev=None, cu_host=None, null_q=False):
    lib = bd.load_library()
    P = FAKE
    return lib.bdgdn_fwd_train(ctypes.byref(desc), None if null_q else P, P, P, P, P, P, P, P, P, P,
                               cu_dev, cu_host, None, P, P, None, None, 0, None)


@pytest.mark.parametrize("kw,status", [
    (dict(h_v=3), bd.BDGDN_ERR_INVALID_ARG),            # h_v % h_qk != 0
    (dict(batch=0), bd.BDGDN_ERR_INVALID_ARG),
    (dict(block=0), bd.BDGDN_ERR_INVALID_ARG),
    (dict(scale=float("nan")), bd.BDGDN_ERR_INVALID_ARG),
    (dict(d_k=96), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(d_v=256), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(block=65), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(dtype=7), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(dtype=bd.BDGDN_F32, block=64), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_BF16), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(out_dtype=5), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(route=9), bd.BDGDN_ERR_INVALID_ARG),
])
def test_fwd_rejects_bad_descriptors(kw, status):
    assert _fwd(_desc(**kw)) == status


def test_fwd_rejects_null_tensor():
    assert _fwd(_desc(), null_q=True) == bd.BDGDN_ERR_INVALID_ARG


def test_fwd_packing_checks():
    cu = (ctypes.c_int32 * 4)(0, 32, 96, 100)
    # misaligned document start (P: document starts must be block-aligned)
    bad = (ctypes.c_int32 * 4)(0, 32, 80, 100)
    d = _desc(seqlen=100, num_seqs=3)
    assert _fwd(d, FAKE, bad) == bd.BDGDN_ERR_UNALIGNED
    # only one of the two copies
    assert _fwd(d, FAKE, None) == bd.BDGDN_ERR_INVALID_ARG
    assert _fwd(d, None, cu) == bd.BDGDN_ERR_INVALID_ARG
    # packed needs batch == 1 and cu[N] == seqlen, non-decreasing offsets
    assert _fwd(_desc(seqlen=100, num_seqs=3, batch=2), FAKE, cu) == bd.BDGDN_ERR_INVALID_ARG
    assert _fwd(_desc(seqlen=128, num_seqs=3), FAKE, cu) == bd.BDGDN_ERR_INVALID_ARG
    dec = (ctypes.c_int32 * 4)(0, 64, 32, 100)
    assert _fwd(d, FAKE, dec) == bd.BDGDN_ERR_INVALID_ARG


def test_workspace_query():
    # RECORDS: one record per (block, v-head): 64 tokens / 32 = 2 blocks x 4 v-heads
    rec = _desc(route=bd.BDGDN_ROUTE_RECORDS)
    ws = bd.bdgdn_fwd_train_workspace(rec)
    assert ws > 0 and ws % (2 * 4) == 0 and (ws // 8) % 256 == 0
    # FUSED runs as one kernel without a workspace for bf16 inputs with blocks up to 32,
    # and with even blocks of 34 .. 64 (two half-block sub-blocks) ...
    assert bd.bdgdn_fwd_train_workspace(_desc()) == 0
    assert bd.bdgdn_fwd_train_workspace(_desc(block=16, d_k=64, d_v=64)) == 0
    assert bd.bdgdn_fwd_train_workspace(_desc(block=64)) == 0
    assert bd.bdgdn_fwd_train_workspace(_desc(block=40)) == 0
    # ... and through the records otherwise (odd blocks above 32, fp32 inputs)
    assert bd.bdgdn_fwd_train_workspace(_desc(block=63)) > 0
    assert bd.bdgdn_fwd_train_workspace(_desc(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32)) > 0
    assert bd.bdgdn_fwd_train_workspace(_desc(route=bd.BDGDN_ROUTE_ONEPASS)) == 0
    assert bd.bdgdn_fwd_train_workspace(_desc(h_v=3)) == 0
    # too small a workspace is refused before any launch
    assert _fwd(rec) == bd.BDGDN_ERR_WORKSPACE
    assert _fwd(_desc(block=63)) == bd.BDGDN_ERR_WORKSPACE


def test_chunked_route_limits_and_workspace():
    """The chunk-parallel schedule: bf16 inputs, d_k = d_v, blocks of at most 32; its
    workspace holds a clean UT record per (block, v-head) and a state per later segment
    start (segments of at least 16 blocks)."""
    ch = dict(route=bd.BDGDN_ROUTE_CHUNKED)
    for kw in (dict(d_k=64, d_v=128), dict(block=64), dict(block=33),
               dict(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32)):
        assert _fwd(_desc(**ch, **kw)) == bd.BDGDN_ERR_UNSUPPORTED, kw
        assert bd.bdgdn_fwd_train_workspace(_desc(**ch, **kw)) == 0
    # every chain one segment (no state pass): no workspace
    assert bd.bdgdn_fwd_train_workspace(_desc(**ch)) == 0
    # 4 x 4096 tokens, 16 heads: 64 chains x 4 tiles, 128 blocks each -> segments of 64 (two
    # workgroups per compute unit)
    big = _desc(**ch, batch=4, seqlen=4096, h_qk=16, h_v=16)
    assert bd.bdgdn_fwd_train_workspace(big) == 512 * 16 * 4352 + (512 // 64) * 16 * 128 * 128 * 4
    # 2 x 1100 tokens, 2 heads, blocks of 32: 70 blocks in 32-column tiles -> segments of 16;
    # records of 4352 bytes per (block, head), a state per (later segment start, head)
    mid = _desc(**ch, batch=2, seqlen=1100, h_qk=2, h_v=2)
    assert bd.bdgdn_fwd_train_workspace(mid) == 70 * 2 * 4352 + (70 // 16) * 2 * 128 * 128 * 4
    assert _fwd(mid) == bd.BDGDN_ERR_WORKSPACE
    # more packed documents than the schedule orders
    cu = (ctypes.c_int32 * 514)(*[32 * i for i in range(514)])
    assert _fwd(_desc(**ch, seqlen=32 * 513, num_seqs=513), cu, cu) == bd.BDGDN_ERR_UNSUPPORTED


def test_split_route_limits_and_workspace():
    """The split schedule runs bf16 inputs with d_k = d_v = 128 and blocks up to 32; its
    workspace holds one fp32 seed state per (block, v-head)."""
    split = dict(route=bd.BDGDN_ROUTE_SPLIT)
    for kw in (dict(d_k=64, d_v=64), dict(d_v=64), dict(block=64),
               dict(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32)):
        assert _fwd(_desc(**split, **kw)) == bd.BDGDN_ERR_UNSUPPORTED, kw
        assert bd.bdgdn_fwd_train_workspace(_desc(**split, **kw)) == 0
    # 64 tokens in blocks of 32 -> 2 blocks; 100 tokens in blocks of 16 -> 7 blocks
    assert bd.bdgdn_fwd_train_workspace(_desc(**split)) == 2 * 4 * 128 * 128 * 4
    assert bd.bdgdn_fwd_train_workspace(_desc(**split, seqlen=100, block=16, batch=3)) == 3 * 7 * 4 * 128 * 128 * 4
    assert _fwd(_desc(**split)) == bd.BDGDN_ERR_WORKSPACE


def _serve(fn, **kw):
    d = dict(num_req=4, h_qk=2, h_v=4, d_k=128, d_v=128, block=32, scale=0.1, dtype=bd.BDGDN_BF16,
             out_dtype=bd.BDGDN_F32)
    d.update(kw)
    desc = bd.ServeDesc(**d)
    lib = bd.load_library()
    P = FAKE
    return getattr(lib, fn)(ctypes.byref(desc), P, None, P, P, P, P, P, P, None)


@pytest.mark.parametrize("fn", ["bdgdn_denoise_step", "bdgdn_commit"])
@pytest.mark.parametrize("kw,status", [
    (dict(h_v=5), bd.BDGDN_ERR_INVALID_ARG),
    (dict(num_req=-1), bd.BDGDN_ERR_INVALID_ARG),
    (dict(d_k=32), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(block=100), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(scale=float("inf")), bd.BDGDN_ERR_INVALID_ARG),
])
def test_serve_rejects_bad_descriptors(fn, kw, status):
    assert _serve(fn, **kw) == status


def test_serve_empty_batch_is_a_no_op():
    assert _serve("bdgdn_denoise_step", num_req=0) == 0
    assert _serve("bdgdn_commit", num_req=0) == 0


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(1, 32, 1, 64, dtype=torch.bfloat16)
    g = torch.zeros(1, 32, 1)
    with pytest.raises(ValueError):
        bd.bdgdn_fwd_train(x, x, x, g, g, x, x, x, g, g, block=32)


def _record(**kw):
    n_record = kw.pop("n_record", 4)
    states = kw.pop("states", FAKE)
    d = dict(num_req=4, h_qk=2, h_v=4, d_k=128, d_v=128, block=8, scale=0.1, dtype=bd.BDGDN_BF16,
             out_dtype=bd.BDGDN_F32)
    d.update(kw)
    P = FAKE
    return bd.load_library().bdgdn_commit_record(ctypes.byref(bd.ServeDesc(**d)), P, None, P, P, P, P, P, None,
                                                 n_record, states, None)


def _accept(**kw):
    n_record = kw.pop("n_record", 4)
    accept = kw.pop("accept", FAKE)
    d = dict(num_req=4, h_qk=2, h_v=4, d_k=128, d_v=128, block=8, scale=0.1, dtype=bd.BDGDN_BF16,
             out_dtype=bd.BDGDN_F32)
    d.update(kw)
    P = FAKE
    return bd.load_library().bdgdn_accept_states(ctypes.byref(bd.ServeDesc(**d)), P, None, P, n_record, accept,
                                                 None)


def test_verify_state_cache_validation():
    assert _record(n_record=0) == bd.BDGDN_ERR_INVALID_ARG
    assert _record(n_record=9) == bd.BDGDN_ERR_INVALID_ARG            # more than the block
    assert _record(states=None) == bd.BDGDN_ERR_INVALID_ARG
    assert _record(d_k=64, d_v=64) == bd.BDGDN_ERR_UNSUPPORTED
    assert _record(block=48, n_record=4) == bd.BDGDN_ERR_UNSUPPORTED  # blocks of up to 32 only
    assert _record(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32) == bd.BDGDN_ERR_UNSUPPORTED
    assert _record(num_req=0) == bd.BDGDN_OK
    assert _accept(n_record=0) == bd.BDGDN_ERR_INVALID_ARG
    assert _accept(accept=None) == bd.BDGDN_ERR_INVALID_ARG
    assert _accept(h_v=5) == bd.BDGDN_ERR_INVALID_ARG
    assert _accept(num_req=0) == bd.BDGDN_OK


def _conv(fn="fwd", cu_dev=None, cu_host=None, null_x=False, ws=None, ws_bytes=0, **kw):
    d = dict(batch=2, seqlen=64, num_seqs=0, channels=256, width=4, block=8, activation=bd.BDGDN_ACT_SILU,
             dtype=bd.BDGDN_BF16)
    d.update(kw)
    desc = bd.ConvDesc(**d)
    lib = bd.load_library()
    P = FAKE
    x = None if null_x else P
    if fn == "fwd":
        return lib.bdgdn_shortconv_fwd(ctypes.byref(desc), x, P, P, None, cu_dev, cu_host, P, P, None)
    return lib.bdgdn_shortconv_bwd(ctypes.byref(desc), x, P, P, None, P, P, cu_dev, cu_host, P, P, P, None,
                                   ws, ws_bytes, None)


@pytest.mark.parametrize("fn", ["fwd", "bwd"])
@pytest.mark.parametrize("kw,status", [
    (dict(width=0), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(width=5), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(channels=258), bd.BDGDN_ERR_UNSUPPORTED),          # bf16 needs multiples of 4
    (dict(channels=0), bd.BDGDN_ERR_INVALID_ARG),
    (dict(block=0), bd.BDGDN_ERR_INVALID_ARG),
    (dict(batch=0), bd.BDGDN_ERR_INVALID_ARG),
    (dict(activation=2), bd.BDGDN_ERR_INVALID_ARG),
    (dict(dtype=7), bd.BDGDN_ERR_UNSUPPORTED),
    (dict(null_x=True), bd.BDGDN_ERR_INVALID_ARG),
])
def test_shortconv_rejects_bad_descriptors(fn, kw, status):
    assert _conv(fn, **kw) == status


def test_shortconv_fp32_channel_rule_and_packing():
    assert _conv(dtype=bd.BDGDN_F32, channels=258, null_x=True) == bd.BDGDN_ERR_INVALID_ARG  # 258 is fine
    cu = (ctypes.c_int32 * 4)(0, 10, 10, 64)
    assert _conv(batch=1, num_seqs=3, cu_dev=FAKE, cu_host=None) == bd.BDGDN_ERR_INVALID_ARG
    assert _conv(batch=2, num_seqs=3, cu_dev=FAKE, cu_host=cu) == bd.BDGDN_ERR_INVALID_ARG
    bad = (ctypes.c_int32 * 4)(0, 20, 10, 64)                     # decreasing
    assert _conv(batch=1, num_seqs=3, cu_dev=FAKE, cu_host=bad, null_x=True) == bd.BDGDN_ERR_INVALID_ARG
    short = (ctypes.c_int32 * 4)(0, 10, 20, 60)                   # does not end at seqlen
    assert _conv(batch=1, num_seqs=3, cu_dev=FAKE, cu_host=short) == bd.BDGDN_ERR_INVALID_ARG


def test_shortconv_workspace():
    lib = bd.load_library()

    def ws(**kw):
        d = dict(batch=2, seqlen=64, num_seqs=0, channels=256, width=4, block=8, activation=1, dtype=0)
        d.update(kw)
        return lib.bdgdn_shortconv_bwd_workspace(ctypes.byref(bd.ConvDesc(**d)))

    # whole (width + 1) x channels fp32 partials, one per group of rows, growing with the rows
    unit = 5 * 256 * 4
    assert ws() > 0 and ws() % unit == 0
    assert ws(seqlen=4096) % unit == 0 and ws(seqlen=4096) > ws()
    assert ws(width=2) % (3 * 256 * 4) == 0
    assert ws(seqlen=0) == 0
    assert ws(width=9) == 0
    assert _conv("bwd", ws=None, ws_bytes=0) == bd.BDGDN_ERR_WORKSPACE
    assert _conv("bwd", ws=FAKE, ws_bytes=ws() - 4) == bd.BDGDN_ERR_WORKSPACE
    assert _conv("bwd", ws=ctypes.c_void_p(0x1004), ws_bytes=ws()) == bd.BDGDN_ERR_WORKSPACE   # misaligned


def test_shortconv_noalloc_validation_and_limit():
    """The no-allocation backward validates like bdgdn_shortconv_bwd and rejects, before any
    HIP call, inputs whose partials exceed the fixed scratch."""
    lib = bd.load_library()
    P = FAKE

    def call(null_x=False, **kw):
        d = dict(batch=2, seqlen=64, num_seqs=0, channels=256, width=4, block=8, activation=bd.BDGDN_ACT_SILU,
                 dtype=bd.BDGDN_BF16)
        d.update(kw)
        desc = bd.ConvDesc(**d)
        return lib.bdgdn_shortconv_bwd_noalloc(ctypes.byref(desc), None if null_x else P, P, P, None, P, P,
                                               None, None, P, P, P, None, None)

    assert call(width=5) == bd.BDGDN_ERR_UNSUPPORTED
    assert call(channels=0) == bd.BDGDN_ERR_INVALID_ARG
    assert call(null_x=True) == bd.BDGDN_ERR_INVALID_ARG
    assert call(activation=3) == bd.BDGDN_ERR_INVALID_ARG
    # partials: (width + 1) x channels fp32 per started group of 1024 rows
    per_group = 5 * 6144 * 4
    groups = bd.BDGDN_NOALLOC_SCRATCH_BYTES // per_group
    fits = dict(batch=1, seqlen=1024 * groups, channels=6144)
    over = dict(batch=1, seqlen=1024 * groups + 1, channels=6144)
    ws = lambda kw: lib.bdgdn_shortconv_bwd_workspace(ctypes.byref(bd.ConvDesc(
        **dict(dict(batch=2, seqlen=64, num_seqs=0, channels=256, width=4, block=8, activation=1, dtype=0), **kw))))
    assert ws(fits) <= bd.BDGDN_NOALLOC_SCRATCH_BYTES < ws(over)
    assert call(**over) == bd.BDGDN_ERR_SCRATCH
    assert call(batch=8, seqlen=1 << 20, channels=512, width=2) == bd.BDGDN_ERR_SCRATCH
    assert "scratch" in bd.bdgdn_status_string(bd.BDGDN_ERR_SCRATCH)


def _bwd(desc, ws=None, ws_bytes=0, null_grad=False, **_):
    lib = bd.load_library()
    P = FAKE
    grads = [P] * 10
    if null_grad:
        grads[3] = None
    return lib.bdgdn_bwd_train(ctypes.byref(desc), P, P, P, P, P, P, P, P, P, P, None, None, None, P, P, None,
                               *grads, None, ws, ws_bytes, None)


def test_bwd_train_validation_and_workspace():
    lib = bd.load_library()
    ok = _desc()
    need = lib.bdgdn_bwd_train_workspace(ctypes.byref(ok))
    # per (block, v-head): an fp16 seed, one fp16 state-gradient term (the scan writes dh
    # over it), U K (32 x 128 fp16), gamma_n; then the range pass
    units = 2 * 4
    body = units * 128 * 128 * (2 + 2) + units * 32 * 128 * 2
    assert body <= need < body + 8 * 1024
    # even blocks of 34 .. 64 positions: noisy blocks of two sub-blocks, the clean stream and
    # the workspace in sub-blocks of half the block (here the same units as blocks of 32)
    assert lib.bdgdn_bwd_train_workspace(ctypes.byref(_desc(block=64))) == need
    need48 = lib.bdgdn_bwd_train_workspace(ctypes.byref(_desc(block=48)))   # 3 sub-blocks of 24
    body48 = 3 * 4 * (128 * 128 * (2 + 2) + 32 * 128 * 2)
    assert body48 <= need48 < body48 + 8 * 1024
    # the other shapes run the per-step backward: a clean state per eighth block start and
    # per chain (sequence, v-head), and per (chain, 16-column tile) eight block-start states
    f32 = _desc(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32)
    groups = 2 // 8 + 1
    gen_need = groups * 4 * 128 * 128 * 4 + 4 * 8 * 8 * 128 * 16 * 4
    assert lib.bdgdn_bwd_train_workspace(ctypes.byref(f32)) == gen_need
    for kw in (dict(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32), dict(d_k=64, d_v=64), dict(block=64),
               dict(d_k=64), dict(block=48, out_dtype=bd.BDGDN_BF16), dict(block=63)):
        d = _desc(**kw)
        assert lib.bdgdn_bwd_train_workspace(ctypes.byref(d)) > 0, kw
        assert _bwd(d) == bd.BDGDN_ERR_WORKSPACE, kw   # every check passes but the workspace
    assert _bwd(_desc(h_v=3)) == bd.BDGDN_ERR_INVALID_ARG
    assert _bwd(ok, null_grad=True) == bd.BDGDN_ERR_INVALID_ARG
    assert _bwd(ok, ws=None, ws_bytes=0) == bd.BDGDN_ERR_WORKSPACE
    assert _bwd(ok, ws=FAKE, ws_bytes=need - 1) == bd.BDGDN_ERR_WORKSPACE


def _seg(desc, cu, k):
    lib = bd.load_library()
    cu_h = None if cu is None else (ctypes.c_int32 * len(cu))(*cu)
    return lib.bdgdn_bwd_train_workspace_segmented(ctypes.byref(desc), cu_h, k)


def test_bwd_segmented_workspace():
    """The time-segmented backward's workspace: checkpoints at the segment starts after the
    first and the state-gradient carry (one fp32 state per (sequence, v-head) each), two
    segment tables, then the per-block layout for the first segment's blocks."""
    lib = bd.load_library()
    state = 128 * 128 * 4
    unit = 128 * 128 * (2 + 2) + 32 * 128 * 2 + 4   # per (block, v-head), as in one pass
    d = _desc(batch=2, seqlen=4096)                    # 128 blocks per sequence, 4 v-heads
    full = lib.bdgdn_bwd_train_workspace(ctypes.byref(d))
    assert _seg(d, None, 1) == full
    for k in (2, 3, 4, 8, 100, 128, 1000):
        S = -(-128 // k)
        n_seg = -(-128 // S)
        body = (n_seg - 1) * 2 * 4 * state + 2 * 4 * state + 2 * n_seg * 3 * 4 + 2 * min(128, S) * 4 * unit
        got = _seg(d, None, k)
        assert body <= got < body + 8 * 1024, k
    assert _seg(d, None, 4) < full // 3     # 32 of 128 blocks per sequence
    assert _seg(d, None, 0) == 0
    # packed: segments of ceil(the longest document's blocks / k); a document contributes
    # min(its blocks, the segment) to the first segment
    cu = [0, 64, 64, 64 + 4096, 64 + 4096 + 1000]      # blocks 2, 0, 128, 32
    p = _desc(seqlen=cu[-1], num_seqs=4)
    S = 32
    body = 3 * 4 * 4 * state + 4 * 4 * state + 2 * 4 * 5 * 4 + (2 + 0 + 32 + 32) * 4 * unit
    assert body <= _seg(p, cu, 4) < body + 8 * 1024
    assert _seg(p, None, 4) == 0                       # packing needed
    assert _seg(p, [0, 64, 64, 4160, 5000], 4) == 0    # offsets must end at seqlen
    # blocks of 64: sub-blocks of 32, segments of an even number of them
    d64 = _desc(seqlen=4096, block=64)                 # 128 sub-blocks
    S = 44                                             # ceil(128 / 3) = 43, made even
    body = 2 * 4 * state + 4 * state + 2 * 3 * 2 * 4 + S * 4 * unit
    assert body <= _seg(d64, None, 3) < body + 8 * 1024
    # the per-step shapes are never segmented
    f32 = _desc(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32, seqlen=4096)
    assert _seg(f32, None, 4) == lib.bdgdn_bwd_train_workspace(ctypes.byref(f32))
    # below every segmented size (and the full one) the call is refused before any launch
    smallest = min(_seg(d, None, k) for k in range(2, 129))
    assert smallest < full
    assert _bwd(d, ws=FAKE, ws_bytes=smallest - 1) == bd.BDGDN_ERR_WORKSPACE


def test_views_validation():
    lib = bd.load_library()
    ok = _desc()
    split = _desc(route=bd.BDGDN_ROUTE_SPLIT)
    assert lib.bdgdn_fwd_train_views_workspace(ctypes.byref(split)) == 2 * 4 * 128 * 128 * 4   # a seed per (block, head)
    assert lib.bdgdn_fwd_train_views_workspace(ctypes.byref(ok)) == 0                          # fused: none
    assert lib.bdgdn_fwd_train_views_workspace(ctypes.byref(_desc(d_k=64, d_v=64))) == 0
    P = FAKE
    views = (bd.NoisyView * 2)(bd.NoisyView(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000),
                               bd.NoisyView(0x1000, 0x1000, 0x1000, 0x1000, None, 0x1000))

    def call(desc, n, ws=None, ws_bytes=0):
        return lib.bdgdn_fwd_train_views(ctypes.byref(desc), P, P, P, P, P, views, n, None, None, None, P, None,
                                         ws, ws_bytes, None)
    assert call(ok, 0) == bd.BDGDN_ERR_INVALID_ARG
    assert call(ok, 17) == bd.BDGDN_ERR_INVALID_ARG
    assert call(ok, 2) == bd.BDGDN_ERR_INVALID_ARG          # view 1 has no beta
    views[1] = bd.NoisyView(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000)
    assert call(split, 2) == bd.BDGDN_ERR_WORKSPACE
    assert call(_desc(route=bd.BDGDN_ROUTE_RECORDS), 2) == bd.BDGDN_ERR_UNSUPPORTED
    assert call(_desc(block=63), 1) == bd.BDGDN_ERR_UNSUPPORTED   # odd blocks above 32: records only


def test_bwd_views_validation():
    lib = bd.load_library()
    ok = _desc()
    need = lib.bdgdn_bwd_train_workspace(ctypes.byref(ok))
    assert lib.bdgdn_bwd_train_views_workspace(ctypes.byref(ok)) == need
    P = FAKE
    full = [0x1000] * 11
    views = (bd.NoisyViewGrad * 2)(bd.NoisyViewGrad(*full), bd.NoisyViewGrad(*full))

    def call(desc, n, ws=None, ws_bytes=0):
        return lib.bdgdn_bwd_train_views(ctypes.byref(desc), P, P, P, P, P, views, n, None, None, None, P, None,
                                         P, P, P, P, P, None, ws, ws_bytes, None)
    assert call(ok, 0) == bd.BDGDN_ERR_INVALID_ARG
    assert call(ok, 17) == bd.BDGDN_ERR_INVALID_ARG
    assert call(ok, 2) == bd.BDGDN_ERR_WORKSPACE             # every pointer given: only the workspace lacks
    assert call(ok, 2, ws=FAKE, ws_bytes=need - 1) == bd.BDGDN_ERR_WORKSPACE
    views[1] = bd.NoisyViewGrad(*(full[:8] + [None] + full[9:]))   # view 1 without dg
    assert call(ok, 2) == bd.BDGDN_ERR_INVALID_ARG
    views[1] = bd.NoisyViewGrad(*(full[:5] + [0x1008] + full[6:]))  # view 1's do not 16-byte aligned
    assert call(ok, 2) == bd.BDGDN_ERR_INVALID_ARG
    views[1] = bd.NoisyViewGrad(*full)
    # the per-step backward takes up to four views
    assert call(_desc(dtype=bd.BDGDN_F32, out_dtype=bd.BDGDN_F32), 2) == bd.BDGDN_ERR_WORKSPACE
    many = (bd.NoisyViewGrad * 5)(*[bd.NoisyViewGrad(*full) for _ in range(5)])

    def call_many(desc, n):
        return lib.bdgdn_bwd_train_views(ctypes.byref(desc), P, P, P, P, P, many, n, None, None, None, P, None,
                                         P, P, P, P, P, None, None, 0, None)
    assert call_many(_desc(block=63), 4) == bd.BDGDN_ERR_WORKSPACE
    assert call_many(_desc(block=63), 5) == bd.BDGDN_ERR_UNSUPPORTED
    assert call_many(_desc(block=64), 5) == bd.BDGDN_ERR_WORKSPACE   # block form: up to 16 views
