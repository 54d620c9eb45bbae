"""Benchmark of the block-diffusion Gated DeltaNet hot path on one MI355X.

A step is one two-stream training forward (bdgdn_fwd_train, clean + noisy streams)
over the 4 x 4096-token, 16-head, d=128, L=32 workload with bf16 inputs, fp32
state and fp32 outputs, inputs resident in HBM.  `value` is tokens/s (clean +
noisy tokens).  The line also carries the roofline of the fused kernel (HBM
bytes the algorithm must move per launch over its measured duration), the
model-FLOP rate against the bf16/fp16 MFMA peak, the denoise_step and commit
bandwidths of the 64-request serving workload, the training backward's time, the
two-stream ShortConv forward and backward bandwidths at the training token shape, and
the fp64 CPU oracle timed on the same workload.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

ROUTES = {"fused": "fused (one kernel: per-block UT transform inside the state scan)",
          "split": "split (clean scan writing fp32 seed states, then the noisy-block kernel)",
          "records": "records (UT-transform kernel, then the scan)"}
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16/bf16 MFMA, TFLOP/s


def algorithmic_bytes_train(w, out_bytes):
    """Bytes the two-stream forward must move once: q, k per q/k head, v and o per
    v head, g and beta per v head, for both streams."""
    in_b = 2 if w.dtype == "bf16" else 4
    per_row = (2 * w.h_qk * w.d_k * in_b + w.h_v * w.d_v * (in_b + out_bytes) + 2 * w.h_v * 4)
    return 2 * w.tokens * per_row


def model_flops_train(w, chunk=64):
    """Work model: clean 6d^2 + 10Cd per (token, v-head) with C = 64, noisy
    2d^2 + 12Ld; the Gram terms (4Cd + 4Ld) once per q/k head."""
    d = w.d_k
    per_v = 6 * d * d + 6 * chunk * d + 2 * d * d + 8 * w.block * d
    per_qk = 4 * chunk * d + 4 * w.block * d
    return w.tokens * (w.h_v * per_v + w.h_qk * per_qk)


def algorithmic_bytes_denoise(w, out_bytes):
    in_b = 2 if w.dtype == "bf16" else 4
    rows = w.requests * w.block
    state = w.requests * w.h_v * w.d_k * w.d_v * 4
    return state + rows * (2 * w.h_qk * w.d_k * in_b + w.h_v * w.d_v * (in_b + out_bytes)
                           + 2 * w.h_v * 4)


def algorithmic_bytes_commit(w):
    """The state pass without outputs: the fp32 state read and written back, and the
    block's k, v, g, beta read once (q is not needed without outputs)."""
    in_b = 2 if w.dtype == "bf16" else 4
    rows = w.requests * w.block
    state = w.requests * w.h_v * w.d_k * w.d_v * 4
    return 2 * state + rows * (w.h_qk * w.d_k * in_b + w.h_v * w.d_v * in_b + 2 * w.h_v * 4)


def algorithmic_bytes_verify(w, n_record):
    """The verify pass (no outputs): the state read and written back, n_record recorded
    states written, the block's k, v, g, beta read."""
    in_b = 2 if w.dtype == "bf16" else 4
    rows = w.requests * w.block
    state = w.requests * w.h_v * w.d_k * w.d_v * 4
    return (2 + n_record) * state + rows * (w.h_qk * w.d_k * in_b + w.h_v * w.d_v * in_b + 2 * w.h_v * 4)


def algorithmic_bytes_conv(w, backward):
    """ShortConv: the forward reads x, xn and writes y, yn; the backward reads x, xn, dy,
    dyn and writes dx, dxn (the filter, bias and their gradients are negligible)."""
    es = 2 if w.dtype == "bf16" else 4
    return (6 if backward else 4) * w.batch * w.seqlen * w.channels * es


def time_launches(fn, steps, warmup, stream):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        fn()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps  # ms per launch


def cpu_baseline(w, inp):
    """The fp64 oracle over the whole workload (every (sequence, v-head) unit, clean and
    noisy streams), its units spread over up to 16 host threads."""
    import oracle
    threads = max(1, min(os.cpu_count() or 1, 16))
    oracle.set_threads(threads)
    keys = ("q", "k", "v", "g", "beta")
    arr = {k: inp[k].double().numpy() for k in inp}
    t0 = time.perf_counter()
    oracle.fwd_train(*[arr[k] for k in keys], *[arr[k + "n"] for k in keys],
                     block=w.block, scale=1.0 / math.sqrt(w.d_k), want_ht=False)
    dt = time.perf_counter() - t0
    tokens = 2 * w.tokens
    return {"value": tokens / dt, "unit": "tokens/s", "cores": oracle.max_threads(),
            "kind": "oracle", "seconds": dt,
            "sample": f"the whole workload: {w.batch} sequences x {w.h_v} v-heads x "
                      f"({w.seqlen} clean + {w.seqlen} noisy) tokens in fp64; value = tokens / wall time"}


# The sources the one-kernel forward is built from (its translation unit and headers).
FUSED_SOURCES = ("common.hpp", "fused.hpp", "fused_kernels.hip", "intra.hpp", "kernels.hpp", "ut.hpp")


def kernel_source_hash():
    """Hash of the one-kernel forward's sources, to tell whether a recorded counter
    measurement still describes the kernel being timed."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2606_01774_amd", "csrc")
    for name in FUSED_SOURCES:
        with open(os.path.join(src, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per forward step from the FETCH_SIZE / WRITE_SIZE counter runs recorded
    under profiles/ (copy-calibrated), or None when the kernels have changed since."""
    path = os.path.join(ROOT, "profiles", "traffic_train_bf16_b4_t4096_h16_d128_l32.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except OSError:
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_step")


def copy_probe(steps):
    """A plain device-to-device copy of 256 MiB, the reference for scaling the byte
    counters (its true traffic is 256 MiB read + 256 MiB written per launch)."""
    import torch
    n = 256 * 1024 * 1024 // 4
    x = torch.ones(n, device="cuda")
    y = torch.empty_like(x)
    for _ in range(steps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n * 4, "launches": steps}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-serve", action="store_true")
    ap.add_argument("--no-conv", action="store_true")
    ap.add_argument("--no-bwd", action="store_true")
    ap.add_argument("--no-views", action="store_true")
    ap.add_argument("--route", choices=sorted(ROUTES), default="fused",
                    help="schedule of the training forward (fused is the performance mode; split and "
                         "records attribute its parts to separate kernels)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run only a 256 MiB device copy (byte-counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    if args.copy_probe:
        copy_probe(args.steps)
        return

    import torch

    import paper_2606_01774_amd as bd
    from paper_2606_01774_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    w = W.TRAIN_4K
    inp = W.make_train(w)
    d = {k: v.to(dev) for k, v in inp.items()}
    scale = 1.0 / math.sqrt(w.d_k)
    o = torch.empty(w.batch, w.seqlen, w.h_v, w.d_v, dtype=torch.float32, device=dev)
    on = torch.empty_like(o)
    route = {"fused": bd.BDGDN_ROUTE_FUSED, "split": bd.BDGDN_ROUTE_SPLIT,
             "records": bd.BDGDN_ROUTE_RECORDS}[args.route]
    desc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, scale=scale, route=route)
    ws = torch.empty(max(256, bd.bdgdn_fwd_train_workspace(desc)), dtype=torch.uint8, device=dev)

    def step():
        bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"],
                           d["qn"], d["kn"], d["vn"], d["gn"], d["betan"],
                           block=w.block, scale=scale, o=o, on=on, workspace=ws, stream=stream, route=route)

    torch.cuda.synchronize()
    ms = time_launches(step, args.steps, args.warmup, stream)
    tokens = 2 * w.tokens
    value = tokens / (ms * 1e-3)
    abytes = algorithmic_bytes_train(w, 4)
    flops = model_flops_train(w)
    achieved = abytes / (ms * 1e-3) / 1e9
    result = {
        "metric": "BD-GDN fwd tokens/s + % bf16 MFMA peak; denoise_step GB/s vs HBM peak",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; q,k L2-normalised N(0,1), v N(0,1), g=-softplus(U(-6,-2)), "
                "beta=sigmoid(U(-2,2)))",
        "config": {"workload": w.name, "batch": w.batch, "seq_len": w.seqlen,
                   "h_qk": w.h_qk, "h_v": w.h_v, "d_k": w.d_k, "d_v": w.d_v, "block": w.block,
                   "inputs": "bf16", "mfma_operands": "fp16", "state": "fp32", "outputs": "fp32",
                   "route": ROUTES[args.route], "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": recorded_traffic(),
                     "kernel": ("bdgdn_fwd_pipelined_kernel (the whole bdgdn_fwd_train step)" if args.route == "fused"
                                else f"the {args.route} schedule (all of its kernels)"),
                     "algorithmic_bytes": abytes, "kernel_source_hash": kernel_source_hash()},
        "mfma": {"model_flop": flops, "tflops": flops / (ms * 1e-3) / 1e12,
                 "frac_of_peak": flops / (ms * 1e-3) / 1e12 / MFMA16_PEAK_TFLOPS},
    }

    if not args.no_serve:
        sw = W.SERVE_64
        pools = [W.make_state_pool(sw.requests, sw.h_v, sw.d_k, sw.d_v, seed=sw.seed + i).to(dev)
                 for i in range(3)]
        blk = {k: v.to(dev) for k, v in W.make_serve_block(sw, 0).items()}
        od = torch.empty(sw.requests, sw.block, sw.h_v, sw.d_v, dtype=torch.float32, device=dev)
        it = [0]

        def dstep():
            pool = pools[it[0] % len(pools)]   # three pools: 384 MiB > the 256 MB MALL
            it[0] += 1
            bd.bdgdn_denoise_step(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                                  scale=scale, o=od, stream=stream)
        dms = time_launches(dstep, 3 * args.steps, args.warmup, stream)
        dbytes = algorithmic_bytes_denoise(sw, 4)
        gbs = dbytes / (dms * 1e-3) / 1e9
        result["denoise_step"] = {"workload": sw.name, "us_per_call": dms * 1e3,
                                  "gb_per_s": gbs, "frac_hbm": gbs / HBM_PEAK_GBS,
                                  "algorithmic_bytes": dbytes,
                                  "tokens_per_s": sw.requests * sw.block / (dms * 1e-3),
                                  "kernel": "bdgdn_k4_denoise_kernel"}

        def cstep():
            pool = pools[it[0] % len(pools)]
            it[0] += 1
            bd.bdgdn_commit(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                            scale=scale, stream=stream)
        cms = time_launches(cstep, 3 * args.steps, args.warmup, stream)
        cbytes = algorithmic_bytes_commit(sw)
        cgbs = cbytes / (cms * 1e-3) / 1e9
        result["commit"] = {"workload": sw.name, "us_per_call": cms * 1e3, "gb_per_s": cgbs,
                            "frac_hbm": cgbs / HBM_PEAK_GBS, "algorithmic_bytes": cbytes,
                            "kernel": "bdgdn_k4_commit_kernel (state written back, no outputs)"}

        # AR-Trust verify round: the verify pass keeping the states before the draft
        # positions, then the accept step (offsets drawn below the horizon, so every
        # request copies one state back)
        vw = W.VERIFY_64
        n_rec = vw.block - 1
        vblk = {k: v.to(dev) for k, v in W.make_serve_block(vw, 0).items()}
        states = torch.empty(vw.requests, n_rec, vw.h_v, vw.d_k, vw.d_v, dtype=torch.float32, device=dev)
        gen = torch.Generator().manual_seed(vw.seed)
        accept = torch.randint(0, n_rec, (vw.requests,), generator=gen, dtype=torch.int32).to(dev)

        def vstep():
            pool = pools[it[0] % len(pools)]
            it[0] += 1
            bd.bdgdn_commit_record(pool, vblk["q"], vblk["k"], vblk["v"], vblk["g"], vblk["beta"],
                                   n_record=n_rec, scale=scale, states=states, stream=stream)
        vms = time_launches(vstep, 3 * args.steps, args.warmup, stream)
        vbytes = algorithmic_bytes_verify(vw, n_rec)

        def astep():
            pool = pools[it[0] % len(pools)]
            it[0] += 1
            bd.bdgdn_accept_states(pool, states, accept, block=vw.block, stream=stream)
        ams = time_launches(astep, 3 * args.steps, args.warmup, stream)
        abytes_acc = 2 * vw.requests * vw.h_v * vw.d_k * vw.d_v * 4
        result["verify"] = {"workload": vw.name, "us_per_call": vms * 1e3,
                            "gb_per_s": vbytes / (vms * 1e-3) / 1e9,
                            "frac_hbm": vbytes / (vms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": vbytes,
                            "kernel": "bdgdn_k4_commit_record_kernel (7 recorded states, no outputs)",
                            "accept_us_per_call": ams * 1e3,
                            "accept_gb_per_s": abytes_acc / (ams * 1e-3) / 1e9}

    if not args.no_views:
        # complementary views: one clean scan seeding two noisy views (the second view drawn
        # with the same recipe), against two calls of the one-kernel forward
        v2 = W.make_custom_train(w.batch, w.seqlen, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype, seed=w.seed + 50)
        views = [{k_: d[k_ + "n"] for k_ in ("q", "k", "v", "g", "beta")},
                 {k_: v2[k_ + "n"].to(dev) for k_ in ("q", "k", "v", "g", "beta")}]
        for vw_ in views:
            vw_["o"] = torch.empty_like(o)
        vdesc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, scale=scale, route=bd.BDGDN_ROUTE_SPLIT)
        vws = torch.empty(bd.bdgdn_fwd_train_views_workspace(vdesc), dtype=torch.uint8, device=dev)
        vms = {}
        for rname, rt in (("fused", bd.BDGDN_ROUTE_FUSED), ("split", bd.BDGDN_ROUTE_SPLIT)):
            def vstep2(rt=rt):
                bd.bdgdn_fwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], views, block=w.block,
                                         scale=scale, o=o, route=rt, workspace=vws, stream=stream)
            vms[rname] = time_launches(vstep2, args.steps, args.warmup, stream)
        result["views"] = {
            "workload": w.name + " + a second noisy view", "n_views": 2,
            "ms_per_call": min(vms.values()), "tokens_per_s": 3 * w.tokens / (min(vms.values()) * 1e-3),
            "fused_ms": vms["fused"], "split_ms": vms["split"],
            "schedules": {"fused": "bdgdn_fwd_pipelined_kernel once per view (clean scan recomputed on chip)",
                          "split": "bdgdn_fwd_pipelined_seeds_kernel (view 0 + seed states) + bdgdn_k3_noisy_kernel"}}

    if not args.no_bwd:
        # the two-stream training backward at the same workload (fp32 upstream gradients)
        gdo = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(5), device=dev)
        gdon = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(6), device=dev)
        bdesc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, scale=scale, out_dtype=torch.float32)
        bws = torch.empty(bd.bdgdn_bwd_train_workspace(bdesc), dtype=torch.uint8, device=dev)
        bgrads = bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                                    d["betan"], gdo, gdon, block=w.block, scale=scale, workspace=bws)

        def bwstep():
            bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                               d["betan"], gdo, gdon, block=w.block, scale=scale, workspace=bws, grads=bgrads,
                               stream=stream)
        bsteps = max(2, args.steps // 4)
        bms = time_launches(bwstep, bsteps, 2, stream)
        # the complementary-view backward: the same clean stream, two noisy views (the second
        # drawn with the same recipe)
        v2b = W.make_custom_train(w.batch, w.seqlen, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype, seed=w.seed + 50)
        gdon2 = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(7), device=dev)
        bviews = [dict({k_: d[k_ + "n"] for k_ in ("q", "k", "v", "g", "beta")}, do=gdon),
                  dict({k_: v2b[k_ + "n"].to(dev) for k_ in ("q", "k", "v", "g", "beta")}, do=gdon2)]
        bvgrads = bd.bdgdn_bwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], bviews, gdo, block=w.block,
                                           scale=scale, workspace=bws)

        def bvstep():
            bd.bdgdn_bwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], bviews, gdo, block=w.block,
                                     scale=scale, grads=bvgrads, workspace=bws, stream=stream)
        bvms = time_launches(bvstep, bsteps, 2, stream)
        result["backward"] = {
            "workload": w.name, "ms_per_call": bms, "tokens_per_s": tokens / (bms * 1e-3), "steps": bsteps,
            "kernels": "bdgdn_k2_scan_states_kernel (seed states) + bdgdn_bwd_noisy_kernel + "
                       "bdgdn_bwd_scan_kernel + bdgdn_bwd_clean_kernel",
            "workspace_bytes": bws.numel(),
            "views2_ms_per_call": bvms, "views2_tokens_per_s": 3 * w.tokens / (bvms * 1e-3)}

    if not args.no_conv:
        # the GDN layer's two-stream ShortConv at the same token shape (channels = the q, k
        # and v projections side by side), forward and backward
        cw = W.CONV_TRAIN
        cin = {k: (None if v is None else v.to(dev)) for k, v in W.make_conv(cw).items()}
        y, yn = torch.empty_like(cin["x"]), torch.empty_like(cin["x"])
        dx, dxn = torch.empty_like(cin["x"]), torch.empty_like(cin["x"])
        dw, db = torch.empty_like(cin["w"]), torch.empty_like(cin["bias"])
        cdesc = bd.make_conv_desc(cin["x"], cin["w"], block=cw.block, activation=cw.act)
        cws = torch.empty(max(256, bd.bdgdn_shortconv_bwd_workspace(cdesc)), dtype=torch.uint8, device=dev)

        def fstep():
            bd.bdgdn_shortconv_fwd(cin["x"], cin["xn"], cin["w"], cin["bias"], block=cw.block, activation=cw.act,
                                   y=y, yn=yn, stream=stream)

        def bstep():
            bd.bdgdn_shortconv_bwd(cin["x"], cin["xn"], cin["w"], cin["bias"], cin["dy"], cin["dyn"],
                                   block=cw.block, activation=cw.act, dx=dx, dxn=dxn, dw=dw, dbias=db,
                                   workspace=cws, stream=stream)
        fms = time_launches(fstep, args.steps, args.warmup, stream)
        bms = time_launches(bstep, args.steps, args.warmup, stream)
        fbytes, bbytes = algorithmic_bytes_conv(cw, backward=False), algorithmic_bytes_conv(cw, backward=True)
        result["shortconv"] = {
            "workload": cw.name,
            "fwd": {"us_per_call": fms * 1e3, "gb_per_s": fbytes / (fms * 1e-3) / 1e9,
                    "frac_hbm": fbytes / (fms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": fbytes,
                    "kernel": "bdgdn_shortconv_fwd_kernel"},
            "bwd": {"us_per_call": bms * 1e3, "gb_per_s": bbytes / (bms * 1e-3) / 1e9,
                    "frac_hbm": bbytes / (bms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": bbytes,
                    "kernel": "bdgdn_shortconv_bwd_kernel + bdgdn_shortconv_reduce_kernel"}}

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, inp)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
