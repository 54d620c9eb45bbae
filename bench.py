"""Benchmark of the block-diffusion Gated DeltaNet hot path on one MI355X.

The headline step is one two-stream training forward (bdgdn_fwd_train, clean + noisy
streams) over the 4 x 4096-token, 16-head, d = 128, L = 32 workload with bf16 inputs,
fp32 state and fp32 outputs, inputs resident in HBM; `value` is tokens/s (clean + noisy
tokens) over K back-to-back steps timed with HIP events on the launch stream.

The roofline numerator is the fixed algorithmic byte model (bf16 q, k, v, o and fp32 g,
beta read or written once: 1032 B per (token, head, stream) at d = 128, plus states
where the interface reads or writes them), whatever output type the kernel writes; the
fp32-output bytes are reported beside it.  The `configs` object measures every
workload (the tiny fp32 case, the training shape, the grouped-value shape, the serving
denoise and commit passes, the packed 128k-token shape) with the same protocol: a
512 MB scratch read before each launch, per-launch HIP events, a trimmed mean of 20
launches, repeated 3 times.  Further sections time the verify-state cache, the
complementary views, the backward and the two-stream ShortConv; `cpu_baseline` times the
fp64 oracle on the host.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                  [--only SECTION[,SECTION...]] [--route fused|split|records]
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
          "records": "records (UT-transform kernel, then the scan)",
          "chunked": "chunked (state pass over the segment starts, then one workgroup per (chain, segment, tile))"}
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16/bf16 MFMA, TFLOP/s
FLUSH_BYTES = 512 * 1024 * 1024
SECTIONS = ("headline", "tiny_f32", "train_4k", "train_4k_bf16_out", "gva_16k", "serve", "varlen_128k", "varlen_128k_bf16_out", "verify", "views", "backward",
            "blocks", "shortconv", "cpu")
SWEEP_BLOCKS = (1, 2, 4, 8, 16, 32)   # the diffusion-block sweep of the route comparison


# ---------------------------------------------------------------- work models
def algorithmic_bytes_train(w, out_bytes=None):
    """Bytes the two-stream forward must move once: q, k per q/k head, v and o per v head,
    g and beta per v head, for both streams.  out_bytes None = the fixed model (o in
    bf16 for bf16 workloads, in the input type otherwise)."""
    in_b = 2 if w.dtype == "bf16" else 4
    ob = in_b if out_bytes is None else out_bytes
    per_row = 2 * w.h_qk * w.d_k * in_b + w.h_v * w.d_v * (in_b + ob) + 2 * w.h_v * 4
    return 2 * w.tokens * per_row


def algorithmic_bytes_bwd(w, up_bytes=4):
    """Bytes the two-stream backward must move once: every forward input read (q, k per q/k
    head, v, g, beta per v head), the upstream gradients of o and o~ read (up_bytes each),
    and the fp32 gradients of every input written, for both streams; the seeds, state
    gradients and any workspace traffic are the schedule's, not counted."""
    in_b = 2 if w.dtype == "bf16" else 4
    read = 2 * w.h_qk * w.d_k * in_b + w.h_v * w.d_v * in_b + 2 * w.h_v * 4 + w.h_v * w.d_v * up_bytes
    written = 4 * (2 * w.h_qk * w.d_k + w.h_v * w.d_v + 2 * w.h_v)
    return 2 * w.tokens * (read + written)


def model_flops_train(w, chunk=64):
    """Work model: clean 6d^2 + 10Cd per (token, v-head) with C = 64, noisy
    2d^2 + 12Ld; the Gram terms (4Cd + 4Ld) once per q/k head; the triangular solve
    excluded."""
    d = w.d_k
    per_v = 6 * d * d + 6 * chunk * d + 2 * d * d + 8 * w.block * d
    per_qk = 4 * chunk * d + 4 * w.block * d
    return w.tokens * (w.h_v * per_v + w.h_qk * per_qk)


def _state_bytes(w):
    return w.requests * w.h_v * w.d_k * w.d_v * 4


def _block_bytes(w, q=True, v=True, o=False, out_bytes=None):
    in_b = 2 if w.dtype == "bf16" else 4
    ob = in_b if out_bytes is None else out_bytes
    rows = w.requests * w.block
    return rows * ((2 if q else 1) * w.h_qk * w.d_k * in_b + (w.h_v * w.d_v * in_b if v else 0)
                   + (w.h_v * w.d_v * ob if o else 0) + 2 * w.h_v * 4)


def algorithmic_bytes_denoise(w, out_bytes=None):
    """The state read once, the block's q, k, v, g, beta read and o written."""
    return _state_bytes(w) + _block_bytes(w, o=True, out_bytes=out_bytes)


def algorithmic_bytes_commit(w, with_outputs, out_bytes=None):
    """The state read and written back and the block's k, v, g, beta read; with outputs
    also q read and the causal o written."""
    return 2 * _state_bytes(w) + _block_bytes(w, q=with_outputs, o=with_outputs, out_bytes=out_bytes)


def model_flops_denoise(w):
    """Noisy block: 2d^2 + 12Ld per (token, v-head)."""
    return w.requests * w.block * w.h_v * (2 * w.d_k * w.d_v + 12 * w.block * w.d_k)


def model_flops_commit(w):
    """Clean pass with the chunk = the block: 6d^2 + 10Ld per (token, v-head)."""
    return w.requests * w.block * w.h_v * (6 * w.d_k * w.d_v + 10 * w.block * w.d_k)


def algorithmic_bytes_verify(w, n_record):
    """The verify pass (no outputs): the state read and written back, n_record recorded
    states written, the block's k, v, g, beta read."""
    return (2 + n_record) * _state_bytes(w) + _block_bytes(w, q=False)


def algorithmic_bytes_conv(w, backward):
    """ShortConv: the forward reads x, xn and writes y, yn; the backward reads x, xn, dy,
    dyn and writes dx, dxn (the filter, bias and their gradients are negligible)."""
    es = 2 if w.dtype == "bf16" else 4
    return (6 if backward else 4) * w.batch * w.seqlen * w.channels * es


# ---------------------------------------------------------------- timing
def time_launches(fn, steps, warmup, stream):
    """Back-to-back launches: ms per launch over `steps` launches after `warmup`."""
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
    return start.elapsed_time(end) / steps


class Flusher:
    """A 512 MB scratch buffer read (summed) before each timed launch, so that no launch
    finds its inputs in the 256 MB MALL or the L2s from the previous one.  It is read, not
    written: a write would leave up to the MALL's size of dirty lines whose write-back then
    falls inside the timed launch (measured on the serving pass: 78 us after a 512 MB fill,
    42 us after this read, 35 us with its pool left warm)."""

    def __init__(self, dev):
        import torch
        self.buf = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)

    def __call__(self):
        self.buf.sum()


PROTOCOL = {"iters": 20, "repeats": 3}


def time_protocol(fn, stream, flush, warmup=5, iters=None, repeats=None, trim=2):
    """The per-config protocol: `warmup` launches, then `repeats` x `iters` launches, each
    after a scratch flush and bracketed by its own HIP events on the launch stream; the
    `trim` fastest and slowest of each repeat dropped, the rest averaged.  Returns ms
    (mean over repeats) and the per-repeat trimmed means."""
    import torch
    iters = PROTOCOL["iters"] if iters is None else min(iters, PROTOCOL["iters"])
    repeats = PROTOCOL["repeats"] if repeats is None else min(repeats, PROTOCOL["repeats"])
    trim = min(trim, (iters - 1) // 2)
    warmup = min(warmup, iters)
    for _ in range(warmup):
        flush()
        fn()
    torch.cuda.synchronize()
    means = []
    for _ in range(repeats):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
        for s, e in ev:
            flush()
            s.record(stream)
            fn()
            e.record(stream)
        torch.cuda.synchronize()
        ts = sorted(s.elapsed_time(e) for s, e in ev)
        kept = ts[trim:len(ts) - trim]
        means.append(sum(kept) / len(kept))
    return sum(means) / len(means), means


def rates(ms, abytes, flops, tokens):
    """Throughput and roofline fractions of one launch of `ms` milliseconds.  The binding
    roofline is min(MFMA peak, AI x HBM bandwidth)."""
    s = ms * 1e-3
    gbs = abytes / s / 1e9
    tfl = flops / s / 1e12
    ai = flops / abytes
    roof_tfl = min(MFMA16_PEAK_TFLOPS, ai * HBM_PEAK_GBS / 1e3)
    return {"ms": ms, "tokens_per_s": tokens / s, "algorithmic_bytes": abytes, "gb_per_s": gbs,
            "frac_hbm": gbs / HBM_PEAK_GBS, "model_flop": flops, "tflops": tfl,
            "frac_mfma": tfl / MFMA16_PEAK_TFLOPS, "arith_intensity": ai,
            "bound": "hbm" if roof_tfl < MFMA16_PEAK_TFLOPS else "mfma",
            "frac_roofline": tfl / roof_tfl}


# ---------------------------------------------------------------- recorded counters
# The sources each measured kernel is built from (translation unit and headers).
KERNEL_SOURCES = {
    "fused": ("common.hpp", "fused.hpp", "fused_kernels.hip", "intra.hpp", "kernels.hpp", "ut.hpp"),
    "chunked": ("common.hpp", "chunked.hpp", "chunked_kernels.hip", "intra.hpp", "kernels.hpp", "ut.hpp"),
    "records": ("common.hpp", "intra.hpp", "scan.hpp", "fwd_scan_kernels.hip", "kernels.hpp", "ut.hpp"),
    "serve": ("common.hpp", "serve.hpp", "serve_kernels.hip", "kernels.hpp", "ut.hpp"),
}


def kernel_source_hash(group="fused"):
    """Hash of a kernel group's sources, to tell whether a recorded counter measurement
    still describes the kernel being timed."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2606_01774_amd", "csrc")
    for name in KERNEL_SOURCES[group]:
        with open(os.path.join(src, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def recorded_traffic(key):
    """HBM bytes per launch of one measured config from the FETCH_SIZE / WRITE_SIZE counter
    runs recorded under profiles/ (copy-calibrated), or None when its kernels have changed
    since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)["configs"][key]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash(rec.get("sources", "fused")):
        return None
    return rec.get("bytes_per_launch")


# The configurations whose HBM traffic is recorded: bench section, kernel (a substring of
# the rocprofv3 kernel name), source group, algorithmic bytes (byte model; with fp32
# outputs where the kernel writes them).
def traffic_targets():
    from paper_2606_01774_amd import workloads as W
    sw = W.SERVE_64
    return {
        "train_4k": ("train_4k", "bdgdn_fwd_pipelined_kernel<float, 128, 32>", "fused", W.TRAIN_4K),
        "gva_16k": ("gva_16k", "bdgdn_fwd_pipelined_pair_kernel<float, 128>", "fused", W.GVA_16K),
        "varlen_128k": ("varlen_128k", "bdgdn_chunk_out_kernel<float, 128, 128, 32>", "chunked", W.VARLEN_128K),
        "serve_denoise": ("serve", "bdgdn_k4_denoise_kernel<float, 32>", "serve", sw),
        "serve_commit": ("serve", "bdgdn_k4_commit_kernel<float, 32, true>", "serve", sw),
        "serve_commit_state_only": ("serve", "bdgdn_k4_commit_kernel<float, 32, false>", "serve", sw),
    }


def _counter_medians(run_dir, counter):
    """Median per kernel name of one counter over the dispatches of a rocprofv3 --pmc run
    (its *counter_collection.csv files under run_dir)."""
    import csv
    import glob
    vals = {}
    for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if row.get("Counter_Name") == counter:
                    vals.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
    return {k: sorted(v)[len(v) // 2] for k, v in vals.items()}


def record_traffic(root):
    """Write profiles/traffic.json and traffic.md from the FETCH_SIZE / WRITE_SIZE counter runs
    under `root`: copy_fetch/, copy_write/ (bench.py --copy-probe) and <section>_fetch/,
    <section>_write/ (bench.py --only <section>).  The counters are scaled by what they read
    for the 256 MiB copy (its true traffic 256 MiB read and 256 MiB written)."""
    copy_bytes = 256 * 1024 * 1024
    cf = max(_counter_medians(os.path.join(root, "copy_fetch"), "FETCH_SIZE").values())
    cw = max(_counter_medians(os.path.join(root, "copy_write"), "WRITE_SIZE").values())
    ff, wf = copy_bytes / 1024 / cf, copy_bytes / 1024 / cw
    out = {"calibration": {"copy_bytes": copy_bytes, "fetch_kib_raw": cf, "write_kib_raw": cw,
                           "fetch_factor": ff, "write_factor": wf}, "configs": {}}
    rows = []
    for key, (section, kernel, group, wl) in traffic_targets().items():
        fm = _counter_medians(os.path.join(root, f"{section}_fetch"), "FETCH_SIZE")
        wm = _counter_medians(os.path.join(root, f"{section}_write"), "WRITE_SIZE")
        fk = [v for k, v in fm.items() if kernel in k]
        wk = [v for k, v in wm.items() if kernel in k]
        if not fk or not wk:
            continue
        rd, wr = fk[0] * 1024 * ff, wk[0] * 1024 * wf
        out["configs"][key] = {"workload": wl.name, "kernel": kernel, "sources": group,
                               "source_hash": kernel_source_hash(group), "fetch_kib_raw": fk[0],
                               "write_kib_raw": wk[0], "read_bytes": rd, "write_bytes": wr,
                               "bytes_per_launch": int(rd + wr)}
        if key.startswith("serve"):
            alg = {"serve_denoise": algorithmic_bytes_denoise(wl, 4),
                   "serve_commit": algorithmic_bytes_commit(wl, True, 4),
                   "serve_commit_state_only": algorithmic_bytes_commit(wl, False)}[key]
            model = f"{alg / 1e6:.1f} (fp32 o)"
        else:
            alg = algorithmic_bytes_train(wl, 4)
            model = f"{algorithmic_bytes_train(wl) / 1e6:.1f} / {alg / 1e6:.1f}"
        rows.append(f"| `{kernel}` | {wl.name} | {fk[0]:.0f} | {wk[0]:.0f} | {rd / 1e6:.1f} | {wr / 1e6:.1f} | "
                    f"{(rd + wr) / 1e6:.1f} | {model} | {100 * (rd + wr) / alg:.1f} % |")
    with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
    md = ["# HBM traffic per launch, every measured configuration", "",
          "Counters per dispatch (median over the dispatches of the run) from two `rocprofv3 --pmc` runs per",
          "configuration, one counter each, scaled by what the same counter reads for a plain 256 MiB device",
          f"copy (`bench.py --copy-probe`): FETCH_SIZE reads {cf:.0f} KiB for the copy's 262144 KiB of reads",
          f"(factor {ff:.4f}), WRITE_SIZE {cw:.0f} KiB (factor {wf:.4f}).", "",
          "Commands (repository root on the MI355X box, `TMPDIR=/tmp`; `<section>` is train_4k, gva_16k, varlen_128k or serve):", "",
          "    cd /tmp && rocprofv3 --pmc FETCH_SIZE --output-format csv -d <root>/<section>_fetch -o run -- \\",
          "        python3 <repo>/bench.py --no-cpu-baseline --only <section> --protocol-iters 3 --protocol-repeats 1",
          "    cd /tmp && rocprofv3 --pmc WRITE_SIZE --output-format csv -d <root>/<section>_write -o run -- \\",
          "        python3 <repo>/bench.py --no-cpu-baseline --only <section> --protocol-iters 3 --protocol-repeats 1",
          "    (and the same two with `bench.py --copy-probe --steps 3` into <root>/copy_fetch, <root>/copy_write)",
          "    python3 <repo>/bench.py --record-traffic <root>", "",
          "| kernel | workload | FETCH_SIZE (KiB) | WRITE_SIZE (KiB) | read (MB) | written (MB) | total (MB) | "
          "algorithmic (MB): byte model / with fp32 o | total / algorithmic with fp32 o |",
          "|---|---|---|---|---|---|---|---|---|", *rows, "",
          "The training byte model counts bf16 q, k, v, o and fp32 g, beta once (1032 B per (token, head, stream));",
          "the kernels write fp32 o, so the bytes they must move are the second figure, which the last column",
          "compares with.  Serving: the state read (and written back by commit) once, the block's q, k, v, g, beta",
          "read and o written (fp32).", "",
          "Recorded in `traffic.json` with the hashes of the kernels' sources; bench.py reports a configuration's",
          "figure as its traffic while those sources are unchanged."]
    with open(os.path.join(ROOT, "profiles", "traffic.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print(json.dumps(out["configs"], indent=1))


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


# ---------------------------------------------------------------- workloads on the device
def train_setup(w, dev, route, out_dtype):
    import torch
    import paper_2606_01774_amd as bd
    from paper_2606_01774_amd import workloads as W
    inp = W.make_train(w)
    d = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    cu = inp.get("cu_seqlens")
    scale = 1.0 / math.sqrt(w.d_k)
    o = torch.empty(w.batch, w.seqlen, w.h_v, w.d_v, dtype=out_dtype, device=dev)
    on = torch.empty_like(o)
    desc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, scale=scale, route=route, out_dtype=out_dtype,
                            num_seqs=0 if cu is None else len(cu) - 1)
    ws = torch.empty(max(256, bd.bdgdn_fwd_train_workspace(desc)), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        bd.bdgdn_fwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                           d["betan"], block=w.block, scale=scale, o=o, on=on, workspace=ws, stream=stream,
                           route=route, cu_seqlens=d.get("cu_seqlens"), cu_seqlens_host=cu)
    return inp, d, step, o


def prefix_pools(sw, dev, n_pools, stream):
    """fp32 state pools [R, h_v, d_k, d_v] with realistic magnitudes: each request's
    state is the clean state after a seeded prefix of 256 tokens (8 blocks of 32),
    run from zero through bdgdn_commit (itself checked against the oracle's causal pass
    in the tests)."""
    import torch
    import paper_2606_01774_amd as bd
    from paper_2606_01774_amd import workloads as W
    pools = []
    for i in range(n_pools):
        pool = torch.zeros(sw.requests, sw.h_v, sw.d_k, sw.d_v, dtype=torch.float32, device=dev)
        for j in range(W.SERVE_PREFIX_BLOCKS):
            blk = {k: v.to(dev) for k, v in W.make_serve_prefix_block(sw, i, j).items()}
            bd.bdgdn_commit(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], stream=stream)
        pools.append(pool)
    torch.cuda.synchronize()
    return pools


# ---------------------------------------------------------------- main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", default=None,
                    help="comma-separated sections to run (" + ", ".join(SECTIONS) + "); default all")
    ap.add_argument("--route", choices=sorted(ROUTES), default="fused",
                    help="schedule of the headline training forward (fused is the performance mode; split and "
                         "records attribute its parts to separate kernels)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run only a 256 MiB device copy (byte-counter calibration)")
    ap.add_argument("--protocol-iters", type=int, default=20,
                    help="launches per repeat of the per-config protocol (fewer for counter runs)")
    ap.add_argument("--protocol-repeats", type=int, default=3)
    ap.add_argument("--record-traffic", metavar="DIR", default=None,
                    help="write profiles/traffic.json and traffic.md from the counter runs under DIR (no GPU)")
    args = ap.parse_args()
    PROTOCOL["iters"], PROTOCOL["repeats"] = max(1, args.protocol_iters), max(1, args.protocol_repeats)
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU (--gpus must be 1); the sharding across GPUs "
                                   "is a design, not a measured path", "n_gpus": args.gpus}))
        sys.exit(2)
    if args.record_traffic:
        record_traffic(args.record_traffic)
        return
    if args.copy_probe:
        copy_probe(args.steps)
        return
    only = set(SECTIONS) if args.only is None else set(args.only.split(","))
    unknown = only - set(SECTIONS)
    if unknown:
        ap.error(f"unknown sections {sorted(unknown)}")
    if args.no_cpu_baseline:
        only.discard("cpu")
    if "verify" in only:
        only.add("serve")   # the verify pass runs on the serving pools

    import torch

    import paper_2606_01774_amd as bd
    from paper_2606_01774_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    flush = Flusher(dev)
    result = {}
    configs = {}

    # ---------------- headline: the training shape, K back-to-back steps
    w = W.TRAIN_4K
    route = {"fused": bd.BDGDN_ROUTE_FUSED, "split": bd.BDGDN_ROUTE_SPLIT,
             "records": bd.BDGDN_ROUTE_RECORDS, "chunked": bd.BDGDN_ROUTE_CHUNKED}[args.route]
    inp = None
    if "headline" in only or "train_4k" in only or "cpu" in only:
        inp, d, step, o = train_setup(w, dev, route, torch.float32)
    if "headline" in only:
        ms = time_launches(step, args.steps, args.warmup, stream)
        tokens = 2 * w.tokens
        abytes = algorithmic_bytes_train(w)
        flops = model_flops_train(w)
        achieved = abytes / (ms * 1e-3) / 1e9
        result.update({
            "metric": "BD-GDN fwd tokens/s + % bf16 MFMA peak; denoise_step GB/s vs HBM peak",
            "value": tokens / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded; q,k L2-normalised N(0,1), v N(0,1), g=-softplus(U(-6,-2)), "
                    "beta=sigmoid(U(-2,2)))",
            "config": {"workload": w.name, "batch": w.batch, "seq_len": w.seqlen,
                       "h_qk": w.h_qk, "h_v": w.h_v, "d_k": w.d_k, "d_v": w.d_v, "block": w.block,
                       "inputs": "bf16", "mfma_operands": "fp16", "state": "fp32", "outputs": "fp32",
                       "route": ROUTES[args.route], "parallelism": "none (1 GPU)"},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBS,
                         "traffic": recorded_traffic("train_4k") if args.route == "fused" else None,
                         "kernel": ("bdgdn_fwd_pipelined_kernel (the whole bdgdn_fwd_train step)"
                                    if args.route == "fused" else f"the {args.route} schedule (all of its kernels)"),
                         "algorithmic_bytes": abytes,
                         "byte_model": "bf16 q, k, v, o and fp32 g, beta of both streams, once: "
                                       "1032 B per (token, head, stream)",
                         "bytes_with_fp32_outputs": algorithmic_bytes_train(w, 4),
                         "frac_with_fp32_output_bytes": algorithmic_bytes_train(w, 4) / (ms * 1e-3) / 1e9
                                                        / HBM_PEAK_GBS,
                         "kernel_source_hash": kernel_source_hash("fused")},
            "mfma": {"model_flop": flops, "tflops": flops / (ms * 1e-3) / 1e12,
                     "frac_of_peak": flops / (ms * 1e-3) / 1e12 / MFMA16_PEAK_TFLOPS,
                     "roofline_tflops": min(MFMA16_PEAK_TFLOPS, flops / abytes * HBM_PEAK_GBS / 1e3)},
        })
        print(f"headline {ms:.4f} ms", file=sys.stderr, flush=True)

    def train_config(key, wl, rt=bd.BDGDN_ROUTE_FUSED, out_dtype=torch.float32, note="", stp=None):
        dd = None
        if stp is None:
            _, dd, stp, _ = train_setup(wl, dev, rt, out_dtype)
        ms, reps = time_protocol(stp, stream, flush)
        r = rates(ms, algorithmic_bytes_train(wl), model_flops_train(wl), 2 * wl.tokens)
        r.update({"workload": wl.name, "repeats_ms": reps, "outputs": str(out_dtype).replace("torch.", ""),
                  "traffic_bytes": recorded_traffic(key)})
        if out_dtype == torch.float32 and wl.dtype == "bf16":
            r["frac_hbm_fp32_output_bytes"] = algorithmic_bytes_train(wl, 4) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS
        if note:
            r["schedule"] = note
        configs[key] = r
        print(f"{key} {ms:.4f} ms", file=sys.stderr, flush=True)
        del dd
        torch.cuda.empty_cache()

    if "tiny_f32" in only:
        train_config("tiny_f32", W.TINY_F32, note="records route (fp32 inputs): UT-transform kernel + scan")
    if "train_4k" in only:
        train_config("train_4k", W.TRAIN_4K, note="bdgdn_fwd_pipelined_kernel (one kernel)",
                     stp=step if route == bd.BDGDN_ROUTE_FUSED else None)
    if "train_4k_bf16_out" in only:
        train_config("train_4k_bf16_out", W.TRAIN_4K, out_dtype=torch.bfloat16,
                     note="bdgdn_fwd_pipelined_kernel, bf16 outputs")
    if "gva_16k" in only:
        train_config("gva_16k", W.GVA_16K, note="bdgdn_fwd_pipelined_pair_kernel (one kernel; each noisy block of 64 "
                                           "spans two 32-position sub-blocks)")
    if "varlen_128k" in only:
        train_config("varlen_128k", W.VARLEN_128K, note="bdgdn_chunk_out_kernel (one workgroup per (document, v-head) over "
                                               "all d_v columns: 512 chains cover the 256 CUs), longest documents first")
    if "varlen_128k_bf16_out" in only:
        # the same kernel writing bf16 outputs: the bytes it moves are then those of the byte model
        train_config("varlen_128k_bf16_out", W.VARLEN_128K, out_dtype=torch.bfloat16,
                     note="bdgdn_chunk_out_kernel, bf16 outputs")

    # ---------------- serving
    if "serve" in only:
        sw = W.SERVE_64
        pools = prefix_pools(sw, dev, 3, stream)   # 3 x 128 MiB > the 256 MB MALL
        blk = {k: v.to(dev) for k, v in W.make_serve_block(sw, 0).items()}
        od = torch.empty(sw.requests, sw.block, sw.h_v, sw.d_v, dtype=torch.float32, device=dev)
        it = [0]

        def dstep():
            pool = pools[it[0] % len(pools)]
            it[0] += 1
            bd.bdgdn_denoise_step(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], o=od, stream=stream)

        ms, reps = time_protocol(dstep, stream, flush)
        r = rates(ms, algorithmic_bytes_denoise(sw), model_flops_denoise(sw), sw.requests * sw.block)
        r.update({"workload": sw.name, "repeats_ms": reps, "kernel": "bdgdn_k4_denoise_kernel",
                  "pools": "3 prefix-state pools rotated (384 MiB)", "traffic_bytes": recorded_traffic("serve_denoise")})
        configs["serve_denoise"] = r
        # warm: one pool, no flush (its 128 MiB state can stay in the MALL between calls)
        it[0] = 0
        one = pools[:1]

        def wstep():
            bd.bdgdn_denoise_step(one[0], blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"], o=od, stream=stream)
        wms, wreps = time_protocol(wstep, stream, lambda: None)
        rw = rates(wms, algorithmic_bytes_denoise(sw), model_flops_denoise(sw), sw.requests * sw.block)
        rw.update({"workload": sw.name, "repeats_ms": wreps, "pools": "one pool, no flush (warm)"})
        configs["serve_denoise_warm"] = rw
        oc = torch.empty_like(od)
        for key, want in (("serve_commit", True), ("serve_commit_state_only", False)):
            def cstep(want=want):
                pool = pools[it[0] % len(pools)]
                it[0] += 1
                bd.bdgdn_commit(pool, blk["q"], blk["k"], blk["v"], blk["g"], blk["beta"],
                                o_causal=oc if want else None, stream=stream)
            cms, creps = time_protocol(cstep, stream, flush)
            rc = rates(cms, algorithmic_bytes_commit(sw, want), model_flops_commit(sw), sw.requests * sw.block)
            rc.update({"workload": sw.name, "repeats_ms": creps, "traffic_bytes": recorded_traffic(key),
                       "kernel": "bdgdn_k4_commit_kernel (" + ("causal outputs" if want else "no outputs") + ")"})
            configs[key] = rc
        print(f"serve denoise {ms * 1e3:.1f} us", file=sys.stderr, flush=True)
        result["denoise_step"] = {"workload": sw.name, "us_per_call": ms * 1e3, "gb_per_s": r["gb_per_s"],
                                  "frac_hbm": r["frac_hbm"], "algorithmic_bytes": r["algorithmic_bytes"],
                                  "tokens_per_s": r["tokens_per_s"], "kernel": "bdgdn_k4_denoise_kernel",
                                  "warm_single_pool_us": wms * 1e3, "traffic_bytes": r["traffic_bytes"]}
        result["commit"] = {"workload": sw.name, "us_per_call": configs["serve_commit"]["ms"] * 1e3,
                            "gb_per_s": configs["serve_commit"]["gb_per_s"],
                            "frac_hbm": configs["serve_commit"]["frac_hbm"],
                            "state_only_us_per_call": configs["serve_commit_state_only"]["ms"] * 1e3,
                            "state_only_frac_hbm": configs["serve_commit_state_only"]["frac_hbm"]}

        if "verify" in only:
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
                                       n_record=n_rec, states=states, stream=stream)
            vms, _ = time_protocol(vstep, stream, flush)
            vbytes = algorithmic_bytes_verify(vw, n_rec)

            def astep():
                pool = pools[it[0] % len(pools)]
                it[0] += 1
                bd.bdgdn_accept_states(pool, states, accept, block=vw.block, stream=stream)
            ams, _ = time_protocol(astep, stream, flush)
            abytes_acc = 2 * vw.requests * vw.h_v * vw.d_k * vw.d_v * 4
            result["verify"] = {"workload": vw.name, "us_per_call": vms * 1e3,
                                "gb_per_s": vbytes / (vms * 1e-3) / 1e9,
                                "frac_hbm": vbytes / (vms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": vbytes,
                                "kernel": "bdgdn_k4_commit_record_kernel (7 recorded states, no outputs)",
                                "accept_us_per_call": ams * 1e3,
                                "accept_gb_per_s": abytes_acc / (ams * 1e-3) / 1e9}
        del pools
        torch.cuda.empty_cache()

    if configs:
        result["configs"] = configs

    if "views" in only or "backward" in only:
        if inp is None:
            inp, d, step, o = train_setup(w, dev, bd.BDGDN_ROUTE_FUSED, torch.float32)
        tokens = 2 * w.tokens
    if "views" in only:
        # complementary views: one clean scan seeding two noisy views (the second view drawn
        # with the same recipe), against two calls of the one-kernel forward
        v2 = W.make_custom_train(w.batch, w.seqlen, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype, seed=w.seed + 50)
        views = [{k_: d[k_ + "n"] for k_ in ("q", "k", "v", "g", "beta")},
                 {k_: v2[k_ + "n"].to(dev) for k_ in ("q", "k", "v", "g", "beta")}]
        for vw_ in views:
            vw_["o"] = torch.empty_like(o)
        vdesc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, route=bd.BDGDN_ROUTE_SPLIT)
        vws = torch.empty(bd.bdgdn_fwd_train_views_workspace(vdesc), dtype=torch.uint8, device=dev)
        vms = {}
        for rname, rt in (("fused", bd.BDGDN_ROUTE_FUSED), ("split", bd.BDGDN_ROUTE_SPLIT)):
            def vstep2(rt=rt):
                bd.bdgdn_fwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], views, block=w.block,
                                         o=o, route=rt, workspace=vws, stream=stream)
            vms[rname] = time_protocol(vstep2, stream, flush)[0]
        result["views"] = {
            "workload": w.name + " + a second noisy view", "n_views": 2,
            "ms_per_call": min(vms.values()), "tokens_per_s": 3 * w.tokens / (min(vms.values()) * 1e-3),
            "fused_ms": vms["fused"], "split_ms": vms["split"],
            "schedules": {"fused": "bdgdn_fwd_pipelined_kernel once per view (clean scan recomputed on chip)",
                          "split": "bdgdn_fwd_pipelined_seeds_kernel (view 0 + seed states) + bdgdn_k3_noisy_kernel"}}
        del vws, views
        torch.cuda.empty_cache()

    if "backward" in only:
        # the two-stream training backward at the same workload (fp32 upstream gradients)
        gdo = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(5), device=dev)
        gdon = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(6), device=dev)
        bdesc = bd.make_fwd_desc(d["q"], d["v"], block=w.block, out_dtype=torch.float32)
        bws = torch.empty(bd.bdgdn_bwd_train_workspace(bdesc), dtype=torch.uint8, device=dev)
        bgrads = bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                                    d["betan"], gdo, gdon, block=w.block, workspace=bws)

        def bwstep():
            bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                               d["betan"], gdo, gdon, block=w.block, workspace=bws, grads=bgrads, stream=stream)
        bms = time_protocol(bwstep, stream, flush, iters=10, repeats=3, trim=1)[0]
        # the complementary-view backward: the same clean stream, two noisy views (the second
        # drawn with the same recipe)
        v2b = W.make_custom_train(w.batch, w.seqlen, w.h_qk, w.h_v, w.d_k, w.d_v, w.dtype, seed=w.seed + 50)
        gdon2 = torch.randn(o.shape, generator=torch.Generator(device=dev).manual_seed(7), device=dev)
        bviews = [dict({k_: d[k_ + "n"] for k_ in ("q", "k", "v", "g", "beta")}, do=gdon),
                  dict({k_: v2b[k_ + "n"].to(dev) for k_ in ("q", "k", "v", "g", "beta")}, do=gdon2)]
        bvgrads = bd.bdgdn_bwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], bviews, gdo, block=w.block,
                                           workspace=bws)

        def bvstep():
            bd.bdgdn_bwd_train_views(d["q"], d["k"], d["v"], d["g"], d["beta"], bviews, gdo, block=w.block,
                                     grads=bvgrads, workspace=bws, stream=stream)
        bvms = time_protocol(bvstep, stream, flush, iters=10, repeats=3, trim=1)[0]
        # the same backward in four time segments (strided clean checkpoints): the workspace
        # the library needs for them, the same gradients bit for bit
        sseg = 4
        sws = torch.empty(bd.bdgdn_bwd_train_workspace_segmented(bdesc, None, sseg), dtype=torch.uint8, device=dev)

        def bsstep():
            bd.bdgdn_bwd_train(d["q"], d["k"], d["v"], d["g"], d["beta"], d["qn"], d["kn"], d["vn"], d["gn"],
                               d["betan"], gdo, gdon, block=w.block, workspace=sws, grads=bgrads, stream=stream)
        bsms = time_protocol(bsstep, stream, flush, iters=10, repeats=3, trim=1)[0]
        bab = algorithmic_bytes_bwd(w)
        result["backward"] = {
            "workload": w.name, "ms_per_call": bms, "tokens_per_s": tokens / (bms * 1e-3),
            "algorithmic_bytes": bab, "frac_hbm": bab / (bms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "byte_model": "inputs and fp32 upstream gradients read, fp32 gradients written, once",
            "kernels": "bdgdn_k2_scan_states_kernel (seed states) + bdgdn_bwd_noisy_kernel + "
                       "bdgdn_bwd_scan_kernel + bdgdn_bwd_clean_kernel",
            "workspace_bytes": bws.numel(),
            "views2_ms_per_call": bvms, "views2_tokens_per_s": 3 * w.tokens / (bvms * 1e-3),
            "segmented": {"segments": sseg, "workspace_bytes": sws.numel(), "ms_per_call": bsms,
                          "tokens_per_s": tokens / (bsms * 1e-3)}}
        del bws, sws, bgrads, bvgrads, bviews
        torch.cuda.empty_cache()
        # the other training workloads: the tiny fp32 one (the per-step fp32 backward), the
        # grouped-value one (blocks of 64: the block form with noisy blocks of two sub-blocks)
        # and the packed 128k one (32 documents)
        per_step = {}
        block_form = ("bdgdn_k2_scan_states_kernel (seed states) + bdgdn_bwd_noisy_kernel + "
                      "bdgdn_bwd_scan_kernel + bdgdn_bwd_clean_kernel")
        paths = {"tiny_f32": ("bdgdn_bwd_gen_ckpt_kernel + bdgdn_bwd_gen_walk_kernel (fp32, per step)", 1, 3, 1),
                 "gva_16k": ("bdgdn_k2_scan_states_kernel (seed states per 32-position sub-block) + "
                        "bdgdn_bwd_pair_kernel + bdgdn_bwd_scan_kernel + bdgdn_bwd_clean_kernel", 3, 10, 3),
                 "varlen_128k": (block_form, 3, 10, 3)}
        for key, pw in (("tiny_f32", W.TINY_F32), ("gva_16k", W.GVA_16K), ("varlen_128k", W.VARLEN_128K)):
            praw = W.make_train(pw)
            pin = {k_: v_.to(dev) for k_, v_ in praw.items() if isinstance(v_, torch.Tensor)}
            pcu = praw.get("cu_seqlens")
            pkw = {} if pcu is None else {"cu_seqlens": pin["cu_seqlens"], "cu_seqlens_host": pcu}
            pshape = (pw.batch, pw.seqlen, pw.h_v, pw.d_v)
            pdo = torch.randn(pshape, generator=torch.Generator(device=dev).manual_seed(8), device=dev)
            pdon = torch.randn(pshape, generator=torch.Generator(device=dev).manual_seed(9), device=dev)
            pdesc = bd.make_fwd_desc(pin["q"], pin["v"], block=pw.block, out_dtype=torch.float32,
                                     num_seqs=0 if pcu is None else len(pcu) - 1)
            pws = torch.empty(bd.bdgdn_bwd_train_workspace(pdesc), dtype=torch.uint8, device=dev)
            pscale = 1.0 / math.sqrt(pw.d_k)
            pargs = [pin[k_] for k_ in ("q", "k", "v", "g", "beta", "qn", "kn", "vn", "gn", "betan")]
            pgrads = bd.bdgdn_bwd_train(*pargs, pdo, pdon, block=pw.block, scale=pscale, workspace=pws, **pkw)

            def pstep():
                bd.bdgdn_bwd_train(*pargs, pdo, pdon, block=pw.block, scale=pscale, workspace=pws, grads=pgrads,
                                   stream=stream, **pkw)
            kern, pwarm, piters, prep = paths[key]
            pms = time_protocol(pstep, stream, flush, warmup=pwarm, iters=piters, repeats=prep,
                                trim=1 if piters >= 10 else 0)[0]
            pab = algorithmic_bytes_bwd(pw)
            per_step[key] = {"workload": pw.name, "ms_per_call": pms, "tokens_per_s": 2 * pw.tokens / (pms * 1e-3),
                             "algorithmic_bytes": pab, "frac_hbm": pab / (pms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                             "workspace_bytes": pws.numel(), "kernels": kern}
            if key != "tiny_f32":   # the block form in eight time segments
                del pws
                pws = torch.empty(bd.bdgdn_bwd_train_workspace_segmented(pdesc, pcu, 8), dtype=torch.uint8,
                                  device=dev)
                psms = time_protocol(pstep, stream, flush, warmup=pwarm, iters=piters, repeats=prep,
                                     trim=1 if piters >= 10 else 0)[0]
                per_step[key]["segmented"] = {"segments": 8, "workspace_bytes": pws.numel(), "ms_per_call": psms,
                                              "tokens_per_s": 2 * pw.tokens / (psms * 1e-3)}
            del pin, pws, pgrads
            torch.cuda.empty_cache()
        result["backward"]["other_workloads"] = per_step

    if "blocks" in only:
        # forward and backward across diffusion-block sizes at one sequence of 4096 clean +
        # 4096 noisy tokens, 16 heads, d = 128 (the shape of the paper's route comparison)
        sin = {k_: v_.to(dev) for k_, v_ in W.make_custom_train(1, 4096, 16, 16, 128, 128, "bf16", seed=91).items()}
        sargs = [sin[k_] for k_ in ("q", "k", "v", "g", "beta", "qn", "kn", "vn", "gn", "betan")]
        sshape = (1, 4096, 16, 128)
        sdo = torch.randn(sshape, generator=torch.Generator(device=dev).manual_seed(10), device=dev)
        sdon = torch.randn(sshape, generator=torch.Generator(device=dev).manual_seed(11), device=dev)
        so, son = torch.empty(sshape, device=dev), torch.empty(sshape, device=dev)
        sweep = {}
        for L in SWEEP_BLOCKS:
            sdesc = bd.make_fwd_desc(sin["q"], sin["v"], block=L, out_dtype=torch.float32)
            fws = bd.bdgdn_fwd_train_workspace(sdesc)
            bws = torch.empty(max(256, bd.bdgdn_bwd_train_workspace(sdesc)), dtype=torch.uint8, device=dev)
            sgrads = bd.bdgdn_bwd_train(*sargs, sdo, sdon, block=L, workspace=bws)

            def sfstep(L=L):
                bd.bdgdn_fwd_train(*sargs, block=L, o=so, on=son, stream=stream)

            def sbstep(L=L):
                bd.bdgdn_bwd_train(*sargs, sdo, sdon, block=L, workspace=bws, grads=sgrads, stream=stream)
            sfms = time_protocol(sfstep, stream, flush)[0]
            sbms = time_protocol(sbstep, stream, flush, iters=5 if L < 8 else 10, repeats=3, trim=1)[0]
            sweep[str(L)] = {
                "fwd_ms": sfms, "bwd_ms": sbms, "fwd_workspace_bytes": fws, "bwd_workspace_bytes": bws.numel(),
                "fwd_schedule": ("bdgdn_fwd_pipelined_small_kernel (32-position clean chunks, %d noisy blocks each)"
                                 % (32 // L)) if L <= 8 else "bdgdn_fwd_pipelined_kernel (one block per step)"}
            del bws, sgrads
            torch.cuda.empty_cache()
            print(f"blocks L={L}: fwd {sfms:.3f} ms, bwd {sbms:.3f} ms", file=sys.stderr, flush=True)
        result["blocks"] = {"workload": "sweep_bf16_b1_t4096_h16_d128 (fp32 outputs, fp32 upstream gradients)",
                            "by_block": sweep}
        del sin, sargs, sdo, sdon, so, son
        torch.cuda.empty_cache()

    if "shortconv" in only:
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
        fms = time_protocol(fstep, stream, flush)[0]
        bms = time_protocol(bstep, stream, flush)[0]
        fbytes, bbytes = algorithmic_bytes_conv(cw, backward=False), algorithmic_bytes_conv(cw, backward=True)
        result["shortconv"] = {
            "workload": cw.name,
            "fwd": {"us_per_call": fms * 1e3, "gb_per_s": fbytes / (fms * 1e-3) / 1e9,
                    "frac_hbm": fbytes / (fms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": fbytes,
                    "kernel": "bdgdn_shortconv_fwd_kernel"},
            "bwd": {"us_per_call": bms * 1e3, "gb_per_s": bbytes / (bms * 1e-3) / 1e9,
                    "frac_hbm": bbytes / (bms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": bbytes,
                    "kernel": "bdgdn_shortconv_bwd_kernel + bdgdn_shortconv_reduce_kernel"}}

    if "cpu" in only:
        result["cpu_baseline"] = cpu_baseline(w, inp)
    print(json.dumps(result))


def cpu_baseline(w, inp):
    """The fp64 oracle, as it stands, on the host: the whole training workload (every
    (sequence, v-head) unit, clean and noisy streams) over up to 16 threads (the host share
    of one GPU), and a one-thread run over a sample of 4 units."""
    import oracle
    threads = max(1, min(os.cpu_count() or 1, 16))
    keys = ("q", "k", "v", "g", "beta")
    arr = {k: inp[k].double().numpy() for k in inp if k != "lengths"}
    scale = 1.0 / math.sqrt(w.d_k)
    oracle.set_threads(threads)
    used = oracle.max_threads()
    t0 = time.perf_counter()
    oracle.fwd_train(*[arr[k] for k in keys], *[arr[k + "n"] for k in keys], block=w.block, scale=scale,
                     want_ht=False)
    dt = time.perf_counter() - t0
    tokens = 2 * w.tokens
    # one thread, a sample of 4 (sequence, v-head) units: sequence 0, heads 0-3
    sample = {k: arr[k][:1, :, :4] for k in arr}
    oracle.set_threads(1)
    t1 = time.perf_counter()
    oracle.fwd_train(*[sample[k] for k in keys], *[sample[k + "n"] for k in keys], block=w.block, scale=scale,
                     want_ht=False)
    dt1 = time.perf_counter() - t1
    oracle.set_threads(threads)
    unit_tokens = 2 * w.seqlen   # clean + noisy tokens of one (sequence, v-head) unit
    return {"value": tokens / dt, "unit": "tokens/s", "cores": used, "kind": "oracle", "seconds": dt,
            "host_cpu_count": os.cpu_count(),
            "sample": f"the whole workload: {w.batch} sequences x {w.h_v} v-heads x "
                      f"({w.seqlen} clean + {w.seqlen} noisy) tokens in fp64 over {used} threads; "
                      "value = tokens / wall time",
            "one_thread": {"units": 4, "seconds": dt1,
                           "value": 4 * unit_tokens / w.h_v / dt1,
                           "unit": "tokens/s (a token = all 16 heads of one position, scaled from 4 heads)",
                           "sample": "sequence 0, v-heads 0-3, 4096 clean + 4096 noisy tokens, one thread"}}


if __name__ == "__main__":
    main()
