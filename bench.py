#!/usr/bin/env python3
"""Throughput of the integer relative-position MHSA block on one MI355X.

A step is one call of the whole block (Q|K|V and position projections, rank-1
bias terms, the attention core with the integer softmax, A.V and the output
projection) on the long-form workload: B=1, T=2500 frames (200 s of audio at
80 ms per frame), d_model=1024, H=8, d_k=128, int8 inputs with heavy-tailed x.
Inputs are resident in HBM before the timed region.

Prints one JSON line.  ``value`` is algorithmic int8 tera-operations per second
(2 x the multiply-accumulates the method needs: projections of the valid rows,
the position projection once, and content + position + A.V over the valid
(query, key) pairs), timed over K steps with no events inside the region, after
untimed calls for --settle-s seconds (the clocks' loaded state) and W warm-up steps.
``stage_ms`` comes from a second pass of steps with per-kernel HIP events on the
launch stream.  ``roofline`` reports the attention core against the dense INT8 MFMA
peak, its average duration measured between two HIP events around back-to-back
launches of the core on the last step's workspace.  ``cpu_baseline`` is the CPU oracle
on the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "int8 rel-pos attention TOPS & encoder frames/sec (T=2500, d=1024, H=8), % INT8 peak"
INT8_PEAK_TOPS = 5000.0  # MI355X dense INT8 MFMA, 5.0 POP/s
HBM_PEAK_GBS = 8000.0


def algorithmic_macs(B, T, d, H, dk, lengths):
    """MACs the method needs for one call: Eq. 7 projections of the valid rows (Q, K,
    V and output), the position projection of the 2T-1 table rows, and the content,
    position and A.V contractions over the valid (query, key) pairs."""
    sl = int(np.sum(lengths))
    sl2 = int(np.sum(np.asarray(lengths, dtype=np.int64) ** 2))
    proj = 4 * sl * d * d
    pos = (2 * T - 1) * d * d
    attn = 3 * H * dk * sl2
    return proj, pos, attn


def kernel_source_hash(csrc: str = None) -> str:
    """Hash of the kernel sources (the HIP files and their shared header; the C-ABI
    glue in ipk_api.cpp does not change what a kernel reads or writes), with comments
    and whitespace left out: only a change to the code itself invalidates a
    measurement taken on it."""
    import glob
    import hashlib
    import re

    h = hashlib.sha256()
    csrc = csrc or os.path.join(ROOT, "paper_2609_30846_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))):
        with open(f, encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        code = " ".join(text.split())
        h.update(os.path.basename(f).encode() + b"\0" + code.encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter measurement
    (FETCH_SIZE + WRITE_SIZE, each scaled by the same counter on a plain copy of
    known size), or None when the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--settle-s", dest="settle_s", type=float, default=0.3,
                    help="seconds of untimed calls before the warm-up steps (clock ramp)")
    ap.add_argument("--workload", default="longform")
    ap.add_argument("--regime", default="literal", choices=["literal", "calibrated"])
    ap.add_argument("--cpu-baseline", dest="cpu_baseline", action="store_true", default=True)
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline", action="store_false")
    ap.add_argument("--no-variants", dest="variants", action="store_false", default=True,
                    help="skip the kept-position-projection and MHSA-module passes")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device (reference kernel for the HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(utterances and heads would shard without exchange; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n}), flush=True)
        return

    from paper_2609_30846_amd import ipk
    from workloads import make_conv, make_ffn, make_residual, make_workload

    ipk.load()  # fails loudly when the HIP library is missing
    wl = make_workload(args.workload, args.regime)
    blk = wl.blocks[0]
    sh = blk.shape
    B, T, d, H, dk = blk.x.shape[0], blk.T, sh.d_model, sh.n_heads, sh.d_k
    lengths = blk.lengths

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    mod = ipk.RelPosAttn.from_block(blk, device=dev)
    x = torch.from_numpy(blk.x).to(dev)
    pe = torch.from_numpy(blk.pos_table).to(dev)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream()

    # the GPU's clocks climb over the first ~0.1 s of sustained load: a short run from
    # idle (20 steps after 5) reads ~10 % slower than the same steps after 0.2 s of
    # load, and does not change once the load has lasted that long.  Untimed calls run
    # for settle_s seconds first, then the W warm-up steps, so the K timed steps see
    # the steady state a serving loop runs at.
    settle_steps, t_settle = 0, time.perf_counter()
    while time.perf_counter() - t_settle < args.settle_s:
        for _ in range(100):
            mod(x, pe, lengths=lengths, y=y, stream=stream)
        settle_steps += 100
        torch.cuda.synchronize()
    settle_s = time.perf_counter() - t_settle
    for _ in range(args.warmup):
        mod(x, pe, lengths=lengths, y=y, stream=stream)
    torch.cuda.synchronize()

    # timed region: K whole steps, bracketed by synchronizations; no per-kernel
    # events inside it (recording them costs the stream about as much as a kernel)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        mod(x, pe, lengths=lengths, y=y, stream=stream)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps

    # stage pass: more steps (at most 200) with per-kernel HIP events recorded by the
    # library on the launch stream (event i at the start of kernel i, the last one at
    # the end of the last kernel); stage_ms comes from it
    nst = ipk.NUM_STAGES
    n_stage = min(args.steps, 200)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nst + 1)] for _ in range(n_stage)]
    for row in evs:
        for e in row:
            e.record(stream)
    torch.cuda.synchronize()
    for k in range(n_stage):
        ipk.ipk_relpos_attn_record_stages(mod.handle, evs[k])
        mod(x, pe, lengths=lengths, y=y, stream=stream)
    torch.cuda.synchronize()

    stage_names = ["projections", "attention", "out_projection"]
    stage_ms = np.zeros(nst)
    for row in evs:
        for i in range(nst):
            stage_ms[i] += row[i].elapsed_time(row[i + 1])
    stage_ms /= n_stage

    # the attention core alone, for the roofline: the library launches the last step's
    # core n_stage more times back to back on its workspace, with one event before and
    # one after the launches.  An event on each kernel stretches the interval it
    # brackets by the stream's event work (the stage pass above reads the core ~9 us
    # longer than a kernel trace of the same run); back-to-back launches carry only the
    # dispatch boundary before each kernel, as the trace does.
    mod.repeat_core(5, stream)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    mod.repeat_core(n_stage, stream)
    c1.record(stream)
    torch.cuda.synchronize()
    core_ms = c0.elapsed_time(c1) / n_stage

    # two variants on the same input, timed like the main region over n_stage steps:
    # the position projection kept on the handle (the paper computes q_P offline), and
    # the MHSA module of Eq. 2 (integer LayerNorm, the block, the residual add)
    def timed(fn, n):
        # settled like the main region: building a variant's inputs leaves the GPU idle
        t_s = time.perf_counter()
        while time.perf_counter() - t_s < args.settle_s:
            for _ in range(20):
                fn()
            torch.cuda.synchronize()
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    if args.variants:
        y_kept = torch.empty_like(x)
        mod.cache_positions(pe, stream=stream)
        ms_kept = timed(lambda: mod(x, None, lengths=lengths, y=y_kept, stream=stream), n_stage)
        z2 = torch.empty_like(x)
        mod.set_residual_from(make_residual(blk, args.regime, seed=wl.seed + 1))
        ms_module = timed(lambda: mod.residual(x, pe, lengths=lengths, z2=z2, stream=stream), n_stage)
        y_kept_matches = bool(torch.equal(y_kept, y))
        # the feed-forward module of Eq. 1 (LayerNorm, W1 with the integer Swish, W2
        # with the half-step residual) on the same rows, d_ff = 4 d
        ffn_par = make_ffn(d, args.regime, seed=wl.seed + 2, S_z=blk.scales["S_x"])
        ffn = ipk.FeedForward(ffn_par, max_rows=B * T, device=dev)
        z_ffn = torch.empty_like(x)
        ms_ffn = timed(lambda: ffn(x, z_out=z_ffn, stream=stream), n_stage)
        ffn_ops = 2 * 2 * B * T * d * ffn_par.d_ff
        ffn.close()
        # the convolution module of Eq. 3 / Eq. 5 (LayerNorm, PW1, GLU + depthwise + INT16
        # BatchNorm + Swish, PW2 with the residual) on the same utterances
        conv_par = make_conv(d, args.regime, seed=wl.seed + 3, S_z=blk.scales["S_x"])
        conv = ipk.ConvModule(conv_par, max_batch=B, max_T=T, device=dev)
        z_conv = torch.empty_like(x)
        ms_conv = timed(lambda: conv(x, lengths=lengths, z_out=z_conv, stream=stream), n_stage)
        conv_ops = 2 * B * T * d * (2 * d + d) + 2 * 9 * B * T * d
        conv.close()
        # the 24-block stack workload (B = 8, T = 500): each block's int8 output feeds the
        # next block; encoder frames per second over whole 24-block passes
        swl = make_workload("stack", args.regime)
        sblk = swl.blocks
        smods = [ipk.RelPosAttn.from_block(b_, device=dev) for b_ in sblk]
        sx = torch.from_numpy(sblk[0].x).to(dev)
        spe = torch.from_numpy(sblk[0].pos_table).to(dev)
        sbuf = [torch.empty_like(sx), torch.empty_like(sx)]

        def stack_pass():
            cur = sx
            for i_, (m_, b_) in enumerate(zip(smods, sblk)):
                m_(cur, spe, lengths=b_.lengths, y=sbuf[i_ % 2], stream=stream)
                cur = sbuf[i_ % 2]

        n_stack = max(1, min(20, n_stage // 10))
        ms_stack = timed(stack_pass, n_stack)
        sB, sT = sblk[0].x.shape[0], sblk[0].T
        s_ops = 0
        for b_ in sblk:
            p_, q_, r_ = algorithmic_macs(sB, sT, d, H, dk, b_.lengths)
            s_ops += 2 * (p_ + q_ + r_)
        for m_ in smods:
            m_.close()
        # the other single-block workloads, timed like the variants: frames per second of
        # whole calls (parity of each is covered by the GPU tests).  The benchmarked
        # workload is timed once more in the other scale regime: the kernels do the same
        # work whatever the values, and at T = 2500 the literal grids leave almost every
        # softmax row without mass (all codes 0), so the calibrated regime shows the time
        # on an input whose attention weights are not degenerate.
        other = {}
        alt = "calibrated" if args.regime == "literal" else "literal"
        for wname, wreg in (("tiny", args.regime), ("parakeet", args.regime), ("batched", args.regime),
                            (args.workload, alt)):
            owl = make_workload(wname, wreg)
            ob = owl.blocks[0]
            om = ipk.RelPosAttn.from_block(ob, device=dev)
            ox = torch.from_numpy(ob.x).to(dev)
            ope = torch.from_numpy(ob.pos_table).to(dev)
            oy = torch.empty_like(ox)
            oms = timed(lambda: om(ox, ope, lengths=ob.lengths, y=oy, stream=stream), n_stage)
            osh = ob.shape
            p_, q_, r_ = algorithmic_macs(ob.x.shape[0], ob.T, osh.d_model, osh.n_heads, osh.d_k, ob.lengths)
            otops = 2 * (p_ + q_ + r_) / (oms * 1e-3) / 1e12
            other[wname if wreg == args.regime else f"{wname}_{wreg}"] = {
                "workload": f"{wname}: B={ob.x.shape[0]} T={ob.T} d_model={osh.d_model} H={osh.n_heads} "
                            f"d_k={osh.d_k}, {wreg} scales, seed {owl.seed}",
                "ms_per_call": round(oms, 5),
                "frames_per_s": round(float(np.sum(ob.lengths)) / (oms * 1e-3), 1),
                "tops": round(otops, 3),
                "pct_int8_peak": round(100.0 * otops / INT8_PEAK_TOPS, 3),
            }
            om.close()

    proj, pos, attn = algorithmic_macs(B, T, d, H, dk, lengths)
    ops = 2 * (proj + pos + attn)
    tops = ops / (ms_step * 1e-3) / 1e12
    frames = float(np.sum(lengths)) / (ms_step * 1e-3)
    attn_tops = 2 * attn / (core_ms * 1e-3) / 1e12

    rec = {
        "metric": METRIC,
        "value": round(tops, 3),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: B={B} T={T} d_model={d} H={H} d_k={dk}, int8 block, "
                        f"{args.regime} scales, seed {wl.seed}",
            "global_batch": B,
            "seq_len": T,
            "parallelism": "none (1 GPU)",
        },
        "frames_per_s": round(frames, 1),
        "pct_int8_peak": round(100.0 * tops / INT8_PEAK_TOPS, 3),
        "algorithmic_ops": ops,
        "stage_ms": {n: round(float(v), 5) for n, v in zip(stage_names, stage_ms)},
        "stage_timing": f"separate pass of {n_stage} steps with per-kernel HIP events on the launch stream",
        "wall_s_timed_region": round(wall, 4),
        "settle": {"seconds": round(settle_s, 3), "steps": settle_steps,
                   "note": "untimed calls before the warm-up steps, until the clocks reach their loaded state"},
        "variants": None if not args.variants else {
            "kept_position_projection": {
                "ms_per_step": round(ms_kept, 5),
                "frames_per_s": round(float(np.sum(lengths)) / (ms_kept * 1e-3), 1),
                "tops_without_position_projection": round(2 * (proj + attn) / (ms_kept * 1e-3) / 1e12, 3),
                "output_equals_per_call_table": y_kept_matches,
            },
            "mhsa_module_layernorm_residual": {
                "ms_per_step": round(ms_module, 5),
                "frames_per_s": round(float(np.sum(lengths)) / (ms_module * 1e-3), 1),
            },
            "ffn_module_minimax_swish": {
                "ms_per_step": round(ms_ffn, 5),
                "rows": B * T,
                "d_ff": ffn_par.d_ff,
                "tops": round(ffn_ops / (ms_ffn * 1e-3) / 1e12, 3),
                "pct_int8_peak": round(100.0 * ffn_ops / (ms_ffn * 1e-3) / 1e12 / INT8_PEAK_TOPS, 3),
            },
            "conv_module_int16_batchnorm": {
                "ms_per_step": round(ms_conv, 5),
                "frames_per_s": round(float(np.sum(lengths)) / (ms_conv * 1e-3), 1),
                "tops": round(conv_ops / (ms_conv * 1e-3) / 1e12, 3),
            },
            "stack_24_blocks": {
                "workload": f"stack: 24 blocks, B={sB} T={sT} d_model={d} H={H}, {args.regime} scales, seed {swl.seed}",
                "ms_per_pass": round(ms_stack, 4),
                "encoder_frames_per_s": round(sB * sT / (ms_stack * 1e-3), 1),
                "tops": round(s_ops / (ms_stack * 1e-3) / 1e12, 3),
                "passes_timed": n_stack,
            },
            "other_workloads": other,
            "timing": f"{n_stage} steps each between two HIP events, after {args.settle_s} s of untimed calls and 5 warm-up steps",
        },
        "roofline": {
            "kernel": "relpos_attn_core",
            "bound": "mfma",
            "achieved": round(attn_tops, 3),
            "peak": INT8_PEAK_TOPS,
            "unit": "TOP/s",
            "frac": round(attn_tops / INT8_PEAK_TOPS, 5),
            "traffic": measured_traffic("relpos_attn_core"),
            "kernel_us": round(1000 * core_ms, 3),
            "timing": f"{n_stage} back-to-back launches of the core on the step's workspace between two HIP events",
        },
    }

    if args.cpu_baseline:
        from oracle import core

        ncores = len(os.sched_getaffinity(0))
        os.environ.setdefault("OMP_NUM_THREADS", str(ncores))
        t1 = time.perf_counter()
        y_ref = core.relpos_attn(blk)
        cpu_s = time.perf_counter() - t1
        exact = bool(np.array_equal(y_ref, y.cpu().numpy()))
        rec["cpu_baseline"] = {
            "value": round(ops / cpu_s / 1e12, 6),
            "unit": "TOPS",
            "cores": core.num_threads(),
            "kind": "oracle",
            "sample": f"one whole call of the same workload ({args.workload}, B={B}, T={T}); "
                      f"{cpu_s:.2f} s; output bit-exact vs GPU: {exact}",
        }
        # the oracle on one thread, one call of the Parakeet-scale block
        pk = make_workload("parakeet", args.regime).blocks[0]
        nthreads = core.num_threads()
        core.set_num_threads(1)
        t1 = time.perf_counter()
        core.relpos_attn(pk)
        pk_s = time.perf_counter() - t1
        core.set_num_threads(nthreads)
        pk_p, pk_q, pk_r = algorithmic_macs(1, pk.T, pk.shape.d_model, pk.shape.n_heads, pk.shape.d_k, pk.lengths)
        rec["cpu_baseline"]["single_thread"] = {
            "workload": f"parakeet: B=1 T={pk.T} d_model={pk.shape.d_model} H={pk.shape.n_heads}",
            "seconds_per_call": round(pk_s, 4),
            "frames_per_s": round(float(np.sum(pk.lengths)) / pk_s, 1),
            "tops": round(2 * (pk_p + pk_q + pk_r) / pk_s / 1e12, 6),
            "cores": 1,
        }
        # the integer block against the float64 block of Eq. 8-9 on the same dequantized
        # inputs, relative L2 per workload, as the oracle measures it (committed analysis)
        gap_path = os.path.join(ROOT, "oracle", "fp_gap_results.json")
        if os.path.exists(gap_path):
            with open(gap_path) as fh:
                gap = json.load(fh)
            rec["oracle_vs_fp_block"] = {
                "rel_l2": {k: round(v["rel_l2"], 4) for k, v in gap["configs"].items()},
                "regime": gap["regime"],
                "target": 0.02,
                "source": "oracle/fp_gap.py (written by python -m oracle.fp_gap)",
            }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
