#!/usr/bin/env python3
"""Benchmark: positions evaluated per second (policy + value) on one MI355X.

One step is one az_eval_batch call over a whole batch of seeded synthetic
positions already resident in device memory: the fused stem + residual tower +
heads + legal-move softmax + tanh value kernel.  Default workload: the 20-block,
128-filter network (5,944,523 parameters) with int8 residual convolutions,
batch 1024.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--tiling 0|1|2|3]

Before the W warm-up steps, untimed calls run for 0.3 s so that the timed
region sees the GPU at its working clock rather than its ramp from idle.

Prints one JSON line on stdout.  --gpus N with N > 1 exits with a message: this
library evaluates on one GPU (positions are independent; a multi-GPU server
would run one handle per GPU on its share of the batch).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import azgen  # noqa: E402

CALIB = os.path.join(ROOT, "tests", "golden", "calib_net20x128_seed1004.npz")
DEPLOYED_SCALES = os.path.join(ROOT, "tests", "golden", "scales_deployed14x160_seed1006.npz")
CSRC = os.path.join(ROOT, "paper_2609_37447_amd", "csrc")


def is_deployed(shape):
    return getattr(shape, "policy_head", "planes") == "fromto"


def kernel_sources(shape, dtype):
    """The source files the kernel of a workload is compiled from."""
    if dtype == "f32":
        main = "az_kernels_f32.hip"
    else:
        main = "az_dep_kernel.h" if is_deployed(shape) else "az_kernels_mfma.hip"
    return [os.path.join(CSRC, f) for f in (main, "az_mfma_common.h", "az_internal.h")]


def kernel_sha(shape, dtype):
    """sha256 over the kernel's source files, in order."""
    h = hashlib.sha256()
    for f in kernel_sources(shape, dtype):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


# Counters of the fused kernel from rocprofv3 --pmc passes (profiles/ holds each
# summary with its commands): HBM traffic as FETCH_SIZE and WRITE_SIZE (KiB per
# dispatch), scaled by what the same counters read for a plain copy kernel of
# known size (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0), and the MFMA busy fraction
# SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE per XCD x 1024 SIMDs).  An entry
# holds for the kernel sources it was taken on only (kernel_sha): any other
# source reports null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
# (workload, tiling, batch): (kernel_sha, FETCH_SIZE KiB, WRITE_SIZE KiB, MFMA busy fraction)
COUNTERS = {
    ("net20x128_int8_b1024", 1, 1024): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 29227.8, 18696.0, 0.5293),
    ("net20x128_int8_b1024", 3, 1024): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 35898.7, 18704.0, 0.5926),
    ("net20x128_int8_b1024", 2, 64): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 24520.8, 1426.0, 0.0997),
    ("net20x128_bf16_b1024", 1, 1024): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 52089.3, 18696.0, 0.6570),
    ("net20x128_bf16_b256", 2, 256): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 48114.3, 4680.0, 0.5021),
    ("net20x128_bf16_b32", 2, 32): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 47036.3, 585.0, 0.0642),
    ("net20x128_fp8_b1024", 1, 1024): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 29304.8, 18696.0, 0.4522),
    ("net24x256_bf16_b1024", 1, 1024): ("7f52e69d56ea062db334372d81332f33ea5f60b0334a17c53cccb4fe8b263aa2", 449866.8, 18704.0, 0.7632),
    ("deployed14x160_int8_b1024", 1, 1024): ("5c99920884a7ae6b6f4b20e9d3a337117dccd2719057c9c6ce14ade7bafdd416", 36532.0, 7552.0, 0.4958),
    ("deployed14x160_int8_b1024", 2, 64): ("5c99920884a7ae6b6f4b20e9d3a337117dccd2719057c9c6ce14ade7bafdd416", 29637.4, 472.0, 0.0743),
    ("deployed14x160_bf16_b1024", 2, 1024): ("5c99920884a7ae6b6f4b20e9d3a337117dccd2719057c9c6ce14ade7bafdd416", 222194.4, 7552.0, 0.4100),
    ("tiny_2x32_f32_b16", 0, 16): ("71a6c293790d7c1ed568fe2a55efb4c240b4ffe70594008f8c4af0194bf047ae", 1010.5, 292.5, 0.0000),
}

# MI355X published dense peaks (FLOP/s) at 2.4 GHz, 256 CUs.
PEAK = {"bf16": 2.5e15, "int8": 5.0e15, "fp8": 5.0e15, "f32_vec": 157.3e12, "f64_vec": 78.6e12}


def mac_counts(shape):
    """Algorithmic multiply-accumulates per position, by layer group (no padding,
    no halo taps, no masked-out logits)."""
    C, F, P, H, NB = shape.in_planes, shape.filters, shape.policy_planes, shape.value_hidden, shape.blocks
    if not is_deployed(shape):
        return {
            "stem": 64 * F * C * 9,
            "tower": 2 * NB * 64 * F * F * 9,
            "head_conv": 64 * F * (P + 1),
            "value_fc": 64 * H + H,
        }
    g = F // 4 if shape.pool_every else 0
    tower, pool_fc = 0, 0
    for j in range(NB):
        pool = shape.is_pool_block(j)
        tower += 64 * F * F * 9 + 64 * F * (F - g if pool else F) * 9
        pool_fc += (F - g) * 2 * g if pool else 0
    D, V = shape.token_dim, shape.value_channels
    return {
        "stem": 64 * F * C * 9,
        "tower": tower,
        "pool_fc": pool_fc,
        "head_conv": 64 * (D + V) * F + 2 * 64 * D * D + 64 * 64 * D + 8 * 4 * D,
        "value_fc": H * V * 64 + 3 * H,
    }


def roofline_peak(shape, dtype):
    """Composite peak: total FLOP / sum_l FLOP_l / peak(dtype_l), each layer group
    priced at the unit it runs on."""
    m = mac_counts(shape)
    if dtype == "f32":
        unit = {k: "f32_vec" for k in m}
    else:
        tower = {"bf16": "bf16", "int8": "int8", "fp8": "fp8"}[dtype]
        unit = {"stem": "bf16", "tower": tower, "head_conv": "bf16", "value_fc": "f32_vec", "pool_fc": "f64_vec"}
    flop = {k: 2.0 * v for k, v in m.items()}
    t_floor = sum(flop[k] / PEAK[unit[k]] for k in flop)
    return sum(flop.values()), sum(flop.values()) / t_floor


def counters_for(w, tiling, B):
    """(scaled HBM bytes per launch, MFMA busy fraction), or (None, None) without
    counters taken on this exact kernel source."""
    e = COUNTERS.get((w.name, tiling, B))
    if e is None or kernel_sha(w.shape, w.dtype) != e[0]:
        return None, None
    return (e[1] * FETCH_SCALE + e[2] * WRITE_SCALE) * 1024.0, e[3]


def load_scales(w):
    if w.dtype not in ("int8", "fp8"):
        return None, None
    if is_deployed(w.shape):
        if w.name != "deployed14x160_int8_b1024":
            raise SystemExit(f"no stored scales for workload {w.name}")
        d = np.load(DEPLOYED_SCALES, allow_pickle=False)
        return d["w_scales_int8"], d["act_scales_int8"]
    if w.shape != azgen.WORKLOADS["net20x128_int8_b1024"].shape or w.index != 4:
        raise SystemExit(f"no stored calibration for workload {w.name}")
    d = np.load(CALIB, allow_pickle=False)
    return d[f"w_scales_{w.dtype}"], d[f"act_scales_{w.dtype}"]


def cpu_baseline(w, blob, ws, acs, planes, legal, budget_s=12.0, chunk=64):
    """The oracle (float64 CPU forward; quantised mode for int8/fp8) on a bounded
    sample of the same workload, chunks of `chunk` positions until budget_s."""
    from threadpoolctl import threadpool_info

    from oracle import az_oracle as O
    from oracle import deployed as OD
    done, t0 = 0, time.perf_counter()
    while True:
        s = done % planes.shape[0]
        pl, lg = planes[s:s + chunk], legal[s:s + chunk]
        if is_deployed(w.shape):
            if w.dtype == "int8":
                OD.forward_quant(w.shape, blob, ws, acs, pl, lg)
            else:
                OD.forward(w.shape, blob, pl, lg)
        elif w.dtype in ("int8", "fp8"):
            O.forward_quant(w.shape, blob, ws, acs, w.dtype, pl, lg)
        else:
            O.forward(w.shape, blob, pl, lg)
        done += pl.shape[0]
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": done / el, "unit": "positions/s", "cores": int(threads), "kind": "oracle",
            "host_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
            "sample": f"{done} positions of the seeded batch in chunks of {chunk}, "
                      f"{el:.1f} s, float64 numpy/BLAS on {threads} threads"
                      + (f" ({w.dtype} quantised network, the plain definition)" if w.dtype in ("int8", "fp8") else "")}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


PIPELINE_LEGS = ("dense_1w4s", "compact_1w4s", "compact_4w2s_b320", "compact_4w2s_b320_graphs")
SETTLE_S = 0.3


def pipeline_rates(az, net, w, planes, legal, batches=100, warm=10, max_legal=256, legs=PIPELINE_LEGS):
    """Positions/s through az_pipeline, host buffers to host buffers: inputs
    copied from pinned memory, evaluation, outputs back in host memory.  The
    library's own worker threads (az_pipeline_drive) share one pipeline; each
    owns some of its slots and keeps them in flight round-robin (wait for the
    slot, resubmit it).  Three set-ups: dense policy, one worker with four slots
    of the full batch; the same with the compact legal-move policy; and four
    workers with two outstanding batches of 320 each, compact (the paper's
    retained actor topology, Section 5.2), once on the pipeline's three shared
    streams and once with each slot replaying its own captured graph.  Each
    worker runs `warm` batches untimed, then `batches` timed ones.  Measured
    after the timed region; never the headline value."""
    B = w.batch
    n_moves = w.shape.n_moves
    res = {"max_legal": max_legal, "driver": "az_pipeline_drive (native worker threads)",
           "bytes_in_per_position": int(planes[0].nbytes + legal[0].nbytes),
           "bytes_out_per_position_dense": int((n_moves + 1) * 4),
           "bytes_out_per_position_compact": int((max_legal + 2) * 4)}
    has = legal.any(axis=1)
    setups = (("dense_1w4s", 1, 4, B, 0, False), ("compact_1w4s", 1, 4, B, max_legal, False),
              ("compact_4w2s_b320", 4, 2, min(320, B), max_legal, False),
              ("compact_4w2s_b320_graphs", 4, 2, min(320, B), max_legal, True))
    for leg, workers, per_worker, batch, K, graphs in setups:
        if leg not in legs:
            continue
        name = leg if "b320" in leg else "%s_b%d" % (leg, B)
        slots = workers * per_worker
        spec = az.spec_from_shape(w.shape, batch)
        pipe = az.Pipeline(net, spec, batch, slots, graphs, max_legal=K)
        try:
            for k in range(slots):
                pipe.views[k][0][:] = planes[:batch]
                pipe.views[k][1][:] = legal[:batch]
            dt = pipe.drive(workers, per_worker, batch, warm, batches)
            # every legal move fits in max_legal here, so compact rows sum to one too
            v = pipe.views[slots - 1]
            assert np.all(np.abs(v[2][:batch][has[:batch]].sum(axis=1) - 1.0) < 1e-3), "pipeline outputs invalid"
        finally:
            pipe.close()
        res[name] = {"positions_per_s": workers * batches * batch / dt, "batches": workers * batches,
                     "warmup_batches": workers * warm}
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="net20x128_int8_b1024", choices=sorted(azgen.WORKLOADS))
    ap.add_argument("--tiling", type=int, default=0, choices=(0, 1, 2, 3))
    ap.add_argument("--batch", type=int, default=0,
                    help="evaluate this many positions per step instead of the workload's batch "
                         "(e.g. 64 for the interactive regime: one outstanding batch of 64)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay measurement")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the host-buffer (PCIe-inclusive) pipeline measurement")
    ap.add_argument("--pipeline-batches", type=int, default=100,
                    help="timed batches per worker in each pipeline set-up (after 10 untimed)")
    ap.add_argument("--pipeline-legs", default=",".join(PIPELINE_LEGS),
                    help="comma-separated pipeline set-ups to measure: " + ", ".join(PIPELINE_LEGS))
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: --gpus {args.gpus} (WORLD_SIZE {world}) requested, but this library "
              "evaluates on one GPU; run one process per GPU with its own share of the batch.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_37447_amd as az

    w = azgen.WORKLOADS[args.workload]
    blob = azgen.workload_weights(w)
    ws, acs = load_scales(w)
    B = args.batch or w.batch
    planes, legal = azgen.make_inputs(w, n=B)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    net = az.az_net_load(az.spec_from_shape(w.shape, B), blob, w.dtype, ws, acs)
    if args.tiling:
        az.az_net_set_tiling(net, args.tiling)
    tiling = az.az_net_tiling_for(net, B)
    pl = torch.from_numpy(planes).to(dev)
    lg = torch.from_numpy(legal).to(dev)
    pol = torch.empty((B, w.shape.n_moves), device=dev)
    val = torch.empty((B,), device=dev)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    def step_on(stream_handle):
        az.az_eval_batch(net, pl.data_ptr(), lg.data_ptr(), B, pol.data_ptr(), val.data_ptr(), stream_handle)

    def step():
        step_on(sp)

    # Before the warm-up steps: untimed calls for at least SETTLE_S seconds.  An
    # idle GPU needs tens of milliseconds of load to reach its working clock, so
    # a short timed region right after a few warm-up steps measures that ramp
    # (20 steps after 5 warm-up ones timed 398 us per batch where 200 after 20
    # timed 334 us on the same box).
    t_settle = time.perf_counter()
    n_settle = 0
    while True:
        for _ in range(8):
            step()
        n_settle += 8
        torch.cuda.synchronize()
        if time.perf_counter() - t_settle >= SETTLE_S:
            break
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    # sanity: every policy row sums to one, values in range
    s = pol.sum(dim=1)
    ok = bool(((s - 1).abs() < 1e-3).all()) and bool((val.abs() <= 1).all())

    # Outside the timed region: per-call device time (each call between its own
    # events) and the replay time of the call captured in a HIP graph.
    pairs = []
    for _ in range(min(args.steps, 100)):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        pairs.append((a, b))
    torch.cuda.synchronize()
    lat = np.array([a.elapsed_time(b) * 1000.0 for a, b in pairs])
    graph_us = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step_on(torch.cuda.current_stream().cuda_stream)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step_on(torch.cuda.current_stream().cuda_stream)
        g.replay()
        torch.cuda.synchronize()
        n_rep = min(args.steps, 100)
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(n_rep):
            g.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) * 1000.0 / n_rep
        del g
    pipeline = None if (args.no_pipeline or B != w.batch) else pipeline_rates(
        az, net, w, planes, legal, args.pipeline_batches, legs=tuple(args.pipeline_legs.split(",")))
    az.az_net_free(net)

    flop_pos, peak = roofline_peak(w.shape, w.dtype)
    achieved = flop_pos * B / (ms * 1e-3)
    traffic, mfma_busy = counters_for(w, tiling, B)
    out = {
        "metric": "positions evaluated/sec (policy+value), one az_eval_batch per step",
        "value": B / (ms * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16", "int8": "int8", "fp8": "fp8_e4m3"}[w.dtype],
        "data": "synthetic (seeded planes, masks and N(0, 2/fan_in) weights)",
        "config": {"workload": w.name, "blocks": w.shape.blocks, "filters": w.shape.filters,
                   "in_planes": w.shape.in_planes, "policy_planes": w.shape.policy_planes,
                   "value_hidden": w.shape.value_hidden, "batch": B, "tiling": tiling,
                   "pool_every": w.shape.pool_every, "policy_head": w.shape.policy_head,
                   "value_head": w.shape.value_head, "n_moves": w.shape.n_moves,
                   "params": w.shape.weight_count(), "flop_per_position": flop_pos},
        "roofline": {"bound": "mfma" if w.dtype != "f32" else "alu", "achieved": achieved / 1e12,
                     "peak": peak / 1e12, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": traffic, "traffic_unit": "bytes per launch",
                     "mfma_busy": mfma_busy},
        "latency_us": {"p10": float(np.percentile(lat, 10)), "p50": float(np.percentile(lat, 50)),
                       "p90": float(np.percentile(lat, 90)), "calls": int(lat.size)},
        "graph_replay_us": graph_us,
        "pipeline_pcie_inclusive": pipeline,
        "outputs_valid": ok,
        "wall_s_timed": wall,
        "settle": {"seconds": SETTLE_S, "calls": n_settle},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, blob, ws, acs, planes, legal, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
