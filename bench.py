"""Benchmark: k-MIP attention forward + backward on one MI355X.

Default workload: one graph of N = 500,000 nodes, H = 4 heads of d = 16,
k = 32 (xyz point-cloud features), forward (score+select, then
gather-softmax-aggregate) and backward (index set held fixed).  A step is one
pass of all of it over the inputs, which are resident in HBM before the timed
region starts.

Prints ONE JSON line on stdout.  Extra detail goes to stderr.
  value        whole-job node-queries per second (N / step time; every head)
  roofline     the score+select kernel against the unit that binds it: the
               work it executes (VALU instructions and MFMA FLOP counted by
               rocprofv3 on the same sources, profiles/select_counters.json)
               over its duration, from HIP events the library records
               around that kernel's launch on the stream it runs on; bound
               is "alu" when the VALU issue rate is the larger fraction of
               its peak, else "mfma"; the kernel skips the key blocks its
               bounds rule out, so its MFMA work is less than a dense scan
               of every (query, key) pair, whose rate over the same time is
               reported separately as the effective rate
  cpu_baseline the float64 CPU oracle on a bounded sample of the same
               workload (not an optimisation target)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "k-MIP attn fwd+bwd queries/s and score TFLOP/s (% bf16 MFMA peak) at N=500k"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
PEAK_VALU_TOPS = 256 * 64 * 2.4e9 / 1e12   # wave64 VALU lane-instructions, 39.3 T/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--config", type=int, default=4, help="workload 1..5 (default 4: N=500k)")
    p.add_argument("--n", type=int, default=None, help="override N (c2: number of graphs)")
    p.add_argument("--k", type=int, default=None, help="override k (configs 3 and 4)")
    p.add_argument("--d", type=int, default=None, help="override the head width d (configs 3 and 4)")
    p.add_argument("--prefilter", action="store_true",
                   help="score + select through the int8 prefilter with an exact re-rank "
                        "(kmip_topk_prefilter; one graph, k <= 32); the select time is then the whole call")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-sample", type=int, default=2048, help="query-heads in the oracle sample")
    p.add_argument("--bwd-variant", type=int, default=0, help="backward: 0 library choice, 1 per-pair atomics, 2 key-sorted segmented, 3 bucketed, 4 key-aggregated")
    p.add_argument("--compare-dense", action="store_true",
                   help="instead of the step benchmark: k-MIP (k=10, d=16, H=1) against dense "
                        "softmax attention (torch SDPA, flash or memory-efficient kernels) over the "
                        "efficiency study's grid of N; prints one JSON line with the table")
    p.add_argument("--dense-exps", type=str, default="2,3,4,4.5,5,5.5,6",
                   help="log10 N of the --compare-dense grid (dense attention only up to --dense-max)")
    p.add_argument("--dense-max", type=float, default=6.0, help="largest log10 N run densely")
    p.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                   help="before the warm-up, run one plain copy kernel that reads and writes MIB MiB "
                        "(the reference for the FETCH_SIZE/WRITE_SIZE counter runs)")
    return p.parse_args()


def measured_counters(config):
    """Counter figures of the score+select kernel on workload `config` from
    profiles/select_counters.json (HBM bytes, MFMA instructions, busy
    fractions per launch), or None when there are none or the select
    sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", "select_counters.json")
    if not os.path.exists(path):
        return None
    import rocprof_summary
    with open(path) as f:
        rec = json.load(f).get(f"c{config}")
    return rec if rec and rec.get("sources_sha256") == rocprof_summary.sources_hash() else None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, sample):
    """Oracle on a seeded sample of query-heads: full-sort selection and the
    aggregate for those rows, plus the backward over the whole batch on a
    fixed index set (it is O(N H k d), a few seconds).  Returns queries/s."""
    import numpy as np
    import oracle

    Qd, Kd, Vd, dOd = (oracle.from_bf16(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    rng = np.random.default_rng(1)
    m = min(sample, w.N * w.H)
    sel = np.sort(rng.choice(w.N * w.H, size=m, replace=False))
    t0 = time.perf_counter()
    idx, _, _ = oracle.topk(Qd, Kd, w.k, offsets=w.offsets, sel=sel)
    oracle.attend(Qd, Kd, Vd, idx, w.scale, sel=sel)
    t_fwd = time.perf_counter() - t0
    # backward on a fixed, valid index set for every query (the first k keys
    # of each graph): its cost does not depend on which keys were selected
    lo = np.zeros(w.N, np.int64) if w.offsets is None else np.repeat(
        w.offsets[:-1].astype(np.int64), np.diff(w.offsets))
    base = (lo[:, None, None] + np.arange(w.k)[None, None, :]).astype(np.int32)
    full_idx = np.broadcast_to(base, (w.N, w.H, w.k)).copy()
    t0 = time.perf_counter()
    oracle.backward(Qd, Kd, Vd, dOd, full_idx, w.scale)
    t_bwd = time.perf_counter() - t0
    per_query = w.H * t_fwd / m + t_bwd / w.N
    return {
        "value": 1.0 / per_query, "unit": "queries/s", "cores": oracle.threads(), "kind": "oracle",
        "cpu_model": cpu_model(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS", "unset"),
        "host_cpus": os.cpu_count(),
        "sample": (f"full-sort top-k + aggregate on {m} seeded query-heads of the same workload "
                   f"({t_fwd:.2f} s), backward on all {w.N * w.H} query-heads ({t_bwd:.2f} s); "
                   f"per node-query cost = H*fwd/query-head + bwd/node"),
    }


def _time_ms(fn, reps):
    """Mean ms of fn() over reps runs after one warm-up, by events on the current stream."""
    import torch
    fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        fn()
    ev[1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / reps


def _peak_bytes(fn):
    """Peak device memory fn() allocates beyond what is already allocated."""
    import torch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    fn()
    torch.cuda.synchronize()
    return torch.cuda.max_memory_allocated() - base


def compare_dense(args):
    """k-MIP attention against dense softmax attention on one MI355X.

    The efficiency study (Section 5.1, "Objective 1", and the detailed
    measurements of Appendix H.2 / I) times one graph with Q, K, V ~ N(0, 1),
    one head, k = 10, over N = 10^2 .. 10^7, for inference (forward) and
    training (forward + backward), with peak memory.  Here d = 16 (the
    smallest head size the library compiles; the paper used 10) and bf16
    inputs.  Dense attention is torch's scaled_dot_product_attention held to
    its flash / memory-efficient kernels (linear memory, no N x N matrix);
    the math fallback is not allowed, so a size it cannot take is reported
    as an error rather than timed on another algorithm."""
    import numpy as np
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel
    import torch.nn.functional as F

    import paper_2604_03815_amd as kmip
    import workloads

    dev = torch.device("cuda:0")
    d, kk = 16, 10
    scale = 1.0 / np.sqrt(d)
    rows = []
    for e in (float(x) for x in args.dense_exps.split(",")):
        N = int(round(10 ** e))
        w = workloads.iid(N, 1, d, kk, seed=args.seed, name="grid")
        q, k, v, g = (torch.from_numpy(getattr(w, n).view(np.int16)).view(torch.bfloat16).to(dev)
                      for n in ("q", "kk", "v", "dout"))
        reps = 5 if N <= 10 ** 5 else (2 if N <= 10 ** 6 else 1)
        row = {"log10_N": e, "N": N}
        ws = kmip.Workspace(dev)
        ws.get(max(kmip.topk_workspace_size(N, 1, d, kk), kmip.bwd_workspace_size(N, 1, d, kk)))
        out = torch.empty((N, 1, d), dtype=torch.float32, device=dev)
        idx = torch.empty((N, 1, kk), dtype=torch.int32, device=dev)
        lse = torch.empty((N, 1), dtype=torch.float32, device=dev)
        grads = [torch.empty((N, 1, d), dtype=torch.float32, device=dev) for _ in range(3)]

        def kmip_inf():
            kmip.topk(q, k, kk, idx=idx, workspace=ws)
            kmip.attend(q, k, v, idx, scale, out=out, lse=lse)

        def kmip_train():
            kmip_inf()
            kmip.bwd(q, k, v, g, idx, lse, scale, dq=grads[0], dk=grads[1], dv=grads[2], workspace=ws)

        row["kmip_inference_ms"] = _time_ms(kmip_inf, reps)
        row["kmip_training_ms"] = _time_ms(kmip_train, reps)
        row["kmip_training_peak_bytes"] = _peak_bytes(kmip_train) + ws.buf.numel() + 4 * (
            out.numel() + idx.numel() + lse.numel() + sum(x.numel() for x in grads))
        if e <= args.dense_max + 1e-9:
            # [batch 1, heads 1, N, d]
            qd, kd, vd, gd = (x.view(N, d).unsqueeze(0).unsqueeze(0) for x in (q, k, v, g))
            try:
                with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                    def dense_inf():
                        with torch.no_grad():
                            F.scaled_dot_product_attention(qd, kd, vd, scale=scale)

                    qg, kg, vg = (x.detach().clone().requires_grad_() for x in (qd, kd, vd))

                    def dense_train():
                        o = F.scaled_dot_product_attention(qg, kg, vg, scale=scale)
                        o.backward(gd)
                        qg.grad = kg.grad = vg.grad = None

                    row["dense_inference_ms"] = _time_ms(dense_inf, reps)
                    row["dense_training_ms"] = _time_ms(dense_train, reps)
                    row["dense_training_peak_bytes"] = _peak_bytes(dense_train) + 3 * 2 * N * d
                    row["speedup_inference"] = row["dense_inference_ms"] / row["kmip_inference_ms"]
                    row["speedup_training"] = row["dense_training_ms"] / row["kmip_training_ms"]
            except RuntimeError as ex:
                row["dense_error"] = str(ex).splitlines()[0][:200]
        log("[dense] " + json.dumps(row))
        rows.append(row)
        del q, k, v, g, out, idx, lse, grads, ws
        torch.cuda.empty_cache()
    result = {
        "metric": "k-MIP vs dense softmax attention, inference and training ms and peak memory",
        "unit": "ms", "higher_is_better": False, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "one graph, H=1, d=16, k=10, Q/K/V/dOut ~ N(0,1) -> bf16, seed "
                               f"{args.seed}; dense = torch SDPA (flash / memory-efficient kernels)",
                   "grid_log10_N": args.dense_exps, "dense_max_log10_N": args.dense_max},
        "rows": rows,
    }
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the k-MIP path here is single-GPU; several graphs would shard by whole "
              "graphs, one large graph by query ranges after an all-gather of K and V)",
              file=sys.stderr)
        sys.exit(2)

    if args.compare_dense:
        compare_dense(args)
        return

    import numpy as np
    import torch

    import paper_2604_03815_amd as kmip
    import workloads

    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    w = workloads.make(args.config, seed=args.seed, n=args.n, k=args.k, d=args.d)
    log(f"[bench] workload c{args.config}: N={w.N} H={w.H} d={w.d} k={w.k} graphs={w.num_graphs} "
        f"(generated in {time.perf_counter() - t0:.1f} s)")

    def dev_t(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = dev_t(w.q), dev_t(w.kk), dev_t(w.v)
    g = dev_t(w.dout) if w.dout is not None else None
    N, H, d, kk = w.N, w.H, w.d, w.k
    idx = torch.empty((N, H, kk), dtype=torch.int32, device=dev)
    out = torch.empty((N, H, d), dtype=torch.float32, device=dev)
    lse = torch.empty((N, H), dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.empty((N, H, d), dtype=torch.float32, device=dev) for _ in range(3))
    backward = w.backward and g is not None
    # one workspace, sized for the larger of the two uses, allocated up front
    ws = kmip.Workspace(dev)
    ws.get(max(kmip.topk_prefilter_workspace_size(N, H, d, kk) if args.prefilter
               else kmip.topk_workspace_size(N, H, d, kk, w.num_graphs),
               kmip.bwd_workspace_size(N, H, d, kk, args.bwd_variant) if backward else 0))
    redone = torch.zeros(1, dtype=torch.int32, device=dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        if args.prefilter:
            if ev is not None:
                ev[4].record()
            kmip.topk_prefilter(q, k, kk, idx=idx, workspace=ws, redone=redone)
            if ev is not None:
                ev[5].record()
                ev[1].record()
            kmip.attend(q, k, v, idx, w.scale, out=out, lse=lse)
        else:
            # the whole forward in one call (its aggregate takes the queries
            # in the select's grouped order); the library records the select
            # kernel's events and the start of the aggregate
            kmip.fwd(q, k, v, kk, w.scale, graph_offsets=w.offsets, workspace=ws, out=out, idx=idx, lse=lse,
                     events=None if ev is None else (ev[4], ev[5], ev[1]))
        if ev is not None:
            ev[2].record()
        if backward:
            kmip.bwd(q, k, v, g, idx, lse, w.scale, variant=args.bwd_variant, dq=dq, dk=dk, dv=dv,
                     workspace=ws)
        if ev is not None:
            ev[3].record()

    if args.calib_copy > 0:
        n = args.calib_copy * 2**20 // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(dev)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # per step: topk start/end, attend end, backward end, select kernel start/end
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    for e in evs:
        for x in e:
            x.record()   # creates the events (the library records some of them)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t0
    peak_mem = torch.cuda.max_memory_allocated(dev)

    t_topk = [e[0].elapsed_time(e[1]) for e in evs]
    t_sel = [e[4].elapsed_time(e[5]) for e in evs]
    t_att = [e[1].elapsed_time(e[2]) for e in evs]
    t_bwd = [e[2].elapsed_time(e[3]) for e in evs]
    ms_step = 1e3 * t_total / args.steps
    sel_ms = sum(t_sel) / len(t_sel)
    pairs = w.score_pairs()
    flops = 2.0 * H * pairs * d
    tflops = flops / (sel_ms * 1e-3) / 1e12
    # MFMA work the kernel actually executed (32x32x16 bf16 MFMAs counted by
    # rocprofv3 on the same sources and workload), when a counter run is on record
    standard = args.n is None and args.seed == 0 and args.k is None and args.d is None and not args.prefilter
    counters = measured_counters(args.config) if standard else None
    executed = counters["mfma_flop_per_launch"] if counters else None
    exec_tflops = None if executed is None else executed / (sel_ms * 1e-3) / 1e12
    topk_ms = sum(t_topk) / len(t_topk)
    att_ms = sum(t_att) / len(t_att)
    bwd_ms = sum(t_bwd) / len(t_bwd) if backward else 0.0
    # algorithmic HBM bytes per call (every operand read once per use, no
    # reuse of gathered key/value rows assumed; bf16 inputs, fp32 outputs)
    nh = N * H
    att_bytes = nh * (2 * d + 4 * kk + 2 * (2 * kk * d) + 4 * d + 4)
    bwd_bytes = nh * (2 * 2 * d + 4 * kk + 4 + 2 * (2 * kk * d) + 3 * 4 * d)
    if args.prefilter:
        nb = (N + 31) // 32
        log(f"[bench] prefilter: {int(redone.item())} of {nb} query blocks redone by the select kernel")
    log(f"[bench] per step: topk {topk_ms:.3f} ms (select kernel {sel_ms:.3f} ms), "
        f"attend {att_ms:.3f} ms, backward {bwd_ms:.3f} ms, "
        f"wall {ms_step:.3f} ms")
    log(f"[bench] score rate {tflops:.1f} TFLOP/s = {100 * tflops / PEAK_BF16_TFLOPS:.1f}% of bf16 peak; "
        f"peak memory {peak_mem / 2**20:.1f} MiB ({peak_mem / N:.0f} B/node)")

    cpu = None
    if not args.no_cpu:
        t0 = time.perf_counter()
        cpu = cpu_baseline(w, args.cpu_sample)
        log(f"[bench] cpu oracle baseline: {cpu['value']:.1f} queries/s on {cpu['cores']} threads "
            f"({time.perf_counter() - t0:.1f} s)")

    # Roofline of the score+select kernel from the work it executes (counted
    # by rocprofv3 on the same sources and workload), against the unit the
    # counters show binding: the VALU when its issue rate exceeds the MFMA
    # busy fraction, else the MFMA.  Without a counter record on file the
    # kernel's executed work is unknown and achieved/frac are null.
    valu = counters.get("valu_instructions_per_launch") if counters else None
    valu_rate = None if valu is None else valu * 64 / (sel_ms * 1e-3) / 1e12     # T lane-instr/s
    valu_frac = None if valu_rate is None else valu_rate / PEAK_VALU_TOPS
    mfma_frac = None if exec_tflops is None else exec_tflops / PEAK_BF16_TFLOPS
    bound = "mfma"
    if valu_frac is not None and mfma_frac is not None and valu_frac > mfma_frac:
        bound = "alu"
    roofline = {
        "bound": bound,
        "achieved": valu_rate if bound == "alu" else exec_tflops,
        "peak": PEAK_VALU_TOPS if bound == "alu" else PEAK_BF16_TFLOPS,
        "unit": "T VALU lane-instr/s" if bound == "alu" else "TFLOP/s",
        "frac": valu_frac if bound == "alu" else mfma_frac,
        "traffic": counters["bytes_per_launch"] if counters else None,
        "kernel": ("select_kernel (score+select) alone, between events recorded around its "
                   "launch; the kmip_topk call also runs the query-grouping, key-tree and "
                   "key-tiling pre-passes (kernel_ms.topk)"),
        "work": ("per launch, from rocprofv3 counters on the same sources and workload "
                 "(null if none is on record): SQ_INSTS_VALU x 64 lanes for the VALU, "
                 "SQ_INSTS_MFMA x 32768 FLOP for the MFMA (the scan of the key blocks the "
                 "bounds do not rule out, plus the bound and seed tiles)"),
        "alu": None if valu is None else {
            "valu_instructions": valu, "achieved": valu_rate, "peak": PEAK_VALU_TOPS,
            "unit": "T VALU lane-instr/s", "frac": valu_frac,
            "peak_is": "256 CUs x 64 lanes x 2.4 GHz (one wave64 VALU instruction per CU per cycle)"},
        "mfma": None if executed is None else {
            "executed_flop": executed, "achieved": exec_tflops, "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": mfma_frac,
            "busy_frac_profiled": counters["mfma_busy_frac"]},
        "effective": {
            "tflops": tflops, "pct_bf16_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
            "flop": flops,
            "what": (f"2*H*sum(n_g^2)*d = {flops:.4g} FLOP, every (query, key) pair of each "
                     "graph (a dense scan), over the select kernel's time; above the peak when "
                     "the bounds skip more than the kernel's shortfall from it"),
        },
        "executed_frac_of_dense": None if executed is None else executed / flops,
    }

    result = {
        "metric": METRIC,
        "value": N / (ms_step * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"c{args.config}{'' if standard else ' with changed sizes'}"
                         f"{'; select through the int8 prefilter' if args.prefilter else ''}: {w.notes}; single MI355X; "
                         f"{'forward+backward' if backward else 'forward only'}"),
            "N": N, "H": H, "d": d, "k": kk, "graphs": w.num_graphs, "score_pairs_per_head": pairs,
            "seed": args.seed, "parallelism": "single GPU",
        },
        "score_tflops": tflops,
        "score_pct_bf16_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "kernel_ms": {"topk": topk_ms, "select_kernel": sel_ms, "attend": att_ms, "backward": bwd_ms},
        "hbm": {
            "attend": {"algorithmic_bytes": att_bytes, "gbs": att_bytes / (att_ms * 1e6),
                       "frac": att_bytes / (att_ms * 1e6) / PEAK_HBM_GBS,
                       "bytes": "N*H*(2d q + 4k idx + 2*2kd gathered key and value rows + 4d out + 4 lse)"},
            "backward": None if not backward else {
                "algorithmic_bytes": bwd_bytes, "gbs": bwd_bytes / (bwd_ms * 1e6),
                "frac": bwd_bytes / (bwd_ms * 1e6) / PEAK_HBM_GBS,
                "bytes": ("N*H*(2*2d q, dO + 4k idx + 4 lse + 2*2kd gathered key and value rows "
                          "+ 3*4d dQ, dK, dV)")},
        },
        "peak_mem_bytes": peak_mem,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
