"""Benchmark of the MAS hot path on one MI355X.

One step = one msao_run over one batch: per-token statistics (and the temporal
term for video), per-modality aggregation and MAS, per-segment top-k selection
and compaction of the kept rows. Inputs are seeded synthetic tensors already
resident in HBM; several replicas of the batch are rotated so that every step
reads from HBM and not from the 256 MB Infinity Cache.

Prints one JSON line (see the repository's design notes for every field).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tokens scored+selected/sec and achieved HBM GB/s vs MI355X peak"
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4, help="workload 1..5 (default 4: tri-modal batch)")
    ap.add_argument("--replicas", type=int, default=0, help="input replicas rotated per step (0: enough for 1 GB)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU time budget of the oracle baseline")
    ap.add_argument("--no-compact", action="store_true", help="time score+select only (no compaction)")
    ap.add_argument("--no-score-select", action="store_true",
                    help="skip the extra score+select-only timing that follows a run with compaction")
    ap.add_argument("--no-entropy", action="store_true",
                    help="skip the draft-confidence kernel and Algorithm 1 measurements")
    ap.add_argument("--entropy-steps", type=int, default=100, help="timed launches of the draft-confidence kernel")
    ap.add_argument("--no-simhash", action="store_true",
                    help="skip the SimHash variant of Eq. 5 on the video clips")
    ap.add_argument("--no-learned", action="store_true",
                    help="skip the learned-head variant (Eq. 3 heads and the Eq. 6 MLP) of the scoring pass")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (calibrates HBM byte counters)")
    ap.add_argument("--streams", type=int, default=3,
                    help="batches in flight: consecutive steps alternate over this many HIP streams")
    return ap.parse_args()


def pack_replicas(w, n_rep, dev):
    """Copy the workload's segments into n_rep contiguous device buffers."""
    import numpy as np
    import torch

    import paper_2604_02945_amd as msao

    offs, total = [], 0
    for s in w.segments:
        offs.append(total)
        total += (s.data.nbytes + 255) // 256 * 256
    host = np.zeros(total, np.uint8)
    for s, o in zip(w.segments, offs):
        host[o:o + s.data.nbytes] = np.ascontiguousarray(s.data).view(np.uint8).reshape(-1)
    first = torch.from_numpy(host).to(dev)
    bufs = [first] + [first.clone() for _ in range(n_rep - 1)]
    reps = []
    for b in bufs:
        segs = []
        for s, o in zip(w.segments, offs):
            nb = s.data.nbytes
            t = b[o:o + nb]
            t = t.view(torch.float32) if s.dtype == "f32" else t.view(torch.bfloat16)
            segs.append(msao.DeviceSegment(t.view(s.n_tokens, s.hidden), s.request, s.modality, s.keep_ratio,
                                           s.n_frames))
        reps.append(segs)
    return reps, total


def algorithmic_bytes(w, kept_count, compact):
    """Bytes the method must move (see the design notes), split by kernel.

    k_score: input rows read once, 16 B/token of statistics (z, l1, l2, info),
    8 B/token more for video tokens (d, res), plus, with compaction, the rows of
    segments that keep every token (written by the scoring pass).
    k_post: 1 B/token keep flag and 4 B per kept index.
    k_gather: the other kept rows, written once."""
    ntok = w.n_tokens
    nvid = sum(s.n_tokens for s in w.segments if s.modality == 2 and s.n_frames >= 2)
    score = w.input_bytes + 16 * ntok + 8 * nvid
    select = ntok * 1 + 4 * int(sum(kept_count))
    fused = gather = 0
    if compact:
        for k, s in zip(kept_count, w.segments):
            rows = int(k) * s.hidden * (4 if s.dtype == "f32" else 2)
            if int(k) == s.n_tokens and s.n_tokens > 0:
                fused += rows
            else:
                gather += rows
    return score + fused, select, gather


def _committed(profile, sources):
    """traffic_bytes_per_launch of a committed rocprofv3 counter summary, or
    None when it is absent or the kernel sources changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    h = hashlib.sha256()
    for f in sources:
        h.update(open(os.path.join(ROOT, "paper_2604_02945_amd", "csrc", f), "rb").read())
    return rec["traffic_bytes_per_launch"] if rec.get("kernel_source_sha256") == h.hexdigest() else None


def committed_traffic(config):
    """HBM bytes per k_score launch on the tri-modal workload (committed counters)."""
    if config != 4:
        return None
    return _committed("k_score_trimodal_traffic.json", ("msao_kernels.hip", "msao_device.h", "msao_internal.h"))


def committed_learned_traffic(config):
    """HBM bytes per learned k_score launch on the tri-modal workload (committed counters)."""
    if config != 4:
        return None
    return _committed("k_score_learned_trimodal_traffic.json",
                      ("msao_kernels.hip", "msao_device.h", "msao_internal.h"))


def committed_simhash_traffic():
    """HBM bytes per k_simhash launch on the video clips (committed counters)."""
    return _committed("k_simhash_video_traffic.json", ("msao_simhash.hip", "msao_device.h", "msao_internal.h"))


def committed_entropy_traffic():
    """HBM bytes per k_entropy launch (committed counters)."""
    return _committed("k_entropy_draft_logits_traffic.json", ("msao_entropy.hip", "msao_internal.h"))


def entropy_bench(args, dev, ctx):
    """Draft confidence (Eq. 9-10) on 1,280 rows x 151,936 bf16 logits (256
    requests x 5 draft tokens over the Qwen2-VL vocabulary), three rotated
    replicas (1.17 GB, so the Infinity Cache is cold), then Algorithm 1's
    per-step loop on the host over the resulting normalised entropies."""
    import numpy as np
    import torch

    import paper_2604_02945_amd as msao
    from workloads import DRAFT_ROWS, DRAFT_VOCAB, draft_logits

    x = draft_logits(DRAFT_ROWS, DRAFT_VOCAB, seed=0, dtype="bf16")
    first = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    reps = [first] + [first.clone() for _ in range(2)]
    rows, V = DRAFT_ROWS, DRAFT_VOCAB
    outs = [{"entropy": torch.empty(rows, device=dev), "entropy_norm": torch.empty(rows, device=dev),
             "draft_token": torch.empty(rows, dtype=torch.int32, device=dev),
             "speculate": torch.empty(rows, dtype=torch.uint8, device=dev)} for _ in reps]
    theta = 0.5
    for i in range(6):
        msao.msao_draft_entropy(reps[i % 3], theta, ctx=ctx, outputs=outs[i % 3])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.entropy_steps):
        msao.msao_draft_entropy(reps[i % 3], theta, ctx=ctx, outputs=outs[i % 3])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.entropy_steps
    ctx.set_profiling(True)
    for i in range(args.entropy_steps):
        msao.msao_draft_entropy(reps[i % 3], theta, ctx=ctx, outputs=outs[i % 3])
    k_ms = ctx.kernel_times()[msao.binding.KERNEL_ENTROPY]
    ctx.set_profiling(False)
    b = rows * V * 2 + rows * (4 + 4 + 4 + 1)
    gbs = b / (k_ms * 1e-3) / 1e9
    hn = outs[0]["entropy_norm"].cpu().numpy()
    # Algorithm 1 on the host: lines 2-3 from the first 500 rows (the paper's
    # calibration-set size), then the per-step loop over the kernel's entropies
    sched = msao.Scheduler(hn[:500])
    theta0, n_draft, p_conf = sched.state.theta, sched.state.n_draft, sched.state.p_conf
    trace = np.tile(hn, 200)
    t0 = time.perf_counter()
    dec, _ = sched.run(trace)
    ns = (time.perf_counter() - t0) / trace.size * 1e9
    res = {
        "workload": f"draft logits {rows} x {V} bf16 (256 requests x 5 draft tokens), 3 rotated replicas",
        "ms_per_launch": ms, "rows_per_s": rows / (ms * 1e-3), "kernel_ms": k_ms,
        "algorithmic_bytes": b, "hbm_gbps": gbs,
        "roofline": {"bound": "hbm", "kernel": "k_entropy", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gbs / PEAK_HBM_GBS, "traffic": committed_entropy_traffic()},
        "speculating_rows": int(outs[0]["speculate"].sum().item()),
        "sched": {"theta0": theta0, "n_draft": n_draft, "p_conf": p_conf, "steps": int(trace.size),
                  "ns_per_step": ns, "sends": int((dec == msao.DECIDE_SEND).sum()),
                  "offloads": int((dec == msao.DECIDE_OFFLOAD).sum())},
    }
    if not args.no_cpu_baseline:
        import oracle
        t0 = time.perf_counter()
        oracle.entropy_rows(x[:64], "bf16")
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": 64 / dt, "unit": "rows/s", "cores": 1, "kind": "oracle",
                               "sample": f"64 rows x {V} of the same logits, single-threaded C oracle (fp64), {dt:.2f} s"}
    del reps, first
    return res


def learned_bench(args, dev, ctx, w, reps, fields):
    """The scoring pass with learned probe heads (Eq. 3: weights on the image
    and audio segments, 3x3 and 1x5 AvgPool) and the Eq. 6 relevance MLP (256
    hidden units over a 1,536-wide prompt embedding plus the 8-entry
    descriptor), over the same rotated replicas, beside the plain scoring pass.
    Random weights: the cost does not depend on their values."""
    import numpy as np
    import torch

    import paper_2604_02945_amd as msao
    from workloads import AUDIO, IMAGE

    rng = np.random.default_rng(5)
    R, n = w.n_requests, len(w.segments)
    heads = []
    for s in w.segments:
        if s.modality in (IMAGE, AUDIO):
            wt = torch.from_numpy((rng.standard_normal(s.hidden) * 1.5 / np.sqrt(s.hidden)).astype(np.float32))
            wt = wt.to(dev).to(torch.bfloat16 if s.dtype == "bf16" else torch.float32)
            heads.append(dict(weight=wt, bias=-0.8 if s.modality == IMAGE else -0.2,
                              grid_w=24 if s.modality == IMAGE else 0, pool=3 if s.modality == IMAGE else 5))
        else:
            heads.append(None)
    pd, hid = 1536, 256
    mlp = {"w1": torch.from_numpy((rng.standard_normal((hid, pd + 8)) * 0.05).astype(np.float32)).to(dev),
           "b1": torch.from_numpy((rng.standard_normal(hid) * 0.1).astype(np.float32)).to(dev),
           "w2": torch.from_numpy((rng.standard_normal(hid) * 0.1).astype(np.float32)).to(dev), "b2": 0.0,
           "prompt": torch.from_numpy(rng.standard_normal((R, pd)).astype(np.float32)).to(dev)}
    outs = [msao.Outputs(segs, R, token_fields=fields, compact=False) for segs in reps]
    steps = max(1, min(args.steps, 100))

    def kernels(fn):
        for i in range(len(reps)):
            fn(i)
        torch.cuda.synchronize()
        ctx.set_profiling(True)
        for i in range(steps):
            fn(i % len(reps))
        torch.cuda.synchronize()
        k = ctx.kernel_times()
        ctx.set_profiling(False)
        return k

    k_plain = kernels(lambda i: msao.msao_mas_score(reps[i], R, w.params, ctx=ctx, outputs=outs[i]))
    k_lrn = kernels(lambda i: msao.msao_mas_score_learned(reps[i], R, w.params, heads=heads, mlp=mlp, ctx=ctx,
                                                          outputs=outs[i]))
    ntok = w.n_tokens
    b_plain = w.input_bytes + 4 * len(fields) * ntok
    b_lrn = b_plain + 4 * ntok          # + the projection or the density importance of every token
    gbs = b_lrn / (k_lrn[msao.binding.KERNEL_SCORE] * 1e-3) / 1e9
    total = k_lrn[msao.binding.KERNEL_SCORE] + k_lrn[msao.binding.KERNEL_HEAD] + k_lrn[msao.binding.KERNEL_POST]
    return {
        "workload": f"{w.name}: heads on image (24x24 grid, pool 3) and audio (1500 frames, pool 5), "
                    f"MLP {hid} x ({pd} + 8)",
        "kernel_ms": {"score_learned": k_lrn[msao.binding.KERNEL_SCORE], "head": k_lrn[msao.binding.KERNEL_HEAD],
                      "post_learned": k_lrn[msao.binding.KERNEL_POST], "score_plain": k_plain[msao.binding.KERNEL_SCORE],
                      "post_plain": k_plain[msao.binding.KERNEL_POST]},
        "gpu_ms_per_call": total,
        "tokens_per_s": ntok / (total * 1e-3),
        "score_overhead": k_lrn[msao.binding.KERNEL_SCORE] / k_plain[msao.binding.KERNEL_SCORE] - 1.0,
        "algorithmic_bytes_score": b_lrn,
        "roofline": {"bound": "hbm", "kernel": "k_score<true>", "achieved": gbs, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "traffic": committed_learned_traffic(w.config)},
    }


def simhash_bench(args, dev, ctx):
    """The SimHash variant of Eq. 5 (K = 32 hyperplanes per token) on the video
    clips (8 x 32 frames x 256 tokens x 1024 bf16, 134 MB), eight rotated
    replicas (1.07 GB, a cold Infinity Cache), beside the bit-sampling
    temporal pass (msao_temporal_redundancy) on the same replicas."""
    import numpy as np
    import torch

    import paper_2604_02945_amd as msao
    from workloads import make_workload, simhash_planes

    w = make_workload(3)
    reps, _ = pack_replicas(w, 8, dev)
    R, K, C = w.n_requests, 32, w.segments[0].hidden
    planes = torch.from_numpy(simhash_planes(K, C, seed=1).view(np.int16)).to(dev).view(torch.bfloat16)
    hashes = [dict(planes=planes, bits=K) for _ in w.segments]
    outs = [msao.Outputs(segs, R, compact=False) for segs in reps]
    sigs = [torch.empty(w.n_tokens, dtype=torch.int64, device=dev) for _ in reps]
    steps = max(1, min(args.steps, 100))

    def kernels(fn):
        for i in range(len(reps)):
            fn(i)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            fn(i % len(reps))
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        ctx.set_profiling(True)
        for i in range(steps):
            fn(i % len(reps))
        torch.cuda.synchronize()
        k = ctx.kernel_times()
        ctx.set_profiling(False)
        return ms, k

    ms_sh, k_sh = kernels(lambda i: msao.msao_temporal_simhash(reps[i], R, hashes, w.params, ctx=ctx, outputs=outs[i],
                                                               sig=sigs[i]))
    ms_bs, k_bs = kernels(lambda i: msao.msao_temporal_redundancy(reps[i], R, w.params, ctx=ctx, outputs=outs[i]))
    # the whole analysis with SimHash in Eq. 5 (score, hash, MAS, selection, compaction) beside msao_run
    routs = [msao.Outputs(segs, R, compact=True) for segs in reps]
    ms_rs, k_rs = kernels(lambda i: msao.msao_run_simhash(reps[i], R, hashes, w.params, ctx=ctx, outputs=routs[i],
                                                          sig=sigs[i]))
    ms_rb, k_rb = kernels(lambda i: msao.msao_run(reps[i], R, w.params, ctx=ctx, outputs=routs[i]))
    ntok = w.n_tokens
    b = w.input_bytes + 8 * ntok               # rows read once, signatures written
    km = k_sh[msao.binding.KERNEL_SIMHASH]
    gbs = b / (km * 1e-3) / 1e9
    flops = 2.0 * ntok * C * K
    res = {
        "workload": f"{w.name}: 8 clips x 32 frames x 256 tokens x 1024 bf16, K = {K} hyperplanes",
        "ms_per_call": ms_sh, "tokens_per_s": ntok / (ms_sh * 1e-3),
        "kernel_ms": {"simhash": km, "hash_post": k_sh[msao.binding.KERNEL_HASH_POST],
                      "bit_sampling_score": k_bs[msao.binding.KERNEL_SCORE],
                      "bit_sampling_post": k_bs[msao.binding.KERNEL_POST]},
        "ms_per_call_bit_sampling": ms_bs,
        "run": {"ms_per_call": ms_rs, "tokens_per_s": ntok / (ms_rs * 1e-3), "ms_per_call_msao_run": ms_rb,
                "kernel_ms": {k: k_rs[getattr(msao.binding, "KERNEL_" + k.upper())]
                              for k in ("score", "clip", "simhash", "hash_post", "post", "gather")},
                "kernel_ms_msao_run": {k: k_rb[getattr(msao.binding, "KERNEL_" + k.upper())]
                                       for k in ("score", "post", "gather")}},
        "algorithmic_bytes": b,
        "mfma_tflops": flops / (km * 1e-3) / 1e12,
        "roofline": {"bound": "hbm", "kernel": "k_simhash", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gbs / PEAK_HBM_GBS, "traffic": committed_simhash_traffic()},
    }
    if not args.no_cpu_baseline:
        import oracle
        seg = w.segments[0]
        hp = simhash_planes(K, C, seed=1)
        t0 = time.perf_counter()
        oracle.temporal_simhash([seg], 1, w.params, [dict(planes=hp, bits=K)])
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": seg.n_tokens / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle",
                               "sample": f"one clip ({seg.n_tokens} tokens) of the same workload, single-threaded C "
                                         f"oracle (fp64 projections), {dt:.2f} s"}
    for o in outs:
        del o
    del reps
    return res


def cpu_baseline(w, budget_s):
    import oracle

    runs, t0 = 0, time.perf_counter()
    t_oracle = 0.0
    while True:
        a = time.perf_counter()
        oracle.run(w.segments, w.n_requests, w.params, compact=True)
        t_oracle += time.perf_counter() - a
        runs += 1
        if time.perf_counter() - t0 > budget_s:
            break
    return {"value": w.n_tokens * runs / t_oracle, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"whole workload ({w.n_tokens} tokens) x {runs} runs of the single-threaded C oracle "
                      f"(fp64 sums, sort-based selection, compaction), {t_oracle:.1f} s",
            "host_cpu": platform.processor() or platform.machine()}


def cpu_baseline_threads(w, budget_s):
    """The same oracle on up to 16 host threads: requests are independent (one
    request's MAS, selection and compaction read only its own segments), so
    each thread runs the unchanged oracle on one request at a time (ctypes
    releases the interpreter lock during the C call)."""
    import dataclasses
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    oracle.lib()
    jobs = []
    for r in range(w.n_requests):
        segs = [dataclasses.replace(s, request=0) for s in w.segments if s.request == r]
        if segs:
            jobs.append(segs)
    threads = max(1, min(16, os.cpu_count() or 1, len(jobs)))
    runs, t0 = 0, time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        while True:
            list(ex.map(lambda segs: oracle.run(segs, 1, w.params, compact=True), jobs))
            runs += 1
            if time.perf_counter() - t0 > budget_s:
                break
    dt = time.perf_counter() - t0
    return {"value": w.n_tokens * runs / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"whole workload ({w.n_tokens} tokens) x {runs} runs, its {len(jobs)} requests spread over "
                      f"{threads} threads of the C oracle, {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the analysis shards by request "
              "with no exchange, so more GPUs would repeat the one-GPU line", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if args.copy_calibration:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": args.steps}), flush=True)
        return

    import paper_2604_02945_amd as msao
    from workloads import CONFIG_NAMES, make_workload

    dev = torch.device("cuda", 0)
    w = make_workload(args.config)
    n_rep = args.replicas or max(2, -(-1_000_000_000 // w.input_bytes))
    reps, buf_bytes = pack_replicas(w, n_rep, dev)
    R, n = w.n_requests, len(w.segments)
    has_video = any(s.modality == 2 and s.n_frames >= 2 for s in w.segments)
    fields = ("z", "l1", "l2", "info", "d", "res") if has_video else ("z", "l1", "l2", "info")
    compact = not args.no_compact
    n_str = max(1, args.streams)
    n_rep = -(-n_rep // n_str) * n_str  # a whole number of replicas per stream
    while len(reps) < n_rep:
        extra, _ = pack_replicas(w, 1, dev)
        reps += extra
    main = torch.cuda.current_stream()
    # steps run on streams of their own (not the default stream, which would
    # serialize with them); the timing events are on the default stream
    streams = [torch.cuda.Stream() for _ in range(n_str)]
    ctxs = [msao.Context(0) for _ in range(n_str)]  # one context per stream

    def make_plans(with_compaction):
        """One plan per replica, each with its own outputs and workspace, so that
        neither the inputs nor the outputs of a step are still in the Infinity Cache."""
        plans, outs = [], []
        for r, segs in enumerate(reps):
            k = r % n_str
            o = msao.Outputs(segs, R, token_fields=fields, compact=with_compaction)
            outs.append(o)
            plans.append((k, msao.Plan(segs, R, o, w.params, ctx=ctxs[k], compact=with_compaction, stream=main)))
        torch.cuda.synchronize()
        return plans, outs

    def run_steps(plans, count, nstreams):
        """Enqueue `count` steps; step i runs plan i % n_rep on its stream."""
        start = torch.cuda.Event()
        start.record(main)
        for st in streams[:nstreams]:
            st.wait_event(start)
        used = set()
        for i in range(count):
            k, plan = plans[i % n_rep]
            k = k if nstreams > 1 else 0
            plan(streams[k])
            used.add(k)
        for k in used:
            ev = torch.cuda.Event()
            ev.record(streams[k])
            main.wait_event(ev)

    def timed(plans, count, nstreams):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        e0.record(main)
        run_steps(plans, count, nstreams)
        e1.record(main)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / count, time.perf_counter() - t

    plans, outs = make_plans(compact)
    run_steps(plans, args.warmup, n_str)
    torch.cuda.synchronize()
    out = outs[0]
    kept_count = out.sel["kept_count"][:n].cpu().numpy()
    kept_total = int(kept_count.sum())

    # timed region: K whole steps over rotated replicas, n_str batches in flight
    ms_step, wall = timed(plans, args.steps, n_str)
    # the same steps one after another on one stream: per-batch latency
    ms_step_serial, _ = timed(plans, args.steps, 1)
    # the same one-stream steps with each replica's plan replayed from a HIP graph
    graphs = []
    for _, plan in plans:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            plan(torch.cuda.current_stream())
        graphs.append(g)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(main)
    for i in range(args.steps):
        graphs[i % n_rep].replay()
    e1.record(main)
    torch.cuda.synchronize()
    ms_step_graph = e0.elapsed_time(e1) / args.steps
    del graphs

    # per-kernel durations: HIP events recorded by the library around each launch,
    # on the stream the kernel is launched on (one stream, so kernels do not overlap)
    for c in ctxs:
        c.set_profiling(True)
    for i in range(args.steps):
        plans[i % n_rep][1](streams[0])
    k_ms = np.mean([np.array(c.kernel_times()) for c in ctxs], axis=0)
    for c in ctxs:
        c.set_profiling(False)

    b_score, b_select, b_compact = algorithmic_bytes(w, kept_count, compact)
    b_step = b_score + b_select + b_compact

    # scoring and selection alone (no compaction), same replicas and streams
    score_select = None
    if compact and not args.no_score_select:
        torch.cuda.synchronize()
        for _, plan in plans:
            plan.close()
        del plans, outs
        plans_ss, _ = make_plans(False)
        run_steps(plans_ss, args.warmup, n_str)
        ms_ss, _ = timed(plans_ss, args.steps, n_str)
        ms_ss_serial, _ = timed(plans_ss, args.steps, 1)
        b_s, b_sel, _ = algorithmic_bytes(w, kept_count, False)
        score_select = {"ms_per_step": ms_ss, "ms_per_step_one_stream": ms_ss_serial,
                        "tokens_per_s": w.n_tokens / (ms_ss * 1e-3), "algorithmic_bytes": b_s + b_sel,
                        "hbm_gbps": (b_s + b_sel) / (ms_ss * 1e-3) / 1e9,
                        "hbm_frac": (b_s + b_sel) / (ms_ss * 1e-3) / 1e9 / PEAK_HBM_GBS}
        plans = plans_ss
    score_gbs = b_score / (k_ms[0] * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": w.n_tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{CONFIG_NAMES[args.config]} (config {args.config})",
            "requests": R, "segments": n, "tokens": w.n_tokens, "input_dtype": sorted({s.dtype for s in w.segments}),
            "input_bytes": w.input_bytes, "kept_tokens": kept_total, "replicas_rotated": n_rep,
            "compaction": compact, "batches_in_flight": n_str,
        },
        "ms_per_step_one_stream": ms_step_serial,
        "ms_per_step_one_stream_graph": ms_step_graph,
        "hbm_gbps_step": b_step / (ms_step * 1e-3) / 1e9,
        "hbm_frac_step": b_step / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBS,
        "algorithmic_bytes": {"score": b_score, "select": b_select, "gather_write": b_compact},
        "kernel_ms": {"score": k_ms[0], "post": k_ms[1], "gather": k_ms[2]},
        "roofline": {"bound": "hbm", "kernel": "k_score", "achieved": score_gbs, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": score_gbs / PEAK_HBM_GBS, "traffic": committed_traffic(args.config)},
        "wall_s_timed": wall,
        "score_select": score_select,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
        line["cpu_baseline_threads"] = cpu_baseline_threads(w, args.cpu_seconds / 2)
    if not args.no_learned:
        line["learned"] = learned_bench(args, dev, ctxs[0], w, reps, fields)
    if not args.no_simhash:
        line["simhash"] = simhash_bench(args, dev, ctxs[0])
    if not args.no_entropy:
        line["entropy"] = entropy_bench(args, dev, ctxs[0])
    for _, plan in plans:
        plan.close()
    for c in ctxs:
        c.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
