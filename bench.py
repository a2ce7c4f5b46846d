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
# untimed launches before each side measurement (draft confidence, learned
# heads, SimHash), about 10-20 ms of GPU work: their inputs are built on the
# host first, and the first launches after that idle stretch ran up to 10 %
# slower than later ones
WARM_LAUNCHES = 300


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
    ap.add_argument("--no-learned-run", action="store_true",
                    help="in the learned block, skip the learned run through selection (every learned scoring "
                         "launch is then of one kind, for counter passes)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (calibrates HBM byte counters)")
    ap.add_argument("--no-configs", action="store_true",
                    help="measure only --config, not the other workloads")
    ap.add_argument("--only-config", action="store_true",
                    help="measure only --config (no other workloads, learned, SimHash or entropy blocks)")
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
    return reps, total, bufs


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


# Sources whose text decides a kernel's memory traffic: its own file, the
# shared device headers and the host planner (work-item sizes, chain split,
# block order, launch shapes).
TRAFFIC_SOURCES = ("msao_device.h", "msao_internal.h", "msao_host.cpp")


def source_hash(kernel_file):
    import hashlib
    h = hashlib.sha256()
    for f in (kernel_file,) + TRAFFIC_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2604_02945_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def _committed(profile, kernel_file):
    """traffic_bytes_per_launch of a committed rocprofv3 counter summary, or
    None when it is absent or the kernel or planner sources changed since it
    was taken."""
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    return rec["traffic_bytes_per_launch"] if rec.get("kernel_source_sha256") == source_hash(kernel_file) else None


TRAFFIC_PROFILES = {  # (config, compacting run) -> counter summary of that scoring launch
    (4, True): "k_score_trimodal_traffic.json",
    (4, False): "k_score_trimodal_scoreonly_traffic.json",
    (3, True): "k_pair_video_traffic.json",
    (3, False): "k_pair_video_scoreonly_traffic.json",
    (5, True): "k_score_highres_traffic.json",
    (5, False): "k_score_highres_scoreonly_traffic.json",
    (2, True): "k_score_imagebatch_traffic.json",
    (2, False): "k_score_imagebatch_scoreonly_traffic.json",
}


# the scoring kernel of each workload: the video clips (bf16, 2 KiB rows) take k_pair
SCORE_KERNEL = {3: "k_pair"}


def committed_traffic(config, compact=True):
    """HBM bytes per scoring launch of a workload (committed counters)."""
    name = TRAFFIC_PROFILES.get((config, compact))
    return _committed(name, "msao_kernels.hip") if name else None


def committed_learned_traffic(config):
    """HBM bytes per learned k_score launch on the tri-modal workload (committed counters)."""
    if config != 4:
        return None
    return _committed("k_score_learned_trimodal_traffic.json", "msao_kernels.hip")


def committed_simhash_traffic():
    """HBM bytes per k_simhash launch on the video clips (committed counters)."""
    return _committed("k_simhash_video_traffic.json", "msao_simhash.hip")


def committed_entropy_traffic():
    """HBM bytes per k_entropy launch (committed counters)."""
    return _committed("k_entropy_draft_logits_traffic.json", "msao_entropy.hip")


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
    # warm-up (the logits are generated on the host first)
    for i in range(WARM_LAUNCHES):
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
        for i in range(max(len(reps), WARM_LAUNCHES)):
            fn(i % len(reps))
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
    res_run = None
    if not args.no_learned_run:
        res_run = learned_run_timing(args, ctx, w, reps, fields, heads, mlp, steps, kernels)
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
        "run_learned": res_run,
        "algorithmic_bytes_score": b_lrn,
        "roofline": {"bound": "hbm", "kernel": "k_score<true>", "achieved": gbs, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "traffic": committed_learned_traffic(w.config)},
    }


def learned_run_timing(args, ctx, w, reps, fields, heads, mlp, steps, kernels):
    """msao_run_learned (image and audio pruned by their Eq. 3 importance,
    compaction) over the same rotated replicas."""
    import torch

    import paper_2604_02945_amd as msao

    R, ntok = w.n_requests, w.n_tokens
    routs = [msao.Outputs(segs, R, token_fields=fields, compact=True) for segs in reps]
    # the arguments marshalled once per replica (a C caller builds them once);
    # every call still plans and uploads its tables
    calls = [msao.binding.prepare_learned(reps[i], R, routs[i], w.params, heads=heads, mlp=mlp, ctx=ctx)[0]
             for i in range(len(reps))]
    for c in calls:
        c()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        calls[i % len(reps)]()
    e1.record()
    torch.cuda.synchronize()
    ms_run = e0.elapsed_time(e1) / steps
    k_run = kernels(lambda i: calls[i]())
    return {"ms_per_call": ms_run, "tokens_per_s": ntok / (ms_run * 1e-3),
            "kernel_ms": {"score": k_run[msao.binding.KERNEL_SCORE], "head": k_run[msao.binding.KERNEL_HEAD],
                          "post_mean_of_request_and_selection": k_run[msao.binding.KERNEL_POST],
                          "gather": k_run[msao.binding.KERNEL_GATHER]}}


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
    reps, _, _ = pack_replicas(w, 8, dev)
    R, K, C = w.n_requests, 32, w.segments[0].hidden
    planes = torch.from_numpy(simhash_planes(K, C, seed=1).view(np.int16)).to(dev).view(torch.bfloat16)
    hashes = [dict(planes=planes, bits=K) for _ in w.segments]
    outs = [msao.Outputs(segs, R, compact=False) for segs in reps]
    sigs = [torch.empty(w.n_tokens, dtype=torch.int64, device=dev) for _ in reps]
    steps = max(1, min(args.steps, 100))

    def kernels(fn):
        for i in range(max(len(reps), WARM_LAUNCHES)):
            fn(i % len(reps))
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

    # every entry point's arguments marshalled once per replica (tables still
    # planned and uploaded per call)
    B = msao.binding
    c_sh = [B.prepare_simhash("msao_temporal_simhash", reps[i], R, hashes, outs[i], sigs[i], w.params, ctx=ctx)
            for i in range(len(reps))]
    c_bs = [B.prepare("msao_temporal_redundancy", reps[i], R, outs[i], w.params, ctx=ctx) for i in range(len(reps))]
    ms_sh, k_sh = kernels(lambda i: c_sh[i]())
    ms_bs, k_bs = kernels(lambda i: c_bs[i]())
    # the whole analysis with SimHash in Eq. 5 (score, hash, MAS, selection, compaction) beside msao_run
    routs = [msao.Outputs(segs, R, compact=True) for segs in reps]
    c_rs = [B.prepare_simhash("msao_run_simhash", reps[i], R, hashes, routs[i], sigs[i], w.params, ctx=ctx)
            for i in range(len(reps))]
    c_rb = [B.prepare("msao_run", reps[i], R, routs[i], w.params, ctx=ctx) for i in range(len(reps))]
    ms_rs, k_rs = kernels(lambda i: c_rs[i]())
    ms_rb, k_rb = kernels(lambda i: c_rb[i]())
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


def host_cpu():
    """The host's logical CPU count and model name (from /proc/cpuinfo)."""
    model = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"host_cpus": os.cpu_count(), "host_cpu_model": model}


def cpu_baseline(w, budget_s, n_requests=None):
    """The oracle, single-threaded, on whole runs of the workload (or of its
    first n_requests requests: requests are independent), for about budget_s."""
    import dataclasses

    import oracle

    segs, R = w.segments, w.n_requests
    if n_requests is not None and n_requests < R:
        segs = [s for s in w.segments if s.request < n_requests]
        R = n_requests
    ntok = sum(s.n_tokens for s in segs)
    runs, t0 = 0, time.perf_counter()
    t_oracle = 0.0
    while True:
        a = time.perf_counter()
        oracle.run(segs, R, w.params, compact=True)
        t_oracle += time.perf_counter() - a
        runs += 1
        if time.perf_counter() - t0 > budget_s:
            break
    what = "whole workload" if R == w.n_requests else f"its first {R} of {w.n_requests} requests"
    res = {"value": ntok * runs / t_oracle, "unit": "tokens/s", "cores": 1, "kind": "oracle",
           "sample": f"{what} ({ntok} tokens) x {runs} runs of the single-threaded C oracle "
                     f"(fp64 sums, sort-based selection, compaction), {t_oracle:.1f} s"}
    res.update(host_cpu())
    return res


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
    res = {"value": w.n_tokens * runs / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"whole workload ({w.n_tokens} tokens) x {runs} runs, its {len(jobs)} requests spread over "
                     f"{threads} threads of the C oracle, {dt:.1f} s"}
    res.update(host_cpu())
    return res


class Bench:
    """Timed steps of one workload: one plan per input replica (each with its
    own outputs and workspace, so that neither a step's inputs nor its outputs
    are still in the Infinity Cache), steps rotating over the replicas, n_str
    batches in flight on as many HIP streams."""

    def __init__(self, w, dev, n_str, replicas=0, max_replicas=128):
        import torch

        import paper_2604_02945_amd as msao

        self.w, self.dev, self.n_str = w, dev, max(1, n_str)
        n_rep = replicas or max(2, -(-1_000_000_000 // w.input_bytes))
        n_rep = min(n_rep, max_replicas)
        n_rep = -(-n_rep // self.n_str) * self.n_str  # a whole number of replicas per stream
        self.reps, self.buf_bytes, self.bufs = pack_replicas(w, n_rep, dev)
        self.n_rep = n_rep
        self.R, self.n = w.n_requests, len(w.segments)
        has_video = any(s.modality == 2 and s.n_frames >= 2 for s in w.segments)
        self.fields = ("z", "l1", "l2", "info", "d", "res") if has_video else ("z", "l1", "l2", "info")
        self.main = torch.cuda.current_stream()
        # steps run on streams of their own (not the default stream, which would
        # serialize with them); the timing events are on the default stream
        self.streams = [torch.cuda.Stream() for _ in range(self.n_str)]
        self.ctxs = [msao.Context(0) for _ in range(self.n_str)]  # one context per stream
        self.plans, self.outs = [], []

    def make_plans(self, compact):
        import torch

        import paper_2604_02945_amd as msao

        self.close_plans()
        for r, segs in enumerate(self.reps):
            k = r % self.n_str
            o = msao.Outputs(segs, self.R, token_fields=self.fields, compact=compact)
            self.outs.append(o)
            self.plans.append((k, msao.Plan(segs, self.R, o, self.w.params, ctx=self.ctxs[k], compact=compact,
                                            stream=self.main)))
        torch.cuda.synchronize()

    def close_plans(self):
        for _, p in self.plans:
            p.close()
        self.plans, self.outs = [], []

    def run_steps(self, count, nstreams):
        """Enqueue `count` steps; step i runs plan i % n_rep on its stream."""
        import torch

        start = torch.cuda.Event()
        start.record(self.main)
        for st in self.streams[:nstreams]:
            st.wait_event(start)
        used = set()
        for i in range(count):
            k, plan = self.plans[i % self.n_rep]
            k = k if nstreams > 1 else 0
            plan(self.streams[k])
            used.add(k)
        for k in used:
            ev = torch.cuda.Event()
            ev.record(self.streams[k])
            self.main.wait_event(ev)

    def timed(self, count, nstreams):
        """Mean ms per step over `count` steps (events on the default stream
        around the whole region), and the host wall time of the region."""
        import torch

        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        e0.record(self.main)
        self.run_steps(count, nstreams)
        e1.record(self.main)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / count, time.perf_counter() - t

    def median_one_stream(self, count):
        """Median over `count` steps on one stream of each step's own duration
        (an event before and after every step on that stream)."""
        import numpy as np
        import torch

        st = self.streams[0]
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(count + 1)]
        ev[0].record(st)
        for i in range(count):
            self.plans[i % self.n_rep][1](st)
            ev[i + 1].record(st)
        torch.cuda.synchronize()
        return float(np.median([ev[i].elapsed_time(ev[i + 1]) for i in range(count)]))

    def kernel_ms(self, count):
        """Mean duration of each kernel: HIP events recorded by the library at
        the kernel's own start and end, on the stream it is launched on (one
        stream, so kernels do not overlap)."""
        import numpy as np

        for c in self.ctxs:
            c.set_profiling(True)
        for i in range(count):
            self.plans[i % self.n_rep][1](self.streams[0])
        per_ctx = np.array([c.kernel_times() for c in self.ctxs])  # each context's mean per kernel (0: none)
        for c in self.ctxs:
            c.set_profiling(False)
        n = (per_ctx > 0).sum(axis=0)
        return np.where(n > 0, per_ctx.sum(axis=0) / np.maximum(n, 1), 0.0)

    def read_ceiling(self, count):
        """A plain streaming read of the replicas' input buffers (the same
        bytes the scoring pass reads), best of four chunk sizes: GB/s of the
        library's read kernel by its own launch events."""
        import torch

        import paper_2604_02945_amd as msao

        c = self.ctxs[0]
        sink = torch.empty(-(-self.buf_bytes // 8192), dtype=torch.int32, device=self.dev)
        best = None
        for kib in (8, 16, 32, 64):
            for buf in self.bufs:
                msao.msao_stream_read(buf, kib, ctx=c, stream=self.streams[0], sink=sink)
            c.set_profiling(True)
            for i in range(count):
                msao.msao_stream_read(self.bufs[i % len(self.bufs)], kib, ctx=c, stream=self.streams[0], sink=sink)
            ms = c.kernel_times()[msao.binding.KERNEL_READ]
            c.set_profiling(False)
            gbs = self.buf_bytes / (ms * 1e-3) / 1e9
            if best is None or gbs > best["gbps"]:
                best = {"gbps": gbs, "ms": ms, "bytes": self.buf_bytes, "chunk_kib": kib}
        best["frac_of_peak"] = best["gbps"] / PEAK_HBM_GBS
        # the fixed cost of a launch by the same events: one wavefront reading 8 KiB
        tiny = self.bufs[0][:8192]
        for _ in range(8):
            msao.msao_stream_read(tiny, 8, ctx=c, stream=self.streams[0], sink=sink)
        c.set_profiling(True)
        for _ in range(count):
            msao.msao_stream_read(tiny, 8, ctx=c, stream=self.streams[0], sink=sink)
        best["launch_floor_ms"] = c.kernel_times()[msao.binding.KERNEL_READ]
        c.set_profiling(False)
        return best

    def close(self):
        self.close_plans()
        for c in self.ctxs:
            c.close()


def measure(w, args, dev, n_str, graph=False, with_compact=True, with_score_select=True, max_replicas=128):
    """Full steps (score, MAS, selection, compaction) and score+select steps of
    workload w: in flight over n_str streams, one after another on one
    stream, per-step medians on one stream, kernel durations, roofline of the
    scoring pass."""
    import numpy as np
    import torch

    b = Bench(w, dev, n_str, args.replicas, max_replicas)
    res = {"replicas_rotated": b.n_rep, "batches_in_flight": b.n_str}
    steps = args.steps
    kept_count = None
    if with_compact:
        b.make_plans(True)
        b.run_steps(args.warmup, b.n_str)
        torch.cuda.synchronize()
        kept_count = b.outs[0].sel["kept_count"][:b.n].cpu().numpy()
        ms_step, wall = b.timed(steps, b.n_str)
        ms_serial, _ = b.timed(steps, 1)
        med = b.median_one_stream(steps)
        k_ms = b.kernel_ms(steps)
        res.update({"ms_per_step": ms_step, "wall_s_timed": wall, "ms_per_step_one_stream": ms_serial,
                    "ms_per_step_one_stream_median": med, "tokens_per_s": w.n_tokens / (ms_step * 1e-3)})
        if graph:
            # the same one-stream steps with each replica's plan replayed from a HIP graph
            graphs = []
            for _, plan in b.plans:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    plan(torch.cuda.current_stream())
                graphs.append(g)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(b.main)
            for i in range(steps):
                graphs[i % b.n_rep].replay()
            e1.record(b.main)
            torch.cuda.synchronize()
            res["ms_per_step_one_stream_graph"] = e0.elapsed_time(e1) / steps
            del graphs
        b_score, b_select, b_compact = algorithmic_bytes(w, kept_count, True)
        b_step = b_score + b_select + b_compact
        score_gbs = b_score / (k_ms[0] * 1e-3) / 1e9
        res.update({
            "kept_tokens": int(kept_count.sum()),
            "hbm_gbps_step": b_step / (ms_step * 1e-3) / 1e9,
            "hbm_frac_step": b_step / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "algorithmic_bytes": {"score": b_score, "select": b_select, "gather_write": b_compact},
            "kernel_ms": {"score": float(k_ms[0]), "post": float(k_ms[1]), "gather": float(k_ms[2])},
            "roofline": {"bound": "hbm", "kernel": SCORE_KERNEL.get(w.config, "k_score"), "achieved": score_gbs,
                         "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": score_gbs / PEAK_HBM_GBS,
                         "traffic": committed_traffic(w.config, compact=True)},
        })
    if with_score_select:
        # scoring and selection alone (no compaction), same replicas and streams
        b.make_plans(False)
        b.run_steps(args.warmup, b.n_str)
        torch.cuda.synchronize()
        if kept_count is None:
            kept_count = b.outs[0].sel["kept_count"][:b.n].cpu().numpy()
            res["kept_tokens"] = int(kept_count.sum())
        ms_ss, _ = b.timed(steps, b.n_str)
        ms_ss_serial, _ = b.timed(steps, 1)
        med_ss = b.median_one_stream(steps)
        k_ss = b.kernel_ms(steps)
        b_s, b_sel, _ = algorithmic_bytes(w, kept_count, False)
        bb = b_s + b_sel
        gbs_s = b_s / (k_ss[0] * 1e-3) / 1e9
        res["score_select"] = {
            "ms_per_step": ms_ss, "ms_per_step_one_stream": ms_ss_serial,
            "ms_per_step_one_stream_median": med_ss,
            "tokens_per_s": w.n_tokens / (ms_ss * 1e-3), "algorithmic_bytes": bb,
            "hbm_gbps": bb / (ms_ss * 1e-3) / 1e9, "hbm_frac": bb / (ms_ss * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "hbm_frac_one_stream": bb / (ms_ss_serial * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "hbm_frac_one_stream_median": bb / (med_ss * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "kernel_ms": {"score": float(k_ss[0]), "post": float(k_ss[1])},
            "roofline": {"bound": "hbm", "kernel": SCORE_KERNEL.get(w.config, "k_score") + " (score only)",
                         "achieved": gbs_s, "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": gbs_s / PEAK_HBM_GBS,
                         "traffic": committed_traffic(w.config, compact=False)},
        }
    res["read_ceiling"] = b.read_ceiling(max(steps, 8))
    b.close()
    return res


def config_block(c, args, dev):
    """One of the other workloads, measured like the headline one (with a
    bounded oracle sample for its CPU baseline)."""
    import torch

    from workloads import CONFIG_NAMES, make_workload

    w = make_workload(c)
    t0 = time.perf_counter()
    res = {"workload": f"{CONFIG_NAMES[c]} (config {c})", "requests": w.n_requests, "segments": len(w.segments),
           "tokens": w.n_tokens, "input_bytes": w.input_bytes}
    res.update(measure(w, args, dev, args.streams, max_replicas=128 if c != 1 else 100))
    if max(s.n_tokens for s in w.segments) >= 4096:
        # the other trade of the selection of large segments: 256-thread blocks
        # (throughput with batches in flight) instead of 1024-thread ones (latency)
        knob, prev = "MSAO_POST_BIG_SEGMENT", os.environ.get("MSAO_POST_BIG_SEGMENT")
        os.environ[knob] = str(2**31 - 1)
        try:
            t = measure(w, args, dev, args.streams, with_compact=False)["score_select"]
        finally:
            if prev is None:
                os.environ.pop(knob)
            else:
                os.environ[knob] = prev
        res["score_select_throughput_mode"] = {
            "knob": f"{knob}={2**31 - 1} (every selection in 256-thread blocks)",
            **{k: t[k] for k in ("ms_per_step", "ms_per_step_one_stream_median", "tokens_per_s", "hbm_frac",
                                 "hbm_frac_one_stream_median", "kernel_ms")}}
    if not args.no_cpu_baseline:
        sample = {1: None, 2: 8, 3: 1, 5: 4}.get(c)
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds / 4, sample)
    res["bench_s"] = time.perf_counter() - t0
    del w
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.only_config:
        args.no_configs = args.no_learned = args.no_simhash = args.no_entropy = True
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the analysis shards by request "
              "with no exchange, so more GPUs would repeat the one-GPU line", file=sys.stderr)
        sys.exit(2)
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

    from workloads import CONFIG_NAMES, make_workload

    dev = torch.device("cuda", 0)
    w = make_workload(args.config)
    compact = not args.no_compact
    m = measure(w, args, dev, args.streams, graph=compact, with_compact=compact,
                with_score_select=not args.no_score_select)
    head = m if compact else m["score_select"]
    line = {
        "metric": METRIC,
        "value": w.n_tokens / (head["ms_per_step"] * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{CONFIG_NAMES[args.config]} (config {args.config})",
            "requests": w.n_requests, "segments": len(w.segments), "tokens": w.n_tokens,
            "input_dtype": sorted({s.dtype for s in w.segments}),
            "input_bytes": w.input_bytes, "kept_tokens": m.get("kept_tokens"), "replicas_rotated": m["replicas_rotated"],
            "compaction": compact, "batches_in_flight": m["batches_in_flight"],
            "timing": f"{m['batches_in_flight']} batches in flight on as many HIP streams; the one_stream "
                      "fields are per-batch latency on one stream",
        },
    }
    for k in ("ms_per_step_one_stream", "ms_per_step_one_stream_median", "ms_per_step_one_stream_graph",
              "hbm_gbps_step", "hbm_frac_step", "algorithmic_bytes", "kernel_ms", "roofline", "wall_s_timed",
              "score_select", "read_ceiling"):
        if k in m:
            line[k] = m[k]
    if "roofline" not in line and "score_select" in m:
        line["roofline"] = m["score_select"]["roofline"]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
        line["cpu_baseline_threads"] = cpu_baseline_threads(w, args.cpu_seconds / 2)
    if not args.no_configs:
        line["configs"] = {}
        for c in (1, 2, 3, 5):
            if c != args.config:
                line["configs"][str(c)] = config_block(c, args, dev)
    ctx = None
    if not (args.no_learned and args.no_simhash and args.no_entropy):
        import paper_2604_02945_amd as msao
        ctx = msao.Context(0)
    if not args.no_learned:
        b = Bench(w, dev, 1, args.replicas)
        line["learned"] = learned_bench(args, dev, ctx, w, b.reps, b.fields)
        b.close()
        del b
    if not args.no_simhash:
        line["simhash"] = simhash_bench(args, dev, ctx)
    if not args.no_entropy:
        line["entropy"] = entropy_bench(args, dev, ctx)
    if ctx is not None:
        ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
