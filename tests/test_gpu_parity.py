"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, on the
same seeded inputs.

Bar: integer outputs (z, d, per-frame D, aggregates, keep flags, kept indices,
keep counts) and compacted rows bit-exact; l1/l2/res within 1e-5 relative for
fp32 inputs and 2e-3 relative for bf16 inputs (sums of non-negative terms, so
a relative bound holds); per-frame sim/gamma and per-modality rho and temporal
term exact (both sides divide the same integers in double and round once);
beta/MAS within 1e-6 relative; informativeness within 1e-5 relative + 2e-6.
Where a MAS-guided keep count sits on a ceil boundary, a keep count from either
side's MAS is accepted and the kept set is checked for the GPU's count.
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from paper_2604_02945_amd import binding as B
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits, make_workload

pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-5, "bf16": 2e-3}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def to_device(segments, dev, pad=0):
    out = []
    for s in segments:
        a = s.data
        if pad:
            a = np.concatenate([a, np.zeros((a.shape[0], pad), a.dtype)], axis=1)
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16 if s.dtype == "bf16" else np.float32)).to(dev)
        if s.dtype == "bf16":
            t = t.view(torch.bfloat16)
        if pad:
            t = t[:, : s.hidden]
        out.append(msao.DeviceSegment(t, s.request, s.modality, s.keep_ratio, s.n_frames))
    return out


def host(t):
    return t.detach().cpu().numpy()


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def token_tolerances(segments):
    rt = np.concatenate([np.full(s.n_tokens, RTOL[s.dtype]) for s in segments]) if segments else np.zeros(0)
    return rt


def assert_close_rel(got, want, rtol, name):
    got = got.astype(np.float64)
    want = want.astype(np.float64)
    both_nan = np.isnan(got) & np.isnan(want)
    same_inf = np.isinf(got) & np.isinf(want) & (np.sign(got) == np.sign(want))
    ok = both_nan | same_inf | (np.abs(got - want) <= rtol * np.abs(want))
    if not ok.all():
        i = int(np.flatnonzero(~ok)[0])
        raise AssertionError(f"{name}[{i}]: got {got[i]!r} want {want[i]!r} ({(~ok).sum()} mismatches)")
    fin = np.isfinite(want) & (want != 0)
    return float(np.max(np.abs(got[fin] - want[fin]) / np.abs(want[fin]))) if fin.any() else 0.0


def compare_scores(segments, R, got, ref, check_tokens=("z", "l1", "l2", "info", "d", "res")):
    rt = token_tolerances(segments)
    errs = {}
    if "z" in check_tokens:
        assert np.array_equal(host(got["z"]).astype(np.uint32), ref["z"]), "z"
    if "d" in check_tokens:
        assert np.array_equal(host(got["d"]).astype(np.uint32), ref["d"]), "d"
    for f in ("l1", "l2", "res"):
        if f in check_tokens:
            errs[f] = assert_close_rel(host(got[f]), ref[f], rt, f)
    if "info" in check_tokens:
        g, w = host(got["info"]).astype(np.float64), ref["info"].astype(np.float64)
        bad = ~(np.abs(g - w) <= 1e-5 * np.abs(w) + 2e-6)
        assert not bad.any(), f"info mismatch at {np.flatnonzero(bad)[:5]}"
    return errs


def compare_frames(got, ref):
    assert np.array_equal(host(got["dframe"]).astype(np.uint64), ref["dframe"]), "dframe"
    assert np.array_equal(host(got["sim"]), ref["sim"]), "sim"
    assert np.array_equal(host(got["gamma"]), ref["gamma"]), "gamma"


def compare_requests(got, ref):
    assert np.array_equal(host(got["agg"]).astype(np.uint64), ref["agg"]), "agg"
    assert np.array_equal(host(got["present"]), ref["present"]), "present"
    assert np.array_equal(host(got["rho"]), ref["rho"]), "rho"
    assert np.array_equal(host(got["temporal"]), ref["temporal"]), "temporal"
    assert np.allclose(host(got["beta"]), ref["beta"], rtol=1e-6, atol=0), "beta"
    assert np.allclose(host(got["mas"]), ref["mas"], rtol=1e-6, atol=1e-7), "mas"


def compare_selection(segments, R, got, ref, p, gpu_mas=None):
    kc = host(got["kept_count"])
    if np.array_equal(kc, ref["k"]):
        assert np.array_equal(host(got["kept_idx"]), ref["kept_idx"]), "kept_idx"
        assert np.array_equal(host(got["keep"]), ref["keep"]), "keep"
        return
    # a MAS-guided count on a ceil boundary: accept the count from the GPU's MAS
    assert gpu_mas is not None, f"keep counts differ: {kc} vs {ref['k']}"
    for i, s in enumerate(segments):
        if kc[i] != ref["k"][i]:
            assert s.keep_ratio < 0
            kappa = 1.0 - float(gpu_mas[s.request * 4 + s.modality])
            if p.get("flags", 0) & oracle.FLAG_SELECT_PER_FRAME and s.n_frames >= 2:
                alt = s.n_frames * oracle.keep_count(kappa, s.tokens_per_frame)
            else:
                alt = oracle.keep_count(kappa, s.n_tokens)
            assert kc[i] == alt
    redo = oracle.select(segments, R, p, ref["z"], ref["d"], gpu_mas)
    assert np.array_equal(kc, redo["k"])
    assert np.array_equal(host(got["kept_idx"]), redo["kept_idx"])
    assert np.array_equal(host(got["keep"]), redo["keep"])


def compare_compaction(dsegs, segments, out, ref_rows, kc):
    rows = msao.compacted_rows(dsegs, out, kc)
    for i, (r, want) in enumerate(zip(rows, ref_rows)):
        g = host(r.view(torch.int16) if r.dtype == torch.bfloat16 else r)
        w = want.view(np.int16) if segments[i].dtype == "bf16" else want
        assert g.shape == w.shape and np.array_equal(g.view(np.uint8), np.ascontiguousarray(w).view(np.uint8)), \
            f"compacted rows of segment {i}"


def run_and_compare(segments, R, params, dev, alpha=None, pad=0, ctx=None, compact=True):
    dsegs = to_device(segments, dev, pad)
    out = msao.msao_run(dsegs, R, params, alpha, ctx=ctx, compact=compact)
    torch.cuda.synchronize()
    got = out.results(R, len(segments))
    ref = oracle.run(segments, R, params, alpha)
    errs = compare_scores(segments, R, got, ref)
    compare_frames(got, ref)
    compare_requests(got, ref)
    compare_selection(segments, R, got, ref, params, gpu_mas=host(got["mas"]))
    if compact:
        compare_compaction(dsegs, segments, out, oracle.compact_rows(segments, host(got["kept_count"]),
                                                                     host(got["kept_idx"])), host(got["kept_count"]))
    return got, ref, errs


# ------------------------------------------------------------- the five workloads

@pytest.mark.parametrize("config", [1, 2, 3, 4])
def test_config_full_size(config, dev):
    log(f"[parity] config {config} full size")
    w = make_workload(config)
    _, ref, errs = run_and_compare(w.segments, w.n_requests, w.params, dev)
    log(f"[parity] config {config}: max rel err {errs}; MAS[:8] {ref['mas'][:8]}")


def test_config5_full_size_fused(dev):
    log("[parity] config 5 full size (1.5 GB, fused run)")
    w = make_workload(5)
    _, ref, errs = run_and_compare(w.segments, w.n_requests, w.params, dev)
    assert np.all(ref["k"] == 720)
    log(f"[parity] config 5: max rel err {errs}")


# ---------------------------------------------------------------- adversarial

def _rand_seg(rng, request, modality, T, P, C, dtype, keep, kind="normal"):
    n = T * P
    if kind == "normal":
        x = rng.standard_normal((n, C)).astype(np.float32)
    elif kind == "relu_bg":
        x = np.maximum(rng.standard_normal((n, C)), 0).astype(np.float32)
        x[rng.random(n) < 0.5] *= np.float32(0.05)
    elif kind == "same":
        x = np.repeat(rng.standard_normal((1, C)).astype(np.float32), n, axis=0)
    elif kind == "zero":
        x = np.zeros((n, C), np.float32)
    elif kind == "special":
        x = rng.standard_normal((n, C)).astype(np.float32)
        specials = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, 0.1, -0.1], np.float32)
        mask = rng.random((n, C)) < 0.05
        x[mask] = rng.choice(specials, size=int(mask.sum()))
    elif kind == "static_video":
        base = rng.standard_normal((P, C)).astype(np.float32)
        frames = [base]
        for _ in range(T - 1):
            frames.append(frames[-1] + np.float32(0.02) * rng.standard_normal((P, C)).astype(np.float32))
        x = np.concatenate(frames)
    else:
        raise ValueError(kind)
    data = x if dtype == "f32" else f32_to_bf16_bits(x)
    return Segment(request, modality, T, P, C, dtype, keep, data)


def adversarial_cases():
    rng = np.random.default_rng(2024)
    cases = {}
    cases["widths"] = [
        _rand_seg(rng, 0, IMAGE, 1, 37, 8, "bf16", 0.5),          # one partial unit, N < 64
        _rand_seg(rng, 0, TEXT, 1, 65, 24, "f32", 1.0),
        _rand_seg(rng, 0, AUDIO, 1, 70, 1288, "bf16", 0.3),       # 161 chunks: ragged third unit
        _rand_seg(rng, 1, IMAGE, 1, 33, 4104, "bf16", 0.2),       # 513 chunks: generic row path
        _rand_seg(rng, 1, AUDIO, 1, 19, 2052, "f32", 0.75),       # 513 chunks (fp32), generic
        _rand_seg(rng, 1, TEXT, 1, 3, 72, "f32", 0.01),
    ]
    cases["video"] = [
        _rand_seg(rng, 0, VIDEO, 2, 9, 1024, "bf16", 0.3),        # T = 2
        _rand_seg(rng, 0, VIDEO, 1, 11, 1024, "bf16", 0.3),       # T = 1: an image
        _rand_seg(rng, 1, VIDEO, 7, 5, 520, "f32", 0.4),          # fp32 chains, ragged units
        _rand_seg(rng, 1, VIDEO, 5, 6, 4096, "bf16", 0.5),        # 8 units: generic chain path
        _rand_seg(rng, 2, VIDEO, 40, 3, 1024, "bf16", 0.25, "static_video"),
        _rand_seg(rng, 2, IMAGE, 1, 50, 1024, "bf16", 0.25, "relu_bg"),
        _rand_seg(rng, 3, VIDEO, 4, 7, 1024, "bf16", 1.0),        # kept whole: rows copied by the scoring pass
    ]
    cases["ties_and_specials"] = [
        _rand_seg(rng, 0, IMAGE, 1, 300, 64, "bf16", 0.37, "same"),   # tie storm
        _rand_seg(rng, 0, AUDIO, 1, 100, 64, "f32", 0.5, "zero"),      # all sparse, all tied
        _rand_seg(rng, 0, TEXT, 1, 200, 256, "f32", 0.5, "special"),   # NaN / inf / -0 / +-tau
        _rand_seg(rng, 1, VIDEO, 6, 16, 64, "bf16", 0.5, "same"),      # identical frames
        _rand_seg(rng, 1, IMAGE, 1, 1, 64, "bf16", 0.5),               # single token
    ]
    cases["keep_extremes"] = [
        _rand_seg(rng, 0, IMAGE, 1, 100, 128, "bf16", 0.0),
        _rand_seg(rng, 0, AUDIO, 1, 100, 128, "bf16", 1.0),
        _rand_seg(rng, 0, TEXT, 1, 100, 128, "bf16", 0.01),            # k = 1
        _rand_seg(rng, 1, IMAGE, 1, 100, 128, "bf16", 0.999),          # k = N
    ]
    cases["empty_and_multi"] = [
        _rand_seg(rng, 0, IMAGE, 1, 0, 64, "bf16", 0.5),
        _rand_seg(rng, 0, IMAGE, 1, 40, 64, "bf16", 0.5, "relu_bg"),
        _rand_seg(rng, 0, IMAGE, 1, 60, 64, "bf16", 0.5),              # two segments, one (r, m)
        _rand_seg(rng, 2, AUDIO, 1, 30, 64, "f32", 0.5),               # request 1 absent
        _rand_seg(rng, 2, VIDEO, 4, 0, 64, "bf16", 0.5),               # empty video
        _rand_seg(rng, 2, VIDEO, 3, 10, 64, "bf16", 0.5),
        _rand_seg(rng, 2, VIDEO, 3, 10, 64, "bf16", 0.5),              # two videos in one (r, m)
    ]
    cases["guided"] = [
        _rand_seg(rng, 0, IMAGE, 1, 576, 1024, "bf16", -1.0, "relu_bg"),
        _rand_seg(rng, 0, AUDIO, 1, 300, 1280, "bf16", -1.0),
        _rand_seg(rng, 0, TEXT, 1, 64, 256, "bf16", -1.0),
        _rand_seg(rng, 1, VIDEO, 8, 32, 1024, "bf16", -1.0, "static_video"),
        _rand_seg(rng, 1, IMAGE, 1, 100, 512, "f32", 0.5),
    ]
    return cases


ADV = adversarial_cases()


@pytest.mark.parametrize("name", sorted(ADV))
def test_adversarial(name, dev):
    segs = ADV[name]
    R = max(s.request for s in segs) + 1
    log(f"[parity] adversarial {name}: {len(segs)} segments, R={R}")
    run_and_compare(segs, R, default_params(), dev)


@pytest.mark.parametrize("variant", ["alpha", "literal", "lambda_s0", "lambda_t0", "tau0", "tau_neg0",
                                     "tau_s_extremes"])
def test_parameter_variants(variant, dev):
    segs = ADV["guided"] + ADV["video"][:3]
    segs = [Segment(s.request if s.request < 2 else 1, s.modality, s.n_frames, s.tokens_per_frame, s.hidden,
                    s.dtype, s.keep_ratio, s.data) for s in segs]
    R = 2
    p = default_params()
    alpha = None
    if variant == "alpha":
        alpha = np.random.default_rng(5).normal(size=R * 4).astype(np.float32)
    elif variant == "literal":
        p["flags"] = oracle.FLAG_TEMPORAL_LITERAL
    elif variant == "lambda_s0":
        p["lambda_s"] = [0.0] * 4
    elif variant == "lambda_t0":
        p["lambda_t"] = [0.0] * 4
    elif variant == "tau0":
        p["tau"] = 0.0
    elif variant == "tau_neg0":
        p["tau"] = -0.0   # |x| <= -0 iff |x| <= 0: zeros inactive, the rest active
    elif variant == "tau_s_extremes":
        p["tau_s"] = 1.0
    log(f"[parity] parameter variant {variant}")
    run_and_compare(segs, R, p, dev, alpha=alpha)


def test_row_stride_padding(dev):
    segs = ADV["widths"][:3] + ADV["video"][:1]
    R = max(s.request for s in segs) + 1
    log("[parity] padded row stride")
    run_and_compare(segs, R, default_params(), dev, pad=24)


# ------------------------------------------------------ separate entry points

def test_separate_entry_points(dev):
    w = make_workload(4, n_requests=3)
    segs = w.segments + ADV["video"]
    segs = [Segment(min(s.request, 2), s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype,
                    -1.0 if i % 4 == 1 else s.keep_ratio, s.data) for i, s in enumerate(segs)]
    R, p = 3, default_params()
    log("[parity] msao_mas_score / temporal_redundancy / select_tokens / compact")
    dsegs = to_device(segs, dev)
    ref = oracle.run(segs, R, p)
    o1 = msao.msao_mas_score(dsegs, R, p)
    torch.cuda.synchronize()
    g1 = o1.results(R, len(segs))
    compare_scores(segs, R, g1, ref)
    compare_frames(g1, ref)
    compare_requests(g1, ref)
    o2 = msao.msao_temporal_redundancy(dsegs, R, p)
    torch.cuda.synchronize()
    g2 = o2.results(R, len(segs))
    assert np.array_equal(host(g2["d"]).astype(np.uint32), ref["d"])
    assert_close_rel(host(g2["res"]), ref["res"], token_tolerances(segs), "res")
    compare_frames(g2, ref)
    assert np.array_equal(host(g2["temporal"]), ref["temporal"])
    # selection from the oracle's z, d and MAS (inputs from the oracle, not from the GPU)
    z = torch.from_numpy(ref["z"].view(np.int32)).to(dev)
    d = torch.from_numpy(ref["d"].view(np.int32)).to(dev)
    mas = torch.from_numpy(ref["mas"]).to(dev)
    o3 = msao.msao_select_tokens(dsegs, R, z, d, mas, p)
    torch.cuda.synchronize()
    g3 = o3.results(R, len(segs))
    assert np.array_equal(host(g3["kept_count"]), ref["k"])
    assert np.array_equal(host(g3["kept_idx"]), ref["kept_idx"])
    assert np.array_equal(host(g3["keep"]), ref["keep"])
    # compaction from the oracle's kept indices
    o4 = msao.Outputs(dsegs, R)
    o4.sel["kept_idx"][: len(ref["kept_idx"])].copy_(torch.from_numpy(ref["kept_idx"]))
    o4.sel["kept_count"][: len(segs)].copy_(torch.from_numpy(ref["k"]))
    msao.msao_compact(dsegs, o4)
    torch.cuda.synchronize()
    compare_compaction(dsegs, segs, o4, oracle.compact_rows(segs, ref["k"], ref["kept_idx"]), ref["k"])


# ------------------------------------------------- determinism and launch shapes

def test_repeat_runs_bitwise_identical(dev):
    w = make_workload(4, n_requests=4)
    segs = w.segments + ADV["video"]
    R = 4
    segs = [Segment(min(s.request, 3), s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype,
                    s.keep_ratio, s.data) for s in segs]
    dsegs = to_device(segs, dev)
    log("[parity] 50 repeated runs")
    first = None
    out = msao.Outputs(dsegs, R)
    call = msao.prepare("msao_run", dsegs, R, out, w.params)
    for i in range(50):
        call()
        torch.cuda.synchronize()
        snap = {k: host(v).copy() for k, v in out.results(R, len(segs)).items()}
        snap["out"] = host(out.out).copy()
        if first is None:
            first = snap
        else:
            for k in first:
                assert np.array_equal(first[k].view(np.uint8), snap[k].view(np.uint8)), (i, k)


def _long_runs():
    """Work items longer than the 64-token store buffer of a wavefront: 16-byte
    rows (512 rows per 8 KiB item) and a 130-frame clip run as one chain."""
    rng = np.random.default_rng(99)
    return [_rand_seg(rng, 0, IMAGE, 1, 300, 8, "bf16", 0.3, "relu_bg"),
            _rand_seg(rng, 0, TEXT, 1, 200, 24, "f32", 0.5),
            _rand_seg(rng, 0, VIDEO, 130, 3, 64, "bf16", 0.4, "static_video"),
            _rand_seg(rng, 1, VIDEO, 70, 2, 4104, "bf16", 0.4)]   # generic chain path


@pytest.mark.parametrize("row_bytes,chain,xcd", [("2048", "4", "1"), ("65536", "32", "0"), ("1", "1", "1"),
                                                 ("8192", "200", "0"), ("8192", "200", "1")])
def test_launch_shapes_same_results(row_bytes, chain, xcd, dev, monkeypatch):
    """Different work-item sizes (rows per wavefront, frames per video run) and
    workgroup orders give the oracle's outputs."""
    segs = make_workload(4, n_requests=2).segments + ADV["video"][:3] + _long_runs()
    R = 3
    log(f"[parity] launch shape rows={row_bytes}B chain={chain} xcd_order={xcd}")
    monkeypatch.setenv("MSAO_ROW_ITEM_BYTES", row_bytes)
    monkeypatch.setenv("MSAO_CHAIN_FRAMES", chain)
    monkeypatch.setenv("MSAO_XCD_ORDER", xcd)
    ctx = B.Context(0)
    run_and_compare(segs, R, default_params(), dev, ctx=ctx)
    run_and_compare(segs, R, default_params(), dev, ctx=ctx, compact=False)
    ctx.close()


def test_selection_beyond_lds_staging(dev):
    """Segments of more than 16,384 tokens: their selection keys do not fit the
    LDS staging area and are recomputed from z and d on every pass."""
    rng = np.random.default_rng(123)
    segs = [_rand_seg(rng, 0, IMAGE, 1, 20000, 16, "bf16", 0.3, "relu_bg"),
            _rand_seg(rng, 0, VIDEO, 80, 300, 64, "bf16", 0.4, "static_video"),
            _rand_seg(rng, 1, AUDIO, 1, 17000, 8, "bf16", -1.0, "relu_bg"),
            _rand_seg(rng, 1, TEXT, 1, 300, 64, "f32", 0.5)]
    log("[parity] selection of segments larger than the LDS key staging")
    run_and_compare(segs, 2, default_params(), dev)


@pytest.mark.parametrize("n_seg", [255, 256])
def test_mid_size_selection_split_threshold(n_seg, dev):
    """Selections of 1,024 to 4,095 tokens are split over several blocks only
    while the launch has fewer than 256 selections: 255 segments take the split
    path, 256 the whole one. Sizes span the split range (a part boundary within
    a wavefront, one token short of the next part), fixed and MAS-guided keeps."""
    rng = np.random.default_rng(400 + n_seg)
    sizes = [1024, 1025, 1535, 1536, 1537, 2303, 2304, 4095] + list(rng.integers(1024, 4096, n_seg - 8))
    mods = (IMAGE, AUDIO, TEXT)
    segs = [_rand_seg(rng, i // 3, mods[i % 3], 1, int(n), 16, "bf16", -1.0 if i % 5 == 0 else 0.35, "relu_bg")
            for i, n in enumerate(sizes)]
    R = (n_seg + 2) // 3
    log(f"[parity] {n_seg} selections of 1,024-4,095 tokens")
    run_and_compare(segs, R, default_params(), dev)


@pytest.mark.parametrize("big", ["1073741824", "1024"])
def test_selection_block_size_knob(big, dev, monkeypatch):
    """MSAO_POST_BIG_SEGMENT moves the threshold of the 1024-thread selection
    blocks: above every selection (the video clips then take 256-thread
    blocks and parts of 768 tokens), or down to 1,024 tokens (the tri-modal
    audio selections take the large blocks). Same results as the oracle."""
    monkeypatch.setenv("MSAO_POST_BIG_SEGMENT", big)
    ctx = B.Context(0)
    segs = make_workload(3, n_requests=3).segments + make_workload(4, n_requests=2).segments
    segs = [Segment(s.request + (3 if s.modality != VIDEO else 0), s.modality, s.n_frames, s.tokens_per_frame,
                    s.hidden, s.dtype, s.keep_ratio, s.data) for s in segs]
    log(f"[parity] MSAO_POST_BIG_SEGMENT={big}")
    run_and_compare(segs, 5, default_params(), dev, ctx=ctx)
    run_and_compare(segs, 5, default_params(), dev, ctx=ctx, compact=False)
    ctx.close()


@pytest.mark.parametrize("keep", [0.49, 0.5])
def test_gather_block_switch(keep, dev):
    """A segment of 200,000 narrow rows keeping 98,001 (gather blocks of eight
    wavefronts) or 100,000 (one-wavefront blocks, above 98,304 rows) beside
    a small image: compacted rows byte-exact either way."""
    rng = np.random.default_rng(int(keep * 100))
    segs = [_rand_seg(rng, 0, AUDIO, 1, 200_000, 8, "bf16", keep, "relu_bg"),
            _rand_seg(rng, 0, IMAGE, 1, 300, 256, "bf16", 0.3)]
    log(f"[parity] gather of {int(200_000 * keep)} rows")
    run_and_compare(segs, 1, default_params(), dev)


def test_plan_runs_match_oracle(dev):
    """msao_plan_create once, msao_plan_run several times (data rewritten in
    place between runs): every run matches the oracle on that run's data."""
    segs = make_workload(4, n_requests=2).segments + ADV["video"][:3] + ADV["guided"][:2]
    R = 3
    p = default_params()
    log("[parity] plan API, three runs with rewritten inputs")
    dsegs = to_device(segs, dev)
    out = msao.Outputs(dsegs, R)
    plan = msao.Plan(dsegs, R, out, p)
    rng = np.random.default_rng(77)
    for run in range(3):
        if run:
            # new data in the same buffers: permute each segment's rows
            for s, ds in zip(segs, dsegs):
                perm = rng.permutation(s.n_tokens)
                s.data = np.ascontiguousarray(s.data[perm])
                src = torch.from_numpy(s.data.view(np.int16 if s.dtype == "bf16" else np.float32)).to(dev)
                ds.data.copy_(src.view(torch.bfloat16) if s.dtype == "bf16" else src)
        plan()
        torch.cuda.synchronize()
        got = out.results(R, len(segs))
        ref = oracle.run(segs, R, p)
        compare_scores(segs, R, got, ref)
        compare_frames(got, ref)
        compare_requests(got, ref)
        compare_selection(segs, R, got, ref, p, gpu_mas=host(got["mas"]))
        kc = host(got["kept_count"])
        compare_compaction(dsegs, segs, out, oracle.compact_rows(segs, kc, host(got["kept_idx"])), kc)
    plan.close()
