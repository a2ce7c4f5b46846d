"""GPU parity of k_pair, the scoring pass of bf16 clips whose rows are 512,
1024, 1536 or 2048 bytes (two patch positions per wavefront over a range of up
to 32 frames, consecutive pairs of positions per block, a ring of four frames
in registers), against the CPU oracle on seeded inputs.

Covers every row width it takes, odd position counts (the last pair holds one
position), pair counts that leave a block part empty, clips shorter than the
ring, clips long enough for several ranges (the halo frame before each range
after the first), padded row strides, identical and
all-zero frames, a batch that mixes k_pair clips with clips and segments of the
other paths (two scoring launches), the temporal-only entry point, and the
same tables with k_pair switched off (MSAO_PAIR=0). Same bar as the other
parity tests: integers bit-exact, bf16 sums within 2e-3 relative.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from paper_2604_02945_amd import binding as B
from test_gpu_parity import (_rand_seg, assert_close_rel, compare_frames, dev, host, log, run_and_compare,  # noqa: F401
                             to_device, token_tolerances)
from workloads import AUDIO, IMAGE, TEXT, VIDEO, default_params

pytestmark = pytest.mark.gpu


def _clips(seed, shapes, kind="normal", keep=0.3):
    rng = np.random.default_rng(seed)
    return [_rand_seg(rng, i % 3, VIDEO, T, P, C, "bf16", keep, kind) for i, (T, P, C) in enumerate(shapes)]


@pytest.mark.parametrize("C", [256, 512, 768, 1024])
def test_row_widths_odd_positions(C, dev):
    """Rows of 1 to 4 units of 512 bytes, odd and even position counts, 2 to 9
    frames (five pairs of positions: three wavefronts of the second block have
    no frames)."""
    segs = _clips(10 + C, [(2, 8, C), (3, 7, C), (5, 9, C), (9, 2, C), (2, 7, C)])
    log(f"[pair] widths C={C}")
    run_and_compare(segs, 3, default_params(), dev)


def test_long_clips_several_time_blocks(dev):
    """70, 130, 64 and 65 frames: ranges of 32 frames (the last one of 6, 2, 32
    and 1), each range after the first reading the frame before it."""
    segs = _clips(31, [(70, 5, 1024), (130, 4, 512), (64, 3, 1024), (65, 2, 256)], kind="static_video")
    log("[pair] long clips")
    run_and_compare(segs, 3, default_params(), dev)


def test_padded_stride(dev):
    segs = _clips(32, [(6, 5, 1024), (33, 4, 512)])
    log("[pair] padded row stride")
    run_and_compare(segs, 2, default_params(), dev, pad=40)


def test_identical_and_zero_frames(dev):
    """Identical frames: d = 0 and res = 0 after frame 0; all-zero frames: z = C."""
    segs = _clips(33, [(12, 6, 1024), (7, 3, 768)], kind="same") + _clips(34, [(10, 4, 512)], kind="zero")
    log("[pair] identical / zero frames")
    got, ref, _ = run_and_compare(segs, 3, default_params(), dev)
    res = host(got["res"])
    n0 = 12 * 6
    assert np.all(res[6:n0] == 0.0) and np.all(host(got["d"])[6:n0] == 0)


def test_mixed_batch_two_launches(dev):
    """k_pair clips with clips of the chain pass (fp32, 64-channel rows, a
    clip kept whole) and image / audio / text segments in one call."""
    rng = np.random.default_rng(35)
    segs = [
        _rand_seg(rng, 0, VIDEO, 8, 6, 1024, "bf16", 0.3, "static_video"),  # k_pair
        _rand_seg(rng, 0, IMAGE, 1, 40, 1024, "bf16", 0.25, "relu_bg"),
        _rand_seg(rng, 1, VIDEO, 5, 3, 520, "f32", 0.4),                    # fp32: chain pass
        _rand_seg(rng, 1, VIDEO, 6, 16, 64, "bf16", 0.5),                   # 128-byte rows: chain pass
        _rand_seg(rng, 1, AUDIO, 1, 30, 1280, "bf16", 0.5),
        _rand_seg(rng, 2, VIDEO, 4, 7, 1024, "bf16", 1.0),                  # kept whole: chain pass copies it
        _rand_seg(rng, 2, VIDEO, 11, 5, 512, "bf16", -1.0),                 # k_pair, MAS-guided
        _rand_seg(rng, 2, TEXT, 1, 20, 256, "bf16", 1.0),
    ]
    log("[pair] mixed batch")
    run_and_compare(segs, 3, default_params(), dev)
    run_and_compare(segs, 3, default_params(), dev, compact=False)


def test_temporal_only_entry_point(dev):
    segs = _clips(36, [(9, 5, 1024), (4, 4, 256)])
    R, p = 2, default_params()
    dsegs = to_device(segs, dev)
    ref = oracle.run(segs, R, p)
    log("[pair] msao_temporal_redundancy")
    o = msao.msao_temporal_redundancy(dsegs, R, p)
    torch.cuda.synchronize()
    g = o.results(R, len(segs))
    assert np.array_equal(host(g["d"]).astype(np.uint32), ref["d"])
    assert_close_rel(host(g["res"]), ref["res"], token_tolerances(segs), "res")
    compare_frames(g, ref)
    assert np.array_equal(host(g["temporal"]), ref["temporal"])


def test_pair_off_same_results(dev, monkeypatch):
    """The same clips scored by the chain pass (MSAO_PAIR=0) and by k_pair give
    the same integers and the oracle's sums."""
    segs = _clips(37, [(32, 10, 1024), (17, 7, 512)], kind="static_video")
    R = 3
    outs = []
    for flag in ("0", "1"):
        monkeypatch.setenv("MSAO_PAIR", flag)
        ctx = B.Context(0)
        log(f"[pair] MSAO_PAIR={flag}")
        got, _, _ = run_and_compare(segs, R, default_params(), dev, ctx=ctx)
        outs.append({k: host(v).copy() for k, v in got.items()})
        ctx.close()
    for k in ("z", "d", "kept_idx", "keep", "kept_count", "agg", "dframe"):
        assert np.array_equal(outs[0][k], outs[1][k]), k


@pytest.mark.parametrize("requests", [1, 2, 4])
def test_small_video_batches_shorter_ranges(requests, dev):
    """One, two and four 32-frame clips of 256 positions: too few pairs of
    positions to give every SIMD a wavefront, so the planner halves the
    frame ranges (8, 8 and 16 frames: each range after the first re-reads
    the frame before it)."""
    from workloads import make_workload
    w = make_workload(3, n_requests=requests)
    log(f"[pair] video batch of {requests} clip(s)")
    run_and_compare(w.segments, requests, w.params, dev)
