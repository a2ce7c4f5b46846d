"""GPU parity of the per-frame selection scope (MSAO_FLAG_SELECT_PER_FRAME):
every frame of a clip keeps its own k_f = ceil(kappa P) tokens. Through the
C ABI against the oracle with the same flag: keep counts, keep flags, kept
indices and compacted rows bit-exact; the statistics are those of the plain
run (checked by run_and_compare as well)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from test_gpu_parity import compare_selection, host, log, run_and_compare, to_device
from workloads import IMAGE, TEXT, VIDEO, Segment, default_params, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def per_frame(p):
    q = dict(p)
    q["flags"] = q.get("flags", 0) | msao.FLAG_SELECT_PER_FRAME
    return q


def with_keep(segs, keep):
    return [Segment(s.request, s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype, keep, s.data)
            for s in segs]


@pytest.mark.parametrize("keep", [0.3, -1.0, 0.0, 1.0])
def test_video_clips_per_frame(keep, dev):
    w = make_workload(3, n_requests=3)
    segs = with_keep(w.segments, keep)
    log(f"[scope] 3 clips x 32 frames x 256 tokens, keep {keep}")
    got, ref, _ = run_and_compare(segs, 3, per_frame(w.params), dev)
    T, P = segs[0].n_frames, segs[0].tokens_per_frame
    kc = host(got["kept_count"])
    assert np.all(kc % T == 0) and np.all(kc // T <= P)


def test_mixed_batch_and_plain_run_unchanged(dev):
    rng = np.random.default_rng(21)
    clip = make_workload(3, n_requests=1).segments[0]
    x = rng.standard_normal((5 * 37, 72)).astype(np.float32)
    small = Segment(1, VIDEO, 5, 37, 72, "f32", 0.45, x)       # ragged frames
    img = make_workload(1).segments[0]
    img = Segment(1, IMAGE, 1, img.tokens_per_frame, img.hidden, img.dtype, 0.5, img.data)
    txt = Segment(0, TEXT, 1, 9, 64, "f32", 1.0, rng.standard_normal((9, 64)).astype(np.float32))
    segs = [clip, small, img, txt]
    p = default_params()
    log("[scope] mixed batch: clip, ragged fp32 clip, image, text")
    run_and_compare(segs, 2, per_frame(p), dev)
    # single-frame segments select as before; the clips differ from the plain run
    a = oracle.run(segs, 2, p)
    b = oracle.run(segs, 2, per_frame(p))
    assert a["k"][2] == b["k"][2] and a["k"][3] == b["k"][3]


def test_select_entry_point_per_frame(dev):
    w = make_workload(3, n_requests=2)
    segs = with_keep(w.segments, -1.0)
    p = per_frame(w.params)
    ref = oracle.run(segs, 2, p)
    dsegs = to_device(segs, dev)
    z = torch.from_numpy(ref["z"].astype(np.int32)).to(dev)
    d = torch.from_numpy(ref["d"].astype(np.int32)).to(dev)
    mas = torch.from_numpy(ref["mas"]).to(dev)
    out = msao.msao_select_tokens(dsegs, 2, z, d, mas, p)
    torch.cuda.synchronize()
    got = out.results(2, len(segs))
    compare_selection(segs, 2, got, ref, p)


def test_plan_per_frame(dev):
    w = make_workload(3, n_requests=2)
    p = per_frame(w.params)
    dsegs = to_device(w.segments, dev)
    o = msao.Outputs(dsegs, 2, compact=True)
    plan = msao.Plan(dsegs, 2, o, p, compact=True)
    ref = oracle.run(w.segments, 2, p)
    for _ in range(2):
        plan()
        torch.cuda.synchronize()
        got = o.results(2, len(dsegs))
        assert np.array_equal(host(got["kept_count"]), ref["k"])
        assert np.array_equal(host(got["kept_idx"]), ref["kept_idx"])
    plan.close()


def test_select_then_compact_per_frame(dev):
    # the standalone compaction does not know the scope: 32 x ceil(0.3 * 256)
    # = 2,464 kept rows per clip exceed ceil(0.3 * 8192) = 2,458, and all of
    # them must be copied
    w = make_workload(3, n_requests=2)
    p = per_frame(w.params)
    ref = oracle.run(w.segments, 2, p)
    assert np.all(ref["k"] == 2464)
    dsegs = to_device(w.segments, dev)
    z = torch.from_numpy(ref["z"].astype(np.int32)).to(dev)
    d = torch.from_numpy(ref["d"].astype(np.int32)).to(dev)
    out = msao.Outputs(dsegs, 2, compact=True)
    msao.msao_select_tokens(dsegs, 2, z, d, None, p, outputs=out)
    msao.msao_compact(dsegs, out)
    torch.cuda.synchronize()
    got = out.results(2, len(dsegs))
    assert np.array_equal(host(got["kept_count"]), ref["k"])
    from test_gpu_parity import compare_compaction
    compare_compaction(dsegs, w.segments, out, oracle.compact_rows(w.segments, ref["k"], ref["kept_idx"]), ref["k"])
