"""msao_run_noalloc (the library's own scratch in place of a workspace)
against msao_run on the same inputs, through the C ABI: two calls in a row,
the second on a smaller table, so the second reads a scratch that still
holds the first call's tables and partials. Every output is compared
element by element: integer outputs, keep flags, kept indices and the
compacted rows bit-exact, and the float outputs too (the same kernels run on
the same inputs in the same order). The smaller call is also checked against
the oracle at the parity bar. A table whose tables exceed the scratch limit
is rejected on the host with nothing enqueued."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from paper_2604_02945_amd import binding as B
from workloads import make_workload

pytestmark = pytest.mark.gpu

FIELDS = ("z", "l1", "l2", "info", "d", "res", "dframe", "sim", "gamma", "agg", "rho", "temporal", "beta", "mas",
          "present", "keep", "kept_idx", "kept_count")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def to_device(w, dev):
    segs = []
    for s in w.segments:
        a = np.ascontiguousarray(s.data)
        t = torch.from_numpy(a.view(np.int16 if s.dtype == "bf16" else np.float32)).to(dev)
        if s.dtype == "bf16":
            t = t.view(torch.bfloat16)
        segs.append(msao.DeviceSegment(t, s.request, s.modality, s.keep_ratio, s.n_frames))
    return segs


def run_both(w, dev, ctx):
    """msao_run (workspace) and msao_run_noalloc (no workspace) on the same
    device inputs; returns both outputs on the host."""
    segs = to_device(w, dev)
    R, n = w.n_requests, len(segs)
    print(f"noalloc: {w.name} ({w.n_tokens} tokens, {n} segments)", flush=True)
    ref = msao.msao_run(segs, R, w.params, ctx=ctx)
    o = msao.Outputs(segs, R, workspace=False)
    assert o.workspace is None
    for v in list(o.tok.values()) + list(o.frm.values()) + list(o.req.values()) + list(o.sel.values()):
        v.fill_(0x5A if v.dtype == torch.uint8 else 7)  # stale values a missed write would leave
    o.out.fill_(0xA5)
    got = msao.msao_run_noalloc(segs, R, w.params, ctx=ctx, outputs=o)
    torch.cuda.synchronize()
    a, b = ref.results(R, n), got.results(R, n)
    return segs, {k: a[k].cpu().numpy() for k in FIELDS}, {k: b[k].cpu().numpy() for k in FIELDS}, ref, got


def check_equal(segs, a, b, ref_out, got_out):
    for k in FIELDS:
        assert a[k].dtype == b[k].dtype and a[k].shape == b[k].shape, k
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), f"{k} differs from msao_run's"
    kc = a["kept_count"]
    for x, y in zip(msao.compacted_rows(segs, ref_out, kc), msao.compacted_rows(segs, got_out, kc)):
        assert torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8)), "compacted rows"


def test_two_calls_second_smaller(dev):
    ctx = msao.Context(0)
    try:
        # call 1: the tri-modal batch (32 requests, 96 segments, 70,528 bf16 tokens)
        w4 = make_workload(4)
        segs, a, b, ro, go = run_both(w4, dev, ctx)
        check_equal(segs, a, b, ro, go)
        del segs, ro, go
        # call 2: one fp32 image and its text (608 tokens) on the same scratch
        w1 = make_workload(1)
        segs, a, b, ro, go = run_both(w1, dev, ctx)
        check_equal(segs, a, b, ro, go)
        ref = oracle.run(w1.segments, w1.n_requests, w1.params)
        assert np.array_equal(b["z"].astype(np.uint32), ref["z"])
        assert np.array_equal(b["kept_count"], ref["k"])
        assert np.array_equal(b["kept_idx"], ref["kept_idx"])
        assert np.array_equal(b["keep"], ref["keep"])
        assert np.allclose(b["l2"], ref["l2"], rtol=1e-5, atol=0)
        assert np.allclose(b["mas"], ref["mas"], rtol=1e-6, atol=1e-7)
        for r, want in zip(msao.compacted_rows(segs, go, ref["k"]), ref["compact"]):
            assert np.array_equal(r.cpu().numpy(), want)
        # call 3: a video batch (temporal chains, per-frame outputs) after the small one
        w3 = make_workload(3)
        segs, a, b, ro, go = run_both(w3, dev, ctx)
        check_equal(segs, a, b, ro, go)
    finally:
        ctx.close()


def test_tables_over_the_limit_are_rejected(dev):
    """600,000 rows of 8 bf16 channels kept at 0.9: one gather entry per kept
    row makes the tables about 2.2 MB, over MSAO_NOALLOC_TABLE_BYTES."""
    ctx = msao.Context(0)
    try:
        t = torch.zeros(600_000, 8, dtype=torch.bfloat16, device=dev)
        segs = [msao.DeviceSegment(t, 0, B.IMAGE, 0.9)]
        o = msao.Outputs(segs, 1, workspace=False)
        o.sel["kept_count"].fill_(-3)
        torch.cuda.synchronize()
        with pytest.raises(msao.MsaoError) as e:
            msao.msao_run_noalloc(segs, 1, ctx=ctx, outputs=o)
        assert e.value.status == 4 and "limits" in str(e.value)
        torch.cuda.synchronize()
        assert int(o.sel["kept_count"][0]) == -3  # nothing was enqueued
    finally:
        ctx.close()


if __name__ == "__main__":
    sys.exit(pytest.main([__file__, "-v"]))
