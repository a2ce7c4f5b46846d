"""A plan whose tables are uploaded on one stream and run on another: the
binding's Plan waits for the upload before it returns, so the first run on a
second stream already reads the whole tables. Outputs must equal a one-shot
msao_run of the same inputs bit for bit."""
import sys

import numpy as np
import pytest
import torch

import paper_2604_02945_amd as msao
from test_gpu_parity import to_device
from workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


@pytest.mark.parametrize("config", [3, 4])
def test_plan_uploaded_on_one_stream_runs_on_another(config, dev):
    w = make_workload(config, n_requests=8 if config == 4 else None)
    R, n = w.n_requests, len(w.segments)
    dsegs = to_device(w.segments, dev)
    print(f"[plan streams] config {config}", flush=True)
    sys.stdout.flush()
    ref = msao.msao_run(dsegs, R, w.params)
    torch.cuda.synchronize()
    want = {k: v.cpu().numpy() for k, v in ref.results(R, n).items()}
    up, run = torch.cuda.Stream(), torch.cuda.Stream()
    o = msao.Outputs(dsegs, R, compact=True)
    # a long kernel queued on the upload stream first, so that an unordered
    # run would see the workspace before the tables arrive
    with torch.cuda.stream(up):
        busy = torch.randn(1 << 24, device=dev)
        for _ in range(4):
            busy = busy * 1.0001 + 0.5
    plan = msao.Plan(dsegs, R, o, w.params, compact=True, stream=up)
    plan(run)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in o.results(R, n).items()}
    for k, v in want.items():
        assert np.array_equal(got[k].view(np.uint8), v.view(np.uint8)), k
    kc = want["kept_count"]
    for x, y in zip(msao.compacted_rows(dsegs, ref, kc), msao.compacted_rows(dsegs, o, kc)):
        assert torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))
    plan.close()
    del busy
