"""A plan run (the three launches of msao_run with the tables already in the
workspace: no upload, no memset) captured into a HIP graph and replayed:
every replay, with eager work and synchronisations between replays and the
outputs cleared eagerly before each one, must reproduce the eager run bit
for bit (statistics, aggregates, MAS, kept indices, compacted rows)."""
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


def snapshot(o, R, n):
    r = o.results(R, n)
    snap = {k: v.clone() for k, v in r.items()}
    snap["out"] = o.out.clone()
    return snap


def clear(o):
    for group in (o.tok, o.frm, o.req, o.sel):
        for t in group.values():
            t.fill_(0)
    o.out.fill_(0)


@pytest.mark.parametrize("config", [1, 4])
def test_plan_replays_from_a_graph(config, dev):
    w = make_workload(config, n_requests=4 if config == 4 else None)
    R, n = w.n_requests, len(w.segments)
    dsegs = to_device(w.segments, dev)
    o = msao.Outputs(dsegs, R, compact=True)
    ctx = msao.Context(0)
    plan = msao.Plan(dsegs, R, o, w.params, ctx=ctx, compact=True)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        plan(s)
    torch.cuda.synchronize()
    want = snapshot(o, R, n)
    print(f"[graph] config {config}: capture", flush=True)
    sys.stdout.flush()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan(torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(4):
        clear(o)
        junk = torch.randn(1 << 20, device=dev).sum()   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(o, R, n)
        for k, v in want.items():
            assert torch.equal(got[k], v), f"replay {rep}: {k}"
        del junk
    plan.close()
    ctx.close()
