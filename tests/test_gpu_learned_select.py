"""GPU parity of the selection by the learned importance (msao_run_learned:
Sec. 4.1.1 pruning of the patches whose Eq. 3 importance M is low) against
the oracle's learned run.

Bar. The scoring outputs equal msao_mas_score_learned's bit for bit (the
same kernels). For a segment without a head the kept indices equal the
oracle's (the exact integer key of msao_run). For a segment with a head the
GPU ranks its own float32 M, whose distance from the oracle's double M is at
most the per-token bound b_i of tests/test_gpu_learned.py (projection
rounding, window mean, sigmoid slope <= 1/4); with v the oracle's k-th
largest M and B = max b_i, every token with oracle M > v + 2B must be kept
and every token with oracle M < v - 2B dropped (the GPU's k-th largest M lies
within B of v), and the kept set must be exactly the k largest of the GPU's
own M, ties by index (a NaN or non-positive M as 0). Keep counts: fixed ones
exact; a MAS-guided one either equals the oracle's or is the ceil of
(1 - MAS) N from the GPU's own MAS (a MAS on a ceil boundary). Compacted
rows equal the input rows at the kept indices, byte for byte."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from test_gpu_learned import head_bound, make_head, to_device
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def device_heads(segs, heads, dev):
    out = []
    for s, h in zip(segs, heads):
        if h is None:
            out.append(None)
            continue
        w = torch.from_numpy(h["weight"].view(np.int16) if s.dtype == "bf16" else h["weight"]).to(dev)
        out.append(dict(weight=w, bias=h["bias"], grid_w=h["grid_w"], pool=h["pool"]))
    return out


def device_mlp(mlp, dev):
    if mlp is None:
        return None
    m = {k: torch.from_numpy(np.ascontiguousarray(mlp[k], dtype=np.float32)).to(dev) for k in ("w1", "b1", "w2", "prompt")}
    m["b2"] = mlp["b2"]
    return m


def imp_rank_key(m):
    """The selection order of importances: NaN and values not above 0 count as 0."""
    m = np.asarray(m, np.float64)
    return np.where(m > 0, m, 0.0)


def top_k(m, k):
    order = np.lexsort((np.arange(m.size), -imp_rank_key(m)))
    return np.sort(order[:k])


def run_and_check(segs, R, heads, mlp, dev, params=None):
    p = params or default_params()
    dsegs = to_device(segs, dev)
    dh, dm = device_heads(segs, heads, dev), device_mlp(mlp, dev)
    log(f"[learned select] {len(segs)} segments, {sum(s.n_tokens for s in segs)} tokens")
    out, extra = msao.msao_run_learned(dsegs, R, p, heads=dh, mlp=dm)
    base, bextra = msao.msao_mas_score_learned(dsegs, R, p, heads=dh, mlp=dm)
    torch.cuda.synchronize()
    n = len(segs)
    g = {k: v.cpu().numpy() for k, v in out.results(R, n).items()}
    b = {k: v.cpu().numpy() for k, v in base.results(R, n).items()}
    imp = extra["importance"].cpu().numpy()
    # the scoring outputs are those of msao_mas_score_learned
    for k in ("z", "l1", "l2", "info", "d", "res", "agg", "rho", "temporal", "beta", "mas", "present"):
        assert np.array_equal(g[k].view(np.uint8), b[k].view(np.uint8)), k
    assert np.array_equal(imp.view(np.uint8), bextra["importance"].cpu().numpy().view(np.uint8))
    ref = oracle.run_learned(segs, R, p, heads, mlp)
    rows = msao.compacted_rows(dsegs, out, g["kept_count"])
    off = 0
    borderline = 0
    for i, s in enumerate(segs):
        N = s.n_tokens
        k = int(g["kept_count"][i])
        kept = g["kept_idx"][off:off + N]
        assert np.all(kept[k:] == -1) and np.all(np.diff(kept[:k]) > 0)
        kept = kept[:k].astype(np.int64)
        if k != int(ref["k"][i]):
            assert s.keep_ratio < 0, f"segment {i}: keep count {k} vs {ref['k'][i]}"
            mas = float(g["mas"][s.request * 4 + s.modality])
            assert k == min(N, math.ceil((1.0 - np.float64(np.float32(mas))) * N))
        per_frame = (p.get("flags", 0) & 2) and s.n_frames >= 2
        units = [(t * s.tokens_per_frame, (t + 1) * s.tokens_per_frame) for t in range(s.n_frames)] if per_frame \
            else [(0, N)]
        ku = k // len(units)
        h = heads[i] if heads is not None else None
        for u0, u1 in units:
            mine = kept[(kept >= u0) & (kept < u1)]
            assert mine.size == ku
            if h is None:
                want = ref["kept_idx"][off:off + N]
                want = want[want >= 0]
                np.testing.assert_array_equal(mine, want[(want >= u0) & (want < u1)])
                continue
            mg = imp[off + u0:off + u1]
            mo = ref["importance"][off + u0:off + u1]
            # exactly the k largest of the GPU's own importance, ties by index
            np.testing.assert_array_equal(mine - u0, top_k(mg, ku))
            if ku == 0 or ku == u1 - u0:
                continue
            bnd = head_bound(s, h["weight"], h["grid_w"], h["pool"])[u0:u1]
            B = float(bnd.max())
            ro = imp_rank_key(mo)
            v = np.sort(ro)[::-1][ku - 1]
            sure_in = np.flatnonzero(ro > v + 2 * B)
            sure_out = np.flatnonzero(ro < v - 2 * B)
            kept_local = mine - u0
            assert np.isin(sure_in, kept_local).all(), f"segment {i}: a clearly important token was dropped"
            assert not np.isin(sure_out, kept_local).any(), f"segment {i}: a clearly unimportant token was kept"
            borderline += (u1 - u0) - sure_in.size - sure_out.size
        # compacted rows are the input rows at the kept indices
        got_rows = rows[i].contiguous().cpu().view(torch.uint8).numpy()
        assert np.array_equal(got_rows.reshape(-1), np.ascontiguousarray(s.data[kept]).view(np.uint8).reshape(-1))
        off += N
    log(f"[learned select] borderline head tokens: {borderline}")
    return g, ref


def trimodal(R, guided=False):
    w = make_workload(4, n_requests=R)
    rng = np.random.default_rng(17)
    heads = []
    for s in w.segments:
        if guided and s.modality in (IMAGE, AUDIO):
            s.keep_ratio = -1.0
        if s.modality == IMAGE:
            heads.append(make_head(s, rng, 24, 3, -0.8)[1])
        elif s.modality == AUDIO:
            heads.append(make_head(s, rng, 0, 5, -0.2)[1])
        else:
            heads.append(None)
    pd, hid = 32, 64
    mlp = {"w1": (rng.standard_normal((hid, pd + 8)) * 0.1).astype(np.float32),
           "b1": (rng.standard_normal(hid) * 0.1).astype(np.float32),
           "w2": (rng.standard_normal(hid) * 0.2).astype(np.float32), "b2": 0.05,
           "prompt": rng.standard_normal((R, pd)).astype(np.float32)}
    return w, heads, mlp


def test_trimodal_fixed_keep_ratios(dev):
    w, heads, mlp = trimodal(6)
    run_and_check(w.segments, 6, heads, mlp, dev, w.params)


def test_trimodal_mas_guided(dev):
    w, heads, mlp = trimodal(6, guided=True)
    run_and_check(w.segments, 6, heads, mlp, dev, w.params)


@pytest.mark.parametrize("per_frame", [False, True])
def test_video_clip_with_a_head(per_frame, dev):
    w = make_workload(3, n_requests=2)
    rng = np.random.default_rng(23)
    heads = [make_head(s, rng, 16, 3, 0.1)[1] for s in w.segments]
    p = dict(w.params)
    p["flags"] = 2 if per_frame else 0
    run_and_check(w.segments, 2, heads, None, dev, p)


def test_nan_rows_and_fp32_segment(dev):
    rng = np.random.default_rng(29)
    x = rng.standard_normal((24 * 24, 520)).astype(np.float32)
    x[[5, 77, 300], 11] = np.nan
    img = Segment(0, IMAGE, 1, 576, 520, "f32", 0.3, x)
    txt = Segment(0, TEXT, 1, 40, 520, "f32", 0.5, rng.standard_normal((40, 520)).astype(np.float32))
    heads = [make_head(img, rng, 24, 1, 0.0)[1], None]
    g, ref = run_and_check([img, txt], 1, heads, None, dev)
    kept = g["kept_idx"][:int(g["kept_count"][0])]
    assert not np.isin([5, 77, 300], kept).any()


def test_argument_errors(dev):
    w, heads, mlp = trimodal(1)
    dsegs = to_device(w.segments, dev)
    dh = device_heads(w.segments, heads, dev)
    bad = [dict(h, pool=4) if h is not None else None for h in dh]
    with pytest.raises(msao.MsaoError) as e:
        msao.msao_run_learned(dsegs, 1, w.params, heads=bad)
    assert e.value.status == 1


@pytest.mark.parametrize("keep", [0.3, -1.0])
def test_clip_with_a_head_beyond_lds_staging(keep, dev):
    """A clip of 18,000 tokens with a head: more keys than the selection
    stages in LDS, so every pass recomputes the importance keys from memory."""
    rng = np.random.default_rng(31)
    T, P, C = 3, 6000, 64
    x = rng.standard_normal((T * P, C)).astype(np.float32)
    clip = Segment(0, VIDEO, T, P, C, "bf16", keep, f32_to_bf16_bits(x))
    img = Segment(0, IMAGE, 1, 576, C, "bf16", 0.25, f32_to_bf16_bits(rng.standard_normal((576, C)).astype(np.float32)))
    heads = [make_head(clip, rng, 100, 3, 0.2)[1], make_head(img, rng, 24, 3, -0.4)[1]]
    run_and_check([clip, img], 1, heads, None, dev)


def test_prepared_call_matches_one_shot(dev):
    """prepare_learned marshals msao_run_learned once: two calls of it give the
    one-shot call's outputs byte for byte (scores, selection, compacted rows)."""
    w, heads, mlp = trimodal(3)
    segs, R, p = w.segments, 3, w.params
    dsegs = to_device(segs, dev)
    dh, dm = device_heads(segs, heads, dev), device_mlp(mlp, dev)
    one, oextra = msao.msao_run_learned(dsegs, R, p, heads=dh, mlp=dm)
    outs = msao.Outputs(dsegs, R)
    call, extra = msao.binding.prepare_learned(dsegs, R, outs, p, heads=dh, mlp=dm)
    log("[learned select] prepared call, twice")
    for _ in range(2):
        call()
        torch.cuda.synchronize()
        a = {k: v.cpu().numpy() for k, v in one.results(R, len(segs)).items()}
        b = {k: v.cpu().numpy() for k, v in outs.results(R, len(segs)).items()}
        for k in a:
            assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k
        assert np.array_equal(oextra["importance"].cpu().numpy().view(np.uint8),
                              extra["importance"].cpu().numpy().view(np.uint8))
        ra = msao.compacted_rows(dsegs, one, a["kept_count"])
        rb = msao.compacted_rows(dsegs, outs, b["kept_count"])
        for x, y in zip(ra, rb):
            assert torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))
