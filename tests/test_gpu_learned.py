"""GPU parity of the learned probe heads (Eq. 3 with caller weights and AvgPool,
Eq. 4 on them, the Eq. 6 relevance MLP on [prompt; z_m]) against the oracle,
through msao_mas_score_learned.

Tolerances. The projection y = w . x is a float32 sum of C products exact in
float32 (bf16 inputs) or rounded once (fp32), so |dy| <= (C + 64) 2^-24
sum_c |w_c x_c|; the window mean and the bias add a few ulps, and sigmoid has
slope <= 1/4, so |dM| <= (C + 80) 2^-26 max over the window of sum_c |w_c x_c|
+ 2^-22. A head token whose oracle importance lies within that bound of
tau_s may fall on either side: the sparse counts may differ by at most the
number of such tokens. Descriptors: z0, z2, z5, z6, z7 are float32 roundings
of doubles computed from exact integers (one ulp, 2^-23 relative); z3 and
z4 come from float32 per-token L1/L2 sums (at most (C/64 + 136) 2^-24
relative, < 3e-5 for C <= 4104). alpha is Eq. 6 in float32: with v the
float32 input [p; z], |d alpha| <= sum_j |w2_j| (IN + 2) 2^-24 (|b1_j| +
sum_k |W1_jk v_k|) + (hidden + 6) 2^-24 sum_j |w2_j relu(h_j)| plus what the
descriptor tolerances carry through W1. The softmax has gradient rows of
1-norm <= 1/2, so |d beta| <= max |d alpha| / 2 + 2^-22, and MAS <= beta
moves by no more.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from paper_2604_02945_amd import binding as B
from workloads import (AUDIO, IMAGE, TEXT, VIDEO, Segment, bf16_bits_to_f32, default_params, f32_to_bf16_bits,
                       make_workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(segments, dev):
    out = []
    for s in segments:
        a = np.ascontiguousarray(s.data)
        t = torch.from_numpy(a.view(np.int16) if s.dtype == "bf16" else a).to(dev)
        if s.dtype == "bf16":
            t = t.view(torch.bfloat16)
        out.append(msao.DeviceSegment(t, s.request, s.modality, s.keep_ratio, s.n_frames))
    return out


def make_head(s, rng, grid_w, pool, bias):
    w32 = (rng.standard_normal(s.hidden) * (1.5 / math.sqrt(s.hidden))).astype(np.float32)
    host = w32 if s.dtype == "f32" else f32_to_bf16_bits(w32)
    return host, dict(weight=host, bias=bias, grid_w=grid_w, pool=pool)


def head_bound(s, w_host, grid_w, pool):
    """Per-token bound on |M_gpu - M_oracle| (see the module docstring)."""
    x = (s.data if s.dtype == "f32" else bf16_bits_to_f32(s.data))[:, :s.hidden].astype(np.float64)
    w = (w_host if s.dtype == "f32" else bf16_bits_to_f32(w_host)).astype(np.float64)
    mag = np.abs(x) @ np.abs(w)
    P = s.tokens_per_frame
    W = grid_w if grid_w > 0 else P
    H = P // W
    r = (pool - 1) // 2
    m = mag.reshape(s.n_frames, H, W)
    win = np.zeros_like(m)
    for di in range(-r, r + 1):
        for dj in range(-r, r + 1):
            if abs(di) >= H or abs(dj) >= W:
                continue  # the shifted window lies outside the grid (and a negative stop would wrap)
            sh = np.full_like(m, 0.0)
            src = m[:, max(0, di):H + min(0, di), max(0, dj):W + min(0, dj)]
            sh[:, max(0, -di):H - max(0, di), max(0, -dj):W - max(0, dj)] = src
            win = np.maximum(win, sh)
    return ((s.hidden + 80) * 2.0 ** -26 * win + 2.0 ** -22).reshape(-1)


def run_case(segs, R, heads, mlp_host, dev, params=None, alpha=None):
    p = params or default_params()
    dsegs = to_device(segs, dev)
    hdev = None
    if heads is not None:
        hdev = []
        for s, h in zip(segs, heads):
            if h is None:
                hdev.append(None)
                continue
            w = torch.from_numpy(h["weight"].view(np.int16) if s.dtype == "bf16" else h["weight"]).to(dev)
            hdev.append(dict(weight=w, bias=h["bias"], grid_w=h["grid_w"], pool=h["pool"]))
    mdev = None
    if mlp_host is not None:
        mdev = {k: torch.from_numpy(np.ascontiguousarray(mlp_host[k], dtype=np.float32)).to(dev)
                for k in ("w1", "b1", "w2", "prompt")}
        mdev["b2"] = mlp_host["b2"]
    out, extra = msao.msao_mas_score_learned(dsegs, R, p, heads=hdev, mlp=mdev, alpha=alpha)
    torch.cuda.synchronize()
    got = out.results(R, len(segs))
    g = {k: v.cpu().numpy() for k, v in got.items()}
    for k in ("importance", "alpha", "desc"):
        g[k] = extra[k].cpu().numpy()
    ref = oracle.run_learned(segs, R, p, heads, mlp_host)
    return g, ref


def alpha_bound(mlp, zr, zg, R):
    """Per-(request, modality) bound on |alpha_gpu - alpha_oracle| (module docstring)."""
    if mlp is None:
        return np.zeros(R * 4)
    w1, b1, w2 = (np.asarray(mlp[k], np.float64) for k in ("w1", "b1", "w2"))
    prompt = np.asarray(mlp["prompt"], np.float64)
    IN, Hd = w1.shape[1], w1.shape[0]
    u = 2.0 ** -24
    dz = np.zeros(8)
    dz[[0, 2, 5, 6, 7]] = 2.0 ** -23
    dz[[3, 4]] = 3e-5
    out = np.zeros(R * 4)
    for x in range(R * 4):
        v = np.concatenate([prompt[x // 4], zr[x]])
        if zr[x, 0] == 0:
            continue
        absv = np.abs(v)
        h = w1 @ v + b1
        hs = np.abs(b1) + np.abs(w1) @ absv
        dzv = np.concatenate([np.zeros(prompt.shape[1]), dz * np.abs(zr[x]) + u * np.abs(zr[x])])
        dh = (IN + 2) * u * hs + np.abs(w1) @ dzv + np.abs(zr[x, 1] - zg[x, 1]) * np.abs(w1[:, prompt.shape[1] + 1])
        out[x] = np.abs(w2) @ dh + (Hd + 6) * u * np.abs(w2) @ np.maximum(h, 0) + u
    return out


def compare(segs, R, heads, g, ref, mlp=None):
    # per-token statistics: exact integers
    assert np.array_equal(g["z"].astype(np.uint32), ref["z"])
    assert np.array_equal(g["d"].astype(np.uint32), ref["d"])
    # importance, and the borderline head tokens per (request, modality)
    border = np.zeros(R * 4, np.int64)
    off = 0
    for i, s in enumerate(segs):
        N = s.n_tokens
        gi, ri = g["importance"][off:off + N], ref["importance"][off:off + N]
        h = heads[i] if heads is not None else None
        if h is None:
            a = s.hidden - ref["z"][off:off + N].astype(np.int64)
            assert np.array_equal(gi, (a / s.hidden).astype(np.float32)), f"density importance of segment {i}"
        else:
            bnd = head_bound(s, h["weight"], h["grid_w"], h["pool"])
            assert np.all(np.abs(gi - ri) <= bnd), f"head importance of segment {i}: {np.max(np.abs(gi - ri) - bnd)}"
            border[s.request * 4 + s.modality] += int(np.sum(np.abs(ri - default_params()["tau_s"]) <= bnd))
        off += N
    agg_g = g["agg"].astype(np.uint64).reshape(-1, 4)
    agg_r = ref["agg"].reshape(-1, 4)
    for c in (0, 2, 3):
        assert np.array_equal(agg_g[:, c], agg_r[:, c])
    dcount = np.abs(agg_g[:, 1].astype(np.int64) - agg_r[:, 1].astype(np.int64))
    assert np.all(dcount <= border), (dcount, border)
    exact_counts = bool(np.all(dcount == 0))
    pres = ref["present"].astype(bool)
    assert np.array_equal(g["present"].astype(bool), pres)
    zg = g["desc"].reshape(-1, 8)
    zr = ref["desc"]
    for k in (0, 2, 5, 6, 7):
        np.testing.assert_allclose(zg[:, k], zr[:, k], rtol=2.0 ** -23, atol=0, err_msg=f"z{k}")
    for k in (3, 4):
        np.testing.assert_allclose(zg[:, k], zr[:, k], rtol=3e-5, atol=0, err_msg=f"z{k}")
    ntok = np.maximum(agg_r[:, 0].astype(np.float64), 1)
    assert np.all(np.abs(zg[:, 1] - zr[:, 1]) <= border / ntok + 2.0 ** -23 * np.abs(zr[:, 1]))
    if exact_counts:
        da = alpha_bound(mlp, zr, zg, R)
        assert np.all(np.abs(g["alpha"] - ref["alpha"]) <= da), (g["alpha"], ref["alpha"], da)
        tb = 0.5 * float(np.max(da)) + 2.0 ** -22
        np.testing.assert_allclose(g["beta"], ref["beta"], rtol=0, atol=tb)
        np.testing.assert_allclose(g["mas"], ref["mas"], rtol=0, atol=tb)
        np.testing.assert_allclose(g["rho"], ref["rho"], rtol=2.0 ** -23, atol=0)
    return exact_counts


def mlp_for(R, P, H, rng):
    return dict(w1=(rng.standard_normal((H, P + 8)) * 0.2).astype(np.float32),
                b1=(rng.standard_normal(H) * 0.1).astype(np.float32),
                w2=(rng.standard_normal(H) * 0.3).astype(np.float32), b2=0.1,
                prompt=rng.standard_normal((R, P)).astype(np.float32))


def test_heads_and_mlp_trimodal(dev):
    w = make_workload(4, n_requests=3)
    rng = np.random.default_rng(11)
    heads = []
    for s in w.segments:
        if s.modality == IMAGE:
            heads.append(make_head(s, rng, 24, 3, -0.8)[1])
        elif s.modality == AUDIO:
            heads.append(make_head(s, rng, 0, 5, -0.2)[1])     # one row of 1500 frames, 1-D window
        else:
            heads.append(None)                                   # text keeps the density test
    mlp = mlp_for(3, 32, 64, rng)
    log("[learned] trimodal, heads on image and audio, MLP 64 x (32 + 8)")
    g, ref = run_case(w.segments, 3, heads, mlp, dev)
    exact = compare(w.segments, 3, heads, g, ref, mlp)
    log(f"[learned] counts exact: {exact}; alpha {np.round(g['alpha'][:4], 4)}")


def test_heads_on_video_and_odd_widths(dev):
    rng = np.random.default_rng(12)
    clip = make_workload(3, n_requests=1).segments[0]
    x = rng.standard_normal((9 * 20, 4104)).astype(np.float32)
    wide = Segment(1, IMAGE, 1, 180, 4104, "bf16", 0.5, f32_to_bf16_bits(x))       # generic row path
    v = rng.standard_normal((4 * 12, 4104)).astype(np.float32)
    wide_clip = Segment(1, VIDEO, 4, 12, 4104, "bf16", 0.5, f32_to_bf16_bits(v))   # generic chain path
    f = rng.standard_normal((30, 520)).astype(np.float32)
    f32seg = Segment(2, AUDIO, 1, 30, 520, "f32", 0.5, f)
    t = rng.standard_normal((7, 64)).astype(np.float32)
    txt = Segment(2, TEXT, 1, 7, 64, "f32", 1.0, t)
    segs = [clip, wide, wide_clip, f32seg, txt]
    heads = [make_head(clip, rng, 16, 3, 0.0)[1], make_head(wide, rng, 20, 5, 0.2)[1],
             make_head(wide_clip, rng, 4, 1, -0.3)[1], make_head(f32seg, rng, 0, 3, 0.1)[1], None]
    mlp = mlp_for(3, 0, 16, rng)
    log("[learned] video clip, generic widths, fp32; MLP without prompt")
    g, ref = run_case(segs, 3, heads, mlp, dev)
    compare(segs, 3, heads, g, ref, mlp)


def test_windows_wider_than_the_grid(dev):
    # pooling windows of 5 and 7 on grids 1 or 2 patches wide (and 1 row
    # high): the window is cut to the grid on every side
    rng = np.random.default_rng(21)
    segs, heads = [], []
    for i, (P, W, pool, dtype) in enumerate([(9, 1, 7, "bf16"), (14, 2, 5, "bf16"), (3, 3, 7, "f32"),
                                             (40, 2, 7, "f32"), (6, 0, 5, "bf16")]):
        x = rng.standard_normal((P, 200)).astype(np.float32)
        s = Segment(i % 2, IMAGE if i % 2 == 0 else AUDIO, 1, P, 200, dtype, 0.5,
                    x if dtype == "f32" else f32_to_bf16_bits(x))
        segs.append(s)
        heads.append(make_head(s, rng, W, pool, float(rng.uniform(-0.5, 0.5)))[1])
    log("[learned] windows wider than the grid")
    g, ref = run_case(segs, 2, heads, None, dev)
    compare(segs, 2, heads, g, ref)


def test_mlp_without_heads_many_requests(dev):
    # the head launch runs only prompt-product blocks; 10 requests make a
    # ragged group of the 8 requests one wavefront serves
    w = make_workload(4, n_requests=10)
    rng = np.random.default_rng(13)
    mlp = mlp_for(10, 200, 96, rng)
    log("[learned] MLP 96 x (200 + 8), no heads, 10 requests")
    g, ref = run_case(w.segments, 10, None, mlp, dev)
    assert compare(w.segments, 10, None, g, ref, mlp)


def test_without_heads_or_mlp_it_is_mas_score(dev):
    w = make_workload(4, n_requests=2)
    alpha = [0.5, -0.25, 0.0, 1.0, 0.0, 0.0, 0.0, 0.0]
    g, ref = run_case(w.segments, 2, None, None, dev, alpha=None)
    compare(w.segments, 2, None, g, ref)
    plain = oracle.run(w.segments, 2, w.params)
    np.testing.assert_allclose(g["mas"], plain["mas"], rtol=0, atol=1e-6)
    # host logits instead of the MLP
    dsegs = to_device(w.segments, dev)
    out, extra = msao.msao_mas_score_learned(dsegs, 2, w.params, alpha=alpha)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.req["beta"].cpu().numpy()[:8], oracle.run(w.segments, 2, w.params,
                                                                             np.array(alpha, np.float32))["beta"],
                               rtol=1e-6, atol=0)


def test_learned_rejects_bad_heads(dev):
    w = make_workload(1)
    dsegs = to_device(w.segments, dev)
    wt = torch.zeros(w.segments[0].hidden, dtype=torch.float32, device=dev)
    for bad, code in ((dict(weight=wt, pool=2), 1), (dict(weight=wt, pool=17), 1), (dict(weight=wt, grid_w=7), 1),
                      (dict(weight=wt[1:], pool=1), 2)):
        with pytest.raises(B.MsaoError) as e:
            msao.msao_mas_score_learned(dsegs, 1, w.params, heads=[bad, None])
        assert e.value.status == code
