"""Pins of the learned probe heads in the oracle (Sec. 4.1.1 Eq. 3 with a
caller 1x1 convolution and AvgPool window; Sec. 4.1.3 Eq. 6 with a caller
MLP on [prompt; z_m]) against library routines, the pooling/convolution
identity computed the other way round, closed forms and the plain path."""
import math

import numpy as np
import pytest
from scipy.special import expit, softmax

import oracle
from workloads import IMAGE, TEXT, VIDEO, AUDIO, Segment, bf16_bits_to_f32, default_params, make_workload


def feats(s):
    x = s.data if s.dtype == "f32" else bf16_bits_to_f32(s.data)
    return x[:, :s.hidden].astype(np.float64)


def wt(s, rng):
    w = (rng.standard_normal(s.hidden) * 0.05).astype(np.float32)
    if s.dtype == "bf16":
        from workloads import f32_to_bf16_bits
        return f32_to_bf16_bits(w)
    return w


def wt64(s, w):
    return (w if s.dtype == "f32" else bf16_bits_to_f32(w)).astype(np.float64)


def test_without_heads_and_mlp_it_is_the_plain_analysis():
    w = make_workload(4, n_requests=2)
    a = oracle.run(w.segments, 2, w.params)
    b = oracle.run_learned(w.segments, 2, w.params)
    for k in ("agg", "rho", "beta", "mas", "present", "z", "d"):
        assert np.array_equal(a[k], b[k]), k
    off = 0
    for s in w.segments:
        N = s.n_tokens
        np.testing.assert_allclose(b["importance"][off:off + N], (s.hidden - a["z"][off:off + N]) / s.hidden,
                                   rtol=0, atol=0)
        off += N
    assert np.all(b["alpha"] == 0.0)


def test_head_without_pooling_is_a_sigmoid_of_a_projection():
    w = make_workload(1)
    rng = np.random.default_rng(1)
    heads = [dict(weight=wt(s, rng), bias=0.25, grid_w=24 if s.modality == IMAGE else 0, pool=1) for s in w.segments]
    o = oracle.run_learned(w.segments, 1, w.params, heads)
    off = 0
    for s, h in zip(w.segments, heads):
        want = expit(feats(s) @ wt64(s, h["weight"]) + 0.25)  # 0.25 is exact in float
        np.testing.assert_allclose(o["importance"][off:off + s.n_tokens], want, rtol=1e-12, atol=1e-15)
        off += s.n_tokens


@pytest.mark.parametrize("pool", [3, 5])
def test_pooled_projection_equals_projected_pooled_features(pool):
    """Conv1x1(AvgPool(F)): average the features over each window cut to the
    grid, then project (this side), against the oracle's average of projections."""
    w = make_workload(3, n_requests=1)           # one clip: 32 frames of a 16 x 16 grid
    s = w.segments[0]
    rng = np.random.default_rng(2)
    h = dict(weight=wt(s, rng), bias=-0.1, grid_w=16, pool=pool)
    o = oracle.run_learned([s], 1, w.params, [h])
    F = feats(s).reshape(s.n_frames, 16, 16, s.hidden)
    wv = wt64(s, h["weight"])
    r = (pool - 1) // 2
    for t in (0, 1, 31):
        for i in range(16):
            for j in range(16):
                win = F[t, max(0, i - r):i + r + 1, max(0, j - r):j + r + 1].reshape(-1, s.hidden)
                want = expit(win.mean(axis=0) @ wv + float(np.float32(-0.1)))   # the bias is a float
                got = o["importance"][t * 256 + i * 16 + j]
                assert got == pytest.approx(want, rel=1e-10), (t, i, j)


def test_pooling_on_a_non_square_grid():
    """A 6 x 10 grid (grid_w = 10), window 3: rows and columns must not swap."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((60, 16)).astype(np.float32)
    s = Segment(0, IMAGE, 1, 60, 16, "f32", 1.0, x)
    wv = rng.standard_normal(16).astype(np.float32)
    o = oracle.run_learned([s], 1, default_params(), [dict(weight=wv, bias=0.0, grid_w=10, pool=3)])
    F = x.astype(np.float64).reshape(6, 10, 16)
    for i in range(6):
        for j in range(10):
            win = F[max(0, i - 1):i + 2, max(0, j - 1):j + 2].reshape(-1, 16)
            assert o["importance"][i * 10 + j] == pytest.approx(expit(win.mean(axis=0) @ wv), rel=1e-12)


def test_pool_window_edges_hand_worked():
    # one frame of a 2 x 3 grid, one channel, weight 1, bias 0; projections 1..6 row-major.
    # 3 x 3 windows cut to the grid: corners average 4 patches, edge middles 6:
    # (0,0): (1+2+4+5)/4 = 3, (0,1): 21/6 = 3.5, (0,2): (2+3+5+6)/4 = 4, row 1 the same.
    x = np.arange(1, 7, dtype=np.float32).reshape(6, 1)
    x = np.concatenate([x, np.zeros((6, 3), np.float32)], axis=1)        # hidden 4, channels 1..3 zero
    s = Segment(0, IMAGE, 1, 6, 4, "f32", 1.0, x)
    h = dict(weight=np.array([1, 0, 0, 0], np.float32), bias=0.0, grid_w=3, pool=3)
    o = oracle.run_learned([s], 1, default_params(), [h])
    np.testing.assert_allclose(o["importance"], expit([3.0, 3.5, 4.0, 3.0, 3.5, 4.0]), rtol=1e-15)


def test_head_bias_extremes_fix_rho():
    w = make_workload(1)
    p = w.params
    img = [s for s in w.segments if s.modality == IMAGE][0]
    rng = np.random.default_rng(3)
    for bias, rho in ((60.0, 0.0), (-60.0, 1.0)):
        o = oracle.run_learned([img], 1, p, [dict(weight=wt(img, rng), bias=bias, grid_w=24, pool=3)])
        assert o["rho"][IMAGE] == rho
        lam = p["lambda_s"][IMAGE]
        assert o["mas"][IMAGE] == pytest.approx(1 - 1.0 * (1 - lam * rho), rel=1e-7)   # beta = 1


def test_descriptor_against_numpy():
    w = make_workload(4, n_requests=1)
    p = w.params
    o = oracle.run_learned(w.segments, 1, p)
    for s in w.segments:
        z = o["desc"][s.modality]
        x = feats(s)
        assert z[0] == 1.0
        assert z[1] == pytest.approx(o["rho"][s.modality], rel=1e-7)
        assert z[2] == pytest.approx(np.mean(np.abs(x) > np.float32(p["tau"])), rel=1e-12)
        assert z[3] == pytest.approx(np.mean(np.abs(x)), rel=1e-6)
        assert z[4] == pytest.approx(math.sqrt(np.mean(x * x)), rel=1e-6)
        assert z[5] == 0.0 and z[6] == 0.0
        assert z[7] == pytest.approx(math.log1p(s.n_tokens) / 16, rel=1e-15)
    assert np.all(o["desc"][VIDEO] == 0.0)                # absent modality


def test_descriptor_temporal_entries():
    w = make_workload(3, n_requests=1)
    o = oracle.run_learned(w.segments, 1, w.params)
    z = o["desc"][VIDEO]
    assert z[6] == 1.0 and z[5] == pytest.approx(o["temporal"][VIDEO], rel=1e-7) and z[5] > 0


def _with(s, data, **kw):
    f = dict(request=s.request, modality=s.modality, n_frames=s.n_frames, tokens_per_frame=s.tokens_per_frame,
             hidden=s.hidden, dtype=s.dtype, keep_ratio=s.keep_ratio)
    f.update(kw)
    return Segment(f["request"], f["modality"], f["n_frames"], f["tokens_per_frame"], f["hidden"], f["dtype"],
                   f["keep_ratio"], data)


def test_descriptor_invariant_under_token_order():
    """Entries 1-4 and 7 are sums over the modality's tokens divided by
    totals: reordering the tokens of an image or audio segment leaves them
    unchanged (up to the order of fp64 sums)."""
    w = make_workload(4, n_requests=1)
    rng = np.random.default_rng(11)
    segs = [s if s.modality == TEXT else _with(s, np.ascontiguousarray(s.data[rng.permutation(s.n_tokens)]))
            for s in w.segments]
    a = oracle.run_learned(w.segments, 1, w.params)["desc"]
    b = oracle.run_learned(segs, 1, w.params)["desc"]
    np.testing.assert_allclose(b, a, rtol=1e-12, atol=0)


def test_descriptor_scales_with_the_features():
    """Doubling every feature (exact in fp32) and tau together keeps the
    activity pattern, so rho and the active fraction stay, while the mean
    magnitude and the root mean square double."""
    w = make_workload(1)
    p = dict(w.params)
    segs2 = []
    for s in w.segments:
        assert s.dtype == "f32"
        segs2.append(_with(s, (s.data * np.float32(2)).astype(np.float32)))
    p2 = dict(p, tau=p["tau"] * 2)
    a = oracle.run_learned(w.segments, 1, p)["desc"]
    b = oracle.run_learned(segs2, 1, p2)["desc"]
    for m in (TEXT, IMAGE):
        np.testing.assert_array_equal(b[m][[0, 1, 2, 5, 6, 7]], a[m][[0, 1, 2, 5, 6, 7]])
        np.testing.assert_allclose(b[m][[3, 4]], 2 * a[m][[3, 4]], rtol=1e-12)


def test_descriptor_of_a_duplicated_segment():
    """Two copies of a segment in one (request, modality): every mean and
    fraction is that of one copy; only the token-count entry moves, to
    ln(1 + 2N) / 16."""
    w = make_workload(4, n_requests=1)
    img = [s for s in w.segments if s.modality == IMAGE][0]
    a = oracle.run_learned([img], 1, w.params)["desc"][IMAGE]
    b = oracle.run_learned([img, img], 1, w.params)["desc"][IMAGE]
    np.testing.assert_allclose(b[:7], a[:7], rtol=1e-12, atol=0)
    assert b[7] == pytest.approx(math.log1p(2 * img.n_tokens) / 16, rel=1e-15)


def mlp_for(R, P, H, rng):
    return dict(w1=rng.standard_normal((H, P + oracle.DESC)).astype(np.float32) * 0.3,
                b1=rng.standard_normal(H).astype(np.float32) * 0.1,
                w2=rng.standard_normal(H).astype(np.float32) * 0.5, b2=0.2,
                prompt=rng.standard_normal((R, P)).astype(np.float32))


def test_mlp_matches_numpy_and_softmax():
    w = make_workload(4, n_requests=3)
    rng = np.random.default_rng(4)
    m = mlp_for(3, 32, 16, rng)
    o = oracle.run_learned(w.segments, 3, w.params, mlp=m)
    for r in range(3):
        pres = [TEXT, IMAGE, AUDIO]
        al = []
        for mod in pres:
            v = np.concatenate([m["prompt"][r].astype(np.float64), o["desc"][r * 4 + mod]])
            hsum = m["w1"].astype(np.float64) @ v + m["b1"]
            want = float(np.maximum(hsum, 0) @ m["w2"].astype(np.float64) + float(np.float32(m["b2"])))
            assert o["alpha"][r * 4 + mod] == pytest.approx(want, rel=1e-10, abs=1e-12)
            al.append(want)
        np.testing.assert_allclose(o["beta"][[r * 4 + mod for mod in pres]], softmax(al), rtol=1e-6)
        assert o["beta"][r * 4 + VIDEO] == 0.0


def test_mlp_closed_form_with_zero_first_layer():
    w = make_workload(1)
    m = dict(w1=np.zeros((4, 5 + oracle.DESC), np.float32), b1=np.array([1.0, -1.0, 2.0, 0.5], np.float32),
             w2=np.array([1.0, 1.0, -0.5, 2.0], np.float32), b2=-0.25, prompt=np.ones((1, 5), np.float32))
    o = oracle.run_learned(w.segments, 1, w.params, mlp=m)
    want = -0.25 + 1.0 * 1.0 + 0.0 + (-0.5) * 2.0 + 2.0 * 0.5     # relu(b1) . w2 + b2 = 0.75
    assert o["alpha"][IMAGE] == pytest.approx(want) and o["alpha"][TEXT] == pytest.approx(want)
    assert o["beta"][IMAGE] == pytest.approx(0.5)
