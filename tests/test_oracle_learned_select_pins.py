"""Pins of the oracle's selection by the learned importance (Sec. 4.1.1: the
patches whose Eq. 3 importance M is low are pruned; a segment with a head
keeps its k tokens of largest M, ties by ascending index, a NaN M counting
as 0; segments without a head keep the plain redundancy selection; a
negative keep ratio takes k = ceil((1 - MAS) N) from the learned MAS).

Routes independent of the oracle's selection code: sorting the raw feature
of a one-channel head (sigmoid is increasing, so M orders the tokens as that
channel does), brute force over all subsets on a small pooled grid with M
recomputed in numpy, closed forms of Eq. 4 and Eq. 7 with saturated heads,
and the plain selection where no segment has a head."""
import itertools
import math

import numpy as np
import pytest
from scipy.special import expit

import oracle
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, bf16_bits_to_f32, default_params, f32_to_bf16_bits, make_workload


def one_channel_head(s, c, bias=0.0):
    w = np.zeros(s.hidden, np.float32)
    w[c] = 1.0
    return dict(weight=w if s.dtype == "f32" else f32_to_bf16_bits(w), bias=bias, grid_w=0, pool=1)


def kept_sets(o, segs):
    out, off = [], 0
    for i, s in enumerate(segs):
        k = int(o["k"][i])
        idx = o["kept_idx"][off:off + s.n_tokens]
        assert np.all(idx[k:] == -1) and np.all(np.diff(idx[:k]) > 0)
        out.append(idx[:k].astype(np.int64))
        off += s.n_tokens
    return out


def image_segment(rng, n_tok, hidden, keep, dtype="f32", request=0, modality=IMAGE, n_frames=1, ties=0):
    x = rng.standard_normal((n_tok, hidden)).astype(np.float32)
    if ties:  # repeat a few values in channel 3, so that ties need the index rule
        x[rng.choice(n_tok, ties, replace=False), 3] = 0.5
    data = x if dtype == "f32" else f32_to_bf16_bits(x)
    return Segment(request, modality, n_frames, n_tok // n_frames, hidden, dtype, keep, data)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("keep", [0.1, 0.25, 0.5, 0.9])
def test_one_channel_head_keeps_the_largest_channel_values(dtype, keep):
    rng = np.random.default_rng(7)
    s = image_segment(rng, 300, 64, keep, dtype, ties=40)
    o = oracle.run_learned([s], 1, default_params(), [one_channel_head(s, 3, bias=-0.5)])
    xc = (s.data if dtype == "f32" else bf16_bits_to_f32(s.data))[:, 3].astype(np.float64)
    order = np.lexsort((np.arange(s.n_tokens), -xc))   # largest value first, then smaller index
    k = math.ceil(np.float64(np.float32(keep)) * s.n_tokens)
    assert int(o["k"][0]) == k
    np.testing.assert_array_equal(kept_sets(o, [s])[0], np.sort(order[:k]))


def test_constant_importance_keeps_the_first_tokens():
    rng = np.random.default_rng(3)
    s = image_segment(rng, 100, 32, 0.37)
    h = dict(weight=np.zeros(32, np.float32), bias=1.5, grid_w=10, pool=3)
    o = oracle.run_learned([s], 1, default_params(), [h])
    k = math.ceil(np.float64(np.float32(0.37)) * 100)
    np.testing.assert_array_equal(kept_sets(o, [s])[0], np.arange(k))


def numpy_importance(x, w, b, grid_w, pool):
    """Eq. 3 recomputed in numpy: window means of the projections over the
    pool x pool square cut to the grid, then the sigmoid."""
    y = x.astype(np.float64) @ w.astype(np.float64)
    P = y.size
    W = grid_w if grid_w > 0 else P
    H = P // W
    g = y.reshape(H, W)
    r = (pool - 1) // 2
    M = np.empty((H, W))
    for i in range(H):
        for j in range(W):
            win = g[max(0, i - r):i + r + 1, max(0, j - r):j + r + 1]
            M[i, j] = expit(win.mean() + b)
    return M.reshape(-1)


@pytest.mark.parametrize("k_ratio", [0.25, 0.5, 0.75])
def test_pooled_head_on_a_small_grid_against_brute_force(k_ratio):
    rng = np.random.default_rng(11)
    s = image_segment(rng, 12, 16, k_ratio)
    w = (rng.standard_normal(16) * 0.3).astype(np.float32)
    h = dict(weight=w, bias=0.1, grid_w=4, pool=3)
    o = oracle.run_learned([s], 1, default_params(), [h])
    M = numpy_importance(s.data, w, 0.1, 4, 3)
    k = int(o["k"][0])
    assert k == math.ceil(np.float64(np.float32(k_ratio)) * 12)
    best = None
    for sub in itertools.combinations(range(12), k):
        rest = [i for i in range(12) if i not in sub]
        # a valid kept set: nothing dropped is more important than anything kept,
        # and among equal importance the smaller index is kept
        if all((M[i] > M[j]) or (M[i] == M[j] and i < j) for i in sub for j in rest):
            assert best is None, "the kept set is unique"
            best = sub
    np.testing.assert_array_equal(kept_sets(o, [s])[0], np.array(best))


def test_nan_importance_is_dropped_first():
    rng = np.random.default_rng(5)
    s = image_segment(rng, 50, 16, 0.5)
    s.data[[2, 9, 30], 0] = np.nan   # NaN rows project to NaN
    o = oracle.run_learned([s], 1, default_params(), [one_channel_head(s, 0)])
    assert np.isnan(o["importance"][[2, 9, 30]]).all()
    kept = kept_sets(o, [s])[0]
    assert not np.isin([2, 9, 30], kept).any()
    # with every token kept but one, the NaN rows come last among the dropped
    s.keep_ratio = 48 / 50
    o = oracle.run_learned([s], 1, default_params(), [one_channel_head(s, 0)])
    dropped = np.setdiff1d(np.arange(50), kept_sets(o, [s])[0])
    np.testing.assert_array_equal(dropped, [9, 30])


def test_mas_guided_keep_counts_from_saturated_heads():
    """Bias +40: M = 1 for every token, nothing is sparse (rho = 0), MAS =
    1 - beta (1 - 0) = 0 with one modality, so k = N. Bias -40: M < tau_s
    everywhere (rho = 1), MAS = 1 - (1 - 0.6) = 0.6, so k = ceil(0.4 N)."""
    rng = np.random.default_rng(9)
    s = image_segment(rng, 200, 32, -1.0)
    for bias, want in ((40.0, 200), (-40.0, math.ceil((1.0 - np.float64(np.float32(0.6))) * 200))):
        h = dict(weight=np.zeros(32, np.float32), bias=bias, grid_w=0, pool=1)
        o = oracle.run_learned([s], 1, default_params(), [h])
        assert float(o["rho"][IMAGE]) == (0.0 if bias > 0 else 1.0)
        assert int(o["k"][0]) == want
        np.testing.assert_array_equal(kept_sets(o, [s])[0], np.arange(want))   # constant M: first tokens


def test_per_frame_scope_ranks_each_frame_by_its_own_importance():
    rng = np.random.default_rng(13)
    s = image_segment(rng, 4 * 30, 32, 0.2, modality=VIDEO, n_frames=4)
    p = default_params()
    p["flags"] = oracle.FLAG_SELECT_PER_FRAME
    o = oracle.run_learned([s], 1, p, [one_channel_head(s, 5)])
    kf = math.ceil(np.float64(np.float32(0.2)) * 30)
    assert int(o["k"][0]) == 4 * kf
    kept = kept_sets(o, [s])[0]
    xc = s.data[:, 5].astype(np.float64)
    for t in range(4):
        f = np.arange(t * 30, (t + 1) * 30)
        want = np.sort(f[np.lexsort((f, -xc[f]))[:kf]])
        np.testing.assert_array_equal(kept[(kept >= t * 30) & (kept < (t + 1) * 30)], want)


def test_segments_without_a_head_keep_the_plain_selection():
    w = make_workload(4, n_requests=3)
    rng = np.random.default_rng(2)
    heads = []
    for s in w.segments:
        if s.modality == AUDIO:
            wv = (rng.standard_normal(s.hidden) * 0.05).astype(np.float32)
            heads.append(dict(weight=f32_to_bf16_bits(wv), bias=-0.3, grid_w=0, pool=5))
        else:
            heads.append(None)
    a = oracle.run(w.segments, 3, w.params)
    b = oracle.run_learned(w.segments, 3, w.params, heads)
    ka, kb = kept_sets(a, w.segments), kept_sets(b, w.segments)
    for s, x, y in zip(w.segments, ka, kb):
        if s.modality != AUDIO:
            np.testing.assert_array_equal(x, y)
    # the audio tracks are ranked by their head instead: the kept set is the
    # k largest importances, ties by index
    off = 0
    for i, s in enumerate(w.segments):
        if s.modality == AUDIO:
            M = b["importance"][off:off + s.n_tokens]
            order = np.lexsort((np.arange(s.n_tokens), -M))
            np.testing.assert_array_equal(kb[i], np.sort(order[:int(b["k"][i])]))
        off += s.n_tokens
    # compacted rows are the kept input rows
    for i, s in enumerate(w.segments):
        np.testing.assert_array_equal(b["compact"][i], s.data[kb[i]])


def test_without_heads_the_selection_is_the_plain_one():
    w = make_workload(3, n_requests=2)
    a = oracle.run(w.segments, 2, w.params)
    b = oracle.run_learned(w.segments, 2, w.params)
    for k in ("k", "keep", "kept_idx"):
        np.testing.assert_array_equal(a[k], b[k])
