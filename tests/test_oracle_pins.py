"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks one oracle step against something other than the oracle
itself: hand-worked values (tests/golden), closed forms, invariants, exact
rational arithmetic, a library routine, or brute force on tiny inputs.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st
from scipy import integrate
from scipy.special import expit, ndtr

import oracle
from workloads import (AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits,
                       make_workload)

F32_TAU = float(np.float32(0.1))


def f32(x):
    return np.asarray(x, dtype=np.float32)


# ---------------------------------------------------------------- O1 widening

def test_bf16_widening_matches_torch():
    """bf16 -> float is exact; pinned against torch's own bfloat16 conversion."""
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint16)
    # drop NaN patterns (their payload handling is library-defined); keep +-inf, +-0, subnormals
    bits = bits[((bits & 0x7FFF) <= 0x7F80)]
    want = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    for i in range(0, bits.size, 97):
        a, l1, l2 = oracle.token_stats(bits[i:i + 1], "bf16", 0.0)
        assert l1 == abs(float(want[i]))
        assert a == (0 if want[i] == 0 else 1)


# ---------------------------------------------------- O2/O3 per-token statistics

def test_hand_worked_token(golden):
    g = golden["token_pair"]
    cur, prev = f32(g["cur"]), f32(g["prev"])
    a, l1, l2 = oracle.token_stats(cur, "f32", g["tau"])
    assert (a, l1, l2) == (g["a_cur"], g["l1_cur"], g["l2_cur"])
    a_p, _, _ = oracle.token_stats(prev, "f32", g["tau"])
    assert a_p == g["a_prev"]


@pytest.mark.parametrize("tau", [0.0, 0.1, 5.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_zero_row_is_fully_sparse(tau, dtype):
    row = np.zeros(96, np.float32) if dtype == "f32" else np.zeros(96, np.uint16)
    assert oracle.token_stats(row, dtype, tau) == (0, 0.0, 0.0)
    neg0 = np.full(96, -0.0, np.float32)
    assert oracle.token_stats(neg0, "f32", tau)[0] == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_negative_zero_threshold_is_zero(dtype):
    """|x| <= -0 holds exactly when |x| <= 0: a threshold of -0 keeps every
    nonzero channel (and NaN) active, the same as +0. (A bf16 threshold taken
    from the float's bits would see -0 as 0x8000, above every magnitude.)"""
    x = f32([0.0, -0.0, 1e-30, -2.5, np.nan, np.inf, 0.0, 3.0])
    row = x if dtype == "f32" else f32_to_bf16_bits(x)
    a_neg = oracle.token_stats(row, dtype, -0.0)[0]
    assert a_neg == oracle.token_stats(row, dtype, 0.0)[0] == 5


def test_activity_boundary_is_inclusive_and_nan_active():
    tau = np.float32(0.1)
    above = np.nextafter(tau, np.float32(1))
    row = f32([tau, -tau, above, -above, np.nan, np.inf, -np.inf, 0.0])
    a, _, _ = oracle.token_stats(row, "f32", float(tau))
    assert a == 5  # |x| == tau is inactive; just above, NaN and +-inf are active


def test_activity_monotone_in_tau_and_symmetric():
    rng = np.random.default_rng(2)
    row = rng.standard_normal(1024).astype(np.float32)
    counts = [oracle.token_stats(row, "f32", t)[0] for t in (0.0, 0.05, 0.1, 0.5, 1.0, 3.0)]
    assert all(x >= y for x, y in zip(counts, counts[1:]))
    assert oracle.token_stats(-row, "f32", 0.1) == oracle.token_stats(row, "f32", 0.1)
    perm = rng.permutation(row.size)
    a0, l10, l20 = oracle.token_stats(row, "f32", 0.1)
    a1, l11, l21 = oracle.token_stats(row[perm], "f32", 0.1)
    assert a0 == a1 and math.isclose(l10, l11, rel_tol=1e-14) and math.isclose(l20, l21, rel_tol=1e-14)


def test_sums_match_correctly_rounded_fsum():
    rng = np.random.default_rng(3)
    row = rng.standard_normal(4096).astype(np.float32)
    _, l1, l2 = oracle.token_stats(row, "f32", 0.1)
    vals = [float(v) for v in row]
    assert math.isclose(l1, math.fsum(abs(v) for v in vals), rel_tol=1e-12)
    assert math.isclose(l2, math.fsum(v * v for v in vals), rel_tol=1e-12)


def test_exact_sums_on_dyadic_values():
    row = f32([k / 8.0 for k in range(-40, 40)])
    a, l1, l2 = oracle.token_stats(row, "f32", 1.0)
    assert l1 == sum(abs(Fraction(k, 8)) for k in range(-40, 40))
    assert l2 == sum(Fraction(k, 8) ** 2 for k in range(-40, 40))
    assert a == sum(1 for k in range(-40, 40) if abs(k) > 8)


def _active_fraction(x, tau=0.1):
    total = 0
    for i in range(x.shape[0]):
        total += oracle.token_stats(x[i], "f32", tau)[0]
    return total / x.size


def test_closed_form_activity_rates():
    """P(active) for the workload distributions, from the normal CDF."""
    rng = np.random.default_rng(4)
    n = 256 * 1024
    g = rng.standard_normal((256, 1024)).astype(np.float32)
    relu = np.maximum(g, 0)
    p_relu = 1 - ndtr(0.1)
    p_norm = 2 * (1 - ndtr(0.1))
    p_bg = 1 - ndtr(2.0)  # ReLU(N(0,1)) * 0.05 active iff x > 2
    for x, p in ((relu, p_relu), (g, p_norm), (relu * np.float32(0.05), p_bg)):
        got = _active_fraction(x)
        assert abs(got - p) < 6 * math.sqrt(p * (1 - p) / n)
    # E|x| = 1/sqrt(2 pi), E x^2 = 1/2 for ReLU(N(0,1))
    s1 = sum(oracle.token_stats(relu[i], "f32", 0.1)[1] for i in range(256)) / n
    s2 = sum(oracle.token_stats(relu[i], "f32", 0.1)[2] for i in range(256)) / n
    assert abs(s1 - 1 / math.sqrt(2 * math.pi)) < 0.004
    assert abs(s2 - 0.5) < 0.004


def test_gelu_activity_rate_by_quadrature():
    """GELU(N(0,1)) activity rate computed by numerical integration over the normal density."""
    x = make_workload(2, n_requests=1).segments[1].data[:32]  # text: GELU, no background
    xf = (x.astype(np.uint32) << 16).view(np.float32)
    # P(|x Phi(x)| > 0.1) for x ~ N(0,1): integrate the density over where the condition holds
    phi = lambda t: math.exp(-t * t / 2) / math.sqrt(2 * math.pi)  # noqa: E731
    cond = lambda t: 1.0 if abs(t * ndtr(t)) > 0.1 else 0.0  # noqa: E731
    p, _ = integrate.quad(lambda t: phi(t) * cond(t), -12, 12, limit=400, points=[-3.0, -0.3, 0.0, 0.3])
    got = _active_fraction(xf)
    assert abs(got - p) < 6 * math.sqrt(p * (1 - p) / xf.size) + 2e-3  # bf16 rounding near the threshold


# ------------------------------------------------------------ O4 temporal term

def test_hand_worked_temporal_pair(golden):
    g = golden["token_pair"]
    cur, prev = f32(g["cur"]), f32(g["prev"])
    assert oracle.temporal_pair(cur, prev, "f32", g["tau"]) == (g["d"], g["res"])
    assert oracle.temporal_pair(cur, None, "f32", g["tau"]) == (g["d_vs_zero"], g["res_vs_zero"])


def test_temporal_invariants():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(2048).astype(np.float32)
    y = rng.standard_normal(2048).astype(np.float32)
    assert oracle.temporal_pair(x, x, "f32", 0.1) == (0, 0.0)          # identical frames
    d, res = oracle.temporal_pair(-x, x, "f32", 0.1)                     # sign-blind activity
    _, _, l2 = oracle.token_stats(x, "f32", 0.1)
    assert d == 0 and math.isclose(res, 4 * l2, rel_tol=1e-12)
    a, _, _ = oracle.token_stats(x, "f32", 0.1)
    assert oracle.temporal_pair(x, None, "f32", 0.1) == (a, l2)          # zero predecessor
    assert oracle.temporal_pair(x, y, "f32", 0.1)[0] == oracle.temporal_pair(y, x, "f32", 0.1)[0]


def test_independent_frames_hamming_rate():
    """Independent N(0,1) frames: E[d/C] = 2p(1-p), p = P(|x| > 0.1)."""
    rng = np.random.default_rng(6)
    n_rows, C = 128, 1024
    x = rng.standard_normal((n_rows, C)).astype(np.float32)
    y = rng.standard_normal((n_rows, C)).astype(np.float32)
    tot = sum(oracle.temporal_pair(x[i], y[i], "f32", 0.1)[0] for i in range(n_rows))
    p = 2 * (1 - ndtr(0.1))
    q = 2 * p * (1 - p)
    assert abs(tot / (n_rows * C) - q) < 6 * math.sqrt(q * (1 - q) / (n_rows * C))


# --------------------------------------------------------------- Eq. 4 sparse

@pytest.mark.parametrize("C", [8, 24, 1000, 1024, 1280, 4096])
@pytest.mark.parametrize("tau_s", [0.0, 0.3, 0.5, 0.7, 1.0])
def test_sparse_test_is_exact_rational_comparison(C, tau_s):
    t = Fraction(float(np.float32(tau_s)))
    for a in range(0, C + 1, max(1, C // 200)):
        assert oracle.is_sparse(a, C, tau_s) == (Fraction(a, C) < t)
    if (t * C).denominator == 1:  # boundary a == tau_s * C must not count (strict <)
        assert not oracle.is_sparse(int(t * C), C, tau_s)


# ----------------------------------------------------------- Sec. 4.1.3 softmax

def test_modal_softmax_special_cases():
    assert list(oracle.modal_softmax([0.3, 1.0, 0, 0], [0, 1, 0, 0])) == [0, 1, 0, 0]
    b = oracle.modal_softmax([0.0, 0.0, 0.0, 0.0], [1, 1, 0, 1])
    assert np.allclose(b, [1 / 3, 1 / 3, 0, 1 / 3], rtol=0, atol=1e-16)
    b = oracle.modal_softmax([0.7, -1.2, 0, 0], [1, 1, 0, 0])
    assert math.isclose(b[0], expit(0.7 + 1.2), rel_tol=1e-14) and math.isclose(b[0] + b[1], 1, rel_tol=1e-15)
    b = oracle.modal_softmax([1000.0, 999.0, 5.0, -1000.0], [1, 1, 1, 1])  # no overflow
    assert math.isclose(b.sum(), 1.0, rel_tol=1e-15) and math.isclose(b[0] / b[1], math.e, rel_tol=1e-12)


# ------------------------------------------------------------------- Eq. 7 MAS

def test_mas_hand_worked(golden):
    for c in golden["mas"]["cases"]:
        got = oracle.mas_value(c["beta"], c["lam_s"], c["rho"], c["lam_t"], c["tterm"], c["has_t"])
        assert math.isclose(got, c["mas"], rel_tol=0, abs_tol=1e-12), c


def test_mas_range_and_monotonicity():
    rng = np.random.default_rng(7)
    for _ in range(2000):
        beta, ls, rho, lt, tt = rng.uniform(0, 1, 5)
        m = oracle.mas_value(beta, ls, rho, lt, tt, 1)
        assert 0.0 <= m <= 1.0
        assert oracle.mas_value(beta, ls, min(1, rho + 0.1), lt, tt, 1) >= m - 1e-15  # more sparsity, more MAS
        assert oracle.mas_value(beta, 0, rho, 0, tt, 1) == pytest.approx(1 - beta, abs=1e-15)
    assert oracle.mas_value(0.37, 1.0, 1.0, 0.0, 0.0, 0) == 1.0


# ------------------------------------------------------- O8/O9 keys and counts

def test_keep_count_pins(golden):
    for N, kappa, k in golden["keep_count"]["cases"]:
        assert oracle.keep_count(float(np.float32(kappa)), N) == k, (N, kappa)


@pytest.mark.parametrize("lam", [0.0, 0.4, 0.5, 0.6, 0.3, 1.0, 0.123456, 0.1, 0.7, 1e-9])
def test_q24_is_round_half_even_of_exact_product(lam):
    exact = Fraction(float(np.float32(lam))) * (1 << 24)
    assert oracle.q24(lam) == round(exact)  # Python's round on Fraction is half-to-even


# ----------------------------------------------------------- O10 selection

def _seg(N, C=16, modality=IMAGE, T=1, keep=0.5):
    P = N // T
    return Segment(0, modality, T, P, C, "f32", keep, np.zeros((N, C), np.float32))


def _brute_force_kept(keys, k):
    best = None
    for sub in itertools.combinations(range(len(keys)), k):
        score = (sum(keys[i] for i in sub), sub)
        if best is None or score < best:
            best = score
    return list(best[1]) if best else []


def test_select_hand_worked(golden):
    g = golden["select"]
    seg = _seg(4, C=16, keep=g["k"] / 4)
    p = default_params()
    p["lambda_s"] = [1.0] * 4
    out = oracle.select([seg], 1, p, np.array(g["keys_as_z"], np.uint32), None, None)
    assert list(out["kept_idx"][: g["k"]]) == g["kept"]


@settings(max_examples=150, deadline=None)
@given(st.integers(1, 11), st.integers(0, 12), st.booleans(), st.data())
def test_select_matches_brute_force(N, k_req, temporal, data):
    k = min(k_req, N)
    C = 8
    T = 2 if (temporal and N % 2 == 0) else 1
    modality = VIDEO if T == 2 else IMAGE
    z = np.array(data.draw(st.lists(st.integers(0, C), min_size=N, max_size=N)), np.uint32)
    d = np.array(data.draw(st.lists(st.integers(0, C), min_size=N, max_size=N)), np.uint32)
    kappa = float(np.float32(k / N))
    seg = Segment(0, modality, T, N // T, C, "f32", kappa, np.zeros((N, C), np.float32))
    p = default_params()
    out = oracle.select([seg], 1, p, z, d if T == 2 else None, None)
    kk = int(out["k"][0])
    assert kk == k or kk == min(N, math.ceil(Fraction(kappa) * N))
    Ls, Lt = oracle.q24(p["lambda_s"][modality]), oracle.q24(p["lambda_t"][modality])
    keys = [Ls * int(z[i]) + (Lt * (C - int(d[i])) if T == 2 else 0) for i in range(N)]
    kept = list(out["kept_idx"][:kk])
    assert kept == _brute_force_kept(keys, kk)
    # counting definition: keep i iff fewer than k pairs (key, j) precede (key_i, i)
    for i in range(N):
        rank = sum(1 for j in range(N) if (keys[j], j) < (keys[i], i))
        assert bool(out["keep"][i]) == (rank < kk)
    assert all(x == -1 for x in out["kept_idx"][kk:])


def test_select_invariants_and_degenerate_ratios():
    rng = np.random.default_rng(8)
    N = 300
    z = rng.integers(0, 16, N).astype(np.uint32)
    p = default_params()
    for kappa, want in ((1.0, N), (0.0, 0)):
        out = oracle.select([_seg(N, keep=kappa)], 1, p, z, None, None)
        assert out["k"][0] == want and out["keep"].sum() == want
    out = oracle.select([_seg(N, keep=0.37)], 1, p, np.full(N, 5, np.uint32), None, None)
    k = out["k"][0]
    assert list(out["kept_idx"][:k]) == list(range(k))  # tie storm: lowest indices
    out = oracle.select([_seg(N, keep=0.37)], 1, p, z, None, None)
    kept = out["kept_idx"][:k]
    assert np.all(np.diff(kept) > 0)
    dropped = np.setdiff1d(np.arange(N), kept)
    assert max((int(z[i]), i) for i in kept) < min((int(z[i]), i) for i in dropped)


def test_mas_guided_keep_count():
    seg = _seg(100, keep=-1.0)
    seg.request = 1
    mas = np.zeros(8, np.float32)
    mas[4 + IMAGE] = np.float32(0.75)
    out = oracle.select([seg], 2, default_params(), np.zeros(100, np.uint32), None, mas)
    assert out["k"][0] == 25


# -------------------------------------------------- whole-run pins on configs

def test_config1_exact_pins():
    w = make_workload(1)
    o = oracle.run(w.segments, w.n_requests, w.params)
    img, txt = w.segments
    bg = img.meta["bg_mask"]
    assert bg.sum() == 345
    assert o["rho"][IMAGE] == np.float32(345 / 576) and o["rho"][TEXT] == 0
    assert o["mas"][IMAGE] == np.float32(0.6796875) and o["mas"][TEXT] == np.float32(0.5)
    assert list(o["present"][:4]) == [1, 1, 0, 0] and o["beta"][IMAGE] == np.float32(0.5)
    assert list(o["k"]) == [288, 32]
    kept = o["kept_idx"][:288]
    assert set(np.flatnonzero(~bg)) <= set(kept.tolist())           # all 231 foreground kept
    kept_bg = [i for i in kept if bg[i]]
    assert len(kept_bg) == 57
    zbg = o["z"][:576][bg]
    assert max(o["z"][i] for i in kept_bg) <= np.sort(zbg)[56]       # the 57 smallest-z background
    agg = o["agg"].reshape(-1, 4, 4)
    assert list(agg[0, IMAGE]) == [576, 345, 0, 0] and list(agg[0, TEXT]) == [32, 0, 0, 0]
    # compaction is a byte copy of the kept rows
    assert np.array_equal(o["compact"][0], img.data[kept])
    assert np.array_equal(o["compact"][1], txt.data)


def test_config4_pins_two_requests():
    w = make_workload(4, n_requests=2)
    o = oracle.run(w.segments, w.n_requests, w.params)
    for r in range(2):
        img = w.segments[3 * r]
        area = int(img.meta["bg_mask"].sum())
        x = r * 4
        assert o["rho"][x + AUDIO] == np.float32(0.4)
        assert o["mas"][x + AUDIO] == np.float32(1 - (1 / 3) * (1 - 0.6 * 0.4))
        assert o["mas"][x + TEXT] == np.float32(1 - 1 / 3)
        assert o["rho"][x + IMAGE] == np.float32(area / 576)
        assert math.isclose(o["mas"][x + IMAGE], 1 - (1 / 3) * (1 - 0.6 * area / 576), rel_tol=1e-6)
        assert math.isclose(o["beta"][x + IMAGE], 1 / 3, rel_tol=1e-7)
    assert list(o["k"]) == [144, 750, 128] * 2


def test_config3_one_clip_pins():
    w = make_workload(3, n_requests=1)
    o = oracle.run(w.segments, 1, w.params)
    seg = w.segments[0]
    P, T, C = 256, 32, 1024
    static = seg.meta["static_mask"]
    assert o["rho"][VIDEO] == 0.0
    # temporal redundancy: static patches barely change, moving ones are independent redraws
    p = 2 * (1 - ndtr(0.1))
    d = o["d"].reshape(T, P)
    moving_rate = d[1:, ~static].mean() / C
    assert abs(moving_rate - 2 * p * (1 - p)) < 0.005
    assert d[1:, static].mean() / C < 0.03
    assert np.array_equal(d[0], C - o["z"].reshape(T, P)[0])          # frame 0: d = a
    assert np.all(o["dframe"][1:] == d[1:].sum(axis=1))
    # Eq. 5 per frame (K = P*C hash bits) equals the mean of the P per-token
    # similarities (K = C each), an identity of bit sampling
    for t in range(T):
        mean_tok = sum(Fraction(C - int(x), C) for x in d[t]) / P
        assert abs(float(o["sim"][t]) - float(mean_tok)) < 1e-7
        assert abs(float(o["gamma"][t]) - float(1 - mean_tok)) < 1e-7
    assert math.isclose(o["temporal"][VIDEO], 1 - d[1:].sum() / ((T - 1) * P * C), rel_tol=1e-6)
    assert 0.93 < o["temporal"][VIDEO] < 0.96 and 0.36 < o["mas"][VIDEO] < 0.40
    # selection: all frame-0 tokens, then moving tokens; no static token beyond frame 0
    k = int(o["k"][0])
    assert k == 2458
    kept = o["kept_idx"][:k]
    assert set(range(P)) <= set(kept.tolist())
    later = kept[kept >= P] % P
    assert not static[later].any()


def test_temporal_literal_flag_and_identical_frames():
    """Single-modality video with lambda_s = 0 and identical frames: MAS = lambda_t
    under the redundancy reading, 0 under the literal one (Eq. 7 with gamma = 1 - sim)."""
    rng = np.random.default_rng(9)
    frame = rng.standard_normal((16, 64)).astype(np.float32)
    data = np.concatenate([frame] * 4)
    seg = Segment(0, VIDEO, 4, 16, 64, "f32", 0.5, data)
    p = default_params()
    p["lambda_s"] = [0.0] * 4
    o = oracle.run([seg], 1, p)
    assert np.all(o["sim"][1:] == 1.0) and np.all(o["gamma"][1:] == 0.0)
    assert o["mas"][VIDEO] == np.float32(0.4)
    p["flags"] = oracle.FLAG_TEMPORAL_LITERAL
    o = oracle.run([seg], 1, p)
    assert o["mas"][VIDEO] == 0.0


def test_video_single_frame_is_an_image_and_empty_segments():
    rng = np.random.default_rng(10)
    x = rng.standard_normal((20, 32)).astype(np.float32)
    segs = [Segment(0, VIDEO, 1, 20, 32, "f32", 0.5, x),
            Segment(0, AUDIO, 3, 0, 32, "f32", 0.5, np.zeros((0, 32), np.float32))]
    o = oracle.run(segs, 1, default_params())
    assert o["d"].sum() == 0 and o["res"].sum() == 0 and o["sim"].size == 0
    assert o["present"][VIDEO] == 1 and o["present"][AUDIO] == 0 and o["temporal"][VIDEO] == 0
    assert o["beta"][VIDEO] == 1.0 and list(o["k"]) == [10, 0]


def test_info_special_cases_and_order():
    """Token informativeness: 1 - lambda_s for an all-inactive token, 1 for an
    all-active one, and it orders tokens like the selection key (kept tokens are
    at least as informative as dropped ones)."""
    rng = np.random.default_rng(12)
    C = 64
    x = rng.standard_normal((40, C)).astype(np.float32)
    x[0] = 0.0
    x[1] = 1.0
    seg = Segment(0, IMAGE, 1, 40, C, "f32", 0.5, x)
    o = oracle.run([seg], 1, default_params())
    lam_s = float(np.float32(0.6))  # lambda is a float32 parameter
    assert o["info"][0] == np.float32(1 - lam_s) and o["info"][1] == 1.0
    kept = o["kept_idx"][: o["k"][0]]
    dropped = np.setdiff1d(np.arange(40), kept)
    assert o["info"][kept].min() >= o["info"][dropped].max()
    # video: frame 0 has e = C - d = z; a repeated frame has e = C
    frame = rng.standard_normal((8, C)).astype(np.float32)
    v = Segment(0, VIDEO, 2, 8, C, "f32", 0.5, np.concatenate([frame, frame]))
    o = oracle.run([v], 1, default_params())
    z0 = o["z"][:8].astype(np.float64)
    assert np.allclose(o["info"][:8], 1 - (0.6 * z0 + 0.4 * z0) / C, rtol=0, atol=1e-6)
    assert np.allclose(o["info"][8:], 1 - (0.6 * z0 + 0.4 * C) / C, rtol=0, atol=1e-6)


def test_multiple_segments_per_modality_aggregate():
    rng = np.random.default_rng(11)
    a = np.maximum(rng.standard_normal((30, 64)), 0).astype(np.float32)
    b = (rng.standard_normal((50, 64)) * 0.01).astype(np.float32)  # all sparse
    segs = [Segment(0, IMAGE, 1, 30, 64, "f32", 0.5, a), Segment(0, IMAGE, 1, 50, 64, "f32", 0.5, b)]
    o = oracle.run(segs, 1, default_params())
    agg = o["agg"].reshape(-1, 4, 4)[0, IMAGE]
    assert agg[0] == 80 and agg[1] == 50
    assert o["rho"][IMAGE] == np.float32(50 / 80)


def test_requests_are_independent():
    """Each request's outputs depend only on its own segments: running the
    requests one at a time (as the threaded CPU baseline does) gives the
    whole table's statistics, MAS, keep counts, kept indices and rows."""
    import dataclasses
    w = make_workload(4, n_requests=5)
    whole = oracle.run(w.segments, w.n_requests, w.params)
    tok = np.cumsum([0] + [s.n_tokens for s in w.segments])
    for r in range(w.n_requests):
        idx = [i for i, s in enumerate(w.segments) if s.request == r]
        segs = [dataclasses.replace(w.segments[i], request=0) for i in idx]
        o = oracle.run(segs, 1, w.params)
        sel = np.concatenate([np.arange(tok[i], tok[i + 1]) for i in idx])
        for k in ("z", "l1", "l2", "info", "keep", "kept_idx"):
            assert np.array_equal(o[k], whole[k][sel]), k
        for k in ("rho", "temporal", "beta", "mas", "present"):
            assert np.array_equal(o[k], whole[k][r * 4:(r + 1) * 4]), k
        assert np.array_equal(o["k"], whole["k"][idx])
        for a, b in zip(o["compact"], [whole["compact"][i] for i in idx]):
            assert np.array_equal(a, b)
