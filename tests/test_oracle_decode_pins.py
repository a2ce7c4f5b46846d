"""Pins of the decoding-side oracle (Sec. 4.2: Eq. 8-10, 12-14, Algorithm 1)
against what the paper and the mathematics fix: closed forms, a library
routine, invariants and hand-worked values (tests/golden/sched_trace.json)."""
import json
import math
import os

import numpy as np
import pytest
from scipy.special import softmax
from scipy.stats import entropy as scipy_entropy

import oracle
from workloads import f32_to_bf16_bits

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def H_of(rows, dtype="f32", vocab=None):
    return oracle.entropy_rows(np.atleast_2d(rows), dtype, vocab)


# ------------------------------------------------------------------ Eq. 9

@pytest.mark.parametrize("V", [1, 2, 7, 1000, 151936])
def test_entropy_of_equal_logits_is_log_vocab(V):
    H, am = H_of(np.full((1, V), 3.25, np.float32))
    assert H[0] == pytest.approx(math.log(V), rel=1e-12, abs=1e-15)
    assert am[0] == 0


def test_entropy_known_distribution():
    # p = (1/2, 1/4, 1/4): H = 1.5 ln 2
    H, _ = H_of(np.log(np.array([[0.5, 0.25, 0.25]])).astype(np.float32))
    assert H[0] == pytest.approx(1.0397207708399179, rel=1e-6)


@pytest.mark.parametrize("a,b", [(0.0, 0.0), (1.0, 0.0), (5.0, -3.0), (-2.0, 7.5)])
def test_binary_entropy_closed_form(a, b):
    row = np.full((1, 64), -np.inf, np.float32)
    row[0, 10], row[0, 40] = a, b
    p = 1.0 / (1.0 + math.exp(float(np.float32(b)) - float(np.float32(a))))
    want = -(p * math.log(p) + (1 - p) * math.log(1 - p))
    H, am = H_of(row)
    assert H[0] == pytest.approx(want, rel=1e-12)
    assert am[0] == (10 if a >= b else 40)


def test_entropy_matches_scipy():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((6, 4096)) * rng.uniform(0.2, 6.0, (6, 1))).astype(np.float32)
    x[2, 17] += 40.0  # a confident row
    H, am = H_of(x)
    for r in range(x.shape[0]):
        want = scipy_entropy(softmax(x[r].astype(np.float64)))
        assert H[r] == pytest.approx(want, rel=1e-9, abs=1e-12)
        assert am[r] == int(np.argmax(x[r]))


def test_entropy_invariances():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((1, 999)).astype(np.float32)
    H0, _ = H_of(x)
    H1, _ = H_of(x + np.float32(4.0))                 # shift (exact in float32 here)
    H2, _ = H_of(x[:, rng.permutation(999)])          # permutation
    pad = np.concatenate([x, np.full((1, 25), -np.inf, np.float32)], axis=1)
    H3, _ = H_of(pad)                                 # -inf logits have probability 0
    assert H1[0] == pytest.approx(H0[0], rel=1e-6)
    assert H2[0] == pytest.approx(H0[0], rel=1e-12)
    assert H3[0] == pytest.approx(H0[0], rel=1e-12)
    assert 0.0 < H0[0] < math.log(999)


def test_entropy_of_a_dominant_logit_vanishes():
    row = np.zeros((1, 500), np.float32)
    row[0, 123] = 200.0
    H, am = H_of(row)
    assert am[0] == 123 and 0.0 <= H[0] < 1e-80


def test_argmax_first_of_equal_maxima_and_bf16_decoding():
    row = np.array([[1.0, 3.0, -2.0, 3.0, 3.0, 0.5, -1.0, 2.0]], np.float32)
    H32, am32 = H_of(row)
    H16, am16 = H_of(f32_to_bf16_bits(row), "bf16")   # every value is exact in bf16
    assert am32[0] == 1 and am16[0] == 1
    assert H16[0] == H32[0]


def test_entropy_vocab_and_stride():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((3, 40)).astype(np.float32)
    H_full, _ = H_of(x[:, :32])
    H_strided, _ = oracle.entropy_rows(x, "f32", vocab=32)   # row stride 40, vocab 32
    assert np.array_equal(H_full, H_strided)


def test_entropy_invalid_rows_are_nan():
    rows = np.zeros((3, 8), np.float32)
    rows[0, 3] = np.nan
    rows[1, 5] = np.inf
    rows[2, :] = -np.inf
    H, _ = H_of(rows)
    assert np.all(np.isnan(H))


def test_normalized_entropy_and_speculate_boundary():
    assert oracle.entropy_normalized(math.log(151936), 151936) == pytest.approx(1.0, rel=1e-15)
    assert oracle.entropy_normalized(0.0, 10) == 0.0
    assert oracle.speculate(0.3, 0.3) and not oracle.speculate(0.30000001, 0.3)   # Eq. 10: <=


# ------------------------------------------------------------ Eq. 8, 12-14

def test_comm_latency_hand_values():
    # 1 MB over 200 Mbps (25e6 B/s) with a 20 ms round trip (Sec. 5.1 link settings)
    assert oracle.comm_latency(1e6, 25e6, 0.02) == pytest.approx(0.06, rel=1e-15)
    assert oracle.comm_latency(0.0, 50e6, 0.02) == pytest.approx(0.02, rel=1e-15)


def test_p_conf_is_the_empirical_cdf():
    h = np.array([0.1, 0.2, 0.3, 0.4])
    assert oracle.p_conf(h, 0.25) == 0.5
    assert oracle.p_conf(h, 0.2) == 0.5          # <= includes the boundary
    assert oracle.p_conf(h, 0.05) == 0.0 and oracle.p_conf(h, 1.0) == 1.0


@pytest.mark.parametrize("P", [0.0, 0.3, 0.7, 0.95])
def test_expected_spec_closed_form_equals_its_series(P):
    t = np.arange(1, 4000, dtype=np.float64)
    series = float(np.sum(t * P ** (t - 1) * (1 - P)))
    assert oracle.expected_spec(P) == pytest.approx(series, rel=1e-9)


def test_expected_spec_diverges_at_one():
    assert math.isinf(oracle.expected_spec(1.0))


def test_expected_e2e_hand_value():
    # prefill max(0.1, 0.05 + 0.08) = 0.13; E[N] = 2 at P = 0.5;
    # 2 * (4*0.01 + 0.5 * 4*0.005) = 0.1; (1 - 0.5) * 0.2 = 0.1; total 0.33
    got = oracle.expected_e2e(0.1, 0.05, 0.08, 0.5, 4, 0.01, 0.005, 0.2)
    assert got == pytest.approx(0.33, rel=1e-12)
    got = oracle.expected_e2e(0.3, 0.05, 0.08, 0.0, 1, 0.01, 0.005, 0.2)   # edge prefill dominates
    assert got == pytest.approx(0.3 + 0.01 + 0.2, rel=1e-12)


# ------------------------------------------------------------ Algorithm 1

def test_quantile_is_the_lower_inverse_cdf():
    rng = np.random.default_rng(8)
    h = rng.permutation(np.arange(1, 501, dtype=np.float64))
    assert oracle.entropy_quantile(h, 0.7) == 350.0      # sorted[ceil(350) - 1]
    assert oracle.entropy_quantile(h, 0.0) == 1.0
    assert oracle.entropy_quantile(h, 1.0) == 500.0
    assert oracle.entropy_quantile(np.array([4.0, 1.0, 3.0, 2.0]), 0.5) == 2.0
    assert oracle.entropy_quantile(np.array([4.0, 1.0, 3.0, 2.0]), 0.51) == 3.0


@pytest.mark.parametrize("P,want", [(0.7, 4), (0.9, 5), (0.5, 2), (0.3, 1), (0.1, 1), (1.0, 5), (0.0, 1)])
def test_n_draft_hand_values(P, want):
    # log(0.2)/log(0.7) = 4.51; log(0.2)/log(0.9) = 15.3 -> N_max 5; log(0.2)/log(0.5) = 2.32;
    # log(0.2)/log(0.3) = 1.34; log(0.2)/log(0.1) = 0.70 -> at least 1
    assert oracle.n_draft(P, 0.8, 5) == want


def test_retention_floor():
    assert np.array_equal(oracle.retention([0.25, 0.6, 0.0, 1.0]), [0.75, 0.4, 1.0, 0.0])


def test_sched_trace_hand_worked():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "sched_trace.json")))
    p = g["params"]
    dec, th, cnt = oracle.sched_run(np.array(g["h_norm"]), p["theta0"], p["n_draft"], p["delta"],
                                    p["theta_min"], p["alpha"])
    assert dec.tolist() == g["decisions"]
    assert th.tolist() == g["theta_after"]          # dyadic values: exact
    c = g["counts"]
    assert cnt.tolist() == [c["held"], c["sends"], c["offloads"], c["tokens_sent"]]


def test_sched_step_rules_on_a_long_trace():
    """Every step follows one of the three branches: hold keeps theta, a send
    moves it toward the mean of the sent entropies (all at most theta, so it
    never rises there), an offload sets max(theta * delta, theta_min) (which
    can lift a theta that the EMA took below theta_min)."""
    rng = np.random.default_rng(9)
    h = rng.uniform(0, 1, 5000)
    n_draft, delta, theta_min, alpha = 3, 0.95, 0.1, 0.1
    dec, th, cnt = oracle.sched_run(h, 0.6, n_draft, delta, theta_min, alpha)
    prev, held = 0.6, []
    for i in range(h.size):
        if dec[i] == oracle.OFFLOAD:
            assert h[i] > prev and th[i] == max(prev * delta, theta_min)
            held = []
        else:
            assert h[i] <= prev
            held.append(h[i])
            if dec[i] == oracle.SEND:
                assert len(held) == n_draft
                assert th[i] == pytest.approx((1 - alpha) * prev + alpha * np.mean(held), rel=1e-12)
                assert th[i] <= prev
                held = []
            else:
                assert len(held) < n_draft and th[i] == prev
        prev = th[i]
    assert cnt[1] * n_draft == cnt[3]
    assert cnt[2] == int(np.sum(dec == oracle.OFFLOAD)) and cnt[1] == int(np.sum(dec == oracle.SEND))
