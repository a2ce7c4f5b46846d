"""Algorithm 1 and the latency model on the host (libmsao.so, no GPU needed)
against the oracle: identical decisions and thresholds, bit for bit, on the
same float entropies; the closed forms of Eq. 8 and 12-14; argument checks."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2604_02945_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INVALID = 1


def params(**kw):
    p = B.sched_default_params()
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def test_default_params_are_the_papers():
    p = B.sched_default_params()
    assert (p.p_target, p.n_max, p.quantile, p.delta) == (0.8, 5, 0.7, 0.95)   # Sec. 5.1 settings
    assert 0.0 <= p.theta_min < 0.7 and 0.0 < p.alpha <= 1.0


def calib(n, seed):
    """Normalised entropies shaped like a draft model's: a confident mass near
    0 and a broad unconfident part (a float32 array)."""
    rng = np.random.default_rng(seed)
    conf = rng.beta(0.6, 8.0, n)
    unconf = rng.beta(4.0, 3.0, n)
    return np.where(rng.random(n) < 0.6, conf, unconf).astype(np.float32)


@pytest.mark.parametrize("n,seed,q", [(500, 1, 0.7), (500, 2, 0.3), (1, 3, 0.7), (7, 4, 0.5), (1000, 5, 1.0),
                                      (999, 6, 0.0)])
def test_init_matches_oracle(n, seed, q):
    h = calib(n, seed)
    s = B.Scheduler(h, params(quantile=q))
    h64 = h.astype(np.float64)
    theta = oracle.entropy_quantile(h64, q)
    P = oracle.p_conf(h64, theta)
    assert s.state.theta == theta
    assert s.state.p_conf == P
    assert s.state.n_draft == oracle.n_draft(P, 0.8, 5)
    assert (s.state.cache, s.state.steps, s.state.sends) == (0, 0, 0)


@pytest.mark.parametrize("seed,n_draft_override", [(11, None), (12, 1), (13, 5)])
def test_steps_match_oracle_bitwise(seed, n_draft_override):
    h_cal = calib(500, seed)
    p = params(alpha=0.15, theta_min=0.02)
    s = B.Scheduler(h_cal, p)
    if n_draft_override is not None:
        s.state.n_draft = n_draft_override
    trace = calib(20000, seed + 100)
    theta0, nd = s.state.theta, s.state.n_draft
    dec, th = s.run(trace)
    odec, oth, ocnt = oracle.sched_run(trace.astype(np.float64), theta0, nd, p.delta, p.theta_min, p.alpha)
    assert np.array_equal(dec, odec)
    assert np.array_equal(th, oth)           # same double arithmetic, same order: bit-identical
    st = s.state
    assert [st.held, st.sends, st.offloads, st.tokens_sent] == ocnt.tolist()
    assert st.steps == trace.size


def test_step_by_step_equals_run():
    h_cal = calib(500, 21)
    trace = calib(300, 22)
    a, b = B.Scheduler(h_cal), B.Scheduler(h_cal)
    dec, th = a.run(trace)
    for i, h in enumerate(trace):
        assert b.step(h) == dec[i]
        assert b.state.theta == th[i]


def test_hand_worked_trace():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "sched_trace.json")))
    p = g["params"]
    s = B.Scheduler(np.array([0.5], np.float32), params(delta=p["delta"], theta_min=p["theta_min"],
                                                         alpha=p["alpha"]))
    s.state.theta, s.state.n_draft = p["theta0"], p["n_draft"]
    dec, th = s.run(np.array(g["h_norm"], np.float32))          # dyadic values: exact in float32
    assert dec.tolist() == g["decisions"] and th.tolist() == g["theta_after"]


def test_nan_entropy_offloads():
    s = B.Scheduler(calib(50, 31))
    t0 = s.state.theta
    assert s.step(float("nan")) == B.DECIDE_OFFLOAD
    assert s.state.theta == max(t0 * 0.95, 0.05)


def test_latency_model_matches_oracle():
    assert B.comm_latency(1e6, 25e6, 0.02) == oracle.comm_latency(1e6, 25e6, 0.02)
    rng = np.random.default_rng(41)
    h = calib(777, 42)
    for theta in (0.0, 0.1, 0.35, 0.9, 1.0):
        assert B.p_conf(h, theta) == oracle.p_conf(h.astype(np.float64), theta)
    for P in (0.0, 0.25, 0.7, 0.999):
        assert B.expected_spec_tokens(P) == oracle.expected_spec(P)
    assert math.isinf(B.expected_spec_tokens(1.0))
    for _ in range(20):
        t = dict(prefill_edge=rng.uniform(0.01, 0.3), prefill_cloud=rng.uniform(0.01, 0.3),
                 comm_offloaded=rng.uniform(0, 0.2), p_conf=rng.uniform(0, 0.99), n_draft=int(rng.integers(1, 6)),
                 t_draft=rng.uniform(0.005, 0.03), t_verify=rng.uniform(0.002, 0.01), t_offload=rng.uniform(0.02, 0.2))
        want = oracle.expected_e2e(t["prefill_edge"], t["prefill_cloud"], t["comm_offloaded"], t["p_conf"],
                                   t["n_draft"], t["t_draft"], t["t_verify"], t["t_offload"])
        assert B.expected_e2e_latency(**t) == pytest.approx(want, rel=1e-15)


def test_retention_floor_matches_oracle():
    mas = np.array([0.0, 0.25, 0.6796875, 1.0], np.float32)
    assert np.array_equal(B.retention_floor(mas), oracle.retention(mas.astype(np.float64)).astype(np.float32))


def test_struct_sizes():
    import ctypes
    assert ctypes.sizeof(B.MsaoSchedParams) == 48
    assert ctypes.sizeof(B.MsaoSchedState) == 72
    assert ctypes.sizeof(B.MsaoLatencyModel) == 64
    assert ctypes.sizeof(B.MsaoEntropyOut) == 32


@pytest.mark.parametrize("field,value", [("p_target", 1.0), ("p_target", 0.0), ("n_max", 0), ("quantile", 1.5),
                                         ("delta", 0.0), ("delta", 1.1), ("theta_min", -0.1),
                                         ("theta_min", float("inf")), ("alpha", 1.5), ("alpha", -0.1)])
def test_init_rejects_bad_params(field, value):
    L = B.lib()
    h = calib(10, 51)
    st = B.MsaoSchedState()
    assert L.msao_sched_init(h.ctypes.data, h.size, B._addr(params(**{field: value})), B._addr(st)) == INVALID


def test_init_rejects_bad_inputs():
    L = B.lib()
    st = B.MsaoSchedState()
    p = params()
    h = np.array([0.1, np.nan], np.float32)
    assert L.msao_sched_init(h.ctypes.data, 2, B._addr(p), B._addr(st)) == INVALID
    assert L.msao_sched_init(h.ctypes.data, 0, B._addr(p), B._addr(st)) == INVALID
    assert L.msao_sched_init(None, 2, B._addr(p), B._addr(st)) == INVALID
    d = B.ctypes.c_int32()
    assert L.msao_sched_step(None, B._addr(p), 0.1, B.ctypes.byref(d)) == INVALID


def test_draft_entropy_rejects_null_context():
    out = B.MsaoEntropyOut()
    assert B.lib().msao_draft_entropy(None, None, 1, 8, 8, B.BF16, 0.5, B._addr(out), None) == INVALID
