"""Pins of the SimHash variant of Eq. 5 in the oracle (Sec. 4.1.2 with
Charikar's random-hyperplane hash: bit k of a token is 1 iff r_k . f >= 0):
a hand-worked clip, the collision probability 1 - theta/pi, exact identities
(scaling keeps every bit, negation flips every bit, the zero frame), the bits
against numpy's projection, and the frame/token similarity identity."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from workloads import IMAGE, VIDEO, Segment, bf16_bits_to_f32, default_params, f32_to_bf16_bits, simhash_planes

HERE = os.path.dirname(os.path.abspath(__file__))


def clip(frames, dtype="f32", request=0):
    x = np.ascontiguousarray(np.concatenate(frames).astype(np.float32))
    T, P, C = len(frames), frames[0].shape[0], frames[0].shape[1]
    data = x if dtype == "f32" else f32_to_bf16_bits(x)
    return Segment(request, VIDEO, T, P, C, dtype, 1.0, data)


def planes_f32(K, C, seed):
    return np.random.default_rng(seed).standard_normal((K, C)).astype(np.float32)


def test_hand_example():
    g = json.load(open(os.path.join(HERE, "golden", "simhash_hand.json")))
    frames = [np.array(f, np.float32) for f in g["frames"]]
    s = clip(frames)
    h = [dict(planes=np.array(g["planes"], np.float32), bits=3)]
    o = oracle.temporal_simhash([s], 1, default_params(), h)
    assert o["sig"].tolist() == g["sig"]
    assert o["d"].tolist() == g["d"]
    assert o["dframe"].tolist() == g["dframe"]
    np.testing.assert_allclose(o["sim"], np.float32(g["sim"]), rtol=0, atol=0)
    np.testing.assert_allclose(o["gamma"], np.float32(g["gamma"]), rtol=0, atol=0)
    x = VIDEO
    assert o["dsum"][x] == g["dsum"] and o["qbits"][x] == g["qbits"]
    assert o["temporal"][x] == np.float32(g["temporal"])
    p = default_params()
    p["flags"] = oracle.FLAG_TEMPORAL_LITERAL
    assert oracle.temporal_simhash([s], 1, p, h)["temporal"][x] == np.float32(g["temporal_literal"])


@pytest.mark.parametrize("theta", [0.1, 0.5, 1.0, 2.0, 3.0])
def test_collision_probability_is_one_minus_angle_over_pi(theta):
    # frame 1's token is frame 0's rotated by theta in a random plane: each
    # of the K bits differs with probability theta / pi (Charikar 2002)
    rng = np.random.default_rng(int(theta * 100))
    P, C, K = 2000, 32, 64
    u = rng.standard_normal((P, C))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    w = rng.standard_normal((P, C))
    w -= np.sum(w * u, axis=1, keepdims=True) * u
    w /= np.linalg.norm(w, axis=1, keepdims=True)
    v = math.cos(theta) * u + math.sin(theta) * w
    o = oracle.temporal_simhash([clip([u, v])], 1, default_params(), [dict(planes=planes_f32(K, C, 1), bits=K)])
    frac = o["d"][P:].astype(np.float64) / K
    # bits of one token share u, so bound the variance of each d/K by 1/4
    assert abs(frac.mean() - theta / math.pi) < 5 * 0.5 / math.sqrt(P)
    assert abs(float(o["sim"][1]) - (1 - frac.mean())) < 1e-6


def test_scaling_keeps_every_bit_and_negation_flips_every_bit():
    rng = np.random.default_rng(3)
    f0 = rng.standard_normal((50, 40)).astype(np.float32)
    s = clip([f0, 2 * f0, -2 * f0, -2 * f0])
    K = 48
    o = oracle.temporal_simhash([s], 1, default_params(), [dict(planes=planes_f32(K, 40, 2), bits=K)])
    d = o["d"].reshape(4, 50)
    assert np.all(d[1] == 0) and np.all(d[2] == K) and np.all(d[3] == 0)
    assert o["sim"].tolist() == [o["sim"][0], 1.0, 0.0, 1.0]
    sig = o["sig"].reshape(4, 50)
    assert np.all(sig[2] == (~sig[1]) & np.uint64((1 << K) - 1))
    # frame 0 against the all-zero frame: the bits that are 0
    assert np.all(d[0] == K - np.array([bin(int(x)).count("1") for x in sig[0]]))


def test_zero_and_nan_rows():
    f0 = np.zeros((3, 8), np.float32)
    f1 = np.zeros((3, 8), np.float32)
    f1[1, 2] = np.nan
    f1[2] = 1.0
    K = 16
    pl = planes_f32(K, 8, 4)
    o = oracle.temporal_simhash([clip([f0, f1])], 1, default_params(), [dict(planes=pl, bits=K)])
    sig = o["sig"].reshape(2, 3)
    assert np.all(sig[0] == (1 << K) - 1)          # every projection 0 -> every bit 1
    assert sig[1, 0] == (1 << K) - 1 and sig[1, 1] == 0   # NaN compares false
    want = sum(1 << k for k in range(K) if float(pl[k].astype(np.float64).sum()) >= 0)
    assert sig[1, 2] == want
    assert o["d"].tolist() == [0, 0, 0, 0, K, K - bin(want).count("1")]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bits_match_numpy_projection(dtype):
    rng = np.random.default_rng(5)
    C, K = 200, 64
    frames = [rng.standard_normal((30, C)).astype(np.float32) for _ in range(3)]
    s = clip(frames, dtype)
    pl = simhash_planes(K, C, seed=9, dtype=dtype)
    o = oracle.temporal_simhash([s], 1, default_params(), [dict(planes=pl, bits=K)])
    x = (s.data if dtype == "f32" else bf16_bits_to_f32(s.data)).astype(np.float64)
    r = (pl if dtype == "f32" else bf16_bits_to_f32(pl)).astype(np.float64)
    y = x @ r.T
    assert np.min(np.abs(y)) > 1e-6   # no ties on this draw, so the sign is unambiguous
    bits = (y >= 0).astype(np.uint64)
    want = np.sum(bits << np.arange(K, dtype=np.uint64), axis=1, dtype=np.uint64)
    assert np.array_equal(o["sig"], want)


def test_frame_similarity_is_the_mean_of_token_similarities():
    rng = np.random.default_rng(6)
    P, C, K = 37, 24, 32
    frames = [rng.standard_normal((P, C)).astype(np.float32) for _ in range(5)]
    o = oracle.temporal_simhash([clip(frames)], 1, default_params(), [dict(planes=planes_f32(K, C, 7), bits=K)])
    d = o["d"].reshape(5, P).astype(np.float64)
    np.testing.assert_allclose(o["sim"], (1 - d / K).mean(axis=1), rtol=0, atol=1e-7)
    assert o["dframe"].tolist() == d.sum(axis=1).astype(np.uint64).tolist()
    assert o["dsum"][VIDEO] == d[1:].sum() and o["qbits"][VIDEO] == 4 * P * K
    assert o["temporal"][VIDEO] == np.float32(1 - d[1:].sum() / (4 * P * K))


def test_only_temporal_segments_are_hashed():
    rng = np.random.default_rng(8)
    img = Segment(0, IMAGE, 1, 6, 16, "f32", 0.5, rng.standard_normal((6, 16)).astype(np.float32))
    one = clip([rng.standard_normal((4, 16)).astype(np.float32)], request=1)       # T = 1: not temporal
    two = clip([rng.standard_normal((4, 16)).astype(np.float32)] * 2, request=1)
    h = [None, None, dict(planes=planes_f32(16, 16, 1), bits=16)]
    o = oracle.temporal_simhash([img, one, two], 2, default_params(), h)
    assert np.all(o["sig"][:10] == 0) and np.all(o["d"][:10] == 0)
    assert np.all(o["d"][14:] == 0)                # identical frames
    assert len(o["sim"]) == 2 and o["sim"][1] == 1.0
    assert o["temporal"][VIDEO] == 0.0 and o["temporal"][4 + VIDEO] == 1.0
    with pytest.raises(RuntimeError):
        oracle.temporal_simhash([img, one, two], 2, default_params(), [None, None, None])
