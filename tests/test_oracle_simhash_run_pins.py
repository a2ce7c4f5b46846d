"""Pins of the whole analysis with SimHash as Eq. 5's hash (oracle.run with
hashes): SimHash's d, counted in K bits per token, replaces bit sampling's d
(C activity bits per token) in D_t, sim, Qbits, the temporal term of Eq. 7,
informativeness and the selection key.

* Reduction to bit sampling. On 0/1 activations with hyperplane k = -e_k,
  SimHash bit k is 1 iff channel k is inactive, the complement of its
  activity bit, and the all-zero frame has all bits 1, the complement of its
  all-0 activity bits; so SimHash's d equals bit sampling's d. With K = C
  every output must equal the bit-sampling run's. With every channel stored
  twice (C = 2K, hyperplanes on the first copy) each Eq. 5 count is half of
  bit sampling's and every ratio (sim, gamma, temporal term, MAS,
  informativeness, the order of the keys and so the selection) is the same.
  A count divided by C instead of K anywhere fails this.
* lambda_t = 0: the hash enters nothing but Eq. 5's own outputs.
* The Eq. 5 entry point (oracle.temporal_simhash) gives the same signatures,
  d, D_t, sim, gamma and temporal term.
* Selection by brute force: the kept tokens are the k smallest pairs of
  (lambda_s z / C + lambda_t (K - d) / K, index), evaluated as exact
  fractions with the Q24 weights.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workloads import IMAGE, TEXT, VIDEO, Segment, default_params, simhash_planes


def binary_clip(rng, T, P, C, request=0, keep=0.5, dup=1):
    x = (rng.random((T * P, C)) < 0.4).astype(np.float32)
    # make neighbouring frames similar so the temporal term is not trivial
    for t in range(1, T):
        keep_rows = rng.random(P) < 0.6
        x[t * P:(t + 1) * P][keep_rows] = x[(t - 1) * P:t * P][keep_rows]
    data = np.ascontiguousarray(np.tile(x, (1, dup)))
    return Segment(request, VIDEO, T, P, C * dup, "f32", keep, data)


def binary_rows(rng, N, C, modality, request=0, keep=0.5, dup=1):
    x = (rng.random((N, C)) < 0.5).astype(np.float32)
    return Segment(request, modality, 1, N, C * dup, "f32", keep, np.ascontiguousarray(np.tile(x, (1, dup))))


def neg_identity(K, C):
    r = np.zeros((K, C), np.float32)
    r[np.arange(K), np.arange(K)] = -1.0
    return r


def table(rng, K, dup):
    segs = [binary_clip(rng, 5, 12, K, request=0, keep=0.4, dup=dup),
            binary_rows(rng, 20, K, IMAGE, request=0, keep=0.25, dup=dup),
            binary_rows(rng, 6, K, TEXT, request=0, keep=1.0, dup=dup),
            binary_clip(rng, 4, 9, K, request=1, keep=-1.0, dup=dup),
            binary_clip(rng, 3, 7, K, request=1, keep=0.5, dup=dup)]
    hashes = [dict(planes=neg_identity(K, K * dup), bits=K) if s.modality == VIDEO else None for s in segs]
    return segs, hashes


@pytest.mark.parametrize("K", [16, 32, 64])
@pytest.mark.parametrize("flags", [0, oracle.FLAG_SELECT_PER_FRAME, oracle.FLAG_TEMPORAL_LITERAL])
def test_reduces_to_bit_sampling_with_k_equal_c(K, flags):
    rng = np.random.default_rng(K + 7 * flags)
    segs, hashes = table(rng, K, 1)
    p = default_params()
    p["flags"] = flags
    a = oracle.run(segs, 2, p)
    b = oracle.run(segs, 2, p, hashes=hashes)
    for key in ("z", "l1", "l2", "info", "d", "res", "dframe", "sim", "gamma", "agg", "rho", "temporal", "beta",
                "mas", "present", "k", "keep", "kept_idx"):
        assert np.array_equal(a[key], b[key]), key
    for ra, rb in zip(a["compact"], b["compact"]):
        assert np.array_equal(ra, rb)


@pytest.mark.parametrize("K", [16, 32])
@pytest.mark.parametrize("flags", [0, oracle.FLAG_SELECT_PER_FRAME])
def test_duplicated_channels_halve_the_counts_and_keep_every_ratio(K, flags):
    rng = np.random.default_rng(100 + K + flags)
    segs, hashes = table(rng, K, 2)
    p = default_params()
    p["flags"] = flags
    p["lambda_s"] = [0.0, 0.6, 0.5, 0.6]   # both terms weigh in the video keys
    a = oracle.run(segs, 2, p)
    b = oracle.run(segs, 2, p, hashes=hashes)
    assert np.array_equal(a["d"], 2 * b["d"])
    assert np.array_equal(a["dframe"], 2 * b["dframe"])
    agg_a, agg_b = a["agg"].reshape(-1, 4), b["agg"].reshape(-1, 4)
    assert np.array_equal(agg_a[:, :2], agg_b[:, :2])
    assert np.array_equal(agg_a[:, 2:], 2 * agg_b[:, 2:])
    for key in ("z", "l1", "l2", "info", "res", "sim", "gamma", "rho", "temporal", "beta", "mas", "present", "k",
                "keep", "kept_idx"):
        assert np.array_equal(a[key], b[key]), key
    assert b["agg"].reshape(-1, 4)[VIDEO, 3] == 4 * 12 * K   # (T - 1) P K of the request-0 clip


def gaussian_table(seed, K):
    rng = np.random.default_rng(seed)
    C = 64
    segs = [Segment(0, VIDEO, 4, 10, C, "f32", 0.3, rng.standard_normal((40, C)).astype(np.float32)),
            Segment(0, IMAGE, 1, 24, C, "f32", 0.5, rng.standard_normal((24, C)).astype(np.float32)),
            Segment(1, VIDEO, 3, 8, C, "f32", -1.0, rng.standard_normal((24, C)).astype(np.float32))]
    hashes = [dict(planes=simhash_planes(K, C, seed=seed + i, dtype="f32"), bits=K) if s.modality == VIDEO
              else None for i, s in enumerate(segs)]
    return segs, hashes


@pytest.mark.parametrize("K", [16, 48])
def test_without_temporal_weight_the_hash_only_changes_eq5(K):
    segs, hashes = gaussian_table(3, K)
    p = default_params()
    p["lambda_t"] = [0.0, 0.0, 0.0, 0.0]
    a = oracle.run(segs, 2, p)
    b = oracle.run(segs, 2, p, hashes=hashes)
    for key in ("z", "l1", "l2", "info", "res", "rho", "beta", "mas", "present", "k", "keep", "kept_idx"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("K", [16, 32, 64])
def test_eq5_outputs_match_the_eq5_entry_point(K):
    segs, hashes = gaussian_table(11, K)
    p = default_params()
    b = oracle.run(segs, 2, p, hashes=hashes)
    e = oracle.temporal_simhash(segs, 2, p, hashes)
    for key in ("sig", "d", "dframe", "sim", "gamma", "temporal"):
        assert np.array_equal(b[key], e[key]), key
    agg = b["agg"].reshape(-1, 4)
    assert np.array_equal(agg[:, 2], e["dsum"]) and np.array_equal(agg[:, 3], e["qbits"])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_selection_is_the_smallest_weighted_redundancy(seed):
    K = 32
    segs, hashes = gaussian_table(20 + seed, K)
    p = default_params()
    p["lambda_s"] = [0.0, 0.6, 0.55, 0.6]
    b = oracle.run(segs, 2, p, hashes=hashes)
    off = 0
    for si, s in enumerate(segs):
        N, C = s.n_tokens, s.hidden
        if s.modality == VIDEO:
            Ls = Fraction(int(oracle.q24(p["lambda_s"][VIDEO])))
            Lt = Fraction(int(oracle.q24(p["lambda_t"][VIDEO])))
            z = b["z"][off:off + N].astype(int)
            d = b["d"][off:off + N].astype(int)
            score = [Ls * z[i] / C + Lt * (K - d[i]) / K for i in range(N)]
            order = sorted(range(N), key=lambda i: (score[i], i))
            k = int(b["k"][si])
            want = sorted(order[:k])
            assert b["kept_idx"][off:off + k].tolist() == want
            assert np.all(b["kept_idx"][off + k:off + N] == -1)
            # informativeness: 1 - (lambda_s z / C + lambda_t (K - d) / K)
            lam_s, lam_t = p["lambda_s"][VIDEO], p["lambda_t"][VIDEO]
            info = 1.0 - (np.float64(np.float32(lam_s)) * z / C + np.float64(np.float32(lam_t)) * (K - d) / K)
            np.testing.assert_allclose(b["info"][off:off + N], info.astype(np.float32), rtol=0, atol=1e-7)
        off += N
