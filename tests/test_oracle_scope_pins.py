"""Pins of the per-frame selection scope in the oracle (the alternative to
per-segment selection: each frame of a clip keeps its own k_f = min(P,
ceil(kappa P)) tokens, the k_f smallest (key, index) pairs of the frame;
Sec. 4.1.1 pruning with the Eq. 11 floor applied per frame): a hand-worked
clip where the two scopes differ, the counting definition of the k smallest
pairs, agreement with per-segment selection when T = 1, and MAS-guided
ratios."""
import math

import numpy as np
import pytest

import oracle
from workloads import IMAGE, VIDEO, Segment, default_params, make_workload


def per_frame(p):
    q = dict(p)
    q["flags"] = q.get("flags", 0) | oracle.FLAG_SELECT_PER_FRAME
    return q


def hand_clip():
    # 2 frames x 3 tokens x 4 fp32 channels, tau = 0.1; a channel of 0 is
    # inactive, of 1 active: z (inactive channels) per token by construction
    z = [[3, 1, 2], [0, 4, 0]]
    rows = []
    for fr in z:
        for zz in fr:
            rows.append([0.0] * zz + [1.0] * (4 - zz))
    return Segment(0, VIDEO, 2, 3, 4, "f32", 0.5, np.array(rows, np.float32))


def test_hand_example_differs_from_per_segment():
    # lambda_t = 0: the key is lambda_s z, so the kept tokens are the fewest
    # inactive channels. Per frame k_f = ceil(0.5 * 3) = 2: frame 0 keeps
    # tokens 1 (z 1) and 2 (z 2), frame 1 keeps 3 and 5 (z 0). Per segment
    # k = ceil(0.5 * 6) = 3 keeps 3, 5 (z 0) and 1 (z 1).
    p = default_params()
    p["lambda_t"] = [0.0, 0.0, 0.0, 0.0]
    s = hand_clip()
    a = oracle.run([s], 1, per_frame(p))
    assert a["z"].tolist() == [3, 1, 2, 0, 4, 0]
    assert a["k"].tolist() == [4]
    assert a["kept_idx"].tolist() == [1, 2, 3, 5, -1, -1]
    assert a["keep"].tolist() == [0, 1, 1, 1, 0, 1]
    b = oracle.run([s], 1, p)
    assert b["k"].tolist() == [3]
    assert b["kept_idx"].tolist() == [1, 3, 5, -1, -1, -1]


def keys_of(seg, p, z, d):
    Ls = oracle.q24(p["lambda_s"][seg.modality])
    Lt = oracle.q24(p["lambda_t"][seg.modality])
    temporal = seg.modality == VIDEO and seg.n_frames >= 2 and seg.tokens_per_frame > 0
    return [Ls * int(zz) + (Lt * (seg.hidden - int(dd)) if temporal else 0) for zz, dd in zip(z, d)]


@pytest.mark.parametrize("keep", [0.0, 0.3, 0.5, 1.0])
def test_counting_definition_per_frame(keep):
    # token i of frame f is kept iff fewer than k_f tokens of its frame have a
    # smaller (key, index) pair
    w = make_workload(3, n_requests=2)
    segs = [Segment(s.request, s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype, keep, s.data)
            for s in w.segments]
    o = oracle.run(segs, 2, per_frame(w.params))
    off = 0
    for i, s in enumerate(segs):
        T, P = s.n_frames, s.tokens_per_frame
        kf = min(P, math.ceil(np.float64(np.float32(keep)) * P))
        assert o["k"][i] == T * kf
        key = keys_of(s, w.params, o["z"][off:off + T * P], o["d"][off:off + T * P])
        keep_flags = o["keep"][off:off + T * P]
        for f in range(T):
            pairs = [(key[f * P + j], f * P + j) for j in range(P)]
            for j in range(P):
                below = sum(1 for q in pairs if q < pairs[j])
                assert keep_flags[f * P + j] == (1 if below < kf else 0)
        kept = o["kept_idx"][off:off + T * P]
        assert kept[:T * kf].tolist() == np.flatnonzero(keep_flags).tolist()
        assert np.all(kept[T * kf:] == -1)
        off += T * P


def test_single_frame_segments_are_unchanged():
    w = make_workload(4, n_requests=3)
    a = oracle.run(w.segments, 3, w.params)
    b = oracle.run(w.segments, 3, per_frame(w.params))
    for k in ("k", "keep", "kept_idx", "mas"):
        assert np.array_equal(a[k], b[k]), k


def test_mas_guided_per_frame():
    w = make_workload(3, n_requests=2)
    segs = [Segment(s.request, s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype, -1.0, s.data)
            for s in w.segments]
    o = oracle.run(segs, 2, per_frame(w.params))
    for i, s in enumerate(segs):
        mas = float(o["mas"][s.request * 4 + s.modality])
        kf = min(s.tokens_per_frame, math.ceil((1.0 - mas) * s.tokens_per_frame))
        assert o["k"][i] == s.n_frames * kf
