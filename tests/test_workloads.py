"""The seeded generators: determinism, prefix property, shapes and masks."""
import hashlib

import numpy as np
import pytest

from workloads import AUDIO, IMAGE, TEXT, VIDEO, bf16_bits_to_f32, f32_to_bf16_bits, make_workload


def _digest(w):
    h = hashlib.sha256()
    for s in w.segments:
        h.update(np.ascontiguousarray(s.data).tobytes())
    return h.hexdigest()


@pytest.mark.parametrize("config,n", [(1, None), (2, 2), (3, 1), (4, 2), (5, 1)])
def test_same_seed_same_bytes(config, n):
    assert _digest(make_workload(config, n_requests=n)) == _digest(make_workload(config, n_requests=n))


def test_other_seed_other_bytes():
    assert _digest(make_workload(1, seed=0)) != _digest(make_workload(1, seed=1))


def test_prefix_of_requests_is_reproducible():
    a = make_workload(4, n_requests=1)
    b = make_workload(4, n_requests=2)
    for s, t in zip(a.segments, b.segments[:3]):
        assert np.array_equal(s.data, t.data)


def test_shapes_and_modalities():
    w = make_workload(4, n_requests=1)
    assert [(s.modality, s.n_tokens, s.hidden, s.dtype, s.keep_ratio) for s in w.segments] == [
        (IMAGE, 576, 1024, "bf16", 0.25), (AUDIO, 1500, 1280, "bf16", 0.5), (TEXT, 128, 4096, "bf16", 1.0)]
    assert w.segments[1].meta["silence_mask"].sum() == 600
    w = make_workload(3, n_requests=1)
    s = w.segments[0]
    assert (s.modality, s.n_frames, s.tokens_per_frame, s.hidden) == (VIDEO, 32, 256, 1024)
    assert s.meta["static_mask"].sum() == 179
    w = make_workload(5, n_requests=1)
    assert w.segments[0].meta["bg_mask"].sum() == 5 * 288
    w = make_workload(1)
    assert w.segments[0].meta["bg_mask"].sum() == 345 and w.segments[0].dtype == "f32"
    w = make_workload(2, n_requests=3)
    for s in w.segments[::2]:
        assert 0.2 * 576 - 1 <= s.meta["bg_mask"].sum() <= 0.8 * 576 + 1


def test_full_sizes():
    # token and byte counts of the full workloads (computed from shapes, nothing drawn)
    expect = {1: (608, 2490368), 2: (40960, 109051904), 3: (65536, 134217728),
              4: (70528, 194183168), 5: (737280, 1509949440)}
    for c, (ntok, nbytes) in expect.items():
        per = {1: [(576, 1024, 4), (32, 1024, 4)], 2: [(576, 1024, 2), (64, 4096, 2)] * 64,
               3: [(8192, 1024, 2)] * 8, 4: [(576, 1024, 2), (1500, 1280, 2), (128, 4096, 2)] * 32,
               5: [(2880, 1024, 2)] * 256}[c]
        assert sum(n for n, _, _ in per) == ntok
        assert sum(n * h * e for n, h, e in per) == nbytes


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, np.inf, 0.0, -0.0], np.float32)
    b = f32_to_bf16_bits(x)
    back = bf16_bits_to_f32(b)
    assert back[0] == 1.0 and back[1] == 1.0  # tie -> even
    assert back[2] == np.float32(1.0 + 2 ** -7)
    assert back[3] == -2.5 and np.isinf(back[4]) and back[5] == 0 and np.signbit(back[6])
    assert np.isnan(bf16_bits_to_f32(f32_to_bf16_bits(np.array([np.nan], np.float32))))[0]
