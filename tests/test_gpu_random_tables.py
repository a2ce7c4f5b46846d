"""Seeded random segment tables through msao_run against the oracle: mixed
modalities, fp32 and bf16, ragged widths (multiples of 8 channels up to
1288), one to nine frames per clip, ragged frame sizes, fixed, zero, full and
MAS-guided keep ratios, padded row strides, several segments per request and
modality, and the literal and per-frame flags. Same bar as the parity tests
(run_and_compare): integers, kept indices and compacted rows bit-exact. The
same kind of tables also go through the SimHash entry points and the learned
heads at their bars; for msao_run_simhash the tables hold integer values, so
that every projection is exact and the whole run is compared bit for bit.
A second set of tables is drawn so that most of its clips take the paired
scoring pass (bf16 rows of 512 to 2,048 bytes, up to 72 frames)."""
import numpy as np
import pytest
import torch

from test_gpu_parity import log, run_and_compare
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def random_table(seed):
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.integers(1, 4))
    segs = []
    for _ in range(int(rng.integers(1, 7))):
        m = int(rng.choice([TEXT, IMAGE, VIDEO, AUDIO]))
        dtype = "bf16" if rng.random() < 0.6 else "f32"
        C = int(rng.integers(1, 162)) * 8
        T = int(rng.integers(1, 10)) if m == VIDEO else 1
        P = int(rng.integers(0, 300 if T > 1 else 900))
        keep = float(rng.choice([0.0, 1.0, -1.0, 0.13, 0.37, 0.5, 0.81]))
        kind = rng.integers(3)
        x = rng.standard_normal((T * P, C)).astype(np.float32)
        if kind == 1:
            x = np.maximum(x, 0) * np.where(rng.random((T * P, 1)) < 0.4, 0.05, 1.0).astype(np.float32)
        elif kind == 2 and T > 1 and P > 0:
            for t in range(1, T):   # slowly drifting frames
                x[t * P:(t + 1) * P] = x[(t - 1) * P:t * P] + 0.02 * rng.standard_normal((P, C)).astype(np.float32)
        data = x if dtype == "f32" else f32_to_bf16_bits(x)
        segs.append(Segment(int(rng.integers(R)), m, T, P, C, dtype, keep, data))
    p = default_params()
    p["flags"] = int(rng.integers(4))            # literal and/or per-frame
    pad = int(rng.choice([0, 0, 8, 24]))
    return segs, R, p, pad


@pytest.mark.parametrize("seed", range(24))
def test_random_table(seed, dev):
    segs, R, p, pad = random_table(seed)
    log(f"[random] seed {seed}: {len(segs)} segments, R {R}, flags {p['flags']}, pad {pad}, "
        f"tokens {sum(s.n_tokens for s in segs)}")
    run_and_compare(segs, R, p, dev, pad=pad)


def random_pair_table(seed):
    """Tables whose clips mostly take k_pair (bf16, 256 to 1,024 channels):
    any frame count from 2 to 72 (ranges of 8 to 32 frames, those after a
    clip's first reading a halo frame; the range length depends on the
    whole batch's pairs of positions), odd and even position counts,
    drifting and redrawn frames, beside a few segments of the other
    passes."""
    rng = np.random.default_rng(3000 + seed)
    R = int(rng.integers(1, 4))
    segs = []
    for _ in range(int(rng.integers(1, 5))):
        T, P = int(rng.integers(2, 73)), int(rng.integers(1, 40))
        C = int(rng.choice([256, 512, 768, 1024]))
        x = rng.standard_normal((T * P, C)).astype(np.float32)
        if rng.random() < 0.5:
            for t in range(1, T):
                x[t * P:(t + 1) * P] = x[(t - 1) * P:t * P] + 0.02 * rng.standard_normal((P, C)).astype(np.float32)
        keep = float(rng.choice([0.3, 0.5, -1.0, 0.07]))
        segs.append(Segment(int(rng.integers(R)), VIDEO, T, P, C, "bf16", keep, f32_to_bf16_bits(x)))
    for _ in range(int(rng.integers(0, 3))):
        m = int(rng.choice([TEXT, IMAGE, AUDIO]))
        C = int(rng.integers(1, 162)) * 8
        P = int(rng.integers(1, 600))
        x = rng.standard_normal((P, C)).astype(np.float32)
        segs.append(Segment(int(rng.integers(R)), m, 1, P, C, "bf16", float(rng.choice([0.25, 1.0, -1.0])),
                            f32_to_bf16_bits(x)))
    p = default_params()
    p["flags"] = int(rng.integers(4))
    pad = int(rng.choice([0, 0, 8, 40]))
    return segs, R, p, pad


@pytest.mark.parametrize("seed", range(32))
def test_random_pair_table(seed, dev):
    segs, R, p, pad = random_pair_table(seed)
    log(f"[random] pair seed {seed}: {len(segs)} segments, R {R}, flags {p['flags']}, pad {pad}, "
        f"shapes {[(s.n_frames, s.tokens_per_frame, s.hidden) for s in segs]}")
    run_and_compare(segs, R, p, dev, pad=pad)


@pytest.mark.parametrize("seed", range(8))
def test_random_table_simhash(seed, dev):
    from test_gpu_simhash import compare as compare_sh, run_case as run_sh
    from workloads import simhash_planes
    segs, R, p, pad = random_table(100 + seed)
    rng = np.random.default_rng(seed)
    hashes = [dict(planes=simhash_planes(int(rng.choice([16, 32, 48, 64])), s.hidden, seed=seed, dtype=s.dtype),
                   bits=0) for s in segs]
    for h in hashes:
        h["bits"] = h["planes"].shape[0]
    log(f"[random] simhash seed {seed}: {len(segs)} segments, R {R}, pad {pad}")
    g, ref = run_sh(segs, R, hashes, dev, params=p, pad=pad)
    compare_sh(segs, hashes, g, ref)


@pytest.mark.parametrize("seed", range(8))
def test_random_table_learned(seed, dev):
    from test_gpu_learned import compare as compare_l, make_head, mlp_for, run_case as run_l
    segs, R, p, _ = random_table(200 + seed)
    rng = np.random.default_rng(50 + seed)
    heads = []
    for s in segs:
        P = s.tokens_per_frame
        if s.n_tokens == 0 or rng.random() < 0.3:
            heads.append(None)
            continue
        divs = [w for w in range(1, P + 1) if P % w == 0]
        grid_w = int(rng.choice(divs)) if rng.random() < 0.7 else 0
        heads.append(make_head(s, rng, grid_w, int(rng.choice([1, 3, 5, 7])), float(rng.uniform(-1, 1)))[1])
    mlp = mlp_for(R, int(rng.choice([0, 16, 100])), int(rng.choice([8, 64])), rng) if rng.random() < 0.7 else None
    log(f"[random] learned seed {seed}: {len(segs)} segments, R {R}, heads {sum(h is not None for h in heads)}, "
        f"mlp {mlp is not None}")
    g, ref = run_l(segs, R, heads, mlp, dev, params=p)
    compare_l(segs, R, heads, g, ref, mlp)


@pytest.mark.parametrize("seed", range(12))
def test_random_table_simhash_run(seed, dev):
    from test_gpu_simhash_run import exact_compare, int_clip, int_planes, int_rows
    segs, R, p, pad = random_table(300 + seed)
    rng = np.random.default_rng(70 + seed)
    isegs = []
    for s in segs:   # the same shapes and parameters with integer values (exact projections)
        x = int_clip(rng, s.n_frames, s.tokens_per_frame, s.hidden) if s.n_frames > 1 else \
            int_rows(rng, s.n_tokens, s.hidden)
        data = x if s.dtype == "f32" else f32_to_bf16_bits(x)
        isegs.append(Segment(s.request, s.modality, s.n_frames, s.tokens_per_frame, s.hidden, s.dtype,
                             s.keep_ratio, data))
    hashes = []
    for s in isegs:
        K = int(rng.choice([16, 32, 48, 64]))
        temporal = s.modality == VIDEO and s.n_frames >= 2 and s.tokens_per_frame > 0
        hashes.append(dict(planes=int_planes(rng, K, s.hidden, s.dtype), bits=K) if temporal else None)
    log(f"[random] simhash run seed {seed}: {len(isegs)} segments, R {R}, flags {p['flags']}, pad {pad}, "
        f"tokens {sum(s.n_tokens for s in isegs)}")
    exact_compare(isegs, R, p, hashes, dev, pad=pad)
