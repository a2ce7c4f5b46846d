"""The largest row the ABI accepts (hidden = 65,536 channels: 128 KiB bf16
rows, 256 KiB fp32 rows) through every entry point that reads rows, each at
its own parity bar: msao_run (row and chain paths, compaction), the SimHash
variant (Eq. 5 alone and the whole run, K = 64, integer inputs so every
projection is exact), and the learned head (Eq. 3) with its projection over
the full width. Also the largest keys: lambda weights of 1.0 (Q24 2^24) at
the full width make L_s z reach 2^40, and under SimHash the key's
multipliers reach L_s K and L_t C."""
import numpy as np
import pytest
import torch

import oracle
from test_gpu_learned import compare as compare_learned, make_head, run_case as run_learned
from test_gpu_parity import log, run_and_compare
from test_gpu_simhash import compare as compare_sh, run_case as run_sh
from test_gpu_simhash_run import encode, exact_compare, int_clip, int_planes, int_rows
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits, simhash_planes

pytestmark = pytest.mark.gpu

CMAX = 65536


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def wide_table(rng):
    def g(n, dtype, relu=False):
        x = rng.standard_normal((n, CMAX)).astype(np.float32)
        if relu:
            x = np.maximum(x, 0) * np.where(rng.random((n, 1)) < 0.5, 0.05, 1.0).astype(np.float32)
        return x if dtype == "f32" else f32_to_bf16_bits(x)
    return [Segment(0, IMAGE, 1, 9, CMAX, "bf16", 0.4, g(9, "bf16", relu=True)),
            Segment(0, VIDEO, 3, 4, CMAX, "bf16", 0.5, g(12, "bf16")),
            Segment(0, TEXT, 1, 3, CMAX, "bf16", 1.0, g(3, "bf16")),
            Segment(1, AUDIO, 1, 5, CMAX, "f32", -1.0, g(5, "f32", relu=True)),
            Segment(1, VIDEO, 2, 3, CMAX, "f32", 0.5, g(6, "f32"))]


@pytest.mark.parametrize("flags", [0, 2])
def test_run_at_maximum_width(flags, dev):
    segs = wide_table(np.random.default_rng(1))
    p = default_params()
    p["flags"] = flags
    log(f"[limits] msao_run at hidden {CMAX}, flags {flags}")
    run_and_compare(segs, 2, p, dev)


def test_run_with_unit_weights_at_maximum_width(dev):
    segs = wide_table(np.random.default_rng(2))
    p = default_params()
    p["lambda_s"] = [1.0] * 4
    p["lambda_t"] = [1.0] * 4
    log("[limits] msao_run at hidden 65536 with lambda 1.0")
    run_and_compare(segs, 2, p, dev)


def test_simhash_at_maximum_width(dev):
    rng = np.random.default_rng(3)
    segs = [Segment(0, VIDEO, 3, 20, CMAX, "bf16", 0.5, encode(int_clip(rng, 3, 20, CMAX), "bf16")),
            Segment(0, IMAGE, 1, 7, CMAX, "bf16", 0.5, encode(int_rows(rng, 7, CMAX), "bf16")),
            Segment(1, VIDEO, 2, 9, CMAX, "f32", -1.0, encode(int_clip(rng, 2, 9, CMAX), "f32"))]
    hashes = [dict(planes=int_planes(rng, 64, CMAX, s.dtype), bits=64) if s.modality == VIDEO else None
              for s in segs]
    p = default_params()
    log("[limits] Eq. 5 with SimHash at hidden 65536, K 64")
    g, ref = run_sh(segs, 2, hashes, dev, p)
    assert compare_sh(segs, hashes, g, ref) >= 0
    assert np.array_equal(g["sig"], ref["sig"]) and np.array_equal(g["d"], ref["d"])
    log("[limits] msao_run_simhash at hidden 65536, K 64")
    p["lambda_s"] = [1.0] * 4
    p["lambda_t"] = [1.0] * 4
    exact_compare(segs, 2, p, hashes, dev)


def test_gaussian_simhash_at_maximum_width(dev):
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3 * 16, CMAX)).astype(np.float32)
    segs = [Segment(0, VIDEO, 3, 16, CMAX, "bf16", 0.5, f32_to_bf16_bits(x))]
    hashes = [dict(planes=simhash_planes(32, CMAX, seed=5), bits=32)]
    g, ref = run_sh(segs, 1, hashes, dev, default_params())
    nb = compare_sh(segs, hashes, g, ref)
    log(f"[limits] Gaussian SimHash at hidden 65536: {nb} borderline bits")


def test_learned_head_at_maximum_width(dev):
    rng = np.random.default_rng(6)
    segs = wide_table(rng)[:2]
    heads = [make_head(segs[0], rng, 3, 3, -0.1)[1], make_head(segs[1], rng, 2, 1, 0.2)[1]]
    log("[limits] learned heads at hidden 65536")
    g, ref = run_learned(segs, 1, heads, None, dev)
    compare_learned(segs, 1, heads, g, ref)
