"""GPU parity of the SimHash variant of Eq. 5 (msao_temporal_simhash) against
the oracle on the same seeded inputs and hyperplanes.

Tolerance. The GPU projects on the matrix cores: bf16 products are exact in
fp32 and accumulated in fp32 (fp32 data: products rounded once), so
|y_gpu - y| <= (C + 2) 2^-24 sum_c |r_kc x_c|. A signature bit whose exact
projection lies within that bound of 0 may differ ("borderline"); every other
bit must match. d of token (t, p) may then differ by at most the borderline
bits of (t, p) and (t-1, p), D_t by the sum over the frame, and sim, gamma and
the temporal term by those counts over P K or Qbits. Every other output is
exact: without borderline bits, d, D_t, sim, gamma and the temporal term equal
the oracle's bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from paper_2604_02945_amd import binding as B
from workloads import (IMAGE, TEXT, VIDEO, Segment, bf16_bits_to_f32, default_params, f32_to_bf16_bits,
                       make_workload, simhash_planes)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_tensor(a, dtype, device):
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16 if dtype == "bf16" else np.float32)).to(device)
    return t.view(torch.bfloat16) if dtype == "bf16" else t


def to_device(segments, device, pad=0):
    out = []
    for s in segments:
        a = s.data
        if pad:
            a = np.concatenate([a, np.zeros((a.shape[0], pad), a.dtype)], axis=1)
        t = dev_tensor(a, s.dtype, device)
        if pad:
            t = t[:, :s.hidden]
        out.append(msao.DeviceSegment(t, s.request, s.modality, s.keep_ratio, s.n_frames))
    return out


def is_temporal(s):
    return s.modality == VIDEO and s.n_frames >= 2 and s.tokens_per_frame > 0


def borderline(segments, hashes):
    """Per token, the number of signature bits whose projection is within the
    fp32 accumulation bound of 0 (0 outside temporal segments)."""
    out = []
    for s, h in zip(segments, hashes):
        if not is_temporal(s):
            out.append(np.zeros(s.n_tokens, np.int64))
            continue
        x = (s.data if s.dtype == "f32" else bf16_bits_to_f32(s.data))[:, :s.hidden].astype(np.float64)
        r = (h["planes"] if s.dtype == "f32" else bf16_bits_to_f32(h["planes"])).astype(np.float64)
        y = x @ r.T
        bound = (s.hidden + 2) * 2.0 ** -24 * (np.abs(x) @ np.abs(r).T)
        out.append(np.sum(np.abs(y) <= bound, axis=1))
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def run_case(segments, R, hashes, device, params=None, pad=0):
    p = params or default_params()
    dsegs = to_device(segments, device, pad)
    dh = [None if h is None else dict(planes=dev_tensor(h["planes"], s.dtype, device), bits=h["bits"])
          for s, h in zip(segments, hashes)]
    out, sig = msao.msao_temporal_simhash(dsegs, R, dh, p)
    torch.cuda.synchronize()
    got = out.results(R, len(segments))
    g = {"sig": sig.cpu().numpy().view(np.uint64), "d": got["d"].cpu().numpy().astype(np.uint32),
         "dframe": got["dframe"].cpu().numpy().astype(np.uint64), "sim": got["sim"].cpu().numpy(),
         "gamma": got["gamma"].cpu().numpy(), "temporal": got["temporal"].cpu().numpy()}
    ref = oracle.temporal_simhash(segments, R, p, hashes)
    return g, ref


def compare(segments, hashes, g, ref):
    nb = borderline(segments, hashes)
    bits = np.array([int(x) for x in (g["sig"] ^ ref["sig"])], dtype=object)
    diff = np.array([bin(int(b)).count("1") for b in bits], np.int64)
    assert np.all(diff <= nb), f"signature bits differ beyond the borderline ones: {np.flatnonzero(diff > nb)[:5]}"
    # d against the same patch of the previous frame
    slack = np.zeros_like(nb)
    frame_slack, frame_bits = [], []
    tslack, tbits = {}, {}
    off = 0
    for si, s in enumerate(segments):
        N = s.n_tokens
        if is_temporal(s):
            P, T = s.tokens_per_frame, s.n_frames
            ss = nb[off:off + N].copy()
            ss[P:] += nb[off:off + N - P]
            slack[off:off + N] = ss
            frame_slack.append(ss.reshape(T, P).sum(axis=1))
            frame_bits.append(np.full(T, P * hashes[si]["bits"]))
            x = s.request * 4 + s.modality
            tslack[x] = tslack.get(x, 0) + int(ss[P:].sum())
            tbits[x] = tbits.get(x, 0) + (T - 1) * P * hashes[si]["bits"]
        off += N
    dd = np.abs(g["d"].astype(np.int64) - ref["d"].astype(np.int64))
    assert np.all(dd <= slack), f"d differs at {np.flatnonzero(dd > slack)[:5]}"
    fs = np.concatenate(frame_slack) if frame_slack else np.zeros(0, np.int64)
    fb = np.concatenate(frame_bits) if frame_bits else np.ones(0)
    dD = np.abs(g["dframe"].astype(np.int64) - ref["dframe"].astype(np.int64))
    assert np.all(dD <= fs), "D_t"
    # sim and gamma: the frame's slack over P K, plus one float32 rounding
    assert np.all(np.abs(g["sim"].astype(np.float64) - ref["sim"]) <= fs / fb + 2.0 ** -24), "sim"
    assert np.all(np.abs(g["gamma"].astype(np.float64) - ref["gamma"]) <= fs / fb + 2.0 ** -24), "gamma"
    for x in range(len(ref["temporal"])):
        tol = tslack.get(x, 0) / tbits[x] + 2.0 ** -24 if x in tbits else 0.0
        assert abs(float(g["temporal"][x]) - float(ref["temporal"][x])) <= tol, f"temporal[{x}]"
    if nb.sum() == 0:
        assert np.array_equal(g["sig"], ref["sig"])
        assert np.array_equal(g["d"], ref["d"])
        assert np.array_equal(g["sim"], ref["sim"]) and np.array_equal(g["gamma"], ref["gamma"])
        assert np.array_equal(g["temporal"], ref["temporal"])
    return int(nb.sum())


@pytest.mark.parametrize("bits", [16, 32, 48, 64])
def test_video_clips(bits, dev):
    w = make_workload(3, n_requests=2)
    hashes = [dict(planes=simhash_planes(bits, s.hidden, seed=1, dtype=s.dtype), bits=bits) for s in w.segments]
    log(f"[simhash] 2 clips x 32 x 256 x 1024 bf16, K = {bits}")
    g, ref = run_case(w.segments, 2, hashes, dev)
    nb = compare(w.segments, hashes, g, ref)
    log(f"[simhash] borderline bits: {nb}; sim[1:4] {g['sim'][1:4]}")


def test_full_size_clips(dev):
    w = make_workload(3)
    hashes = [dict(planes=simhash_planes(32, s.hidden, seed=2, dtype=s.dtype), bits=32) for s in w.segments]
    log("[simhash] all 8 clips, K = 32")
    g, ref = run_case(w.segments, w.n_requests, hashes, dev)
    compare(w.segments, hashes, g, ref)


def test_ragged_widths_fp32_padding_and_mixed_segments(dev):
    rng = np.random.default_rng(31)
    segs, hashes = [], []

    def add(seg, bits):
        segs.append(seg)
        hashes.append(None if bits is None else dict(planes=simhash_planes(bits, seg.hidden, seed=len(segs),
                                                                         dtype=seg.dtype), bits=bits))

    add(Segment(0, IMAGE, 1, 20, 64, "f32", 0.5, rng.standard_normal((20, 64)).astype(np.float32)), None)
    add(Segment(0, VIDEO, 3, 37, 520, "f32", 0.5, rng.standard_normal((111, 520)).astype(np.float32)), 48)
    add(Segment(1, VIDEO, 4, 9, 1288, "bf16", 0.5,
                f32_to_bf16_bits(rng.standard_normal((36, 1288)).astype(np.float32))), 16)
    add(Segment(1, VIDEO, 1, 8, 64, "bf16", 0.5, f32_to_bf16_bits(rng.standard_normal((8, 64)).astype(np.float32))),
        None)                                                   # one frame: not temporal
    add(Segment(1, TEXT, 1, 5, 32, "f32", 1.0, rng.standard_normal((5, 32)).astype(np.float32)), None)
    add(Segment(2, VIDEO, 2, 70, 8, "bf16", 0.5, f32_to_bf16_bits(rng.standard_normal((140, 8)).astype(np.float32))),
        64)                                                     # 8 channels: one 16-byte chunk per row
    log("[simhash] ragged widths, fp32, a padded row stride, mixed segments")
    for pad in (0, 8):
        g, ref = run_case(segs, 3, hashes, dev, pad=pad)
        compare(segs, hashes, g, ref)
    p = default_params()
    p["flags"] = msao.FLAG_TEMPORAL_LITERAL
    g, ref = run_case(segs, 3, hashes, dev, params=p)
    compare(segs, hashes, g, ref)


def test_scaled_frames_have_no_differing_bits(dev):
    # y(2 x) = 2 y(x) exactly in any summation order, so every bit repeats
    rng = np.random.default_rng(33)
    f0 = rng.standard_normal((64, 256)).astype(np.float32)
    f0 = bf16_bits_to_f32(f32_to_bf16_bits(f0))
    x = np.concatenate([f0, 2 * f0, 4 * f0])
    s = Segment(0, VIDEO, 3, 64, 256, "bf16", 0.5, f32_to_bf16_bits(x))
    h = [dict(planes=simhash_planes(64, 256, seed=5), bits=64)]
    g, ref = run_case([s], 1, h, dev)
    assert np.all(g["d"][64:] == 0) and np.all(g["sim"][1:] == 1.0)
    compare([s], h, g, ref)


def test_rejects_bad_hashes(dev):
    w = make_workload(3, n_requests=1)
    dsegs = to_device(w.segments, dev)
    pl = torch.zeros((32, 1024), dtype=torch.bfloat16, device=dev)
    for bad, code in (([None], 1), ([dict(planes=pl, bits=24)], 1), ([dict(planes=pl.view(-1)[1:], bits=16)], 2)):
        with pytest.raises(B.MsaoError) as e:
            msao.msao_temporal_simhash(dsegs, 1, bad)
        assert e.value.status == code
