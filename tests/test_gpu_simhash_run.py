"""GPU parity of the whole analysis with SimHash as Eq. 5's hash
(msao_run_simhash) against the oracle (oracle.run with hashes), through the
fused clip pass (the default) and through the two-pass path.

Exact cases. Integer activations (|x| <= 3) and hyperplanes (entries -1, 0,
1) make every projection an integer of magnitude below 2^24, which the
matrix cores' fp32 accumulation reproduces whatever the order, zeros
included. Then every signature bit, d, D_t, sim, gamma, aggregate, the
temporal term, rho, MAS, keep count, kept index and compacted row equals the
oracle's bit for bit; beta within 1e-6 relative, informativeness within 1e-5
relative + 2e-6, l1, l2 and res within the other parity tests' bounds.

Gaussian cases (the video workload's statistics). A signature bit may differ
where the exact projection lies within the fp32 accumulation bound of 0 (the
borderline bits of the SimHash parity tests). d, D_t, sim, gamma, Dsum and the
temporal term are held to the slack those bits allow, MAS to beta lambda_t
times the temporal term's slack, and informativeness to lambda_t times the
token's d slack over K. The selection is checked for what is valid for the
GPU's own z and d: its keep count (from the fixed ratio, or from the GPU's
MAS), and the k smallest (key, index) pairs with key = L_s z K + L_t (K - d) C;
the compacted rows are the input rows at the kept indices, bitwise.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2604_02945_amd as msao
from test_gpu_parity import (compare_compaction, compare_frames, compare_requests, compare_scores, host, log,
                             to_device)
from test_gpu_simhash import borderline, dev_tensor
from workloads import AUDIO, IMAGE, TEXT, VIDEO, Segment, default_params, f32_to_bf16_bits, make_workload, \
    simhash_planes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def is_temporal(s):
    return s.modality == VIDEO and s.n_frames >= 2 and s.tokens_per_frame > 0


def encode(x, dtype):
    return np.ascontiguousarray(x) if dtype == "f32" else f32_to_bf16_bits(np.ascontiguousarray(x))


def int_rows(rng, n, C):
    x = rng.integers(-3, 4, size=(n, C)).astype(np.float32)
    x[rng.random((n, C)) < 0.5] = 0.0
    return x


def int_clip(rng, T, P, C):
    """Frames whose patches repeat (d = 0), change a few channels, or are new."""
    x = int_rows(rng, T * P, C)
    for t in range(1, T):
        kind = rng.integers(3, size=P)
        cur, prev = x[t * P:(t + 1) * P], x[(t - 1) * P:t * P]
        cur[kind == 0] = prev[kind == 0]
        few = np.flatnonzero(kind == 1)
        cur[few] = prev[few]
        for q in few:
            ch = rng.integers(C, size=max(1, C // 16))
            cur[q, ch] = rng.integers(-3, 4, size=ch.size)
    return x


def int_planes(rng, K, C, dtype):
    return encode(rng.integers(-1, 2, size=(K, C)).astype(np.float32), dtype)


def hashes_for(segments, planes_of):
    return [planes_of(i, s) if is_temporal(s) else None for i, s in enumerate(segments)]


def gpu_run(segments, R, params, hashes, dev, alpha=None, pad=0, compact=True, ctx=None):
    dsegs = to_device(segments, dev, pad)
    dh = [None if h is None else dict(planes=dev_tensor(h["planes"], s.dtype, dev), bits=h["bits"])
          for s, h in zip(segments, hashes)]
    out, sig = msao.msao_run_simhash(dsegs, R, dh, params, alpha, ctx=ctx, compact=compact)
    torch.cuda.synchronize()
    got = out.results(R, len(segments))
    got["sig"] = sig
    return dsegs, out, got


def exact_compare(segments, R, p, hashes, dev, alpha=None, pad=0, ctx=None):
    dsegs, out, got = gpu_run(segments, R, p, hashes, dev, alpha, pad, ctx=ctx)
    ref = oracle.run(segments, R, p, alpha, hashes=hashes)
    assert np.array_equal(host(got["sig"]).view(np.uint64), ref["sig"]), "sig"
    compare_scores(segments, R, got, ref)
    compare_frames(got, ref)
    compare_requests(got, ref)
    assert np.array_equal(host(got["kept_count"]), ref["k"]), "kept_count"
    assert np.array_equal(host(got["kept_idx"]), ref["kept_idx"]), "kept_idx"
    assert np.array_equal(host(got["keep"]), ref["keep"]), "keep"
    compare_compaction(dsegs, segments, out, ref["compact"], ref["k"])
    return got, ref


def mixed_int_table(seed, K, dtype):
    rng = np.random.default_rng(seed)
    C = 200
    segs = [Segment(0, VIDEO, 5, 37, C, dtype, 0.4, encode(int_clip(rng, 5, 37, C), dtype)),
            Segment(0, IMAGE, 1, 50, C, dtype, 0.25, encode(int_rows(rng, 50, C), dtype)),
            Segment(0, TEXT, 1, 9, C, dtype, 1.0, encode(int_rows(rng, 9, C), dtype)),
            Segment(1, VIDEO, 3, 64, C, dtype, -1.0, encode(int_clip(rng, 3, 64, C), dtype)),
            Segment(1, VIDEO, 1, 20, C, dtype, 0.5, encode(int_rows(rng, 20, C), dtype)),
            Segment(1, AUDIO, 1, 33, C, dtype, 0.5, encode(int_rows(rng, 33, C), dtype)),
            Segment(1, VIDEO, 2, 130, C, dtype, 0.3, encode(int_clip(rng, 2, 130, C), dtype))]
    hashes = hashes_for(segs, lambda i, s: dict(planes=int_planes(rng, K, C, dtype), bits=K))
    return segs, hashes


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("flags", [0, 1, 2])
@pytest.mark.parametrize("K", [16, 32, 48, 64])
def test_exact_mixed_table(K, flags, dtype, dev):
    segs, hashes = mixed_int_table(K * 10 + flags, K, dtype)
    p = default_params()
    p["flags"] = flags
    log(f"[simhash-run] exact mixed table K {K} flags {flags} {dtype}")
    got, ref = exact_compare(segs, 2, p, hashes, dev, alpha=[0.3, -0.2, 0.5, 0.0, 0.1, 0.0, 0.4, -0.3])
    agg = ref["agg"].reshape(-1, 4)
    assert agg[1 * 4 + VIDEO, 3] == (2 * 64 + 1 * 130) * K   # Qbits in K-bit units


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_exact_negative_zero_threshold(dtype, dev):
    """tau = -0 is the threshold 0: half of every integer row is exact zeros
    (inactive), the rest active, in the fused clip pass as in the rest."""
    segs, hashes = mixed_int_table(77, 32, dtype)
    p = default_params()
    p["tau"] = -0.0
    log(f"[simhash-run] exact mixed table with tau -0 {dtype}")
    got, ref = exact_compare(segs, 2, p, hashes, dev)
    z0 = oracle.run(segs, 2, dict(p, tau=0.0), hashes=hashes)["z"]
    assert np.array_equal(ref["z"], z0)


@pytest.mark.parametrize("K", [16, 64])
def test_exact_unfused_path(K, dev, monkeypatch):
    # MSAO_CLIP_FUSE=0: the clips are scored by k_score and hashed by k_simhash
    # (two passes over their rows), the path taken when a clip's 16-frame tiles
    # do not fit a 32-bit buffer resource
    monkeypatch.setenv("MSAO_CLIP_FUSE", "0")
    ctx = msao.Context(0)
    try:
        for flags in (0, 2):
            segs, hashes = mixed_int_table(500 + K + flags, K, "bf16")
            p = default_params()
            p["flags"] = flags
            log(f"[simhash-run] unfused path K {K} flags {flags}")
            exact_compare(segs, 2, p, hashes, dev, ctx=ctx)
    finally:
        ctx.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_exact_tile_boundaries(dtype, dev):
    # clips whose frame counts sit at the fused pass's tile boundaries (tiles
    # of at most 15 new frames, split evenly: 15 = one tile, 16 = 8 + 8,
    # 17 = 9 + 8, 30 = 15 + 15, 31 = 11 + 10 + 10), positions not a multiple
    # of the tiles per block, one signature width (the fused path)
    rng = np.random.default_rng(77)
    C, K = 136 if dtype == "f32" else 144, 48
    segs = []
    for r, (T, P) in enumerate([(15, 9), (16, 5), (17, 3), (30, 7), (31, 2), (2, 11)]):
        segs.append(Segment(r % 3, VIDEO, T, P, C, dtype, [0.3, -1.0, 0.5][r % 3],
                            encode(int_clip(rng, T, P, C), dtype)))
    hashes = hashes_for(segs, lambda i, s: dict(planes=int_planes(rng, K, C, dtype), bits=K))
    for flags in (0, 2):
        p = default_params()
        p["flags"] = flags
        log(f"[simhash-run] tile boundaries {dtype} flags {flags}")
        exact_compare(segs, 3, p, hashes, dev)


def test_exact_every_tile_height(dev):
    # clips of 2..17 frames: a tile holds r = 3..16 rows (its new frames and
    # their predecessor), and the statistics give each 16-lane group
    # ceil(r / 4) consecutive rows, so every group height (1..4) and every
    # split of the rows over the groups occurs; both element types, every
    # signature width
    for T in range(2, 18):
        rng = np.random.default_rng(300 + T)
        dtype = "bf16" if T % 2 == 0 else "f32"
        K = [16, 32, 48, 64][T % 4]
        C = [8, 40, 200, 72][T % 4]
        P = 1 + T % 7
        segs = [Segment(0, VIDEO, T, P, C, dtype, 0.4, encode(int_clip(rng, T, P, C), dtype)),
                Segment(1, VIDEO, T, 5, C, dtype, -1.0, encode(int_clip(rng, T, 5, C), dtype))]
        hashes = hashes_for(segs, lambda i, s: dict(planes=int_planes(rng, K, C, dtype), bits=K))
        p = default_params()
        p["flags"] = T % 3
        log(f"[simhash-run] tile height T {T} {dtype} K {K} C {C}")
        exact_compare(segs, 2, p, hashes, dev)


def test_exact_padded_rows_and_weights(dev):
    rng = np.random.default_rng(5)
    C = 264
    segs = [Segment(0, VIDEO, 4, 45, C, "bf16", 0.35, encode(int_clip(rng, 4, 45, C), "bf16")),
            Segment(0, IMAGE, 1, 40, C, "bf16", -1.0, encode(int_rows(rng, 40, C), "bf16"))]
    hashes = hashes_for(segs, lambda i, s: dict(planes=int_planes(rng, 48, C, "bf16"), bits=48))
    p = default_params()
    p["lambda_s"] = [0.0, 0.6, 0.3, 0.6]
    p["lambda_t"] = [0.0, 0.0, 0.7, 0.0]
    log("[simhash-run] exact padded rows")
    exact_compare(segs, 1, p, hashes, dev, pad=24)
    p["lambda_s"] = [0.0, 0.6, 0.0, 0.6]   # temporal term alone orders the clip
    exact_compare(segs, 1, p, hashes, dev, pad=24)


@pytest.mark.parametrize("flags", [0, 2])
def test_exact_clip_beyond_lds_staging(flags, dev):
    # 72 x 256 = 18,432 tokens: the selection re-reads z and d instead of staging keys
    rng = np.random.default_rng(9)
    C = 256
    segs = [Segment(0, VIDEO, 72, 256, C, "bf16", 0.3, encode(int_clip(rng, 72, 256, C), "bf16"))]
    hashes = [dict(planes=int_planes(rng, 32, C, "bf16"), bits=32)]
    p = default_params()
    p["flags"] = flags
    log(f"[simhash-run] exact clip of 18432 tokens, flags {flags}")
    exact_compare(segs, 1, p, hashes, dev)


def test_without_clips_equals_msao_run(dev):
    rng = np.random.default_rng(3)
    segs = [Segment(0, IMAGE, 1, 70, 128, "bf16", 0.5, encode(rng.standard_normal((70, 128)).astype(np.float32),
                                                              "bf16")),
            Segment(0, VIDEO, 1, 30, 128, "f32", -1.0, rng.standard_normal((30, 128)).astype(np.float32))]
    p = default_params()
    dsegs = to_device(segs, dev)
    a = msao.msao_run(dsegs, 1, p).results(1, 2)
    out, sig = msao.msao_run_simhash(dsegs, 1, [None, None], p)
    b = out.results(1, 2)
    torch.cuda.synchronize()
    assert sig.numel() == 100 and int(torch.count_nonzero(sig)) == 0   # signatures written, all zero
    for k in ("z", "l1", "l2", "info", "d", "res", "agg", "rho", "temporal", "beta", "mas", "present", "keep",
              "kept_idx", "kept_count"):
        assert torch.equal(a[k], b[k]), k


# ------------------------------------------------------------ Gaussian inputs

def valid_selection(segments, R, p, got, hashes):
    z = host(got["z"]).astype(np.int64)
    d = host(got["d"]).astype(np.int64)
    kc = host(got["kept_count"])
    kept = host(got["kept_idx"])
    keep = host(got["keep"])
    mas = host(got["mas"])
    per_frame = p.get("flags", 0) & oracle.FLAG_SELECT_PER_FRAME
    off = 0
    for i, s in enumerate(segments):
        N, C = s.n_tokens, s.hidden
        kappa = float(np.float32(s.keep_ratio)) if s.keep_ratio >= 0 else 1.0 - float(mas[s.request * 4 + s.modality])
        framed = per_frame and s.n_frames >= 2 and s.tokens_per_frame > 0
        units = [(t * s.tokens_per_frame, s.tokens_per_frame) for t in range(s.n_frames)] if framed else [(0, N)]
        kk = [oracle.keep_count(kappa, n) for _, n in units]
        assert kc[i] == sum(kk), f"keep count of segment {i}"
        Ls = int(oracle.q24(p["lambda_s"][s.modality]))
        Lt = int(oracle.q24(p["lambda_t"][s.modality]))
        if is_temporal(s):
            K = hashes[i]["bits"]
            key = Ls * z[off:off + N] * K + Lt * (K - d[off:off + N]) * C
        else:
            key = Ls * z[off:off + N]
        want = []
        for (a, n), k in zip(units, kk):
            order = sorted(range(a, a + n), key=lambda j: (int(key[j]), j))
            want.extend(order[:k])
        want = sorted(want)
        assert kept[off:off + kc[i]].tolist() == want, f"kept indices of segment {i}"
        assert np.all(kept[off + kc[i]:off + N] == -1)
        flags = np.zeros(N, np.uint8)
        flags[want] = 1
        assert np.array_equal(keep[off:off + N], flags)
        off += N


def gaussian_compare(segments, R, p, hashes, dev, pad=0):
    dsegs, out, got = gpu_run(segments, R, p, hashes, dev, pad=pad)
    ref = oracle.run(segments, R, p, hashes=hashes, compact=False)
    compare_scores(segments, R, got, ref, check_tokens=("z", "l1", "l2", "res"))
    nb = borderline(segments, hashes)
    sig_g = host(got["sig"]).view(np.uint64)
    diff = np.array([bin(int(v)).count("1") for v in (sig_g ^ ref["sig"])], np.int64)
    assert np.all(diff <= nb), "signature bits differ beyond the borderline ones"
    slack = np.zeros_like(nb)
    frame_slack, frame_bits, tslack, tbits = [], [], {}, {}
    info_tol = np.zeros(len(nb))
    off = 0
    for si, s in enumerate(segments):
        N = s.n_tokens
        if is_temporal(s):
            P, T, K = s.tokens_per_frame, s.n_frames, hashes[si]["bits"]
            ss = nb[off:off + N].copy()
            ss[P:] += nb[off:off + N - P]
            slack[off:off + N] = ss
            frame_slack.append(ss.reshape(T, P).sum(axis=1))
            frame_bits.append(np.full(T, P * K))
            x = s.request * 4 + s.modality
            tslack[x] = tslack.get(x, 0) + int(ss[P:].sum())
            tbits[x] = tbits.get(x, 0) + (T - 1) * P * K
            info_tol[off:off + N] = p["lambda_t"][s.modality] * ss / K
        off += N
    g_d = host(got["d"]).astype(np.int64)
    assert np.all(np.abs(g_d - ref["d"].astype(np.int64)) <= slack), "d"
    fs = np.concatenate(frame_slack) if frame_slack else np.zeros(0, np.int64)
    fb = np.concatenate(frame_bits) if frame_bits else np.ones(0)
    g_D = host(got["dframe"]).astype(np.int64)
    assert np.all(np.abs(g_D - ref["dframe"].astype(np.int64)) <= fs), "D_t"
    for f in ("sim", "gamma"):
        assert np.all(np.abs(host(got[f]).astype(np.float64) - ref[f]) <= fs / fb + 2.0 ** -24), f
    g_info, w_info = host(got["info"]).astype(np.float64), ref["info"].astype(np.float64)
    assert np.all(np.abs(g_info - w_info) <= 1e-5 * np.abs(w_info) + 2e-6 + info_tol), "info"
    g_agg = host(got["agg"]).astype(np.int64).reshape(-1, 4)
    r_agg = ref["agg"].astype(np.int64).reshape(-1, 4)
    assert np.array_equal(g_agg[:, [0, 1, 3]], r_agg[:, [0, 1, 3]]), "Ntok, Nsparse, Qbits"
    assert np.array_equal(host(got["rho"]), ref["rho"]), "rho"
    assert np.array_equal(host(got["present"]), ref["present"]), "present"
    assert np.allclose(host(got["beta"]), ref["beta"], rtol=1e-6, atol=0), "beta"
    g_t, g_mas = host(got["temporal"]), host(got["mas"])
    for x in range(len(ref["temporal"])):
        ts = tslack.get(x, 0)
        assert abs(int(g_agg[x, 2]) - int(r_agg[x, 2])) <= ts, f"Dsum[{x}]"
        tt = ts / tbits[x] + 2.0 ** -24 if x in tbits else 0.0
        assert abs(float(g_t[x]) - float(ref["temporal"][x])) <= tt, f"temporal[{x}]"
        mt = float(ref["beta"][x]) * p["lambda_t"][x % 4] * tt + 1e-6 * abs(float(ref["mas"][x])) + 1e-7
        assert abs(float(g_mas[x]) - float(ref["mas"][x])) <= mt, f"mas[{x}]"
    valid_selection(segments, R, p, got, hashes)
    rows = msao.compacted_rows(dsegs, out, host(got["kept_count"]))
    kept, kc = host(got["kept_idx"]), host(got["kept_count"])
    off = 0
    for i, (s, r) in enumerate(zip(segments, rows)):
        want = np.ascontiguousarray(s.data[kept[off:off + kc[i]], :s.hidden])
        g = host(r.view(torch.int16) if r.dtype == torch.bfloat16 else r)
        assert np.array_equal(g.view(np.uint8), want.view(np.uint8)), f"compacted rows of segment {i}"
        off += s.n_tokens
    if nb.sum() == 0:
        assert np.array_equal(host(got["kept_idx"]), ref["kept_idx"])
    return int(nb.sum())


@pytest.mark.parametrize("flags", [0, 2])
@pytest.mark.parametrize("K", [16, 32, 64])
def test_gaussian_mixed_table(K, flags, dev):
    rng = np.random.default_rng(40 + K + flags)
    segs = []
    for r, (T, P, C, dtype, keep) in enumerate([(6, 48, 256, "bf16", 0.3), (4, 70, 136, "f32", -1.0),
                                                (3, 100, 512, "bf16", 0.5)]):
        x = rng.standard_normal((T * P, C)).astype(np.float32)
        for t in range(1, T):   # 70 % of the patches drift slowly
            st = rng.random(P) < 0.7
            x[t * P:(t + 1) * P][st] = x[(t - 1) * P:t * P][st] + 0.02 * rng.standard_normal((st.sum(), C))
        segs.append(Segment(r % 2, VIDEO, T, P, C, dtype, keep, encode(x, dtype)))
    segs.append(Segment(0, IMAGE, 1, 90, 256, "bf16", 0.25,
                        encode(np.maximum(rng.standard_normal((90, 256)), 0).astype(np.float32), "bf16")))
    hashes = hashes_for(segs, lambda i, s: dict(planes=simhash_planes(K, s.hidden, seed=i, dtype=s.dtype), bits=K))
    p = default_params()
    p["flags"] = flags
    nb = gaussian_compare(segs, 2, p, hashes, dev)
    log(f"[simhash-run] gaussian K {K} flags {flags}: {nb} borderline bits")


def test_video_workload_full_size(dev):
    w = make_workload(3)
    hashes = [dict(planes=simhash_planes(32, s.hidden, seed=100 + i, dtype=s.dtype), bits=32)
              for i, s in enumerate(w.segments)]
    log("[simhash-run] video workload, 8 clips x 32 x 256 x 1024 bf16, K 32")
    nb = gaussian_compare(w.segments, w.n_requests, w.params, hashes, dev)
    log(f"[simhash-run] full size: {nb} borderline bits")


def test_errors_write_nothing(dev):
    rng = np.random.default_rng(1)
    C = 64
    segs = [Segment(0, VIDEO, 3, 16, C, "f32", 0.5, rng.standard_normal((48, C)).astype(np.float32))]
    dsegs = to_device(segs, dev)
    out = msao.Outputs(dsegs, 1)
    out.sel["kept_count"].fill_(-7)
    with pytest.raises(msao.MsaoError, match="hash of segment 0"):
        msao.msao_run_simhash(dsegs, 1, [None], outputs=out)
    planes = torch.zeros((24, C), dtype=torch.float32, device=dev)
    with pytest.raises(msao.MsaoError, match="bits must be"):
        msao.msao_run_simhash(dsegs, 1, [dict(planes=planes, bits=24)], outputs=out)
    torch.cuda.synchronize()
    assert int(out.sel["kept_count"][0]) == -7


def test_prepared_calls_match_one_shot(dev):
    """prepare_simhash marshals msao_run_simhash / msao_temporal_simhash once:
    two calls of each give the one-shot calls' outputs byte for byte."""
    segs, hashes = mixed_int_table(77, 32, "bf16")
    R, p = 2, default_params()
    dsegs = to_device(segs, dev)
    dh = [None if h is None else dict(planes=dev_tensor(h["planes"], s.dtype, dev), bits=h["bits"])
          for s, h in zip(segs, hashes)]
    ntok = sum(s.n_tokens for s in segs)
    log("[simhash-run] prepared calls, twice each")
    one, sig1 = msao.msao_run_simhash(dsegs, R, dh, p)
    t_one, tsig1 = msao.msao_temporal_simhash(dsegs, R, dh, p)
    o_run = msao.Outputs(dsegs, R)
    o_tmp = msao.Outputs(dsegs, R, compact=False)
    sig2 = torch.empty(ntok, dtype=torch.int64, device=dev)
    tsig2 = torch.empty(ntok, dtype=torch.int64, device=dev)
    run = msao.binding.prepare_simhash("msao_run_simhash", dsegs, R, dh, o_run, sig2, p)
    tmp = msao.binding.prepare_simhash("msao_temporal_simhash", dsegs, R, dh, o_tmp, tsig2, p)
    for _ in range(2):
        run()
        tmp()
        torch.cuda.synchronize()
        a, b = one.results(R, len(segs)), o_run.results(R, len(segs))
        for k in a:
            assert torch.equal(a[k].view(torch.uint8), b[k].view(torch.uint8)), k
        assert torch.equal(sig1, sig2)
        ra = msao.compacted_rows(dsegs, one, host(a["kept_count"]))
        rb = msao.compacted_rows(dsegs, o_run, host(b["kept_count"]))
        for x, y in zip(ra, rb):
            assert torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))
        assert torch.equal(tsig1, tsig2)
        assert torch.equal(t_one.tok["d"], o_tmp.tok["d"])
        assert torch.equal(t_one.req["temporal"], o_tmp.req["temporal"])
        for k in ("dframe", "sim", "gamma"):
            assert torch.equal(t_one.frm[k], o_tmp.frm[k]), k
