"""The whole hot path from C on the GPU: tests/c/abi_gpu_run (built by the
package's build step with gcc against include/msao.h, the HIP C API and
libmsao.so; no Python or framework in the process) runs msao_run on inputs
written here and dumps its outputs, which are compared with the oracle on
the same inputs: z, d, per-frame D_t, sim, aggregates, keep flags, kept
indices, keep counts and compacted rows bit-exact, MAS within 1e-6."""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from workloads import Segment, make_workload

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "c", "abi_gpu_run")


def run_client(segs, R, flags, tmp_path):
    if not os.path.exists(CLIENT):
        pytest.fail("tests/c/abi_gpu_run is not built (run the build step first)")
    ind, outd = tmp_path / "in", tmp_path / "out"
    ind.mkdir()
    outd.mkdir()
    with open(ind / "segments.txt", "w") as f:
        f.write(f"{len(segs)} {R} {flags}\n")
        for i, s in enumerate(segs):
            np.ascontiguousarray(s.data).tofile(ind / f"seg{i}.bin")
            f.write(f"{s.request} {s.modality} {s.n_frames} {s.tokens_per_frame} {s.hidden} "
                    f"{0 if s.dtype == 'f32' else 1} {float(np.float32(s.keep_ratio))!r} seg{i}.bin\n")
    print(f"[c-client] {len(segs)} segments, flags {flags}", flush=True)
    sys.stdout.flush()
    r = subprocess.run([CLIENT, str(ind), str(outd)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    return lambda name, dt: np.fromfile(outd / name, dt)


def compare(segs, R, flags, tmp_path):
    got = run_client(segs, R, flags, tmp_path)
    p = make_workload(1).params
    p["flags"] = flags
    ref = oracle.run(segs, R, p)
    assert np.array_equal(got("z.bin", np.uint32), ref["z"])
    assert np.array_equal(got("d.bin", np.uint32), ref["d"])
    assert np.array_equal(got("dframe.bin", np.uint64), ref["dframe"])
    assert np.array_equal(got("sim.bin", np.float32), ref["sim"])
    assert np.array_equal(got("agg.bin", np.uint64), ref["agg"])
    np.testing.assert_allclose(got("mas.bin", np.float32), ref["mas"], rtol=1e-6, atol=1e-7)
    kc = got("kept_count.bin", np.int32)
    assert np.array_equal(kc, ref["k"])
    assert np.array_equal(got("kept_idx.bin", np.int32), ref["kept_idx"])
    assert np.array_equal(got("keep.bin", np.uint8), ref["keep"])
    out = got("out.bin", np.uint8)
    offs = got("offsets.bin", np.int64)
    for i, (s, want) in enumerate(zip(segs, oracle.compact_rows(segs, ref["k"], ref["kept_idx"]))):
        w = np.ascontiguousarray(want).view(np.uint8).reshape(-1)
        assert np.array_equal(out[offs[i]:offs[i] + w.size], w), f"compacted rows of segment {i}"


def test_c_client_trimodal(tmp_path):
    w = make_workload(4, n_requests=2)
    compare(w.segments, 2, 0, tmp_path)


def test_c_client_fp32_image_and_text(tmp_path):
    w = make_workload(1)
    compare(w.segments, 1, 0, tmp_path)


def test_c_client_video_per_frame_scope(tmp_path):
    w = make_workload(3, n_requests=1)
    compare(w.segments, 1, oracle.FLAG_SELECT_PER_FRAME, tmp_path)
