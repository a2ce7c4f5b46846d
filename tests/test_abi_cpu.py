"""The C ABI on the CPU: library loads, exports every declared symbol, and
rejects invalid calls with specific status codes before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2604_02945_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, ALIGN, WS, UNSUP, HIP = range(6)


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "msao.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(msao_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    L = B.lib()
    names = _declared_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(L, name), name
    assert {n for n, _, _ in B.SIGNATURES} == set(names)


def test_struct_layouts_match_header():
    assert ctypes.sizeof(B.MsaoSegment) == 48
    assert ctypes.sizeof(B.MsaoParams) == 44
    assert ctypes.sizeof(B.MsaoTokenOut) == 48
    assert ctypes.sizeof(B.MsaoSpatialHead) == 24
    assert ctypes.sizeof(B.MsaoModalMlp) == 48


def test_default_params_are_the_papers():
    p = B.default_params()
    assert p["tau_s"] == pytest.approx(0.3) and p["tau"] == pytest.approx(0.1)
    assert p["lambda_s"] == pytest.approx([0, 0.6, 0.6, 0.6]) and p["lambda_t"] == pytest.approx([0, 0, 0.4, 0])
    assert p["flags"] == 0


def test_status_strings():
    L = B.lib()
    assert L.msao_status_string(0) == b"MSAO_OK" and L.msao_status_string(5) == b"MSAO_ERR_HIP"


FAKE = 0x10000  # a 16-byte aligned address; validation never dereferences data


def seg(**kw):
    s = B.MsaoSegment()
    s.data = kw.get("data", FAKE)
    s.row_stride = kw.get("row_stride", 1024)
    s.request = kw.get("request", 0)
    s.modality = kw.get("modality", B.IMAGE)
    s.n_frames = kw.get("n_frames", 1)
    s.tokens_per_frame = kw.get("tokens_per_frame", 576)
    s.hidden = kw.get("hidden", 1024)
    s.dtype = kw.get("dtype", B.BF16)
    s.keep_ratio = kw.get("keep_ratio", 0.25)
    return s


def validate(segs, R=1, params=None):
    arr = (B.MsaoSegment * max(1, len(segs)))(*segs)
    p = params or B.lib().msao_default_params()
    return B.lib().msao_validate(arr, len(segs), R, ctypes.byref(p))


def test_valid_table():
    assert validate([seg(), seg(modality=B.VIDEO, n_frames=32, tokens_per_frame=256),
                     seg(modality=B.TEXT, hidden=4096, row_stride=4096, keep_ratio=1.0),
                     seg(dtype=B.F32, keep_ratio=-1.0), seg(tokens_per_frame=0, data=0)]) == OK


@pytest.mark.parametrize("kw,code", [
    (dict(modality=4), INVALID), (dict(modality=-1), INVALID), (dict(dtype=2), INVALID),
    (dict(request=1), INVALID), (dict(request=-1), INVALID), (dict(n_frames=0), INVALID),
    (dict(n_frames=2), INVALID),                       # frames on a non-video segment
    (dict(tokens_per_frame=-1), INVALID), (dict(hidden=0), INVALID), (dict(hidden=70000, row_stride=70000), INVALID),
    (dict(hidden=1020, row_stride=1024), ALIGN),        # bf16 rows must be whole 16-byte chunks
    (dict(hidden=1022, row_stride=1024, dtype=B.F32), ALIGN),
    (dict(keep_ratio=float("nan")), INVALID), (dict(keep_ratio=1.5), INVALID),
    (dict(data=0), INVALID), (dict(row_stride=1000), INVALID),
    (dict(data=FAKE + 8), ALIGN), (dict(row_stride=1028), ALIGN),
    (dict(modality=B.VIDEO, n_frames=1 << 16, tokens_per_frame=1 << 16), UNSUP),
])
def test_invalid_segments(kw, code):
    assert validate([seg(**kw)]) == code
    assert B.lib().msao_last_error_global()  # a message is recorded


@pytest.mark.parametrize("field,value", [("tau", -0.1), ("tau", float("nan")), ("tau", float("inf")),
                                         ("tau_s", 1.5), ("tau_s", -0.01), ("flags", 6)])
def test_invalid_params(field, value):
    p = B.lib().msao_default_params()
    setattr(p, field, value)
    assert validate([seg()], params=p) == INVALID


def test_invalid_lambda_and_counts():
    p = B.lib().msao_default_params()
    p.lambda_t[2] = 1.25
    assert validate([seg()], params=p) == INVALID
    L = B.lib()
    assert L.msao_validate(None, 1, 1, ctypes.byref(L.msao_default_params())) == INVALID
    arr = (B.MsaoSegment * 1)(seg())
    assert L.msao_validate(arr, -1, 1, ctypes.byref(L.msao_default_params())) == INVALID
    assert L.msao_validate(arr, 1, 1, None) == INVALID


def test_sizes_and_layout():
    L = B.lib()
    segs = [seg(), seg(modality=B.VIDEO, n_frames=4, tokens_per_frame=10),
            seg(modality=B.TEXT, keep_ratio=-1.0, tokens_per_frame=7)]
    arr = (B.MsaoSegment * 3)(*segs)
    nt, nf = ctypes.c_int64(), ctypes.c_int64()
    assert L.msao_count(arr, 3, ctypes.byref(nt), ctypes.byref(nf)) == OK
    assert (nt.value, nf.value) == (576 + 40 + 7, 4)
    ws = ctypes.c_size_t()
    assert L.msao_workspace_size(arr, 3, 1, ctypes.byref(ws)) == OK
    assert ws.value >= 16 * (576 + 40 + 7) and ws.value % 16 == 0
    off = (ctypes.c_int64 * 3)()
    total = ctypes.c_int64()
    assert L.msao_compact_layout(arr, 3, off, ctypes.byref(total)) == OK
    # image: ceil(0.25*576) = 144 rows; video: max(ceil(0.25*40), 4*ceil(0.25*10)) = 12 rows (room for
    # the per-frame scope); guided text: all 7 rows
    assert off[0] == 0 and off[1] == 144 * 2048 and off[2] == 144 * 2048 + 12 * 2048
    assert total.value == off[2] + 7 * 2048 + (256 - (7 * 2048) % 256) % 256
    assert all(o % 256 == 0 for o in off)


def test_entry_points_reject_null_context():
    L = B.lib()
    arr = (B.MsaoSegment * 1)(seg())
    p = L.msao_default_params()
    assert L.msao_mas_score(None, arr, 1, 1, ctypes.byref(p), None, None, None, None, None, 0, None) == INVALID
    assert L.msao_run(None, arr, 1, 1, ctypes.byref(p), None, None, None, None, None, None, None, 0, None, 0,
                      None) == INVALID
    assert L.msao_select_tokens(None, arr, 1, 1, ctypes.byref(p), None, None, None, None, None, 0, None) == INVALID


# entry points whose first argument is the context (or the plan): every one
# rejects a NULL one before touching any other argument
CTX_ENTRY_POINTS = ["msao_mas_score", "msao_temporal_redundancy", "msao_select_tokens", "msao_compact", "msao_run",
                    "msao_run_noalloc", "msao_plan_create", "msao_plan_run", "msao_mas_score_learned",
                    "msao_run_learned", "msao_temporal_simhash", "msao_run_simhash", "msao_draft_entropy",
                    "msao_stream_read", "msao_set_profiling", "msao_kernel_times"]


@pytest.mark.parametrize("name", CTX_ENTRY_POINTS)
def test_every_entry_point_rejects_a_null_context(name):
    L = B.lib()
    fn = getattr(L, name)
    args = []
    for t in fn.argtypes:
        if t in (ctypes.c_int, ctypes.c_int64, ctypes.c_size_t):
            args.append(0)
        elif t in (ctypes.c_float, ctypes.c_double):
            args.append(0.0)
        else:
            args.append(None)
    assert fn(*args) == INVALID


def test_create_without_device_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    h = ctypes.c_void_p()
    assert B.lib().msao_create(ctypes.byref(h), 0) == HIP
    assert h.value is None


def test_product_package_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2604_02945_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "libmsao_oracle" not in text and "msao_oracle" not in text, f
