"""Thin ctypes binding of libmsao.so (the C ABI in include/msao.h).

Argument marshalling only: torch provides device memory and the current
stream; every step of the analysis runs in the library's HIP kernels. The
library must be built in-tree (paper_2604_02945_amd/build.py); importing this
module never falls back to anything else.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, List, Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmsao.so")

NMOD = 4
TEXT, IMAGE, VIDEO, AUDIO = 0, 1, 2, 3
F32, BF16 = 0, 1
FLAG_TEMPORAL_LITERAL = 1
FLAG_SELECT_PER_FRAME = 2
(KERNEL_SCORE, KERNEL_POST, KERNEL_GATHER, KERNEL_ENTROPY, KERNEL_HEAD, KERNEL_SIMHASH, KERNEL_HASH_POST,
 KERNEL_CLIP, KERNEL_READ, NUM_KERNELS) = 0, 1, 2, 3, 4, 5, 6, 7, 8, 9
MODAL_DESC = 8
DECIDE_HOLD, DECIDE_SEND, DECIDE_OFFLOAD = 0, 1, 2

STATUS = {0: "MSAO_OK", 1: "MSAO_ERR_INVALID_ARG", 2: "MSAO_ERR_ALIGNMENT", 3: "MSAO_ERR_WORKSPACE",
          4: "MSAO_ERR_UNSUPPORTED", 5: "MSAO_ERR_HIP"}

_P = ctypes.c_void_p


class MsaoSegment(ctypes.Structure):
    _fields_ = [("data", _P), ("row_stride", ctypes.c_int64), ("request", ctypes.c_int32),
                ("modality", ctypes.c_int32), ("n_frames", ctypes.c_int32),
                ("tokens_per_frame", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("keep_ratio", ctypes.c_float)]


class MsaoParams(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("tau_s", ctypes.c_float),
                ("lambda_s", ctypes.c_float * NMOD), ("lambda_t", ctypes.c_float * NMOD),
                ("flags", ctypes.c_uint32)]


class MsaoTokenOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("z", "l1", "l2", "info", "d", "res")]


class MsaoFrameOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("dframe", "sim", "gamma")]


class MsaoReqOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("agg", "rho", "temporal", "beta", "mas", "present")]


class MsaoSelectOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("keep", "kept_idx", "kept_count")]


class MsaoSpatialHead(ctypes.Structure):
    _fields_ = [("weight", _P), ("bias", ctypes.c_float), ("grid_w", ctypes.c_int32), ("pool", ctypes.c_int32)]


class MsaoModalMlp(ctypes.Structure):
    _fields_ = [("w1", _P), ("b1", _P), ("w2", _P), ("b2", ctypes.c_float), ("hidden", ctypes.c_int32),
                ("prompt_dim", ctypes.c_int32), ("prompt", _P)]


class MsaoSimHash(ctypes.Structure):
    _fields_ = [("planes", _P), ("bits", ctypes.c_int32)]


class MsaoEntropyOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("entropy", "entropy_norm", "draft_token", "speculate")]


class MsaoSchedParams(ctypes.Structure):
    _fields_ = [("p_target", ctypes.c_double), ("n_max", ctypes.c_int32), ("quantile", ctypes.c_double),
                ("delta", ctypes.c_double), ("theta_min", ctypes.c_double), ("alpha", ctypes.c_double)]


class MsaoSchedState(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("p_conf", ctypes.c_double), ("n_draft", ctypes.c_int32),
                ("cache", ctypes.c_int32), ("cache_h", ctypes.c_double), ("steps", ctypes.c_int64),
                ("held", ctypes.c_int64), ("sends", ctypes.c_int64), ("offloads", ctypes.c_int64),
                ("tokens_sent", ctypes.c_int64)]


class MsaoLatencyModel(ctypes.Structure):
    _fields_ = [("prefill_edge", ctypes.c_double), ("prefill_cloud", ctypes.c_double),
                ("comm_offloaded", ctypes.c_double), ("p_conf", ctypes.c_double), ("n_draft", ctypes.c_int32),
                ("t_draft", ctypes.c_double), ("t_verify", ctypes.c_double), ("t_offload", ctypes.c_double)]


class MsaoError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None

# (name, restype, argtypes) of every entry point in include/msao.h
SIGNATURES = [
    ("msao_create", ctypes.c_int, [ctypes.POINTER(_P), ctypes.c_int]),
    ("msao_destroy", None, [_P]),
    ("msao_last_error", ctypes.c_char_p, [_P]),
    ("msao_last_error_global", ctypes.c_char_p, []),
    ("msao_status_string", ctypes.c_char_p, [ctypes.c_int]),
    ("msao_default_params", MsaoParams, []),
    ("msao_validate", ctypes.c_int, [_P, ctypes.c_int, ctypes.c_int, _P]),
    ("msao_count", ctypes.c_int, [_P, ctypes.c_int, _P, _P]),
    ("msao_workspace_size", ctypes.c_int, [_P, ctypes.c_int, ctypes.c_int, _P]),
    ("msao_compact_layout", ctypes.c_int, [_P, ctypes.c_int, _P, _P]),
    ("msao_mas_score", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                      ctypes.c_size_t, _P]),
    ("msao_temporal_redundancy", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                                ctypes.c_size_t, _P]),
    ("msao_select_tokens", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                          ctypes.c_size_t, _P]),
    ("msao_compact", ctypes.c_int, [_P, _P, ctypes.c_int, _P, _P, _P, _P, ctypes.c_int64, _P,
                                    ctypes.c_size_t, _P]),
    ("msao_run", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P,
                                ctypes.c_int64, _P, ctypes.c_size_t, _P]),
    ("msao_run_noalloc", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P,
                                        ctypes.c_int64, _P]),
    ("msao_plan_create", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, ctypes.c_size_t, _P,
                                        ctypes.POINTER(_P)]),
    ("msao_plan_run", ctypes.c_int, [_P, _P, _P, _P, _P, _P, ctypes.c_int64, _P]),
    ("msao_plan_destroy", None, [_P]),
    ("msao_set_profiling", ctypes.c_int, [_P, ctypes.c_int]),
    ("msao_kernel_times", ctypes.c_int, [_P, _P]),
    ("msao_mas_score_learned", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P,
                                              _P, _P, _P, ctypes.c_size_t, _P]),
    ("msao_run_learned", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                        _P, _P, _P, ctypes.c_int64, _P, ctypes.c_size_t, _P]),
    ("msao_temporal_simhash", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P,
                                             ctypes.c_size_t, _P]),
    ("msao_run_simhash", ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                        ctypes.c_int64, _P, ctypes.c_size_t, _P]),
    ("msao_draft_entropy", ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                          ctypes.c_float, _P, _P]),
    ("msao_stream_read", ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int, _P, ctypes.c_int64, _P]),
    ("msao_sched_default_params", MsaoSchedParams, []),
    ("msao_sched_init", ctypes.c_int, [_P, ctypes.c_int64, _P, _P]),
    ("msao_sched_step", ctypes.c_int, [_P, _P, ctypes.c_float, _P]),
    ("msao_sched_run", ctypes.c_int, [_P, _P, _P, ctypes.c_int64, _P, _P]),
    ("msao_retention_floor", ctypes.c_int, [_P, ctypes.c_int, _P]),
    ("msao_comm_latency", ctypes.c_double, [ctypes.c_double, ctypes.c_double, ctypes.c_double]),
    ("msao_p_conf", ctypes.c_double, [_P, ctypes.c_int64, ctypes.c_double]),
    ("msao_expected_spec_tokens", ctypes.c_double, [ctypes.c_double]),
    ("msao_expected_e2e_latency", ctypes.c_double, [_P]),
]


def lib() -> ctypes.CDLL:
    """Load the in-tree libmsao.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2604_02945_amd/build.py "
                               "(or __graft_entry__.build()); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _addr(struct) -> ctypes.c_void_p:
    return ctypes.cast(ctypes.byref(struct), ctypes.c_void_p)


def default_params() -> dict:
    p = lib().msao_default_params()
    return {"tau": p.tau, "tau_s": p.tau_s, "lambda_s": list(p.lambda_s), "lambda_t": list(p.lambda_t),
            "flags": p.flags}


def params_struct(p: Optional[dict]) -> MsaoParams:
    if p is None:
        return lib().msao_default_params()
    q = MsaoParams()
    q.tau, q.tau_s = p["tau"], p["tau_s"]
    for m in range(NMOD):
        q.lambda_s[m] = p["lambda_s"][m]
        q.lambda_t[m] = p["lambda_t"][m]
    q.flags = p.get("flags", 0)
    return q


@dataclasses.dataclass
class DeviceSegment:
    """A modality-tagged activation tensor on the device.

    `data` is [rows, hidden] (row stride may exceed hidden) with rows = n_frames
    * tokens_per_frame, float32 or bfloat16.
    """
    data: torch.Tensor
    request: int
    modality: int
    keep_ratio: float
    n_frames: int = 1

    @property
    def rows(self) -> int:
        return int(self.data.shape[0])


def segment_table(segments: Sequence[DeviceSegment]):
    arr = (MsaoSegment * max(1, len(segments)))()
    for i, s in enumerate(segments):
        t = s.data
        if t.dim() != 2:
            raise ValueError("segment data must be a 2-D [rows, hidden] tensor")
        if t.dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("segment data must be float32 or bfloat16")
        if t.numel() and t.stride(1) != 1:
            raise ValueError("rows must be contiguous")
        if s.rows % s.n_frames:
            raise ValueError("rows must be a multiple of n_frames")
        arr[i].data = t.data_ptr() if t.numel() else None
        arr[i].row_stride = t.stride(0) if t.shape[0] > 1 else t.shape[1]
        arr[i].request = s.request
        arr[i].modality = s.modality
        arr[i].n_frames = s.n_frames
        arr[i].tokens_per_frame = s.rows // s.n_frames
        arr[i].hidden = t.shape[1]
        arr[i].dtype = F32 if t.dtype == torch.float32 else BF16
        arr[i].keep_ratio = s.keep_ratio
    return arr


def _check(status: int, ctx: Optional["Context"] = None):
    if status != 0:
        msg = (lib().msao_last_error(ctx.handle) if ctx is not None else lib().msao_last_error_global()) or b""
        raise MsaoError(status, msg.decode())


class Context:
    """An msao_ctx bound to one device; one per concurrently used stream."""

    def __init__(self, device: int = 0):
        h = ctypes.c_void_p()
        _check(lib().msao_create(ctypes.byref(h), device))
        self.handle = h
        self.device = device

    def close(self):
        if getattr(self, "handle", None):
            lib().msao_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_profiling(self, enable: bool):
        _check(lib().msao_set_profiling(self.handle, 1 if enable else 0), self)

    def kernel_times(self) -> List[float]:
        ms = (ctypes.c_float * NUM_KERNELS)()
        _check(lib().msao_kernel_times(self.handle, ms), self)
        return list(ms)


_default_ctx: Dict[int, Context] = {}


def default_context(device: int) -> Context:
    if device not in _default_ctx:
        _default_ctx[device] = Context(device)
    return _default_ctx[device]


def sizes(segments: Sequence[DeviceSegment], n_requests: int):
    """(total tokens, total temporal frames, workspace bytes) of a segment table."""
    segt = segment_table(segments)
    nt, nf = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().msao_count(segt, len(segments), ctypes.byref(nt), ctypes.byref(nf)))
    ws = ctypes.c_size_t()
    _check(lib().msao_workspace_size(segt, len(segments), n_requests, ctypes.byref(ws)))
    return nt.value, nf.value, ws.value


def compact_layout(segments: Sequence[DeviceSegment]):
    segt = segment_table(segments)
    off = (ctypes.c_int64 * max(1, len(segments)))()
    total = ctypes.c_int64()
    _check(lib().msao_compact_layout(segt, len(segments), off, ctypes.byref(total)))
    return [off[i] for i in range(len(segments))], total.value


def _workspace(nbytes: int, device) -> torch.Tensor:
    buf = torch.empty(max(nbytes, 1) + 256, dtype=torch.uint8, device=device)
    shift = (-buf.data_ptr()) % 256
    return buf[shift:shift + max(nbytes, 1)]


def _device_of(segments) -> torch.device:
    for s in segments:
        return s.data.device
    return torch.device("cuda", torch.cuda.current_device())


class Outputs:
    """Device buffers of every output of the analysis for one segment table."""

    def __init__(self, segments: Sequence[DeviceSegment], n_requests: int, device=None,
                 token_fields=("z", "l1", "l2", "info", "d", "res"), compact: bool = True,
                 workspace: bool = True):
        device = device or _device_of(segments)
        ntok, nfr, ws = sizes(segments, n_requests)
        self.ntok, self.nframes, self.ws_bytes = ntok, nfr, ws
        R, n = n_requests, len(segments)
        e = lambda k, dt: torch.empty(max(k, 1), dtype=dt, device=device)  # noqa: E731
        tk = {"z": torch.int32, "l1": torch.float32, "l2": torch.float32, "info": torch.float32,
              "d": torch.int32, "res": torch.float32}
        self.tok = {f: e(ntok, tk[f]) for f in token_fields}
        self.frm = {"dframe": e(nfr, torch.int64), "sim": e(nfr, torch.float32), "gamma": e(nfr, torch.float32)}
        self.req = {"agg": e(R * NMOD * 4, torch.int64), "rho": e(R * NMOD, torch.float32),
                    "temporal": e(R * NMOD, torch.float32), "beta": e(R * NMOD, torch.float32),
                    "mas": e(R * NMOD, torch.float32), "present": e(R * NMOD, torch.uint8)}
        self.sel = {"keep": e(ntok, torch.uint8), "kept_idx": e(ntok, torch.int32),
                    "kept_count": e(n, torch.int32)}
        # msao_run_noalloc takes no workspace (workspace=False leaves it out)
        self.workspace = _workspace(ws, device) if workspace else None
        self.out = None
        self.out_off = None
        if compact:
            offs, total = compact_layout(segments)
            self.out = e(total, torch.uint8)
            self.out_off = (ctypes.c_int64 * max(1, n))(*offs)
            self.out_bytes = total
        self._structs()

    def _structs(self):
        g = lambda d, k: _ptr(d.get(k))  # noqa: E731
        self.c_tok = MsaoTokenOut(*[g(self.tok, k) for k in ("z", "l1", "l2", "info", "d", "res")])
        self.c_frm = MsaoFrameOut(*[g(self.frm, k) for k in ("dframe", "sim", "gamma")])
        self.c_req = MsaoReqOut(*[g(self.req, k) for k in ("agg", "rho", "temporal", "beta", "mas", "present")])
        self.c_sel = MsaoSelectOut(*[g(self.sel, k) for k in ("keep", "kept_idx", "kept_count")])

    def results(self, n_requests: int, n_segments: int) -> dict:
        """Outputs trimmed to their logical sizes (still on the device)."""
        R, n, nt, nf = n_requests, n_segments, self.ntok, self.nframes
        r = {k: v[:nt] for k, v in self.tok.items()}
        r.update({k: v[:nf] for k, v in self.frm.items()})
        r.update({k: v[: (R * NMOD * 4 if k == "agg" else R * NMOD)] for k, v in self.req.items()})
        r["keep"] = self.sel["keep"][:nt]
        r["kept_idx"] = self.sel["kept_idx"][:nt]
        r["kept_count"] = self.sel["kept_count"][:n]
        return r


def _stream_ptr(stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Call:
    """Prepared arguments of one entry point, reusable across launches (the
    segment table and output pointers are marshalled once)."""

    def __init__(self, fn_name: str, args: list, ctx: Context, keep_alive: list):
        self.fn = getattr(lib(), fn_name)
        self.args = args
        self.ctx = ctx
        self.keep_alive = keep_alive

    def __call__(self, stream=None):
        _check(self.fn(*self.args[:-1], _stream_ptr(stream)), self.ctx)


def prepare(entry: str, segments: Sequence[DeviceSegment], n_requests: int, outputs: Outputs,
            params: Optional[dict] = None, alpha: Optional[Sequence[float]] = None,
            ctx: Optional[Context] = None, mas: Optional[torch.Tensor] = None,
            z: Optional[torch.Tensor] = None, d: Optional[torch.Tensor] = None,
            compact: bool = True) -> Call:
    """Marshal the arguments of entry point `entry` (msao_run, msao_mas_score, ...)."""
    device = _device_of(segments)
    ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
    segt = segment_table(segments)
    prm = params_struct(params)
    n, R = len(segments), n_requests
    al = None
    if alpha is not None:
        vals = list(alpha)
        if len(vals) != R * NMOD:
            raise ValueError("alpha needs n_requests * 4 logits")
        al = (ctypes.c_float * len(vals))(*vals)
    o = outputs
    ws = _ptr(o.workspace)
    wsb = ctypes.c_size_t(o.ws_bytes)
    keep = [segt, prm, al, o, mas, z, d]
    if entry == "msao_run":
        out = _ptr(o.out) if (compact and o.out is not None) else None
        off = o.out_off if (compact and o.out is not None) else None
        ob = ctypes.c_int64(o.out_bytes if out is not None else 0)
        args = [ctx.handle, segt, n, R, _addr(prm), al, _addr(o.c_tok), _addr(o.c_frm), _addr(o.c_req),
                _addr(o.c_sel), out, off, ob, ws, wsb, None]
    elif entry == "msao_run_noalloc":
        out = _ptr(o.out) if (compact and o.out is not None) else None
        off = o.out_off if (compact and o.out is not None) else None
        ob = ctypes.c_int64(o.out_bytes if out is not None else 0)
        args = [ctx.handle, segt, n, R, _addr(prm), al, _addr(o.c_tok), _addr(o.c_frm), _addr(o.c_req),
                _addr(o.c_sel), out, off, ob, None]
    elif entry == "msao_mas_score":
        args = [ctx.handle, segt, n, R, _addr(prm), al, _addr(o.c_tok), _addr(o.c_frm), _addr(o.c_req),
                ws, wsb, None]
    elif entry == "msao_temporal_redundancy":
        args = [ctx.handle, segt, n, R, _addr(prm), _ptr(o.tok.get("d")), _ptr(o.tok.get("res")),
                _addr(o.c_frm), _ptr(o.req["temporal"]), ws, wsb, None]
    elif entry == "msao_select_tokens":
        zz = z if z is not None else o.tok["z"]
        dd = d if d is not None else o.tok.get("d")
        args = [ctx.handle, segt, n, R, _addr(prm), _ptr(zz), _ptr(dd), _ptr(mas), _addr(o.c_sel),
                ws, wsb, None]
    elif entry == "msao_compact":
        args = [ctx.handle, segt, n, _ptr(o.sel["kept_idx"]), _ptr(o.sel["kept_count"]), _ptr(o.out),
                o.out_off, ctypes.c_int64(o.out_bytes), ws, wsb, None]
    else:
        raise ValueError(f"unknown entry point {entry}")
    return Call(entry, args, ctx, keep)


class Plan:
    """msao_plan: the tables of one segment table uploaded once into the
    workspace of `outputs`; each call enqueues the three launches of msao_run
    with no host-to-device copy. The segments' input buffers and `outputs`
    must outlive the plan. The upload is enqueued on `stream` (the current
    stream when None) and waited for before the constructor returns, so runs
    may then be launched on any stream."""

    def __init__(self, segments: Sequence[DeviceSegment], n_requests: int, outputs: Outputs,
                 params: Optional[dict] = None, alpha: Optional[Sequence[float]] = None,
                 ctx: Optional[Context] = None, compact: bool = True, stream=None):
        device = _device_of(segments)
        self.ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
        self.segt = segment_table(segments)
        self.prm = params_struct(params)
        n, R = len(segments), n_requests
        self.al = None
        if alpha is not None:
            vals = list(alpha)
            if len(vals) != R * NMOD:
                raise ValueError("alpha needs n_requests * 4 logits")
            self.al = (ctypes.c_float * len(vals))(*vals)
        o = self.outputs = outputs
        self.compact = compact and o.out is not None
        h = ctypes.c_void_p()
        up = stream if stream is not None else torch.cuda.current_stream(device)
        _check(lib().msao_plan_create(self.ctx.handle, self.segt, n, R, _addr(self.prm), self.al,
                                      o.out_off if self.compact else None, _ptr(o.workspace),
                                      ctypes.c_size_t(o.ws_bytes), _stream_ptr(up), ctypes.byref(h)), self.ctx)
        self.handle = h
        # the tables must be in the workspace before a run on another stream reads them
        up.synchronize()
        self.segments = list(segments)
        self._args = [h, _addr(o.c_tok), _addr(o.c_frm), _addr(o.c_req), _addr(o.c_sel),
                      _ptr(o.out) if self.compact else None,
                      ctypes.c_int64(o.out_bytes if self.compact else 0)]

    def __call__(self, stream=None):
        _check(lib().msao_plan_run(*self._args, _stream_ptr(stream)), self.ctx)

    def close(self):
        if getattr(self, "handle", None):
            lib().msao_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _one_shot(entry, segments, n_requests, params=None, alpha=None, ctx=None, outputs=None, stream=None,
              compact=True, **kw):
    o = outputs or Outputs(segments, n_requests, compact=compact)
    prepare(entry, segments, n_requests, o, params, alpha, ctx, compact=compact, **kw)(stream)
    return o


def msao_mas_score(segments, n_requests, params=None, alpha=None, ctx=None, outputs=None, stream=None):
    """Per-token statistics, per-frame terms and per-modality MAS (Sec. 4.1)."""
    return _one_shot("msao_mas_score", segments, n_requests, params, alpha, ctx, outputs, stream, compact=False)


def msao_temporal_redundancy(segments, n_requests, params=None, ctx=None, outputs=None, stream=None):
    """Eq. 5 terms only: d, res, per-frame D/sim/gamma, temporal term per (request, modality)."""
    return _one_shot("msao_temporal_redundancy", segments, n_requests, params, None, ctx, outputs, stream,
                     compact=False)


def msao_temporal_simhash(segments, n_requests, hashes, params=None, ctx=None, outputs=None, stream=None, sig=None):
    """Eq. 5 with SimHash: hashes[s] = dict(planes=[bits, hidden] device
    tensor in the segment's dtype, bits) for temporal segments (None
    elsewhere). Fills outputs.tok["d"], outputs.frm and outputs.req["temporal"];
    returns (outputs, sig) with sig the [total tokens] int64 signatures."""
    device = _device_of(segments)
    ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
    o = outputs or Outputs(segments, n_requests, compact=False)
    segt = segment_table(segments)
    prm = params_struct(params)
    n = len(segments)
    harr, keep = _hash_array(hashes, n)
    if sig is None:
        sig = torch.empty(max(o.ntok, 1), dtype=torch.int64, device=device)[:o.ntok]
    st = stream if stream is not None else torch.cuda.current_stream(device)
    _check(lib().msao_temporal_simhash(ctx.handle, segt, n, n_requests, _addr(prm), ctypes.cast(harr, _P),
                                       _ptr(sig) if o.ntok else None, _ptr(o.tok["d"]) if o.ntok else None,
                                       _addr(o.c_frm), _ptr(o.req["temporal"]), _ptr(o.workspace),
                                       ctypes.c_size_t(o.ws_bytes), ctypes.c_void_p(st.cuda_stream)), ctx)
    return o, sig


def _hash_array(hashes, n):
    harr = (MsaoSimHash * max(1, n))()
    keep = [harr]
    for i, h in enumerate(hashes):
        if h is None:
            continue
        keep.append(h["planes"])
        harr[i] = MsaoSimHash(h["planes"].data_ptr(), int(h["bits"]))
    return harr, keep


def msao_run_simhash(segments, n_requests, hashes, params=None, alpha=None, ctx=None, outputs=None, stream=None,
                     compact=True, sig=None):
    """msao_run with SimHash as Eq. 5's hash (hashes as for
    msao_temporal_simhash): returns (outputs, sig)."""
    device = _device_of(segments)
    ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
    o = outputs or Outputs(segments, n_requests, compact=compact)
    segt = segment_table(segments)
    prm = params_struct(params)
    n, R = len(segments), n_requests
    harr, keep = _hash_array(hashes, n)
    al = None
    if alpha is not None:
        vals = list(alpha)
        if len(vals) != R * NMOD:
            raise ValueError("alpha needs n_requests * 4 logits")
        al = (ctypes.c_float * len(vals))(*vals)
    if sig is None:
        sig = torch.empty(max(o.ntok, 1), dtype=torch.int64, device=device)[:o.ntok]
    use_out = compact and o.out is not None
    st = stream if stream is not None else torch.cuda.current_stream(device)
    _check(lib().msao_run_simhash(ctx.handle, segt, n, R, _addr(prm), ctypes.cast(harr, _P), al, _addr(o.c_tok),
                                  _ptr(sig) if o.ntok else None, _addr(o.c_frm), _addr(o.c_req), _addr(o.c_sel),
                                  _ptr(o.out) if use_out else None, o.out_off if use_out else None,
                                  ctypes.c_int64(o.out_bytes if use_out else 0), _ptr(o.workspace),
                                  ctypes.c_size_t(o.ws_bytes), ctypes.c_void_p(st.cuda_stream)), ctx)
    del keep
    return o, sig


def prepare_simhash(entry, segments, n_requests, hashes, outputs, sig, params=None, alpha=None, ctx=None,
                    compact=True) -> Call:
    """msao_run_simhash's or msao_temporal_simhash's arguments (entry) marshalled
    once, as prepare() does for the other entry points; sig is the caller's
    [total tokens] int64 signature tensor."""
    device = _device_of(segments)
    ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
    o = outputs
    segt = segment_table(segments)
    prm = params_struct(params)
    n, R = len(segments), n_requests
    harr, keep = _hash_array(hashes, n)
    al = None
    if alpha is not None:
        vals = list(alpha)
        if len(vals) != R * NMOD:
            raise ValueError("alpha needs n_requests * 4 logits")
        al = (ctypes.c_float * len(vals))(*vals)
    keep += [segt, prm, al, o, sig]
    if entry == "msao_run_simhash":
        use_out = compact and o.out is not None
        args = [ctx.handle, segt, n, R, _addr(prm), ctypes.cast(harr, _P), al, _addr(o.c_tok),
                _ptr(sig) if o.ntok else None, _addr(o.c_frm), _addr(o.c_req), _addr(o.c_sel),
                _ptr(o.out) if use_out else None, o.out_off if use_out else None,
                ctypes.c_int64(o.out_bytes if use_out else 0), _ptr(o.workspace), ctypes.c_size_t(o.ws_bytes), None]
    elif entry == "msao_temporal_simhash":
        args = [ctx.handle, segt, n, R, _addr(prm), ctypes.cast(harr, _P), _ptr(sig) if o.ntok else None,
                _ptr(o.tok["d"]) if o.ntok else None, _addr(o.c_frm), _ptr(o.req["temporal"]), _ptr(o.workspace),
                ctypes.c_size_t(o.ws_bytes), None]
    else:
        raise ValueError(f"unknown SimHash entry point {entry}")
    return Call(entry, args, ctx, keep)


def msao_select_tokens(segments, n_requests, z, d=None, mas=None, params=None, ctx=None, outputs=None,
                       stream=None):
    """Per-segment top-k selection from z (and d); mas for MAS-guided keep ratios."""
    return _one_shot("msao_select_tokens", segments, n_requests, params, None, ctx, outputs, stream,
                     compact=False, z=z, d=d, mas=mas)


def msao_compact(segments, outputs, ctx=None, stream=None):
    """Packed copy of the kept rows named by outputs.sel (kept_idx, kept_count)."""
    n_req = max((s.request for s in segments), default=-1) + 1
    prepare("msao_compact", segments, n_req, outputs, None, None, ctx)(stream)
    return outputs


def msao_run(segments, n_requests, params=None, alpha=None, ctx=None, outputs=None, stream=None, compact=True):
    """Scoring, MAS, selection and compaction in one call."""
    return _one_shot("msao_run", segments, n_requests, params, alpha, ctx, outputs, stream, compact=compact)


def msao_run_noalloc(segments, n_requests, params=None, alpha=None, ctx=None, outputs=None, stream=None,
                     compact=True):
    """msao_run on the library's own scratch (no workspace; the call
    allocates nothing). `outputs` may be built with workspace=False."""
    return _one_shot("msao_run_noalloc", segments, n_requests, params, alpha, ctx, outputs, stream,
                     compact=compact)


def compacted_rows(segments: Sequence[DeviceSegment], outputs: Outputs, kept_count) -> list:
    """Views of each segment's packed kept rows in outputs.out (after synchronising)."""
    offs, _ = compact_layout(segments)
    rows = []
    for s, off, k in zip(segments, offs, kept_count):
        es = 4 if s.data.dtype == torch.float32 else 2
        nb = int(k) * s.data.shape[1] * es
        view = outputs.out[off:off + nb]
        rows.append(view.view(s.data.dtype).view(int(k), s.data.shape[1]))
    return rows


# ---- Sec. 4.2: draft confidence (GPU) and Algorithm 1 (host) ------------------

def msao_draft_entropy(logits: torch.Tensor, theta: float, vocab: Optional[int] = None, ctx: Optional[Context] = None,
                       stream=None, outputs: Optional[Dict[str, torch.Tensor]] = None) -> Dict[str, torch.Tensor]:
    """Eq. 9-10 per row of a [rows, row_stride] float32/bfloat16 device tensor
    (the first `vocab` columns are the logits). Returns device tensors
    entropy (nats), entropy_norm, draft_token and speculate."""
    if logits.dim() != 2 or logits.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("logits must be a 2-D float32 or bfloat16 tensor")
    if logits.numel() and logits.stride(1) != 1:
        raise ValueError("rows must be contiguous")
    rows = int(logits.shape[0])
    V = int(logits.shape[1]) if vocab is None else int(vocab)
    stride = int(logits.stride(0)) if rows > 1 else int(logits.shape[1])
    dev = logits.device
    if ctx is None:
        ctx = default_context(dev.index if dev.index is not None else torch.cuda.current_device())
    o = outputs or {"entropy": torch.empty(rows, dtype=torch.float32, device=dev),
                    "entropy_norm": torch.empty(rows, dtype=torch.float32, device=dev),
                    "draft_token": torch.empty(rows, dtype=torch.int32, device=dev),
                    "speculate": torch.empty(rows, dtype=torch.uint8, device=dev)}
    out = MsaoEntropyOut(*[_ptr(o.get(k)) for k in ("entropy", "entropy_norm", "draft_token", "speculate")])
    st = stream if stream is not None else torch.cuda.current_stream(dev)
    dt = F32 if logits.dtype == torch.float32 else BF16
    _check(lib().msao_draft_entropy(ctx.handle, _ptr(logits) if logits.numel() else None, rows, V, stride, dt,
                                    float(theta), _addr(out), ctypes.c_void_p(st.cuda_stream)), ctx)
    return o


def msao_stream_read(data: torch.Tensor, chunk_kib: int = 8, ctx: Optional[Context] = None, stream=None,
                     sink: Optional[torch.Tensor] = None) -> torch.Tensor:
    """A plain streaming read of a contiguous device tensor (the read
    ceiling of the HBM-bound passes); returns the sink of one XOR per
    wavefront."""
    nbytes = data.numel() * data.element_size()
    dev = data.device
    if ctx is None:
        ctx = default_context(dev.index if dev.index is not None else torch.cuda.current_device())
    waves = -(-nbytes // (chunk_kib * 1024))
    if sink is None:
        sink = torch.empty(max(waves, 1), dtype=torch.int32, device=dev)
    st = stream if stream is not None else torch.cuda.current_stream(dev)
    _check(lib().msao_stream_read(ctx.handle, _ptr(data), nbytes, int(chunk_kib), _ptr(sink), sink.numel(),
                                  ctypes.c_void_p(st.cuda_stream)), ctx)
    return sink


def sched_default_params() -> MsaoSchedParams:
    return lib().msao_sched_default_params()


def _host_f32(x):
    import numpy as np
    return np.ascontiguousarray(x, dtype=np.float32)


class Scheduler:
    """Algorithm 1 for one request: line 2-3 from calibration entropies, then
    the per-step hold / send / offload loop (host code in libmsao.so)."""

    def __init__(self, calib_h_norm, params: Optional[MsaoSchedParams] = None):
        self.params = params if params is not None else sched_default_params()
        self.state = MsaoSchedState()
        h = _host_f32(calib_h_norm)
        _check(lib().msao_sched_init(h.ctypes.data, h.size, _addr(self.params), _addr(self.state)))

    def step(self, h_norm: float) -> int:
        d = ctypes.c_int32()
        _check(lib().msao_sched_step(_addr(self.state), _addr(self.params), float(h_norm), ctypes.byref(d)))
        return d.value

    def run(self, h_norm):
        import numpy as np
        h = _host_f32(h_norm)
        dec = np.zeros(h.size, np.int8)
        th = np.zeros(h.size, np.float64)
        _check(lib().msao_sched_run(_addr(self.state), _addr(self.params), h.ctypes.data, h.size,
                                    dec.ctypes.data, th.ctypes.data))
        return dec, th


def retention_floor(mas):
    import numpy as np
    m = _host_f32(mas)
    b = np.zeros_like(m)
    _check(lib().msao_retention_floor(m.ctypes.data, m.size, b.ctypes.data))
    return b


def comm_latency(data_bytes: float, bandwidth_bytes_per_s: float, rtt_s: float) -> float:
    return lib().msao_comm_latency(data_bytes, bandwidth_bytes_per_s, rtt_s)


def p_conf(h_norm, theta: float) -> float:
    h = _host_f32(h_norm)
    return lib().msao_p_conf(h.ctypes.data, h.size, theta)


def expected_spec_tokens(p: float) -> float:
    return lib().msao_expected_spec_tokens(p)


def expected_e2e_latency(**terms) -> float:
    m = MsaoLatencyModel(**terms)
    return lib().msao_expected_e2e_latency(_addr(m))


# ---- Sec. 4.1.1 Eq. 3 and Sec. 4.1.3 Eq. 6 with caller weights ----------------

def _learned_args(segments, n_requests, params, heads, mlp, alpha, ctx):
    """Marshalled heads, MLP and logits of a learned call (and what must stay alive)."""
    device = _device_of(segments)
    ctx = ctx or default_context(device.index if device.index is not None else torch.cuda.current_device())
    segt = segment_table(segments)
    prm = params_struct(params)
    n = len(segments)
    keep = [segt, prm]
    harr = None
    if heads is not None:
        harr = (MsaoSpatialHead * max(1, n))()
        for i, h in enumerate(heads):
            if h is None:
                continue
            w = h["weight"]
            keep.append(w)
            harr[i] = MsaoSpatialHead(w.data_ptr(), float(h.get("bias", 0.0)), int(h.get("grid_w", 0)),
                                      int(h.get("pool", 1)))
        keep.append(harr)
    m = None
    if mlp is not None:
        m = MsaoModalMlp(mlp["w1"].data_ptr(), mlp["b1"].data_ptr(), mlp["w2"].data_ptr(), float(mlp.get("b2", 0.0)),
                         int(mlp["b1"].numel()), int(mlp["prompt"].shape[1]) if mlp.get("prompt") is not None else 0,
                         mlp["prompt"].data_ptr() if mlp.get("prompt") is not None else None)
        keep.append(m)
    al = None
    if alpha is not None:
        vals = list(alpha)
        al = (ctypes.c_float * len(vals))(*vals)
        keep.append(al)
    return device, ctx, segt, prm, harr, m, al, keep


def _learned_extra(o, n_requests, device):
    R = n_requests
    return {"importance": torch.empty(max(o.ntok, 1), dtype=torch.float32, device=device)[:o.ntok],
            "alpha": torch.empty(R * NMOD, dtype=torch.float32, device=device),
            "desc": torch.empty(R * NMOD * MODAL_DESC, dtype=torch.float32, device=device)}


def msao_mas_score_learned(segments, n_requests, params=None, heads=None, mlp=None, alpha=None, ctx=None,
                           outputs=None, stream=None):
    """msao_mas_score with learned probe heads: heads[s] is None or a dict
    (weight=[hidden] device tensor in the segment's dtype, bias, grid_w, pool);
    mlp is None or a dict of device float32 tensors (w1 [hidden, prompt_dim +
    8], b1, w2, prompt [n_requests, prompt_dim]) and b2. Returns
    (outputs, extra) with extra = importance, alpha and desc device tensors."""
    device, ctx, segt, prm, harr, m, al, keep = _learned_args(segments, n_requests, params, heads, mlp, alpha, ctx)
    o = outputs or Outputs(segments, n_requests, compact=False)
    n, R = len(segments), n_requests
    extra = _learned_extra(o, R, device)
    st = stream if stream is not None else torch.cuda.current_stream(device)
    _check(lib().msao_mas_score_learned(ctx.handle, segt, n, R, _addr(prm),
                                        ctypes.cast(harr, _P) if harr is not None else None,
                                        _addr(m) if m is not None else None, al, _addr(o.c_tok),
                                        _ptr(extra["importance"]) if o.ntok else None, _addr(o.c_frm),
                                        _addr(o.c_req), _ptr(extra["alpha"]), _ptr(extra["desc"]),
                                        _ptr(o.workspace), ctypes.c_size_t(o.ws_bytes), ctypes.c_void_p(st.cuda_stream)),
           ctx)
    extra["_keep"] = keep
    return o, extra


def prepare_learned(segments, n_requests, outputs, params=None, heads=None, mlp=None, alpha=None, ctx=None,
                    compact=True):
    """msao_run_learned's arguments marshalled once (as prepare() does for the
    other entry points): returns (call, extra); each call(stream) enqueues one
    run on the same outputs and extra buffers (tables still uploaded per call)."""
    device, ctx, segt, prm, harr, m, al, keep = _learned_args(segments, n_requests, params, heads, mlp, alpha, ctx)
    o = outputs
    n, R = len(segments), n_requests
    extra = _learned_extra(o, R, device)
    use_out = compact and o.out is not None
    args = [ctx.handle, segt, n, R, _addr(prm), ctypes.cast(harr, _P) if harr is not None else None,
            _addr(m) if m is not None else None, al, _addr(o.c_tok),
            _ptr(extra["importance"]) if o.ntok else None, _addr(o.c_frm), _addr(o.c_req),
            _ptr(extra["alpha"]), _ptr(extra["desc"]), _addr(o.c_sel),
            _ptr(o.out) if use_out else None, o.out_off if use_out else None,
            ctypes.c_int64(o.out_bytes if use_out else 0), _ptr(o.workspace), ctypes.c_size_t(o.ws_bytes), None]
    return Call("msao_run_learned", args, ctx, keep + [o, extra]), extra


def msao_run_learned(segments, n_requests, params=None, heads=None, mlp=None, alpha=None, ctx=None, outputs=None,
                     stream=None, compact=True):
    """msao_mas_score_learned plus the selection and compaction of msao_run,
    with segments that have a head ranked by their Eq. 3 importance (heads
    and mlp as for msao_mas_score_learned). Returns (outputs, extra)."""
    device, ctx, segt, prm, harr, m, al, keep = _learned_args(segments, n_requests, params, heads, mlp, alpha, ctx)
    o = outputs or Outputs(segments, n_requests, compact=compact)
    n, R = len(segments), n_requests
    extra = _learned_extra(o, R, device)
    use_out = compact and o.out is not None
    st = stream if stream is not None else torch.cuda.current_stream(device)
    _check(lib().msao_run_learned(ctx.handle, segt, n, R, _addr(prm),
                                  ctypes.cast(harr, _P) if harr is not None else None,
                                  _addr(m) if m is not None else None, al, _addr(o.c_tok),
                                  _ptr(extra["importance"]) if o.ntok else None, _addr(o.c_frm), _addr(o.c_req),
                                  _ptr(extra["alpha"]), _ptr(extra["desc"]), _addr(o.c_sel),
                                  _ptr(o.out) if use_out else None, o.out_off if use_out else None,
                                  ctypes.c_int64(o.out_bytes if use_out else 0), _ptr(o.workspace),
                                  ctypes.c_size_t(o.ws_bytes), ctypes.c_void_p(st.cuda_stream)), ctx)
    extra["_keep"] = keep
    return o, extra
