"""Seeded synthetic workloads shaped like the paper's image, video and audio inputs.

The paper evaluates on VQAv2 and MMBench with Qwen2-VL encoders (Sec. 5.1.1);
neither the datasets nor the encoders are available, so these generators stand
in for the early-layer activations the probing module reads (Sec. 4.1). Each
configuration follows the shapes and value distributions stated for the five
benchmark workloads; every tensor is drawn from numpy's PCG64 seeded with
SeedSequence([seed, config, request, segment]), so any prefix of requests is
reproducible on its own.

Values are drawn in float32 (float64 where a distribution needs it) and stored
either as float32 or as bf16 bit patterns (uint16, round-to-nearest-even).
"""
from __future__ import annotations

import dataclasses
import os
from typing import List, Optional

import numpy as np
from scipy.special import ndtr

TEXT, IMAGE, VIDEO, AUDIO = 0, 1, 2, 3
MODALITY_NAMES = ("text", "image", "video", "audio")

CONFIG_NAMES = {
    1: "single-image-fp32",
    2: "image-batch-bf16",
    3: "video-batch-bf16",
    4: "trimodal-batch-bf16",
    5: "highres-fused-bf16",
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    if nan.any():
        rounded[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x0040)).astype(np.uint16)
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Segment:
    """One modality-tagged activation tensor of one request.

    `data` is [n_frames * tokens_per_frame, hidden] (row t*P + p is token p of
    frame t), float32 or uint16 bf16 bit patterns.
    """
    request: int
    modality: int
    n_frames: int
    tokens_per_frame: int
    hidden: int
    dtype: str  # "f32" or "bf16"
    keep_ratio: float
    data: np.ndarray
    meta: dict = dataclasses.field(default_factory=dict)  # generator masks, for statistical pins

    @property
    def n_tokens(self) -> int:
        return self.n_frames * self.tokens_per_frame

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


@dataclasses.dataclass
class Workload:
    name: str
    config: int
    n_requests: int
    segments: List[Segment]
    params: dict
    alpha: Optional[np.ndarray] = None  # [R, 4] float32 logits or None (all zero)

    @property
    def n_tokens(self) -> int:
        return sum(s.n_tokens for s in self.segments)

    @property
    def input_bytes(self) -> int:
        return sum(s.n_tokens * s.hidden * s.elt_bytes for s in self.segments)


def default_params() -> dict:
    """Sec. 5.1.4 parameters: tau_s = 0.3, lambda_spatial = 0.6, lambda_temp = 0.4.

    The element threshold tau = 0.1 is the workloads' value (the paper has no
    element threshold). lambda_spatial applies to image, video and audio;
    lambda_temp to video only (text is dense, Sec. 1).
    """
    return {
        "tau": 0.1,
        "tau_s": 0.3,
        "lambda_s": [0.0, 0.6, 0.6, 0.6],
        "lambda_t": [0.0, 0.0, 0.4, 0.0],
        "flags": 0,
    }


def _rng(seed: int, config: int, request: int, segment: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, config, request, segment])))


def _gelu(x: np.ndarray) -> np.ndarray:
    # exact (erf) form: x * Phi(x), evaluated in float64 then stored as float32
    return (x.astype(np.float64) * ndtr(x.astype(np.float64))).astype(np.float32)


def _rect_for_area(rng: np.random.Generator, grid_h: int, grid_w: int, area: float):
    """A seeded axis-aligned rectangle inside the grid whose area is nearest `area`."""
    best = None
    cands = []
    for h in range(1, grid_h + 1):
        for w in range(1, grid_w + 1):
            err = abs(h * w - area)
            if best is None or err < best - 1e-12:
                best, cands = err, [(h, w)]
            elif abs(err - best) <= 1e-12:
                cands.append((h, w))
    h, w = cands[int(rng.integers(len(cands)))]
    top = int(rng.integers(grid_h - h + 1))
    left = int(rng.integers(grid_w - w + 1))
    mask = np.zeros((grid_h, grid_w), dtype=bool)
    mask[top:top + h, left:left + w] = True
    return mask.reshape(-1)


def _encode(x: np.ndarray, dtype: str) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32) if dtype == "f32" else f32_to_bf16_bits(x)


def _image_relu(rng, n_tok, hidden, bg_mask, bg_scale=0.05):
    x = rng.standard_normal((n_tok, hidden), dtype=np.float32)
    np.maximum(x, 0.0, out=x)
    x[bg_mask] *= np.float32(bg_scale)
    return x


def _image_gelu(rng, n_tok, hidden, bg_mask, bg_scale=0.05):
    x = _gelu(rng.standard_normal((n_tok, hidden), dtype=np.float32))
    x[bg_mask] *= np.float32(bg_scale)
    return x


def _config1(seed, r):
    segs = []
    rng = _rng(seed, 1, r, 0)
    h, w = (15, 23) if rng.integers(2) == 0 else (23, 15)
    top = int(rng.integers(24 - h + 1))
    left = int(rng.integers(24 - w + 1))
    mask = np.zeros((24, 24), dtype=bool)
    mask[top:top + h, left:left + w] = True
    mask = mask.reshape(-1)
    img = _image_relu(rng, 576, 1024, mask)
    segs.append(Segment(r, IMAGE, 1, 576, 1024, "f32", 0.5, _encode(img, "f32"),
                        {"bg_mask": mask}))
    rng_t = _rng(seed, 1, r, 1)
    txt = np.maximum(rng_t.standard_normal((32, 1024), dtype=np.float32), 0.0)
    segs.append(Segment(r, TEXT, 1, 32, 1024, "f32", 1.0, _encode(txt, "f32")))
    return segs


def _image_bf16_gelu_segment(seed, config, r, seg_id, keep):
    rng = _rng(seed, config, r, seg_id)
    frac = float(rng.uniform(0.2, 0.8))
    mask = _rect_for_area(rng, 24, 24, frac * 576)
    img = _image_gelu(rng, 576, 1024, mask)
    return Segment(r, IMAGE, 1, 576, 1024, "bf16", keep, _encode(img, "bf16"), {"bg_mask": mask})


def _text_bf16_gelu_segment(seed, config, r, seg_id, n_tok):
    rng = _rng(seed, config, r, seg_id)
    txt = _gelu(rng.standard_normal((n_tok, 4096), dtype=np.float32))
    return Segment(r, TEXT, 1, n_tok, 4096, "bf16", 1.0, _encode(txt, "bf16"))


def _config2(seed, r):
    return [_image_bf16_gelu_segment(seed, 2, r, 0, 0.25), _text_bf16_gelu_segment(seed, 2, r, 1, 64)]


def video_clip(rng, n_frames, grid, hidden, static_frac=0.7, step_sigma=0.02):
    """Frame 0 ~ N(0,1); static patches follow a float32 random walk with
    N(0, step_sigma^2) steps; moving patches are redrawn every frame. Each
    frame is rounded to bf16 independently. Returns ([T*P, hidden] uint16, static mask [P])."""
    P = grid * grid
    n_static = int(round(static_frac * P))
    static = np.zeros(P, dtype=bool)
    static[rng.choice(P, size=n_static, replace=False)] = True
    out = np.empty((n_frames * P, hidden), dtype=np.uint16)
    cur = rng.standard_normal((P, hidden), dtype=np.float32)
    out[0:P] = f32_to_bf16_bits(cur)
    n_moving = P - n_static
    for t in range(1, n_frames):
        step = rng.standard_normal((n_static, hidden), dtype=np.float32) * np.float32(step_sigma)
        cur[static] = cur[static] + step
        cur[~static] = rng.standard_normal((n_moving, hidden), dtype=np.float32)
        out[t * P:(t + 1) * P] = f32_to_bf16_bits(cur)
    return out, static


def _config3(seed, r):
    rng = _rng(seed, 3, r, 0)
    data, static = video_clip(rng, 32, 16, 1024)
    return [Segment(r, VIDEO, 32, 256, 1024, "bf16", 0.3, data, {"static_mask": static})]


def silence_runs(rng, n_frames, n_silent, n_runs):
    """Seeded non-overlapping runs of `n_silent` frames in total, in `n_runs` pieces."""
    cuts = np.sort(rng.choice(np.arange(1, n_silent), size=n_runs - 1, replace=False))
    lens = np.diff(np.concatenate([[0], cuts, [n_silent]]))
    gaps = rng.multinomial(n_frames - n_silent, [1.0 / (n_runs + 1)] * (n_runs + 1))
    mask = np.zeros(n_frames, dtype=bool)
    pos = 0
    for i in range(n_runs):
        pos += int(gaps[i])
        mask[pos:pos + int(lens[i])] = True
        pos += int(lens[i])
    return mask


def _config4(seed, r):
    segs = [_image_bf16_gelu_segment(seed, 4, r, 0, 0.25)]
    rng = _rng(seed, 4, r, 1)
    mask = silence_runs(rng, 1500, 600, 4)
    aud = rng.standard_normal((1500, 1280), dtype=np.float32)
    aud[mask] *= np.float32(1e-3)
    segs.append(Segment(r, AUDIO, 1, 1500, 1280, "bf16", 0.5, _encode(aud, "bf16"),
                        {"silence_mask": mask}))
    segs.append(_text_bf16_gelu_segment(seed, 4, r, 2, 128))
    return segs


def _config5(seed, r):
    shapes = [(12, 24), (16, 18), (18, 16), (24, 12)]
    rng = _rng(seed, 5, r, 0)
    masks = []
    for _tile in range(5):
        h, w = shapes[int(rng.integers(4))]
        top = int(rng.integers(24 - h + 1))
        left = int(rng.integers(24 - w + 1))
        m = np.zeros((24, 24), dtype=bool)
        m[top:top + h, left:left + w] = True
        masks.append(m.reshape(-1))
    bg = np.concatenate(masks)
    img = _image_relu(rng, 2880, 1024, bg)
    return [Segment(r, IMAGE, 1, 2880, 1024, "bf16", 0.25, _encode(img, "bf16"), {"bg_mask": bg})]


_FULL_REQUESTS = {1: 1, 2: 64, 3: 8, 4: 32, 5: 256}
_BUILDERS = {1: _config1, 2: _config2, 3: _config3, 4: _config4, 5: _config5}


def make_workload(config: int, seed: int = 0, n_requests: Optional[int] = None, threads: int = 0) -> Workload:
    """Build benchmark workload `config` (1..5); `n_requests` takes a prefix of its requests.

    Requests are drawn independently (each from its own seeded generator), so
    they may be built on several threads (numpy's generators and ufuncs release
    the interpreter lock on large arrays); the result is the same for any
    `threads` (0: up to 16, the host's cores permitting)."""
    from concurrent.futures import ThreadPoolExecutor

    full = _FULL_REQUESTS[config]
    n = full if n_requests is None else min(int(n_requests), full)
    nt = threads if threads > 0 else max(1, min(16, os.cpu_count() or 1))
    build = _BUILDERS[config]
    if nt == 1 or n <= 1:
        parts = [build(seed, r) for r in range(n)]
    else:
        with ThreadPoolExecutor(min(nt, n)) as ex:
            parts = list(ex.map(lambda r: build(seed, r), range(n)))
    segs = [s for p in parts for s in p]
    return Workload(CONFIG_NAMES[config], config, n, segs, default_params(), None)


# ---- draft-model logits (Sec. 4.2) --------------------------------------------

DRAFT_VOCAB = 151936          # the Qwen2-VL output vocabulary (embedding rows, padded)
DRAFT_ROWS = 1280             # 256 requests x N_max = 5 draft tokens per speculative round


def draft_logits(rows: int = DRAFT_ROWS, vocab: int = DRAFT_VOCAB, seed: int = 0, dtype: str = "bf16",
                 row_stride: Optional[int] = None) -> np.ndarray:
    """Synthetic logits of a draft model, [rows, row_stride] (float32, or bf16
    bit patterns), standing in for the per-step output distributions of the
    paper's Qwen2-VL-2B draft model (Sec. 5.1), which is not available.

    Recipe per row r (PCG64 seeded with SeedSequence([seed, 6, rows, vocab])):
    background logits N(0, sigma_r^2) with sigma_r ~ U(0.5, 2.5); one peak
    token at a uniform index raised by b_r ~ U(0, 30); three runner-up tokens
    (fewer when the vocabulary is smaller) raised by b_r - U(1, 8). Small b_r gives a flat, unconfident row (normalised
    entropy near 1), large b_r a confident one (near 0), so the rows span the
    whole threshold range of Algorithm 1. Columns past `vocab` (when
    row_stride > vocab) are filled with NaN so that reading them would show."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 6, rows, vocab])))
    stride = vocab if row_stride is None else row_stride
    sigma = rng.uniform(0.5, 2.5, rows).astype(np.float32)
    boost = rng.uniform(0.0, 30.0, rows).astype(np.float32)
    k = min(4, vocab)                          # boosted tokens per row (the peak and its runners-up)
    if vocab <= 64:
        idx = np.stack([rng.permutation(vocab)[:k] for _ in range(rows)]) if rows else np.zeros((0, k), np.int64)
    else:
        idx = rng.integers(0, vocab, (rows, k))
        for r in range(rows):                  # distinct tokens; collisions are rare for a large vocabulary
            while len(set(idx[r].tolist())) < k:
                idx[r] = rng.integers(0, vocab, k)
    runner = rng.uniform(1.0, 8.0, (rows, k - 1)).astype(np.float32)
    x = np.full((rows, stride), np.nan, np.float32)
    x[:, :vocab] = rng.standard_normal((rows, vocab), dtype=np.float32)
    x[:, :vocab] *= sigma[:, None]
    r_ix = np.arange(rows)
    x[r_ix, idx[:, 0]] += boost
    if k > 1:
        x[r_ix[:, None], idx[:, 1:]] += boost[:, None] - runner
    return x if dtype == "f32" else f32_to_bf16_bits(x)


# ---- SimHash hyperplanes (Sec. 4.1.2 variant) -----------------------------------

def simhash_planes(bits: int, hidden: int, seed: int = 0, dtype: str = "bf16") -> np.ndarray:
    """[bits, hidden] random hyperplanes with N(0, 1) entries drawn in float32,
    encoded like segment data (float32, or bf16 bit patterns)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7, bits, hidden])))
    return _encode(rng.standard_normal((bits, hidden), dtype=np.float32), dtype)
