"""Seeded synthetic inputs: weights W, calibration activations X and frames P.

Recipe (every draw from numpy's PCG64, keyed by [seed, tag, index]):

* W (d_out x d_in) = sigma * N(0, 1) in float32; then exactly floor(frac * d_out * d_in)
  positions, uniform without replacement, are multiplied by the outlier scale.  With a
  Student-t fraction, each entry is drawn with that probability from sigma * t(4)
  instead.  The result is rounded once (round-to-nearest-even) to the device dtype.
* X (n x d_in) = N(0, 1) in float32, produced in chunks of CHUNK tokens (chunk c from
  its own stream, so any chunk can be regenerated alone); a fixed set of outlier
  channels (columns, uniform without replacement) is multiplied by the outlier scale;
  then rounded to the device dtype.
* P: a Parseval tight fusion frame (see tff.py) with its own rotation seed; the input
  frame is shared by all layers that read the same X.

Every array is returned both as the exact values (float32/float64 holding
device-representable numbers) and, for upload, in its device storage type.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
import os

import numpy as np

from . import tff
from .configs import Workload, Layer, frame_k

CHUNK = 8192
TAG_W, TAG_X, TAG_XCH, TAG_POUT, TAG_PIN = 1, 2, 3, 4, 5


def round_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_device_storage(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to the device dtype; return the storage array
    (float32 / float16 / uint16 bf16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(x32, dtype=np.float32)
    if dtype == "f16":
        return x32.astype(np.float16)
    if dtype == "bf16":
        return round_bf16_bits(x32)
    raise ValueError(dtype)


def storage_to_f32(s: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float32 values of a device-storage array."""
    if dtype == "bf16":
        return bf16_bits_to_f32(s)
    return s.astype(np.float32)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def make_weight(wl: Workload, li: int) -> np.ndarray:
    """Layer li's weight, in device storage (see to_device_storage)."""
    L: Layer = wl.layers[li]
    rng = np.random.default_rng([wl.seed, TAG_W, li])
    shape = (L.d_out, L.d_in)
    W = rng.standard_normal(shape, dtype=np.float32)
    if L.t4_frac > 0:
        pick = rng.random(shape) < L.t4_frac
        W[pick] = rng.standard_t(4, size=int(pick.sum())).astype(np.float32)
    W *= np.float32(L.w_sigma)
    if L.outlier_frac > 0:
        m = int(np.floor(L.outlier_frac * L.d_out * L.d_in))
        idx = rng.choice(L.d_out * L.d_in, size=m, replace=False)
        W.reshape(-1)[idx] *= np.float32(L.outlier_scale)
    return to_device_storage(W, wl.w_dtype)


def x_outlier_channels(wl: Workload, d_in: int) -> np.ndarray:
    rng = np.random.default_rng([wl.seed, TAG_XCH])
    return np.sort(rng.choice(d_in, size=wl.x_outlier_channels, replace=False))


def make_x_chunk(wl: Workload, c: int, d_in: int, n_tokens: int | None = None) -> np.ndarray:
    """Tokens [c*CHUNK, min((c+1)*CHUNK, n)) of X in device storage."""
    n = wl.n_tokens if n_tokens is None else n_tokens
    t0 = c * CHUNK
    rows = min(CHUNK, n - t0)
    if rows <= 0:
        raise ValueError("chunk out of range")
    rng = np.random.default_rng([wl.seed, TAG_X, c])
    X = rng.standard_normal((rows, d_in), dtype=np.float32)
    ch = x_outlier_channels(wl, d_in)
    X[:, ch] *= np.float32(wl.x_outlier_scale)
    return to_device_storage(X, wl.x_dtype)


def n_chunks(n_tokens: int) -> int:
    return (n_tokens + CHUNK - 1) // CHUNK


def make_x(wl: Workload, d_in: int, n_tokens: int | None = None, out: np.ndarray | None = None):
    """All of X (n x d_in) in device storage, generated chunk-parallel."""
    n = wl.n_tokens if n_tokens is None else n_tokens
    sdt = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[wl.x_dtype]
    if out is None:
        out = np.empty((n, d_in), dtype=sdt)

    def fill(c):
        ch = make_x_chunk(wl, c, d_in, n)
        out[c * CHUNK: c * CHUNK + ch.shape[0]] = ch

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fill, range(n_chunks(n))))
    return out


def make_frame(wl: Workload, d: int, tag: int, index: int = 0, dtype=np.float64) -> np.ndarray:
    """Dense Parseval frame P (d x K) for dimension d (float64, or its float32 rounding)."""
    k = frame_k(wl, d)
    ss = np.random.SeedSequence([wl.seed, tag, index])
    return tff.parseval_frame(k, wl.rho, d, ss, dtype=dtype)


def make_frames(wl: Workload, li: int, dtype=np.float64):
    """(P_out, P_in) for layer li; P_in is shared by all layers of the workload."""
    L = wl.layers[li]
    P_out = make_frame(wl, L.d_out, TAG_POUT, li, dtype)
    P_in = make_frame(wl, L.d_in, TAG_PIN, 0, dtype)
    return P_out, P_in


def frame_factors(wl: Workload, d: int, tag: int, index: int = 0):
    """(k, rho, R1, R2): the construction parameters of make_frame(wl, d, tag, index), whose
    rotation is R1 (x) R2 with exactly these (float64) factors."""
    k = frame_k(wl, d)
    R1, R2 = tff.rotation_factors(d, np.random.SeedSequence([wl.seed, tag, index]))
    return k, wl.rho, R1, R2


def layer_frame_factors(wl: Workload, li: int):
    """frame_factors of (P_out, P_in) of layer li, as make_frames builds them."""
    L = wl.layers[li]
    return frame_factors(wl, L.d_out, TAG_POUT, li), frame_factors(wl, L.d_in, TAG_PIN, 0)


def frame_f32(P: np.ndarray) -> np.ndarray:
    """The frame as the float32 matrix handed to the device (RNE from float64)."""
    return np.ascontiguousarray(P, dtype=np.float32)
