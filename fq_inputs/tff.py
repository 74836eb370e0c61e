"""Tight fusion frame (TFF) construction: the frame inputs P of the quantization pass.

The paper treats the TFF as a black-box input (Sec. 2.2, "Constructing TFFs") and
sketches the construction in its appendix ("Synopsis of Construction of Tight Fusion
Frames"):

1. spectral tetris builds a unit-norm tight frame F (rho x d) for C^rho: unit columns,
   orthogonal rows, every row of squared norm d/rho, made of 1s and 2x2 blocks T(x);
2. every row of F, multiplied entrywise by the modulation vector (w^(j*s))_j with
   w = exp(2*pi*i/k), spans subspace s (s = 0..k-1);
3. the entrywise map x+iy -> [[x, -y], [y, x]] takes a complex (k, rho, d) TFF to a real
   (k, 2*rho, 2*d) one.

The resulting real basis is then scaled so that the frame is Parseval (weights w_i
absorbed, Sec. 3 "To reduce notational clutter ...") and hit by a seeded random rotation
(Sec. 2.2 remarks; appendix "Computational Complexity during Inference", where
P = R(T)).  Column order of P is subspace-major, P = [P_1 ... P_k] (Sec. 3).

Nothing here is arithmetic of the quantization method itself; the frame is an input.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction
import math
import os
import threading

import numpy as np

_BLAS_LOCK = threading.Lock()


def t_block(x: float) -> np.ndarray:
    """The 2x2 spectral-tetris block T(x) (appendix, Spectral Tetris).

    T(x) = 1/sqrt(2) [[sqrt(x), sqrt(x)], [sqrt(2-x), -sqrt(2-x)]], so that
    T T^T = diag(x, 2-x).  Requires 0 < x < 2.
    """
    if not (0.0 < x < 2.0):
        raise ValueError("T(x) needs 0 < x < 2")
    a = math.sqrt(x / 2.0)
    b = math.sqrt((2.0 - x) / 2.0)
    return np.array([[a, a], [b, -b]], dtype=np.float64)


def spectral_tetris_layout(rho: int, d: int):
    """Exact bookkeeping of spectral tetris for a rho x d unit-norm tight frame.

    Returns a list of entries (row, col, sq, sign): F[row, col] = sign * sqrt(sq) with sq an
    exact Fraction.  Rows are filled left to right: while the row still needs at least 1
    of squared norm, place a 1; a remaining need 0 < x < 1 is closed with T(x) spanning
    this row and the next, which then starts with the need reduced by 2 - x.
    Fails (ValueError) when a block would overfill a row; d >= 2*rho always succeeds.
    """
    if rho <= 0 or d <= 0:
        raise ValueError("rho and d must be positive")
    if d < rho:
        raise ValueError("a frame for C^rho needs at least rho vectors")
    target = Fraction(d, rho)
    entries = []
    col = 0
    carry = Fraction(0)
    for row in range(rho):
        need = target - carry
        carry = Fraction(0)
        if need < 0:
            raise ValueError("spectral tetris: a 2x2 block overfilled the next row")
        while need >= 1:
            entries.append((row, col, Fraction(1), 1))
            col += 1
            need -= 1
        if need > 0:
            if row + 1 >= rho:
                raise ValueError("spectral tetris ran out of rows")
            x = need
            entries.append((row, col, x / 2, 1))
            entries.append((row, col + 1, x / 2, 1))
            entries.append((row + 1, col, (2 - x) / 2, 1))
            entries.append((row + 1, col + 1, (2 - x) / 2, -1))
            col += 2
            carry = 2 - x
    if col != d:
        raise ValueError(f"spectral tetris filled {col} columns, expected {d}")
    return entries


def spectral_tetris(rho: int, d: int) -> np.ndarray:
    """The rho x d unit-norm tight frame F of spectral tetris, as float64."""
    F = np.zeros((rho, d), dtype=np.float64)
    for r, c, sq, sgn in spectral_tetris_layout(rho, d):
        F[r, c] = sgn * math.sqrt(float(sq))
    return F


def row_supports(F: np.ndarray):
    return [np.flatnonzero(F[r]) for r in range(F.shape[0])]


def modulation_is_tight(F: np.ndarray, k: int) -> bool:
    """Whether modulating F by the k-th roots of unity yields a tight fusion frame.

    The modulated subspaces are mutually consistent (each subspace basis orthogonal and
    the frame operator a multiple of I) exactly when no row of F has two support columns
    congruent mod k; a row whose support spans at most k consecutive columns satisfies it.
    """
    for sup in row_supports(F):
        res = np.mod(sup, k)
        if len(np.unique(res)) != len(res):
            return False
    return True


def _base_frame(k: int, rho_c: int, d_c: int) -> np.ndarray:
    F = spectral_tetris(rho_c, d_c) if d_c != rho_c else np.eye(rho_c)
    if not modulation_is_tight(F, k):
        raise ValueError(f"no tight modulation for (k={k}, rho={rho_c}, d={d_c})")
    return F


def complex_tff(k: int, rho_c: int, d_c: int, subspaces=None) -> np.ndarray:
    """Complex (k, rho_c, d_c) TFF: array B[s] (d_c x rho_c), orthonormal columns.

    Subspace s is spanned by the rows of F modulated by (w^(j*s))_j, w = exp(2*pi*i/k),
    each divided by sqrt(d_c/rho_c) to make it unit norm.  subspaces: optional range of
    s to build (default all k).
    """
    F = _base_frame(k, rho_c, d_c)
    j = np.arange(d_c)
    norm = math.sqrt(d_c / rho_c)
    ss = range(k) if subspaces is None else subspaces
    B = np.empty((len(ss), d_c, rho_c), dtype=np.complex128)
    for i, s in enumerate(ss):
        w = np.exp(2j * np.pi * s * j / k)
        B[i] = (F * w[None, :]).T / norm
    return B


def realify(B: np.ndarray) -> np.ndarray:
    """Entrywise x+iy -> [[x, -y], [y, x]]: a (d_c x rho_c) complex block becomes a
    (2 d_c x 2 rho_c) real block; complex row j -> real rows 2j, 2j+1 and complex
    column c -> real columns 2c, 2c+1."""
    d_c, rho_c = B.shape[-2:]
    out = np.empty(B.shape[:-2] + (2 * d_c, 2 * rho_c), dtype=np.float64)
    out[..., 0::2, 0::2] = B.real
    out[..., 0::2, 1::2] = -B.imag
    out[..., 1::2, 0::2] = B.imag
    out[..., 1::2, 1::2] = B.real
    return out


def real_tff_basis(k: int, rho: int, d: int, subspaces=None) -> np.ndarray:
    """Real (k, rho, d) TFF as a d x (k*rho) matrix T = [T_1 ... T_k], each T_i with
    orthonormal columns; sum_i T_i T_i^T = (k*rho/d) I_d.  rho and d must be even
    (realification of a complex (k, rho/2, d/2) TFF).  subspaces: optional range of i
    (the matching column blocks only)."""
    if rho % 2 or d % 2:
        raise ValueError("the real construction needs even rho and d")
    B = complex_tff(k, rho // 2, d // 2, subspaces)
    R = realify(B)  # n x d x rho
    return np.ascontiguousarray(R.transpose(1, 0, 2).reshape(d, R.shape[0] * rho))


def valid_k_for(rho: int, d: int, k: int) -> bool:
    """(k, rho, d) is constructible here (spectral tetris + tight modulation)."""
    try:
        rho_c, d_c = rho // 2, d // 2
        if rho % 2 or d % 2:
            return False
        F = spectral_tetris(rho_c, d_c) if d_c != rho_c else np.eye(rho_c)
        return modulation_is_tight(F, k)
    except ValueError:
        return False


def choose_k(d: int, r: float, rho: int = 16) -> int:
    """Number of subspaces for a target redundancy r = k*rho/d (Sec. 2.2 remarks: pick a
    valid (k, rho); if none, lower r).  k = round(r*d/rho), decreased until valid."""
    k = int(round(r * d / rho))
    while k >= 1:
        if valid_k_for(rho, d, k):
            return k
        k -= 1
    raise ValueError("no valid k")


def haar_orthogonal(n: int, rng: np.random.Generator) -> np.ndarray:
    """Haar-distributed n x n orthogonal matrix: QR of a Gaussian matrix with the signs of
    R's diagonal moved into Q."""
    if n == 1:
        return np.array([[1.0 if rng.standard_normal() >= 0 else -1.0]])
    G = rng.standard_normal((n, n))
    Q, Rm = np.linalg.qr(G)
    return Q * np.sign(np.diag(Rm))[None, :]


def kron_factors(d: int):
    """Split d = d1 * d2 with d1 <= d2 and d1 as close to sqrt(d) as possible."""
    best = 1
    for a in range(1, int(math.isqrt(d)) + 1):
        if d % a == 0:
            best = a
    return best, d // best


def rotation_factors(d: int, seed_seq) -> tuple[np.ndarray, np.ndarray]:
    """Seeded random rotation R = R1 (x) R2 (Kronecker product of two Haar factors)."""
    d1, d2 = kron_factors(d)
    rng = np.random.default_rng(seed_seq)
    return haar_orthogonal(d1, rng), haar_orthogonal(d2, rng)


def apply_rotation(R1: np.ndarray, R2: np.ndarray, T: np.ndarray) -> np.ndarray:
    """(R1 (x) R2) @ T without forming the Kronecker product: each column t of T is
    reshaped row-major to d1 x d2 and mapped to R1 t R2^T (two large matrix products)."""
    d1, d2 = R1.shape[0], R2.shape[0]
    K = T.shape[1]
    M = np.ascontiguousarray(T.T).reshape(K, d1, d2)
    with _BLAS_LOCK:      # the BLAS is threaded itself and not safe for concurrent callers
        A = np.tensordot(R1, M, axes=([1], [1]))             # (d1, K, d2)
        B = (A.reshape(d1 * K, d2) @ R2.T).reshape(d1, K, d2)
    return np.ascontiguousarray(B.transpose(1, 0, 2).reshape(K, d1 * d2).T)


def parseval_frame(k: int, rho: int, d: int, seed_seq=None, rotate: bool = True,
                   dtype=np.float64) -> np.ndarray:
    """Dense d x (k*rho) Parseval fusion frame P = R T sqrt(d/(k rho)).

    P P^T = I_d; column block i (rho columns) is an orthogonal basis of subspace i scaled
    by its weight w_i = sqrt(d/(k rho)).  Built in float64, a group of subspaces at a
    time (the rotation acts on each column separately), and stored as dtype (float32:
    round-to-nearest of the float64 frame).
    """
    scale = math.sqrt(d / (k * rho))
    if k == 1 and rho == d:
        T = np.eye(d) * scale
        if rotate:
            R1, R2 = rotation_factors(d, seed_seq)
            T = apply_rotation(R1, R2, T)
        return np.asarray(T, dtype=dtype)
    if rotate:
        R1, R2 = rotation_factors(d, seed_seq)
    out = np.empty((d, k * rho), dtype=dtype)
    group = max(1, 2048 // rho)

    def build(s0):
        s1 = min(k, s0 + group)
        T = real_tff_basis(k, rho, d, range(s0, s1)) * scale
        if rotate:
            T = apply_rotation(R1, R2, T)
        out[:, s0 * rho: s1 * rho] = T

    starts = range(0, k, group)
    if len(starts) == 1:
        build(0)
    else:
        with ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(build, starts))
    return out
