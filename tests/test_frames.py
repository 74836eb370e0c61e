"""Pins for the frame inputs (tight fusion frames) against values the paper prints."""
import json
import math
import os

import numpy as np
import pytest

from fq_inputs import tff, WORKLOADS, frame_k

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_t_block_identity():
    for x in (0.25, 0.5, 0.75, 1.0, 1.5, 1.9):
        T = tff.t_block(x)
        np.testing.assert_allclose(T @ T.T, np.diag([x, 2 - x]), atol=1e-15)


def test_spectral_tetris_5_4_11_matches_printed_F():
    g = _load("tff_5_4_11.json")
    v = np.array(g["F_sq8_signed"], dtype=np.float64)
    F_gold = np.sign(v) * np.sqrt(np.abs(v) / 8.0)
    F = tff.spectral_tetris(4, 11)
    np.testing.assert_allclose(F, F_gold, atol=1e-15)
    # unit-norm columns, orthogonal rows of squared norm 11/4
    np.testing.assert_allclose((F ** 2).sum(axis=0), np.ones(11), atol=1e-14)
    np.testing.assert_allclose(F @ F.T, (11 / 4) * np.eye(4), atol=1e-14)


def test_modulated_5_4_11_table():
    g = _load("tff_5_4_11.json")
    F = tff.spectral_tetris(4, 11)
    B = tff.complex_tff(5, 4, 11) * math.sqrt(11 / 4)        # un-normalised rows of F * w^(j s)
    w = np.exp(2j * np.pi / 5)
    for key, (c0, exps) in g["modulated_exponents"]["rows"].items():
        row = int(key)
        r, s = divmod(row, 5)
        vec = B[s][:, r]                                      # subspace s, basis vector r
        nz = np.flatnonzero(np.abs(vec) > 1e-12)
        assert nz[0] == c0 and len(nz) == len(exps)
        expect = F[r, nz] * w ** np.array(exps)
        np.testing.assert_allclose(vec[nz], expect, atol=1e-13)
    # tight: sum_s B_s B_s^* = (k rho / d) I
    Bn = tff.complex_tff(5, 4, 11)
    S = sum(Bs @ Bs.conj().T for Bs in Bn)
    np.testing.assert_allclose(S, (20 / 11) * np.eye(11), atol=1e-13)


def test_example1_frame_coefficients_projections():
    g = _load("example1.json")
    P = tff.parseval_frame(3, 2, 4, rotate=False)             # 4 x 6, Parseval
    x = np.array(g["x"])
    blocks = [P[:, 2 * i:2 * i + 2] for i in range(3)]
    order = [0, 2, 1]                                        # printed subspace i <- s = order[i]
    for i, s in enumerate(order):
        Pi = blocks[s]
        printed = np.array(g["synthesis_blocks"][i])
        # printed values are truncated (not rounded) to 2 decimals
        assert np.all(np.abs(Pi - printed) < 0.01)
        assert np.all(np.abs(printed) <= np.abs(Pi) + 1e-12)
        c = Pi.T @ x
        cp = np.array(g["coefficients"][i])
        assert np.all(np.abs(c - cp) < 0.01) and np.all(np.abs(cp) <= np.abs(c) + 1e-12)
        proj = Pi @ c
        np.testing.assert_allclose(proj, g["projections"][i], atol=5e-5)
    # Parseval: the projections sum back to x
    np.testing.assert_allclose(P @ (P.T @ x), x, atol=1e-14)
    np.testing.assert_allclose(P @ P.T, np.eye(4), atol=1e-14)


FRAME_DIMS = sorted({(d, frame_k(wl, d)) for wl in WORKLOADS.values()
                     for L in wl.layers for d in (L.d_out, L.d_in) if d <= 4096})


@pytest.mark.parametrize("d,k", FRAME_DIMS)
def test_tff_identity_workload_frames(d, k):
    rho = 16
    T = tff.real_tff_basis(k, rho, d)
    # each subspace basis is orthonormal, and sum_i T_i T_i^T = (k rho / d) I
    for i in range(0, k, max(1, k // 7)):
        Ti = T[:, i * rho:(i + 1) * rho]
        np.testing.assert_allclose(Ti.T @ Ti, np.eye(rho), atol=1e-12)
    np.testing.assert_allclose(T @ T.T, (k * rho / d) * np.eye(d), atol=1e-11)
    P = tff.parseval_frame(k, rho, d, np.random.SeedSequence(5))
    np.testing.assert_allclose(P @ P.T, np.eye(d), atol=1e-11)


def test_invalid_triple_rejected():
    # (k=16, rho=18, d=256): the complex (16, 9, 128) spectral tetris has a row whose
    # support spans more than 16 columns, so the modulation is not tight.
    assert not tff.valid_k_for(18, 256, 16)
    assert tff.valid_k_for(16, 256, 18)


def test_noise_robustness_redundancy():
    """Sec. 2.1, Example 1 epilogue: with white noise on the FF coefficients at 10 dB,
    reconstruction MSE falls by 33% at r = 1.5 and 50% at r = 2 (MSE ~ 1/r for Parseval
    frames)."""
    rng = np.random.default_rng(3)
    d, rho = 16, 4
    mse = {}
    for k in (4, 6, 8):                       # r = 1, 1.5, 2
        P = tff.parseval_frame(k, rho, d, np.random.SeedSequence(k))
        K = P.shape[1]
        X = rng.standard_normal((20000, d))
        C = X @ P
        sig_pow = (C ** 2).mean()
        noise = rng.standard_normal(C.shape) * math.sqrt(sig_pow / 10.0)
        Xr = (C + noise) @ P.T
        mse[K / d] = ((Xr - X) ** 2).mean()
    assert abs(1 - mse[1.5] / mse[1.0] - 1 / 3) < 0.03
    assert abs(1 - mse[2.0] / mse[1.0] - 1 / 2) < 0.03
