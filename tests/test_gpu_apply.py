"""Layer outputs from the codes and the frames (fq_frame_apply) against the oracle's
Y = X Theta^T.

Tolerance (relative Frobenius): every step is an fp32 dot product with fp32 accumulation
(d_in, K_in and K_out terms), the partial sums over d_in are combined in fp64; the
products are exact up to one rounding each.  Small shapes: 1e-5; the Llama-7B up_proj
shape (K_out = 12112 terms in the last step): 1e-4, the bound the layer outputs of the
pass are held to.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import WORKLOADS, gen, tff
from fq_testutil import need_gpu, upload, rel_fro

pytestmark = pytest.mark.gpu


def _problem(rng, d_out, d_in, k_out, k_in, rho=4):
    Po = gen.frame_f32(tff.parseval_frame(k_out, rho, d_out, np.random.SeedSequence(5)))
    Pi = gen.frame_f32(tff.parseval_frame(k_in, rho, d_in, np.random.SeedSequence(6)))
    K_out, K_in = Po.shape[1], Pi.shape[1]
    codes = rng.integers(0, 4, size=(K_out, K_in))
    scale = rng.uniform(0.01, 0.1, K_out).astype(np.float32)
    zero = rng.integers(0, 4, K_out).astype(np.float32)
    return Po, Pi, codes, scale, zero


def _apply(torch, fq, Xs, xdt, codes, scale, zero, Po, Pi, ws=None):
    X = upload(Xs, xdt)
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    Y = fq.fq_frame_apply(X, words, torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda(),
                          torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda(), ws=ws)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


@pytest.mark.parametrize("xdt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("n", [1, 3, 8, 11])
def test_frame_apply_parity(xdt, n):
    """Ragged shapes (K_in = 148, K_out = 220: partial code words, unaligned rows), every
    token-block size, and 11 tokens (two blocks)."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(n * 13 + len(xdt))
    Po, Pi, codes, scale, zero = _problem(rng, 200, 136, 55, 37)
    Xs = gen.to_device_storage(rng.standard_normal((n, 136)).astype(np.float32), xdt)
    Yg = _apply(torch, fq, Xs, xdt, codes, scale, zero, Po, Pi)
    Yo = O.frame_apply(gen.storage_to_f32(Xs, xdt), codes, scale.astype(np.float64),
                       zero.astype(np.float64), Po, Pi)
    assert Yg.shape == (n, 200)
    assert rel_fro(Yg, Yo) < 1e-5


def test_frame_apply_strided_and_poisoned_workspace():
    """X as a column slice of a wider buffer; the workspace filled with NaN bytes."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(41)
    Po, Pi, codes, scale, zero = _problem(rng, 264, 200, 72, 55)
    wide = rng.standard_normal((5, 232)).astype(np.float32)
    X = torch.from_numpy(wide).cuda()[:, :200]
    ws = torch.full((fq.fq_frame_apply_workspace_bytes(200, Po.shape[1], Pi.shape[1]),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    Y = fq.fq_frame_apply(X, words, torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda(),
                          torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda(), ws=ws)
    torch.cuda.synchronize()
    Yo = O.frame_apply(wide[:, :200].astype(np.float64), codes, scale.astype(np.float64),
                       zero.astype(np.float64), Po, Pi)
    assert rel_fro(Y.cpu().numpy(), Yo) < 1e-5


def test_frame_apply_matches_synthesis():
    """Same outputs as forming Theta^ with fq_frame_synthesis and multiplying."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(42)
    Po, Pi, codes, scale, zero = _problem(rng, 520, 264, 143, 72)
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    sc, ze = torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda()
    P_out, P_in = torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda()
    Wh = torch.empty((520, 264), dtype=torch.float32, device="cuda")
    fq.fq_frame_synthesis(words, sc, ze, P_out, P_in, Wh)
    X = torch.from_numpy(rng.standard_normal((6, 264)).astype(np.float32)).cuda()
    Y = fq.fq_frame_apply(X, words, sc, ze, P_out, P_in)
    torch.cuda.synchronize()
    Yw = X.double().cpu() @ Wh.double().cpu().T
    assert rel_fro(Y.cpu().numpy(), Yw.numpy()) < 1e-5


def test_frame_apply_empty_and_errors():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(43)
    Po, Pi, codes, scale, zero = _problem(rng, 40, 24, 12, 8)
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    sc, ze = torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda()
    P_out, P_in = torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda()
    X = torch.zeros((0, 24), dtype=torch.float32, device="cuda")
    assert fq.fq_frame_apply(X, words, sc, ze, P_out, P_in).shape == (0, 40)
    with pytest.raises(ValueError):
        fq.fq_frame_apply(torch.zeros((2, 23), device="cuda"), words, sc, ze, P_out, P_in)


@pytest.mark.parametrize("n", [1, 8])
def test_frame_apply_llama7b_up_sampled(n):
    """The Llama-2-7B up_proj shape (d_out 11008, d_in 4096, K 12112 x 4512) in the launch
    configuration the benchmark times; 64 sampled output channels against the oracle's
    definition (Theta^ restricted to those rows of P_out)."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    wl = WORKLOADS["llama7b"]
    Po, Pi = gen.make_frames(wl, 1, np.float32)
    rng = np.random.default_rng(44 + n)
    K_out, K_in = Po.shape[1], Pi.shape[1]
    codes = rng.integers(0, 4, size=(K_out, K_in))
    scale = rng.uniform(0.01, 0.1, K_out).astype(np.float32)
    zero = rng.integers(0, 4, K_out).astype(np.float32)
    Xs = gen.to_device_storage(rng.standard_normal((n, Pi.shape[0])).astype(np.float32), "bf16")
    Yg = _apply(torch, fq, Xs, "bf16", codes, scale, zero, Po, Pi)
    rows = np.sort(rng.choice(Po.shape[0], 64, replace=False))
    Yo = O.frame_apply(gen.storage_to_f32(Xs, "bf16"), codes, scale.astype(np.float64),
                       zero.astype(np.float64), Po[rows], Pi)
    assert Yg.shape == (n, Po.shape[0])
    assert rel_fro(Yg[:, rows], Yo) < 1e-4
    assert np.isfinite(Yg).all()
