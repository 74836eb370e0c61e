"""3- and 4-bit grids on the device (fq_quantize_frames with bits 3 and 4,
fq_frame_synthesis_nbit) against the oracle, under the same bar as the 2-bit pass: codes
bit-exact outside the near-tie window of a teacher-forced replay, scale equal to 2e-7 and
zero exactly; the synthesized weights within 1e-5 relative Frobenius of the oracle's.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import tff
from fq_testutil import need_gpu, rel_fro, replay_rows, check_codes

pytestmark = pytest.mark.gpu


def _ff_problem(rng, K_out, d_in, k_in, rho=4, n=600):
    Pi = tff.parseval_frame(k_in, rho, d_in, np.random.SeedSequence(11))
    X = rng.standard_normal((n, d_in))
    X[:, 3] *= 20.0
    Ht = (Pi.T @ (X.T @ X) @ Pi).astype(np.float32)
    Ht = np.triu(Ht) + np.triu(Ht, 1).T
    D = (rng.standard_normal((K_out, Pi.shape[1])) * 0.02 + 0.001).astype(np.float32)
    big = rng.random(D.shape) < 0.01
    D[big] *= 10
    return D, Ht


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("K_out,d_in,k_in,block", [(70, 64, 18, 128), (300, 136, 37, 7),
                                                   (200, 256, 70, 200)])
def test_quantize_nbit_teacher_forced(bits, K_out, d_in, k_in, block):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(K_out + block + bits)
    D, Ht = _ff_problem(rng, K_out, d_in, k_in)
    K_in = D.shape[1]
    codes = torch.empty((K_out, fq.fq.words_per_row(K_in, bits)), dtype=torch.int32, device="cuda")
    scale = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    zero = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    fq.fq_quantize_frames(torch.from_numpy(D).cuda(), torch.from_numpy(Ht).cuda(), codes, scale,
                          zero, bits=bits, block=block)
    torch.cuda.synchronize()
    cg = O.unpack_bits(codes.cpu().numpy().view(np.uint32), K_in, bits)
    assert cg.max() <= (1 << bits) - 1
    r = replay_rows(D, Ht, cg, bits=bits, block=block)
    assert check_codes(r, cg, scale.cpu().numpy(), zero.cpu().numpy()) <= 2
    # the bits beyond the last code of every row are zero
    w = codes.cpu().numpy().view(np.uint32)
    used = K_in - (w.shape[1] - 1) * (32 // bits)
    if bits * used < 32:
        assert not np.any(w[:, -1] >> np.uint32(bits * used))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_synthesis_nbit(bits):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(30 + bits)
    Po = tff.parseval_frame(55, 4, 200, np.random.SeedSequence(5))
    Pi = tff.parseval_frame(37, 4, 136, np.random.SeedSequence(6))
    K_out, K_in = Po.shape[1], Pi.shape[1]
    codes = rng.integers(0, 1 << bits, size=(K_out, K_in))
    scale = rng.uniform(0.01, 0.1, K_out).astype(np.float32)
    zero = rng.integers(0, 1 << bits, K_out).astype(np.float32)
    words = torch.from_numpy(O.pack_bits(codes, bits).view(np.int32)).cuda()
    Wh = torch.empty((200, 136), dtype=torch.float32, device="cuda")
    fq.fq_frame_synthesis(words, torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda(),
                          torch.from_numpy(Po.astype(np.float32)).cuda(),
                          torch.from_numpy(Pi.astype(np.float32)).cuda(), Wh, bits=bits)
    torch.cuda.synchronize()
    Wo = O.synthesis(codes, scale.astype(np.float64), zero.astype(np.float64),
                     Po.astype(np.float32).astype(np.float64), Pi.astype(np.float32).astype(np.float64))
    assert rel_fro(Wh.cpu().numpy(), Wo) < 1e-5


def test_nbit_rejects_other_widths():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    D = torch.zeros((8, 16), device="cuda")
    Ht = torch.eye(16, device="cuda")
    codes = torch.empty((8, fq.fq.words_per_row(16, 5)), dtype=torch.int32, device="cuda")
    sc = torch.empty(8, device="cuda")
    with pytest.raises(fq.FQError):
        fq.fq_quantize_frames(D, Ht, codes, sc, sc.clone(), bits=5)


def _tff_frame(torch, fq, d, k, rho, seed):
    P = tff.parseval_frame(k, rho, d, np.random.SeedSequence(seed))
    R1, R2 = tff.rotation_factors(d, np.random.SeedSequence(seed))
    return fq.Frame(d, k, rho, torch.from_numpy(R1.astype(np.float32)).cuda(),
                    torch.from_numpy(R2.astype(np.float32)).cuda()), P


@pytest.mark.parametrize("n", [1, 3, 8, 11])
def test_inference_4bit_codes(n):
    """Layer outputs from 4-bit codes (fq_frame_apply and fq_frame_apply_tff with bits 4)
    against the oracle's frame_apply within 1e-5 relative Frobenius, the bar of the 2-bit
    calls.  K_in = 148: a half-filled last word, and a padded U row one word longer than a
    code row."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo, Po = _tff_frame(torch, fq, 200, 55, 4, 5)
    Fi, Pi = _tff_frame(torch, fq, 136, 37, 4, 6)
    rng = np.random.default_rng(40 + n)
    codes = rng.integers(0, 16, size=(Fo.K, Fi.K))
    scale = rng.uniform(0.01, 0.1, Fo.K).astype(np.float32)
    zero = rng.integers(0, 16, Fo.K).astype(np.float32)
    words = torch.from_numpy(O.pack_bits(codes, 4).view(np.int32)).cuda()
    sc, ze = torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda()
    X = rng.standard_normal((n, 136)).astype(np.float32)
    Xd = torch.from_numpy(X).cuda()
    Yo = O.frame_apply(X.astype(np.float64), codes, scale.astype(np.float64),
                       zero.astype(np.float64), Po, Pi)
    Yt = fq.fq_frame_apply_tff(Xd, words, sc, ze, Fo, Fi, bits=4)
    Yd = fq.fq_frame_apply(Xd, words, sc, ze, torch.from_numpy(Po.astype(np.float32)).cuda(),
                           torch.from_numpy(Pi.astype(np.float32)).cuda(), bits=4)
    torch.cuda.synchronize()
    assert rel_fro(Yt.cpu().numpy(), Yo) < 1e-5
    assert rel_fro(Yd.cpu().numpy(), Yo) < 1e-5


def test_inference_rejects_3bit_codes():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo, _ = _tff_frame(torch, fq, 64, 16, 4, 1)
    X = torch.zeros((1, 64), device="cuda")
    words = torch.zeros((64, fq.fq.words_per_row(64, 3)), dtype=torch.int32, device="cuda")
    sc = torch.ones(64, device="cuda")
    with pytest.raises(fq.FQError):
        fq.fq_frame_apply_tff(X, words, sc, sc, Fo, Fo, bits=3)


@pytest.mark.parametrize("n", [1, 8])
def test_inference_4bit_llama7b_up(n):
    """Llama-2-7B up_proj frames, 4-bit codes: the structured and the dense call agree within
    1e-5, and 32 sampled output channels match the oracle within 1e-5 of their norm."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    from fq_inputs import WORKLOADS, gen
    wl = WORKLOADS["llama7b"]
    L = wl.layers[1]
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, 1)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    Fo = fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o))
    Fi = fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i))
    Po, Pi = gen.make_frames(wl, 1)
    rng = np.random.default_rng(7 + n)
    codes = rng.integers(0, 16, size=(Fo.K, Fi.K))
    scale = rng.uniform(0.001, 0.01, Fo.K).astype(np.float32)
    zero = rng.integers(0, 16, Fo.K).astype(np.float32)
    words = torch.from_numpy(O.pack_bits(codes, 4).view(np.int32)).cuda()
    sc, ze = torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda()
    X = rng.standard_normal((n, L.d_in)).astype(np.float32)
    Xd = torch.from_numpy(X).cuda()
    Yt = fq.fq_frame_apply_tff(Xd, words, sc, ze, Fo, Fi, bits=4)
    Yd = fq.fq_frame_apply(Xd, words, sc, ze, up(Po), up(Pi), bits=4)
    torch.cuda.synchronize()
    Ytn, Ydn = Yt.cpu().numpy(), Yd.cpu().numpy()
    assert rel_fro(Ytn, Ydn.astype(np.float64)) < 1e-5
    rows = rng.choice(L.d_out, 32, replace=False)
    U = X.astype(np.float64) @ Pi
    V = U @ ((codes - zero[:, None]) * scale.astype(np.float64)[:, None]).T
    Yo = V @ Po[rows].T
    assert rel_fro(Ytn[:, rows], Yo) < 1e-5
