"""Rounded activations on the device (fq_act_quantize, fq_frame_apply_tff_actq) against
the oracle.

The rounding decisions are compared bit for bit: the oracle takes them in float32 on the
device's own U (the analysis output, which fq_tff_analysis reproduces exactly), as the
device does.  The layer outputs then differ only by the float32 synthesis and final scaling
(the integer products are exact): relative Frobenius <= 1e-5, 1e-4 at the Llama-7B up_proj
shape.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import WORKLOADS, gen, tff
from fq_testutil import need_gpu, upload, rel_fro

pytestmark = pytest.mark.gpu


def _frame(torch, fq, d, k, rho, seed):
    P = tff.parseval_frame(k, rho, d, np.random.SeedSequence(seed))
    R1, R2 = tff.rotation_factors(d, np.random.SeedSequence(seed))
    F = fq.Frame(d, k, rho, torch.from_numpy(R1.astype(np.float32)).cuda(),
                 torch.from_numpy(R2.astype(np.float32)).cuda())
    return F, P


@pytest.mark.parametrize("bits", [8, 6, 2])
def test_act_quantize_bit_exact(bits):
    """Random rows, a zero row, a row of exact ties (multiples of Delta/2 with Delta = 1)
    and a ragged width."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(bits)
    qmax = 2 ** (bits - 1) - 1
    U = rng.standard_normal((7, 301)).astype(np.float32) * rng.uniform(0.01, 100, (7, 1)).astype(np.float32)
    U[2] = 0.0
    U[4] = (rng.integers(-2 * qmax, 2 * qmax + 1, 301) / 2.0).astype(np.float32)
    U[4, 0] = qmax
    Cq, d = fq.fq_act_quantize(torch.from_numpy(U).cuda(), bits)
    torch.cuda.synchronize()
    Co, do = O.activation_rtn(U, bits)
    np.testing.assert_array_equal(d.cpu().numpy(), do)
    np.testing.assert_array_equal(Cq.cpu().numpy().astype(np.int64), Co)


@pytest.mark.parametrize("cbits,bits", [(2, 8), (2, 6), (4, 4), (4, 8)])
@pytest.mark.parametrize("xdt", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 3, 8, 11])
def test_frame_apply_tff_actq_parity(cbits, bits, xdt, n):
    """2-bit codes with 8- and 6-bit activations, 4-bit codes with 4- and 8-bit activations
    (the appendix's W4/A4); K_in = 148 (partial code words for both widths)."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo, Po = _frame(torch, fq, 200, 55, 4, 5)
    Fi, _ = _frame(torch, fq, 136, 37, 4, 6)
    rng = np.random.default_rng(3 * n + bits + len(xdt) + 7 * cbits)
    codes = rng.integers(0, 1 << cbits, size=(220, 148))
    scale = rng.uniform(0.01, 0.1, 220).astype(np.float32)
    zero = rng.integers(0, 1 << cbits, 220).astype(np.float32)
    Xs = gen.to_device_storage(rng.standard_normal((n, 136)).astype(np.float32), xdt)
    X = upload(Xs, xdt)
    ws = torch.full((fq.fq_frame_apply_tff_actq_workspace_bytes(Fo, Fi),), 0xFF, dtype=torch.uint8,
                    device="cuda")
    words = torch.from_numpy(O.pack_bits(codes, cbits).view(np.int32)).cuda()
    Y = fq.fq_frame_apply_tff_actq(X, words, torch.from_numpy(scale).cuda(),
                                   torch.from_numpy(zero).cuda(), Fo, Fi, bits, ws=ws, bits=cbits)
    U = fq.fq_tff_analysis(X, Fi)
    torch.cuda.synchronize()
    Yo = O.frame_apply_rtn_activations(U.cpu().numpy(), codes, scale.astype(np.float64),
                                       zero.astype(np.float64), Po, bits)
    assert rel_fro(Y.cpu().numpy(), Yo) < 1e-5


def test_frame_apply_tff_actq_empty_and_errors():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo, _ = _frame(torch, fq, 64, 16, 4, 1)
    Fi, _ = _frame(torch, fq, 64, 16, 4, 2)
    words = torch.zeros((64, 4), dtype=torch.int32, device="cuda")
    sc = torch.ones(64, device="cuda")
    assert fq.fq_frame_apply_tff_actq(torch.zeros((0, 64), device="cuda"), words, sc, sc, Fo, Fi).shape == (0, 64)
    with pytest.raises(fq.FQError):
        fq.fq_frame_apply_tff_actq(torch.zeros((1, 64), device="cuda"), words, sc, sc, Fo, Fi, 9)
    Y = fq.fq_frame_apply_tff_actq(torch.zeros((2, 64), device="cuda"), words, sc, sc, Fo, Fi)
    torch.cuda.synchronize()
    assert float(Y.abs().max()) == 0.0          # a zero input rounds to a zero row


@pytest.mark.parametrize("n", [1, 8])
def test_frame_apply_tff_actq_llama7b_up_sampled(n):
    """The Llama-2-7B up_proj frames at 8-bit activations, in the benchmark's launch
    configuration, on 64 sampled output channels."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    wl = WORKLOADS["llama7b"]
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, 1)
    Fo = fq.Frame(11008, ko, ro, torch.from_numpy(R1o.astype(np.float32)).cuda(),
                  torch.from_numpy(R2o.astype(np.float32)).cuda())
    Fi = fq.Frame(4096, ki, ri, torch.from_numpy(R1i.astype(np.float32)).cuda(),
                  torch.from_numpy(R2i.astype(np.float32)).cuda())
    Po, _ = gen.make_frames(wl, 1)
    rng = np.random.default_rng(70 + n)
    codes = rng.integers(0, 4, size=(Fo.K, Fi.K))
    scale = rng.uniform(0.01, 0.1, Fo.K).astype(np.float32)
    zero = rng.integers(0, 4, Fo.K).astype(np.float32)
    X = upload(gen.to_device_storage(rng.standard_normal((n, 4096)).astype(np.float32), "bf16"), "bf16")
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    Y = fq.fq_frame_apply_tff_actq(X, words, torch.from_numpy(scale).cuda(),
                                   torch.from_numpy(zero).cuda(), Fo, Fi, 8)
    U = fq.fq_tff_analysis(X, Fi)
    torch.cuda.synchronize()
    rows = np.sort(rng.choice(11008, 64, replace=False))
    Yo = O.frame_apply_rtn_activations(U.cpu().numpy(), codes, scale.astype(np.float64),
                                       zero.astype(np.float64), Po[rows], 8)
    Yg = Y.cpu().numpy()
    assert rel_fro(Yg[:, rows], Yo) < 1e-4
    assert np.isfinite(Yg).all()
