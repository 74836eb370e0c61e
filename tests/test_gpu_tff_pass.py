"""The analysis and the synthesis with both frames given by their construction
(fq_frame_analysis_tff, fq_frame_synthesis_tff) against the oracle's D = P_out^T W P_in,
Ht = P_in^T H P_in and W_hat = P_out diag(scale)(Q - zero) P_in^T with the dense float64
frames the input generator builds from the same (k, rho, d) and rotation seed.

Bar: 1e-5 relative Frobenius for D, Ht and W_hat, the bar of the dense entry points.  The
device takes the rotation factors in fp32, rotates with fp32 sums of d1 + d2 terms and
forms the DFT blocks as fp32-accumulated products of bf16 (hi, lo) pairs (relative error
of a pair 2^-17, of the dropped lo x lo term 2^-16 of the product): a few 1e-6 at most.
Shapes cover pads of both block sizes (2m and 2k not multiples of 32), odd d1 / d2, and
the Llama-2-7B up_proj layer at full size, where the structured results are also held to
the dense entry points' and to sampled float64 entries.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import WORKLOADS, gen, tff
from fq_testutil import need_gpu, upload, rel_fro

pytestmark = pytest.mark.gpu

# (d_out, k_out, d_in, k_in, rho)
SHAPES = [(200, 55, 136, 37, 4), (520, 143, 264, 72, 4), (64, 16, 256, 18, 16),
          (264, 72, 200, 55, 4)]


def _frame(torch, fq, d, k, rho, seed):
    P = tff.parseval_frame(k, rho, d, np.random.SeedSequence(seed))
    R1, R2 = tff.rotation_factors(d, np.random.SeedSequence(seed))
    F = fq.Frame(d, k, rho, torch.from_numpy(R1.astype(np.float32)).cuda(),
                 torch.from_numpy(R2.astype(np.float32)).cuda())
    return F, P


def _poisoned(torch, nbytes):
    return torch.full((max(int(nbytes), 256),), 0xFF, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("wt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_analysis_tff_parity(wt, shape):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    d_out, k_out, d_in, k_in, rho = shape
    Fo, Po = _frame(torch, fq, d_out, k_out, rho, 21)
    Fi, Pi = _frame(torch, fq, d_in, k_in, rho, 22)
    rng = np.random.default_rng(d_out + d_in)
    Ws = gen.to_device_storage((rng.standard_normal((d_out, d_in)) * 0.02).astype(np.float32), wt)
    Xs = rng.standard_normal((400, d_in)).astype(np.float32)
    Xs[:, 3] *= 20.0
    Hn = O.hessian(Xs.astype(np.float64)).astype(np.float32)
    D = torch.empty((Fo.K, Fi.K), dtype=torch.float32, device="cuda")
    Ht = torch.empty((Fi.K, Fi.K), dtype=torch.float32, device="cuda")
    dt = {"f32": fq.FQ_F32, "f16": fq.FQ_F16, "bf16": fq.FQ_BF16}[wt]
    ws = _poisoned(torch, fq.fq_frame_analysis_tff_workspace_bytes(dt, Fo, Fi))
    fq.fq_frame_analysis_tff(upload(Ws, wt), Fo, Fi, torch.from_numpy(Hn).cuda(), D, Ht, ws=ws)
    torch.cuda.synchronize()
    Do, Hto = O.frame_analysis(gen.storage_to_f32(Ws, wt), Po, Pi, Hn)
    assert rel_fro(D.cpu().numpy(), Do) < 1e-5
    Htg = Ht.cpu().numpy()
    assert rel_fro(Htg, Hto) < 1e-5
    np.testing.assert_array_equal(Htg, Htg.T)


def test_analysis_tff_one_output_at_a_time():
    """D alone (H NULL) and Ht alone (W NULL) give the results of the joint call."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo, _ = _frame(torch, fq, 200, 55, 4, 31)
    Fi, _ = _frame(torch, fq, 136, 37, 4, 32)
    rng = np.random.default_rng(33)
    W = torch.from_numpy(rng.standard_normal((200, 136)).astype(np.float32)).cuda()
    A = rng.standard_normal((300, 136))
    H = torch.from_numpy((A.T @ A).astype(np.float32)).cuda()
    D1, Ht1 = fq.fq_frame_analysis_tff(W, Fo, Fi, H,
                                       torch.empty((Fo.K, Fi.K), device="cuda"),
                                       torch.empty((Fi.K, Fi.K), device="cuda"))
    D2, _ = fq.fq_frame_analysis_tff(W, Fo, Fi, None, torch.empty((Fo.K, Fi.K), device="cuda"))
    _, Ht2 = fq.fq_frame_analysis_tff(None, Fo, Fi, H, None, torch.empty((Fi.K, Fi.K), device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(D1, D2) and torch.equal(Ht1, Ht2)


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("shape", SHAPES)
def test_synthesis_tff_parity(bits, shape):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    d_out, k_out, d_in, k_in, rho = shape
    Fo, Po = _frame(torch, fq, d_out, k_out, rho, 41)
    Fi, Pi = _frame(torch, fq, d_in, k_in, rho, 42)
    rng = np.random.default_rng(10 * bits + d_out)
    codes = rng.integers(0, 1 << bits, size=(Fo.K, Fi.K))
    scale = rng.uniform(0.01, 0.1, Fo.K).astype(np.float32)
    zero = rng.integers(0, 1 << bits, Fo.K).astype(np.float32)
    words = torch.from_numpy(O.pack_bits(codes, bits).view(np.int32)).cuda()
    ws = _poisoned(torch, fq.fq_frame_synthesis_tff_workspace_bytes(Fo, Fi))
    Wh = fq.fq_frame_synthesis_tff(words, torch.from_numpy(scale).cuda(),
                                   torch.from_numpy(zero).cuda(), Fo, Fi, ws=ws, bits=bits)
    torch.cuda.synchronize()
    Wo = O.synthesis(codes, scale.astype(np.float64), zero.astype(np.float64), Po, Pi)
    assert Wh.shape == (d_out, d_in)
    assert rel_fro(Wh.cpu().numpy(), Wo) < 1e-5


def test_tff_pass_llama7b_up_full_size():
    """Llama-2-7B up_proj (d_out 11008, d_in 4096, K_out 12112, K_in 4512), bf16 weights: the
    structured D, Ht and W_hat against the dense entry points with the fp32 frames (1e-5
    relative Frobenius) and 64 sampled entries of D and of W_hat against float64 sums."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    wl = WORKLOADS["llama7b"]
    li = 1
    L = wl.layers[li]
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, li)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    Fo = fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o))
    Fi = fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i))
    Po, Pi = gen.make_frames(wl, li)
    rng = np.random.default_rng(77)
    Wn = (rng.standard_normal((L.d_out, L.d_in)) * 0.02).astype(np.float32)
    Ws = gen.to_device_storage(Wn, "bf16")
    W = upload(Ws, "bf16")
    A = rng.standard_normal((2048, L.d_in)).astype(np.float32)
    H = torch.from_numpy(A.T @ A).cuda()
    Dt = torch.empty((Fo.K, Fi.K), device="cuda")
    Htt = torch.empty((Fi.K, Fi.K), device="cuda")
    fq.fq_frame_analysis_tff(W, Fo, Fi, H, Dt, Htt)
    P_out, P_in = up(Po), up(Pi)
    Dd = torch.empty_like(Dt)
    Htd = torch.empty_like(Htt)
    fq.fq_frame_analysis(W, P_out, P_in, H, Dd, Htd)
    torch.cuda.synchronize()
    rel = lambda a, b: float(torch.linalg.norm((a - b).double()) / torch.linalg.norm(b.double()))
    assert rel(Dt, Dd) < 1e-5
    assert rel(Htt, Htd) < 1e-5
    # sampled entries of D in float64 from the float64 frames
    Wf = gen.storage_to_f32(Ws, "bf16").astype(np.float64)
    ii = rng.integers(0, Fo.K, 64)
    jj = rng.integers(0, Fi.K, 64)
    ref = np.einsum("ij,ij->j", Po[:, ii], Wf @ Pi[:, jj])
    got = Dt.cpu().numpy()[ii, jj]
    scale_d = float(torch.linalg.norm(Dd.double())) / np.sqrt(Fo.K * Fi.K)
    assert np.max(np.abs(got - ref)) < 1e-4 * scale_d
    del Dd, Htd, Htt, H, A
    # synthesis from random 2-bit codes
    codes = rng.integers(0, 4, size=(Fo.K, Fi.K))
    scale = rng.uniform(0.01, 0.1, Fo.K).astype(np.float32)
    zero = rng.integers(0, 4, Fo.K).astype(np.float32)
    words = torch.from_numpy(O.pack_bits(codes, 2).view(np.int32)).cuda()
    sc, ze = torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda()
    Wt = fq.fq_frame_synthesis_tff(words, sc, ze, Fo, Fi)
    Wd = torch.empty_like(Wt)
    fq.fq_frame_synthesis(words, sc, ze, P_out, P_in, Wd)
    torch.cuda.synchronize()
    assert rel(Wt, Wd) < 1e-5
    ri_ = rng.integers(0, L.d_out, 64)
    ci_ = rng.integers(0, L.d_in, 64)
    N = (codes - zero[:, None]) * scale.astype(np.float64)[:, None]
    ref_w = np.einsum("ij,ij->j", Po[ri_, :].T, N @ Pi[ci_, :].T)
    got_w = Wt.cpu().numpy()[ri_, ci_]
    scale_w = float(torch.linalg.norm(Wd.double())) / np.sqrt(L.d_out * L.d_in)
    assert np.max(np.abs(got_w - ref_w)) < 1e-4 * scale_w


@pytest.mark.parametrize("two_streams", [False, True])
def test_pipeline_with_structured_frames(two_streams):
    """The whole pass with frames given by their construction: D and Ht against the oracle,
    the codes replayed row by row on the device's own D and Ht (bit-exact outside the
    near-tie window), W_hat against the oracle's synthesis of the device's codes."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    from fq_testutil import replay_rows, check_codes, unpack_codes
    d_out, d_in = 520, 264
    Fo, Po = _frame(torch, fq, d_out, 143, 4, 51)
    Fi, Pi = _frame(torch, fq, d_in, 72, 4, 52)
    rng = np.random.default_rng(53)
    Wn = (rng.standard_normal((d_out, d_in)) * 0.02).astype(np.float32)
    Xn = rng.standard_normal((700, d_in)).astype(np.float32)
    Xn[:, 5] *= 30.0
    W, X = torch.from_numpy(Wn).cuda(), torch.from_numpy(Xn).cuda()
    b = LayerBuffers(d_out, d_in, Fo.K, Fi.K, torch.float32, torch.float32, 700,
                     frames=(Fo, Fi))
    side = torch.cuda.Stream() if two_streams else None
    quantize_layer(W, X, None, None, b, side_stream=side)
    torch.cuda.synchronize()
    Hg = b.H.cpu().numpy()
    Do, Hto = O.frame_analysis(Wn, Po, Pi, Hg)
    Dg, Htg = b.D.cpu().numpy(), b.Ht.cpu().numpy()
    assert rel_fro(Dg, Do) < 1e-5 and rel_fro(Htg, Hto) < 1e-5
    cg = unpack_codes(b.codes, Fi.K)
    r = replay_rows(Dg, Htg, cg)
    check_codes(r, cg, b.scale.cpu().numpy(), b.zero.cpu().numpy(), words=b.codes.cpu().numpy())
    Who = O.synthesis(cg, b.scale.cpu().numpy().astype(np.float64),
                      b.zero.cpu().numpy().astype(np.float64), Po, Pi)
    assert rel_fro(b.W_hat.cpu().numpy(), Who) < 1e-5
