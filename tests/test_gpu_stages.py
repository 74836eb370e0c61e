"""Device parity of each ABI call against the CPU oracle on small and ragged shapes.

Tolerances (relative Frobenius), derived from the arithmetic:
  * H = X^T X: f16/bf16 products are exact in fp32, partial sums run in fp32 over at most
    one K-split of tokens and are combined in fp64; an fp32 X is split into two bf16 terms
    (three products kept, error <= 3 * 2^-17 per product).  Bound used: 1e-5.
  * D, H~, W^: two chained contractions whose fp32 operands are split into bf16 pairs
    (per-product relative error about 2^-17, uncorrelated across terms).  Bound: 1e-5
    per contraction pair.
  * codes: bit-exact wherever the oracle's pre-rounding value is more than 1e-6 (code
    units) from a rounding boundary (teacher-forced replay on the device's D and H~).
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import tff, gen
from fq_testutil import need_gpu, upload, rel_fro, unpack_codes, replay_rows, check_codes

pytestmark = pytest.mark.gpu


def _fq():
    import paper_2403_06082_amd as fq
    return fq


def _rand_storage(rng, shape, dtype, scale=1.0):
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    return gen.to_device_storage(x, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("n,d", [(77, 100), (512, 256), (1000, 520), (3000, 264), (2048, 264), (4096, 520)])
def test_hessian_parity(dtype, n, d):
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(n * 7 + d)
    Xs = _rand_storage(rng, (n, d), dtype)
    Xs_np = gen.storage_to_f32(Xs, dtype).astype(np.float64)
    X = upload(Xs, dtype)
    H = torch.empty((d, d), dtype=torch.float32, device="cuda")
    fq.fq_hessian_accumulate(X, H)
    torch.cuda.synchronize()
    Hg = H.cpu().numpy().astype(np.float64)
    Ho = O.hessian(Xs_np)
    assert rel_fro(Hg, Ho) < 1e-5
    np.testing.assert_array_equal(Hg, Hg.T)
    # accumulate: H += X^T X
    fq.fq_hessian_accumulate(X, H, accumulate=True)
    torch.cuda.synchronize()
    assert rel_fro(H.cpu().numpy(), 2 * Ho) < 1e-5


def test_hessian_empty_and_strided():
    torch = need_gpu()
    fq = _fq()
    H = torch.full((40, 40), 7.0, dtype=torch.float32, device="cuda")
    X = torch.zeros((0, 40), dtype=torch.bfloat16, device="cuda")
    fq.fq_hessian_accumulate(X, H)
    torch.cuda.synchronize()
    assert float(H.abs().max()) == 0.0
    # a row stride larger than d_in (a column slice of a wider buffer)
    rng = np.random.default_rng(5)
    big = _rand_storage(rng, (300, 72), "bf16")
    Xb = upload(big, "bf16")[:, :64]
    H2 = torch.empty((64, 64), dtype=torch.float32, device="cuda")
    fq.fq_hessian_accumulate(Xb, H2)
    torch.cuda.synchronize()
    Ho = O.hessian(gen.storage_to_f32(big, "bf16")[:, :64].astype(np.float64))
    assert rel_fro(H2.cpu().numpy(), Ho) < 1e-5


def _frames(d_out, d_in, k_out, k_in, rho=4, seed=0):
    Po = tff.parseval_frame(k_out, rho, d_out, np.random.SeedSequence(seed))
    Pi = tff.parseval_frame(k_in, rho, d_in, np.random.SeedSequence(seed + 1))
    return gen.frame_f32(Po), gen.frame_f32(Pi)


@pytest.mark.parametrize("wt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("d_out,d_in,k_out,k_in", [(200, 136, 55, 37), (520, 264, 143, 72)])
def test_analysis_parity(wt, d_out, d_in, k_out, k_in):
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(d_out)
    Po, Pi = _frames(d_out, d_in, k_out, k_in)
    Ws = _rand_storage(rng, (d_out, d_in), wt, 0.02)
    Xs = _rand_storage(rng, (400, d_in), "f32")
    Hn = O.hessian(Xs.astype(np.float64)).astype(np.float32)
    W, P_out, P_in, H = upload(Ws, wt), torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda(), torch.from_numpy(Hn).cuda()
    K_out, K_in = Po.shape[1], Pi.shape[1]
    D = torch.empty((K_out, K_in), dtype=torch.float32, device="cuda")
    Ht = torch.empty((K_in, K_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_analysis(W, P_out, P_in, H, D, Ht)
    torch.cuda.synchronize()
    Do, Hto = O.frame_analysis(gen.storage_to_f32(Ws, wt), Po, Pi, Hn)
    assert rel_fro(D.cpu().numpy(), Do) < 1e-5
    Htg = Ht.cpu().numpy()
    assert rel_fro(Htg, Hto) < 1e-5
    np.testing.assert_array_equal(Htg, Htg.T)


def test_synthesis_parity():
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(3)
    d_out, d_in = 264, 200
    Po, Pi = _frames(d_out, d_in, 72, 55)
    K_out, K_in = Po.shape[1], Pi.shape[1]
    codes = rng.integers(0, 4, size=(K_out, K_in))
    scale = rng.uniform(0.01, 0.1, K_out).astype(np.float32)
    zero = rng.integers(0, 4, K_out).astype(np.float32)
    words = O.pack2(codes)
    Wh = torch.empty((d_out, d_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_synthesis(torch.from_numpy(words.view(np.int32)).cuda(), torch.from_numpy(scale).cuda(),
                          torch.from_numpy(zero).cuda(), torch.from_numpy(Po).cuda(),
                          torch.from_numpy(Pi).cuda(), Wh)
    torch.cuda.synchronize()
    Who = O.synthesis(codes, scale.astype(np.float64), zero.astype(np.float64), Po, Pi)
    assert rel_fro(Wh.cpu().numpy(), Who) < 1e-5


def _ff_problem(rng, K_out, d_in, k_in, rho=4, n=600):
    Pi = tff.parseval_frame(k_in, rho, d_in, np.random.SeedSequence(11))
    X = rng.standard_normal((n, d_in))
    X[:, 3] *= 20.0
    Ht = (Pi.T @ (X.T @ X) @ Pi).astype(np.float32)
    Ht = np.triu(Ht) + np.triu(Ht, 1).T            # exactly symmetric
    D = (rng.standard_normal((K_out, Pi.shape[1])) * 0.02 + 0.001).astype(np.float32)
    big = rng.random(D.shape) < 0.01
    D[big] *= 10
    return D, Ht


def _quantize(torch, fq, D, Ht, block, **kw):
    K_out, K_in = D.shape
    codes = torch.empty((K_out, fq.fq.words_per_row(K_in, kw.get("bits", 2))), dtype=torch.int32,
                        device="cuda")
    scale = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    zero = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    fq.fq_quantize_frames(torch.from_numpy(D).cuda(), torch.from_numpy(Ht).cuda(), codes, scale,
                          zero, block=block, **kw)
    torch.cuda.synchronize()
    w = codes.cpu().numpy().view(np.uint32)
    return O.unpack2(w, K_in), scale.cpu().numpy(), zero.cpu().numpy(), w


@pytest.mark.parametrize("K_out,d_in,k_in,block", [(70, 64, 18, 128), (300, 136, 37, 7),
                                                   (130, 200, 55, 128), (200, 256, 70, 200),
                                                   (64, 96, 25, 1),
                                                   # K_in = 1100: two updates beyond a
                                                   # 512-column span on the LDS-ring
                                                   # kernel (interior and clamped edge
                                                   # column tiles, ragged rows)
                                                   (300, 1024, 275, 128)])
def test_quantize_teacher_forced(K_out, d_in, k_in, block):
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(K_out + block)
    D, Ht = _ff_problem(rng, K_out, d_in, k_in)
    cg, sg, zg, words = _quantize(torch, fq, D, Ht, block)
    r = replay_rows(D, Ht, cg, block=block)
    ties = check_codes(r, cg, sg, zg, words=words)
    assert ties <= 2


def test_quantize_odd_row_length():
    """K_in = 1101: the rows of R have an odd length, so the LDS-ring kernel copies B a
    dword per lane in every column tile."""
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(1101)
    A = rng.standard_normal((600, 1101))
    A[:, 3] *= 20.0
    Ht = (A.T @ A).astype(np.float32)
    Ht = np.triu(Ht) + np.triu(Ht, 1).T            # exactly symmetric
    D = (rng.standard_normal((260, 1101)) * 0.02 + 0.001).astype(np.float32)
    cg, sg, zg, words = _quantize(torch, fq, D, Ht, 128)
    r = replay_rows(D, Ht, cg, block=128)
    assert check_codes(r, cg, sg, zg, words=words) <= 2


def test_quantize_identity_hessian_is_rtn():
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(2)
    D = (rng.standard_normal((90, 77)) * 0.05 + 0.002).astype(np.float32)
    Ht = np.eye(77, dtype=np.float32)
    cg, sg, zg, words = _quantize(torch, fq, D, Ht, 128)
    mu, sigma, lo, hi = O.clip_bounds(D.astype(np.float64))
    Dc = O.apply_clip(D.astype(np.float64), lo, hi)
    s, z = O.row_grid(Dc)
    q, _ = O.rtn_codes(Dc, s[:, None], z[:, None])
    np.testing.assert_array_equal(cg, q)
    # K_in = 77: the last word of every row holds 13 codes and 3 zero pad fields
    np.testing.assert_array_equal(words, O.pack2(q))


def test_quantize_no_clip_and_dead_column():
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(4)
    D, Ht = _ff_problem(rng, 50, 64, 18)
    Ht[5, :] = 0
    Ht[:, 5] = 0
    cg, sg, zg, words = _quantize(torch, fq, D, Ht, 16, clip_sigmas=float("inf"))
    r = replay_rows(D, Ht, cg, block=16, clip_sigmas=float("inf"))
    check_codes(r, cg, sg, zg, words=words)       # K_in = 72: half-filled last words


def test_quantize_errors():
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(6)
    D, Ht = _ff_problem(rng, 40, 64, 18)     # K_in = 72 > rank(Ht) = 64
    with pytest.raises(fq.FQError) as ei:
        _quantize(torch, fq, D, Ht - np.float32(1e-3) * np.eye(72, dtype=np.float32) * Ht.max(), 128, damp=0.0)
    assert ei.value.status == 3
    Dn = D.copy()
    Dn[3, 4] = np.nan
    with pytest.raises(fq.FQError) as ei:
        _quantize(torch, fq, Dn, Ht, 128)
    assert ei.value.status == 4
    with pytest.raises(fq.FQError) as ei:
        _quantize(torch, fq, D, Ht, 128, bits=5)
    assert ei.value.status == 2


@pytest.mark.parametrize("wt", ["bf16", "f32"])
def test_poisoned_workspaces(wt):
    """Every workspace filled with NaN bytes before the call: no output may depend on
    workspace contents the call did not write itself (padding lanes and columns included)."""
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(77)
    d_out, d_in, k_out, k_in = 520, 264, 143, 72     # ragged: fallback and padded paths
    Po, Pi = _frames(d_out, d_in, k_out, k_in)
    K_out, K_in = Po.shape[1], Pi.shape[1]
    Ws = _rand_storage(rng, (d_out, d_in), wt, 0.02)
    Xs = _rand_storage(rng, (300, d_in), wt)
    X = upload(Xs, wt)
    W, P_out, P_in = upload(Ws, wt), torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda()

    def poisoned(nbytes):
        return torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")

    dt = {"bf16": fq.FQ_BF16, "f32": fq.FQ_F32}[wt]
    H = torch.empty((d_in, d_in), dtype=torch.float32, device="cuda")
    fq.fq_hessian_accumulate(X, H, ws=poisoned(fq.fq_hessian_workspace_bytes(dt, 300, d_in)))
    D = torch.empty((K_out, K_in), dtype=torch.float32, device="cuda")
    Ht = torch.empty((K_in, K_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_analysis(W, P_out, P_in, H, D, Ht,
                         ws=poisoned(fq.fq_frame_analysis_workspace_bytes(dt, d_out, d_in, K_out, K_in)))
    codes = torch.empty((K_out, (K_in + 15) // 16), dtype=torch.int32, device="cuda")
    scale = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    zero = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    fq.fq_quantize_frames(D, Ht, codes, scale, zero,
                          ws=poisoned(fq.fq_quantize_frames_workspace_bytes(K_out, K_in, 128)))
    Wh = torch.empty((d_out, d_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_synthesis(codes, scale, zero, P_out, P_in, Wh,
                          ws=poisoned(fq.fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in)))
    torch.cuda.synchronize()
    Ho = O.hessian(gen.storage_to_f32(Xs, wt).astype(np.float64))
    Hg = H.cpu().numpy()
    assert rel_fro(Hg, Ho) < 1e-5
    Do, Hto = O.frame_analysis(gen.storage_to_f32(Ws, wt), Po, Pi, Hg)
    Dg, Htg = D.cpu().numpy(), Ht.cpu().numpy()
    assert rel_fro(Dg, Do) < 1e-5 and rel_fro(Htg, Hto) < 1e-5
    cg = unpack_codes(codes, K_in)
    r = replay_rows(Dg, Htg, cg)
    check_codes(r, cg, scale.cpu().numpy(), zero.cpu().numpy())
    Who = O.synthesis(cg, scale.cpu().numpy().astype(np.float64),
                      zero.cpu().numpy().astype(np.float64), Po, Pi)
    assert rel_fro(Wh.cpu().numpy(), Who) < 1e-5


def _max_tile_rel(A, B, t=256):
    """Largest relative Frobenius error over the 256 x 256 output tiles."""
    worst = 0.0
    for i in range(0, A.shape[0], t):
        for j in range(0, A.shape[1], t):
            worst = max(worst, rel_fro(A[i:i + t, j:j + t], B[i:i + t, j:j + t]))
    return worst


@pytest.mark.parametrize("d_out,d_in,wt", [(1000, 4100, "f32"), (4100, 1000, "bf16")])
def test_short_last_round_products(d_out, d_in, wt):
    """Products with 17 x 17 output tiles leave a last round of 33 tiles on 256 compute
    units; those are computed as K-slices in a scratch area and reduced.  Every tile,
    the reduced ones included, is checked, with NaN-filled workspaces."""
    torch = need_gpu()
    fq = _fq()
    rng = np.random.default_rng(d_out + d_in)
    k = 1050                                     # K_out = K_in = 4200: 17 tiles
    Po, Pi = _frames(d_out, d_in, k, k)
    K_out, K_in = Po.shape[1], Pi.shape[1]
    Ws = _rand_storage(rng, (d_out, d_in), wt, 0.02)
    Xs = _rand_storage(rng, (300, d_in), "f32")
    Hn = O.hessian(Xs.astype(np.float64)).astype(np.float32)
    W, P_out, P_in = upload(Ws, wt), torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda()
    H = torch.from_numpy(Hn).cuda()
    dt = {"bf16": fq.FQ_BF16, "f32": fq.FQ_F32}[wt]

    def poisoned(nbytes):
        return torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")

    D = torch.empty((K_out, K_in), dtype=torch.float32, device="cuda")
    Ht = torch.empty((K_in, K_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_analysis(W, P_out, P_in, H, D, Ht,
                         ws=poisoned(fq.fq_frame_analysis_workspace_bytes(dt, d_out, d_in, K_out, K_in)))
    codes = rng.integers(0, 4, size=(K_out, K_in))
    scale = rng.uniform(0.01, 0.1, K_out).astype(np.float32)
    zero = rng.integers(0, 4, K_out).astype(np.float32)
    Wh = torch.empty((d_out, d_in), dtype=torch.float32, device="cuda")
    fq.fq_frame_synthesis(torch.from_numpy(O.pack2(codes).view(np.int32)).cuda(),
                          torch.from_numpy(scale).cuda(), torch.from_numpy(zero).cuda(), P_out,
                          P_in, Wh,
                          ws=poisoned(fq.fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in)))
    torch.cuda.synchronize()
    Do, Hto = O.frame_analysis(gen.storage_to_f32(Ws, wt), Po, Pi, Hn)
    assert _max_tile_rel(D.cpu().numpy(), Do) < 1e-5
    assert _max_tile_rel(Ht.cpu().numpy(), Hto) < 1e-5
    Who = O.synthesis(codes, scale.astype(np.float64), zero.astype(np.float64), Po, Pi)
    assert _max_tile_rel(Wh.cpu().numpy(), Who) < 1e-5
