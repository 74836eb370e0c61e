"""Rotation factors drawn on the device from a seed (fq_tff_rotation_factors) against the
oracle's seeded_haar (Philox4x32-10, Box-Muller, positive-diagonal QR; the oracle's
generator is pinned to the published known-answer vectors).

Bar: every entry within 1e-6 of the oracle's float64 factor. The device rounds fp64 to
fp32 (relative 2^-24 on entries below 1). The two QRs differ by rounding order only, a
few 1e-15 on these sizes, because the positive-diagonal QR is unique. Orthogonality of the
device factors is checked to 1e-5. A frame generated on the device from the seeded factors
is checked against the dense frame the input generator builds from the oracle's factors.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import tff
from fq_testutil import need_gpu, rel_fro

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("d1,d2", [(1, 5), (8, 17), (16, 16), (64, 64), (86, 128), (128, 224)])
@pytest.mark.parametrize("seed", [0, 2 ** 40 + 12345])
def test_seeded_factors_match_oracle(d1, d2, seed):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    R1, R2 = fq.fq_tff_rotation_factors(seed, d1, d2)
    torch.cuda.synchronize()
    for R, f, n in ((R1, 0, d1), (R2, 1, d2)):
        Rg = R.cpu().numpy().astype(np.float64)
        Ro = O.seeded_haar(seed, f, n)
        assert np.max(np.abs(Rg - Ro)) < 1e-6
        np.testing.assert_allclose(Rg.T @ Rg, np.eye(n), atol=1e-5)


def test_seeded_factors_repeat_and_reuse_workspace():
    """Two calls on one workspace give identical factors; another seed gives others."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    ws = torch.full((fq.fq_tff_rotation_factors_workspace_bytes(86, 128),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    a1, a2 = fq.fq_tff_rotation_factors(5, 86, 128, ws=ws)
    b1, b2 = fq.fq_tff_rotation_factors(5, 86, 128, ws=ws)
    c1, _ = fq.fq_tff_rotation_factors(6, 86, 128, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(a1, b1) and torch.equal(a2, b2)
    assert not torch.equal(a1, c1)


@pytest.mark.parametrize("d,k,rho", [(200, 55, 4), (256, 18, 16)])
def test_frame_from_seed(d, k, rho):
    """fq_tff_materialize with the seeded factors equals the dense frame built from the
    oracle's factors and the unrotated construction, within 1e-5 relative Frobenius."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    d1, d2 = tff.kron_factors(d)
    seed = 99
    R1, R2 = fq.fq_tff_rotation_factors(seed, d1, d2)
    F = fq.Frame(d, k, rho, R1, R2)
    P = fq.fq_tff_materialize(F)
    torch.cuda.synchronize()
    T = tff.parseval_frame(k, rho, d, rotate=False)
    Po = tff.apply_rotation(O.seeded_haar(seed, 0, d1), O.seeded_haar(seed, 1, d2), T)
    assert rel_fro(P.cpu().numpy(), Po) < 1e-5


def test_pass_with_frames_from_seed():
    """The whole pass with both frames regenerated from (d, r, rho, seed) alone
    (fq.Frame.from_seed: fq_tff_choose, then fq_tff_rotation_factors): D and H~ against the
    oracle's products with the dense frames built from the oracle's own seeded factors, the
    codes replayed row by row on the device's D and H~, W^ against the oracle's synthesis
    of the device's codes."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    from fq_testutil import replay_rows, check_codes, unpack_codes
    d_out, d_in, r, rho, seed = 520, 264, 1.1, 4, 2 ** 33 + 7
    Fo = fq.Frame.from_seed(d_out, r, rho, seed)
    Fi = fq.Frame.from_seed(d_in, r, rho, seed + 1)
    torch.cuda.synchronize()

    def dense(F, s):
        d1, d2 = F.R1.shape[0], F.R2.shape[0]
        T = tff.parseval_frame(F.k, F.rho, F.d, rotate=False)
        return tff.apply_rotation(O.seeded_haar(s, 0, d1), O.seeded_haar(s, 1, d2), T)

    assert (Fo.k, Fi.k) == (O.tff_choose_k(d_out, r, rho), O.tff_choose_k(d_in, r, rho)) == (143, 73)
    Po, Pi = dense(Fo, seed), dense(Fi, seed + 1)
    rng = np.random.default_rng(61)
    Wn = (rng.standard_normal((d_out, d_in)) * 0.02).astype(np.float32)
    Xn = rng.standard_normal((900, d_in)).astype(np.float32)
    Xn[:, 7] *= 30.0
    W, X = torch.from_numpy(Wn).cuda(), torch.from_numpy(Xn).cuda()
    b = LayerBuffers(d_out, d_in, Fo.K, Fi.K, torch.float32, torch.float32, 900, frames=(Fo, Fi))
    quantize_layer(W, X, None, None, b, side_stream=torch.cuda.Stream())
    torch.cuda.synchronize()
    Do, Hto = O.frame_analysis(Wn, Po, Pi, b.H.cpu().numpy())
    Dg, Htg = b.D.cpu().numpy(), b.Ht.cpu().numpy()
    assert rel_fro(Dg, Do) < 1e-5 and rel_fro(Htg, Hto) < 1e-5
    cg = unpack_codes(b.codes, Fi.K)
    r_ = replay_rows(Dg, Htg, cg)
    check_codes(r_, cg, b.scale.cpu().numpy(), b.zero.cpu().numpy(), words=b.codes.cpu().numpy())
    Who = O.synthesis(cg, b.scale.cpu().numpy().astype(np.float64),
                      b.zero.cpu().numpy().astype(np.float64), Po, Pi)
    assert rel_fro(b.W_hat.cpu().numpy(), Who) < 1e-5
