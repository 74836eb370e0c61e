"""Diagonal Wiener filter at synthesis (fq_wiener_gains) against the oracle's
wiener_row_gains on the same D, H~ and codes.

Tolerance: the gains are ratios of two row sums of D^ H~ products; on the device D^ H~ runs
on bf16 MFMA with the codes exact and H~ as a bf16 pair (relative error about 2^-17 per
entry, uncorrelated across the sum) and fp32 accumulation, the row sums in fp64.  Both
sums carry a relative error of a few 1e-6, so each gain is held to 2e-5 relative; the
filtered scale to that plus the fp32 rounding of the product.
"""
import numpy as np
import pytest

import oracle as O
from fq_inputs import WORKLOADS, gen, tff
from fq_testutil import need_gpu

pytestmark = pytest.mark.gpu


def _problem(rng, K_out, d_in, K_in, bits):
    """D (K_out x K_in), a singular frame-space H~ (rank d_in < K_in), random codes of
    `bits` bits with random per-row scale and zero; row 3 dequantizes to zero."""
    k = K_in // 4
    P = tff.parseval_frame(k, 4, d_in, np.random.SeedSequence(K_in))
    X = rng.standard_normal((3 * d_in, d_in))
    X[:, 1] *= 20.0
    Ht = (P.T @ (X.T @ X) @ P).astype(np.float32)
    Ht = np.triu(Ht) + np.triu(Ht, 1).T                    # exactly symmetric
    maxq = 2 ** bits - 1
    codes = rng.integers(0, maxq + 1, size=(K_out, K_in))
    zero = rng.integers(0, maxq + 1, K_out).astype(np.float32)
    codes[3] = zero[3]
    scale = rng.uniform(0.01, 0.05, K_out).astype(np.float32)
    Dh = O.dequant(codes, scale.astype(np.float64), zero.astype(np.float64))
    D = (Dh + rng.standard_normal(Dh.shape) * 0.3 * scale[:, None]).astype(np.float32)
    return D, Ht, codes, scale, zero


def _run(torch, fq, D, Ht, codes, scale, zero, bits, alias=False):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    words = t(O.pack_bits(codes, bits).view(np.int32))
    sc = t(scale)
    so = sc if alias else torch.full_like(sc, float("nan"))
    ws = torch.full((fq.lib().fq_wiener_gains_workspace_bytes(*D.shape),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    g = fq.fq_wiener_gains(t(D), t(Ht), words, sc, t(zero), scale_out=so, ws=ws, bits=bits)
    torch.cuda.synchronize()
    return g.cpu().numpy().astype(np.float64), so.cpu().numpy()


@pytest.mark.parametrize("K_out,d_in,K_in,bits", [(70, 64, 72, 2), (300, 1000, 1100, 2),
                                                  (130, 800, 880, 3), (257, 120, 136, 4)])
def test_wiener_gains_parity(K_out, d_in, K_in, bits):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(K_out + K_in + bits)
    D, Ht, codes, scale, zero = _problem(rng, K_out, d_in, K_in, bits)
    g, so = _run(torch, fq, D, Ht, codes, scale, zero, bits)
    Dh = O.dequant(codes, scale.astype(np.float64), zero.astype(np.float64))
    go = O.wiener_row_gains(D.astype(np.float64), Dh, Ht.astype(np.float64))
    assert go[3] == 1.0 and g[3] == 1.0                    # a row of zero weights keeps g = 1
    np.testing.assert_allclose(g, go, rtol=2e-5, atol=0)
    np.testing.assert_allclose(so, scale * go, rtol=2.1e-5, atol=0)


def test_wiener_gains_scale_in_place_and_errors():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(5)
    D, Ht, codes, scale, zero = _problem(rng, 40, 64, 72, 2)
    g, so = _run(torch, fq, D, Ht, codes, scale, zero, 2, alias=True)
    # scale_out is fp32(g scale) with g unrounded; g itself was returned rounded to fp32
    np.testing.assert_allclose(so, scale.astype(np.float64) * g, rtol=2.5e-7)
    with pytest.raises(fq.FQError):
        _run(torch, fq, D, Ht, codes, scale, zero, 5)
    with pytest.raises(fq.FQError):
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        w = t(O.pack2(codes).view(np.int32))
        tiny = torch.empty(16, dtype=torch.uint8, device="cuda")
        fq.fq_wiener_gains(t(D), t(Ht), w, t(scale), t(zero), ws=tiny)


def test_wiener_filtered_pass_lowers_proxy_loss():
    """The filter on the device's own pass (ViT-B qkv layer, structured frames): gains
    against the oracle on the device's D, H~ and codes, and the filtered proxy loss
    ||(D - diag(g) D^) C||^2 (= tr(R H~ R^T)) below the unfiltered one."""
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    wl = WORKLOADS["vitb"]
    L = wl.layers[0]
    X = torch.from_numpy(gen.make_x(wl, L.d_in)).cuda()
    W = torch.from_numpy(gen.make_weight(wl, 0)).cuda()
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, 0)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    F = (fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o)), fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i)))
    b = LayerBuffers(L.d_out, L.d_in, F[0].K, F[1].K, W.dtype, X.dtype, X.shape[0], frames=F)
    quantize_layer(W, X, None, None, b)
    g = fq.fq_wiener_gains(b.D, b.Ht, b.codes, b.scale, b.zero)
    torch.cuda.synchronize()
    D = b.D.cpu().numpy().astype(np.float64)
    Ht = b.Ht.cpu().numpy().astype(np.float64)
    cg = O.unpack2(b.codes.cpu().numpy().view(np.uint32), F[1].K)
    Dh = O.dequant(cg, b.scale.cpu().numpy().astype(np.float64), b.zero.cpu().numpy().astype(np.float64))
    go = O.wiener_row_gains(D, Dh, Ht)
    np.testing.assert_allclose(g.cpu().numpy(), go, rtol=2e-5, atol=0)
    R0, R1 = D - Dh, D - go[:, None] * Dh
    loss0 = np.einsum("ij,jk,ik->", R0, Ht, R0)
    loss1 = np.einsum("ij,jk,ik->", R1, Ht, R1)
    assert loss1 < loss0
