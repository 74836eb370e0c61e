"""End-to-end device runs of the per-layer pass on the small workloads, checked stage by
stage against the oracle (each oracle stage fed the device's own upstream outputs), then
codes by teacher-forced replay, then the reconstructed weights and layer outputs."""
import numpy as np
import pytest

import oracle as O
from fq_inputs import WORKLOADS, gen
from fq_testutil import need_gpu, upload, rel_fro, unpack_codes, replay_rows, check_codes

pytestmark = pytest.mark.gpu


def run_workload(key, independent=True):
    torch = need_gpu()
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    wl = WORKLOADS[key]
    d_in = wl.layers[0].d_in
    Xs = gen.make_x(wl, d_in)
    X = upload(Xs, wl.x_dtype)
    X64 = gen.storage_to_f32(Xs, wl.x_dtype).astype(np.float64)
    H_o = O.hessian(X64)
    Ht_gpu = None
    out = []
    for li, L in enumerate(wl.layers):
        Po64, Pi64 = gen.make_frames(wl, li)
        Po, Pi = gen.frame_f32(Po64), gen.frame_f32(Pi64)
        Ws = gen.make_weight(wl, li)
        W64 = gen.storage_to_f32(Ws, wl.w_dtype).astype(np.float64)
        K_out, K_in = Po.shape[1], Pi.shape[1]
        W = upload(Ws, wl.w_dtype)
        bufs = LayerBuffers(L.d_out, L.d_in, K_out, K_in, W.dtype, X.dtype, X.shape[0], wl.block)
        P_out, P_in = torch.from_numpy(Po).cuda(), torch.from_numpy(Pi).cuda()
        if li == 0:
            quantize_layer(W, X, P_out, P_in, bufs, block=wl.block, damp=wl.damp,
                           clip_sigmas=wl.clip_sigmas)
            Hg = bufs.H.cpu().numpy().astype(np.float64)
            Ht_gpu = bufs.Ht
            H_share = bufs.H
        else:
            quantize_layer(W, None, P_out, P_in, bufs, H=H_share, Ht=Ht_gpu, block=wl.block,
                           damp=wl.damp, clip_sigmas=wl.clip_sigmas)
        torch.cuda.synchronize()
        Dg = bufs.D.cpu().numpy()
        Htg = Ht_gpu.cpu().numpy()
        # stage 1 / 2: oracle on exact inputs (Ht from the device's H)
        if li == 0:
            assert rel_fro(Hg, H_o) < 1e-5, "H"
        D_o, Ht_o = O.frame_analysis(W64, Po, Pi, Hg)
        assert rel_fro(Dg, D_o) < 1e-5, "D"
        if li == 0:
            assert rel_fro(Htg, Ht_o) < 1e-5, "Ht"
        # stage 3: teacher-forced replay on the device's D and Ht
        cg = unpack_codes(bufs.codes, K_in)
        sg, zg = bufs.scale.cpu().numpy(), bufs.zero.cpu().numpy()
        r = replay_rows(Dg, Htg, cg, block=wl.block, damp=wl.damp, clip_sigmas=wl.clip_sigmas)
        ties = check_codes(r, cg, sg, zg, words=bufs.codes.cpu().numpy())
        # stage 4 and layer outputs, from the replayed codes
        Wh_o = O.synthesis(r["codes"], r["scale"], r["zero"], Po, Pi)
        Whg = bufs.W_hat.cpu().numpy()
        assert rel_fro(Whg, Wh_o) < 1e-4, "W_hat"
        xs = X64[:: max(1, X64.shape[0] // 2048)]
        assert rel_fro(xs @ Whg.T.astype(np.float64), xs @ Wh_o.T) < 1e-4, "Y"
        info = {"layer": L.name, "ties": ties}
        if independent:
            # fully independent oracle run (informational): code agreement and proxy loss
            ind = O.quantize_layer(W64, None, Po, Pi, bits=wl.bits, block=wl.block,
                                   damp=wl.damp, clip_sigmas=wl.clip_sigmas, H=H_o)
            info["code_mismatch_frac"] = float((ind["codes"] != cg).mean())
            Dh_g = O.dequant(cg, sg.astype(np.float64), zg.astype(np.float64))
            Dh_o = O.dequant(ind["codes"], ind["scale"], ind["zero"])
            info["proxy_loss_ratio"] = (O.proxy_loss(ind["D"], Dh_g, ind["Ht"]) /
                                        O.proxy_loss(ind["D"], Dh_o, ind["Ht"]))
            assert info["code_mismatch_frac"] < 0.01
            assert abs(info["proxy_loss_ratio"] - 1) < 0.01
        print(key, info)
        out.append(info)
    return out


def test_pipeline_tiny256():
    run_workload("tiny256")


def test_pipeline_vitb():
    run_workload("vitb")


@pytest.mark.parametrize("key", ["tiny256", "vitb"])
def test_two_stream_order_is_bit_identical(key):
    """D formed on a second stream while the main stream factors H~ (prepare / apply)
    gives exactly the outputs of the one-stream order, also when the second stream is kept
    off part of the device (fq_side_stream_create)."""
    torch = need_gpu()
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    wl = WORKLOADS[key]
    L = wl.layers[0]
    X = upload(gen.make_x(wl, L.d_in), wl.x_dtype)
    Po64, Pi64 = gen.make_frames(wl, 0)
    P_out, P_in = torch.from_numpy(gen.frame_f32(Po64)).cuda(), torch.from_numpy(gen.frame_f32(Pi64)).cuda()
    W = upload(gen.make_weight(wl, 0), wl.w_dtype)
    K_out, K_in = P_out.shape[1], P_in.shape[1]
    outs = []
    import paper_2403_06082_amd as fq
    part = fq.SideStream(128)         # kernels kept off 128 compute units
    sides = {0: None, 1: torch.cuda.Stream(), 2: torch.cuda.Stream(), 3: part.stream}
    for two in (0, 1, 2, 3):
        bufs = LayerBuffers(L.d_out, L.d_in, K_out, K_in, W.dtype, X.dtype, X.shape[0], wl.block)
        quantize_layer(W, X, P_out, P_in, bufs, block=wl.block, damp=wl.damp,
                       clip_sigmas=wl.clip_sigmas, side_stream=sides[two])
        torch.cuda.synchronize()
        outs.append({k: getattr(bufs, k).cpu().numpy() for k in
                     ("H", "D", "Ht", "codes", "scale", "zero", "W_hat")})
    for o in outs[1:]:
        for k, v in o.items():
            np.testing.assert_array_equal(v, outs[0][k], err_msg=k)


def test_side_stream_create_and_errors():
    """fq_side_stream_create: a usable stream for reserves across [0, CUs / 2]; a reserve
    out of range and a NULL handle are refused."""
    torch = need_gpu()
    import ctypes
    import paper_2403_06082_amd as fq
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    for reserve in (0, 1, n_cu // 4, n_cu // 2, 3 * n_cu // 4):
        print(f"reserve {reserve} of {n_cu}", flush=True)
        s = fq.SideStream(reserve)
        x = torch.arange(1 << 20, dtype=torch.float32, device="cuda")
        with torch.cuda.stream(s.stream):
            y = x * 2.0 + 1.0
        s.stream.synchronize()
        assert torch.equal(y, x * 2.0 + 1.0)
        del s
    h = ctypes.c_void_p()
    for bad in (-1, 3 * n_cu // 4 + 1, n_cu):
        assert fq.lib().fq_side_stream_create(bad, ctypes.byref(h)) == 1
    assert fq.lib().fq_side_stream_create(0, None) == 1
    assert fq.lib().fq_side_stream_destroy(None) == 1


def test_prepare_apply_match_fused_call():
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    rng = np.random.default_rng(12)
    K_out, K_in = 300, 200
    A = rng.standard_normal((400, K_in))
    Ht = torch.from_numpy((A.T @ A).astype(np.float32)).cuda()
    Ht = (Ht + Ht.T) / 2
    D = torch.from_numpy((rng.standard_normal((K_out, K_in)) * 0.02).astype(np.float32)).cuda()
    res = []
    for split in ("fused", "prepare+apply", "prepare|grid+round", "round_async+status"):
        codes = torch.empty((K_out, (K_in + 15) // 16), dtype=torch.int32, device="cuda")
        scale = torch.empty((K_out,), dtype=torch.float32, device="cuda")
        zero = torch.empty((K_out,), dtype=torch.float32, device="cuda")
        ws = torch.full((fq.fq_quantize_frames_workspace_bytes(K_out, K_in, 128),), 0xFF,
                        dtype=torch.uint8, device="cuda")
        if split == "prepare+apply":
            s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
            fq.fq_quantize_prepare(Ht, K_out, ws, stream=s1)
            ev = torch.cuda.Event()
            ev.record(s1)
            s2.wait_event(ev)
            fq.fq_quantize_apply(D, codes, scale, zero, ws, stream=s2)
        elif split == "prepare|grid+round":
            # the grid beside prepare on its own stream, the rounding after both
            s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
            fq.fq_quantize_grid(D, scale, zero, ws, stream=s2)
            fq.fq_quantize_prepare(Ht, K_out, ws, stream=s1)
            ev = torch.cuda.Event()
            ev.record(s2)
            s1.wait_event(ev)
            fq.fq_quantize_round(D, codes, ws, stream=s1)
        elif split == "round_async+status":
            fq.fq_quantize_prepare(Ht, K_out, ws)
            fq.fq_quantize_grid(D, scale, zero, ws)
            fq.fq_quantize_round_async(D, codes, ws)
            fq.fq_quantize_status(K_out, K_in, ws)
        else:
            fq.fq_quantize_frames(D, Ht, codes, scale, zero, ws=ws)
        torch.cuda.synchronize()
        res.append((codes.cpu().numpy(), scale.cpu().numpy(), zero.cpu().numpy()))
    for r in res[1:]:
        for a, b in zip(res[0], r):
            np.testing.assert_array_equal(a, b)
    # a non-finite D found by the grid is reported by the rounding, also when the grid ran
    # beside prepare (prepare clears only its own checks)
    ws = torch.empty((fq.fq_quantize_frames_workspace_bytes(K_out, K_in, 128),), dtype=torch.uint8,
                     device="cuda")
    Dn = D.clone()
    Dn[3, 7] = float("inf")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    fq.fq_quantize_grid(Dn, scale, zero, ws, stream=s2)
    fq.fq_quantize_prepare(Ht, K_out, ws, stream=s1)
    ev = torch.cuda.Event()
    ev.record(s2)
    s1.wait_event(ev)
    with pytest.raises(fq.FQError) as ei:
        fq.fq_quantize_round(Dn, codes, ws, stream=s1)
    assert ei.value.status == 4
    # the same check reported by fq_quantize_status after the asynchronous rounding
    fq.fq_quantize_grid(Dn, scale, zero, ws, stream=s1)
    fq.fq_quantize_round_async(Dn, codes, ws, stream=s1)
    with pytest.raises(fq.FQError) as ei:
        fq.fq_quantize_status(K_out, K_in, ws, stream=s1)
    assert ei.value.status == 4
    # one factor, several applies: a non-finite D is reported by its own apply only
    ws = torch.empty((fq.fq_quantize_frames_workspace_bytes(K_out, K_in, 128),), dtype=torch.uint8,
                     device="cuda")
    fq.fq_quantize_prepare(Ht, K_out, ws)
    Dn = D.clone()
    Dn[7, 3] = float("nan")
    with pytest.raises(fq.FQError) as ei:
        fq.fq_quantize_apply(Dn, codes, scale, zero, ws)
    assert ei.value.status == 4
    for _ in range(2):
        fq.fq_quantize_apply(D, codes, scale, zero, ws)
        torch.cuda.synchronize()
        for a, b in zip(res[0], (codes.cpu().numpy(), scale.cpu().numpy(), zero.cpu().numpy())):
            np.testing.assert_array_equal(a, b)
    # a non-positive-definite H~ found by prepare is reported by apply
    bad = -torch.eye(K_in, dtype=torch.float32, device="cuda")
    ws = torch.empty((fq.fq_quantize_frames_workspace_bytes(K_out, K_in, 128),), dtype=torch.uint8,
                     device="cuda")
    fq.fq_quantize_prepare(bad, K_out, ws, damp=0.0)
    with pytest.raises(fq.FQError) as ei:
        fq.fq_quantize_apply(D, codes, scale, zero, ws)
    assert ei.value.status == 3
