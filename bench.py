"""Benchmark: FrameQuant's per-layer quantization pass on one MI355X.

One step = the whole pass on one layer with its inputs resident in HBM:
    H = X^T X (262,144 tokens)  ->  D = P_l^T W P_prev, H~ = P_prev^T H P_prev
    ->  clip + grid + OPTQ 2-bit rounding (fp64)  ->  W^ = P_l D^ P_prev^T
on the Llama-2-7B-shaped up_proj layer (11008 x 4096 bf16, X 262,144 x 4096 bf16,
frames r = 1.1: K_out x K_in = 12112 x 4512, block 128).  Inputs are synthetic and
seeded (fq_inputs).  The frames are applied from their construction (rotation and
per-block DFT; --frames dense multiplies by the d x K matrices instead, and the pass with
the other choice is timed beside the headline).  With --streams 2 (the default) D is
formed on a second stream while the main stream factors H~.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--streams 1|2]
                    [--frames structured|dense] [--no-cpu-baseline]

Prints one JSON line.  value = quantized weights per second (d_out * d_in / step time).
"roofline" is the dominant kernel's algorithmic throughput against its MFMA peak, timed
with HIP events on its own launch stream inside the timed region; "kernels" lists every
kernel group the same way.  "cpu_baseline" is the float64 CPU oracle timed on a bounded
sample of the same workload on this host, extrapolated stage by stage.  "inference" times
the quantized layer's outputs for 1 and 8 tokens (fq_frame_apply on the pass's own codes)
against HBM bandwidth, with its own roofline and CPU-oracle baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "quantized weights/sec per layer (Llama-7B-shaped 11008×4096); MFMA % of peak"
PEAK = {"bf16": 2500.0, "f32": 157.3, "f64": 78.6, "hbm": 8000.0}   # TFLOP/s ..., GB/s


def algorithmic_work(n, d_out, d_in, K_out, K_in, block, rho=None, rot=None):
    """Algorithmic flops (bytes for the memory-bound kernels) per launch group and step.
    With structured frames (rho, and rot = (d1_out + d2_out, d1_in + d2_in)): the per-block
    DFT products, 4 d k flops per transformed row (k = K / rho), and the rotations,
    2 d (d1 + d2) flops per row, over the rows each stage transforms (D: d_out rows of W,
    then K_in columns; Ht: d_in, then K_in; W_hat: K_out code rows, then d_in columns)."""
    gptq_upd = 0
    for o1 in range(0, K_in, block):
        o2 = min(o1 + block, K_in)
        for i1 in range(o1, o2, 128):
            i2 = min(i1 + 128, o2)
            gptq_upd += 2 * K_out * (i2 - i1) * (o2 - i2)
        gptq_upd += 2 * K_out * (o2 - o1) * (K_in - o2)
    # the device applies the same residual terms regrouped: inside spans of
    # block * ceil(512 / block) columns after every chunk, beyond a span once per span
    span = block * -(-512 // block)
    gptq_lazy = sum(2 * K_out * (min(s1 + span, K_in) - s1) * (K_in - min(s1 + span, K_in))
                    for s1 in range(0, K_in, span))
    chol = 0
    for k0 in range(0, K_in, 64):
        kb = min(64, K_in - k0)
        rest = K_in - k0 - kb
        chol += rest * (rest + 1) * kb          # lower-triangle rank-kb update, 2 flops/FMA
    extra = {}
    if rho is not None:
        k_out, k_in = K_out // rho, K_in // rho
        rows_in = d_out + d_in + K_in + K_out        # rows transformed by the input frame
        rows_out = K_in + d_in                       # rows transformed by the output frame
        extra["tffp_dft"] = ("bf16", 4 * d_in * k_in * rows_in + 4 * d_out * k_out * rows_out)
        extra["tffp_rotate"] = ("f32", 2 * d_in * rot[1] * rows_in + 2 * d_out * rot[0] * rows_out)
    return {
        **extra,
        "gemm_hessian": ("bf16", n * d_in * (d_in + 1)),
        "gemm_analysis_w1": ("bf16", 2 * K_out * d_out * d_in),
        "gemm_analysis_w2": ("bf16", 2 * K_out * d_in * K_in),
        "gemm_analysis_h1": ("bf16", 2 * d_in * d_in * K_in),
        "gemm_analysis_h2": ("bf16", K_in * (K_in + 1) * d_in),
        "gemm_synthesis_1": ("bf16", 2 * d_out * K_out * K_in),
        "gemm_synthesis_2": ("bf16", 2 * d_out * K_in * d_in),
        "gptq_update": ("f64", gptq_upd),
        "gptq_update_lazy": ("f64", gptq_lazy),
        "gptq_update_span": ("f64", gptq_upd - gptq_lazy),
        "chol_syrk": ("f64", chol),
        "gptq_block": ("f64", K_out * K_in * 128),     # in-block FMAs (upper bound)
        "pack2": ("hbm", K_out * K_in + K_out * ((K_in + 15) // 16) * 4),
    }


def mfma_passes(w_dtype):
    """bf16 MFMA passes per product: an fp32 operand is a bf16 (hi, lo) pair; a product
    takes 3 passes (hi.hi + hi.lo + lo.hi), 2 when one side is exact in one bf16 plane
    (bf16 weights, codes - zero), 1 for the Hessian of 16-bit calibration data."""
    return {"gemm_hessian": 1, "gemm_analysis_w1": 2 if w_dtype == "bf16" else 3,
            "gemm_analysis_w2": 3, "gemm_analysis_h1": 3, "gemm_analysis_h2": 3,
            "gemm_synthesis_1": 2, "gemm_synthesis_2": 3}


KERNEL_GROUPS = ["gemm_hessian", "gemm_analysis_w1", "gemm_analysis_w2", "gemm_analysis_h1",
                 "gemm_analysis_h2", "gemm_synthesis_1", "gemm_synthesis_2", "tffp_rotate",
                 "tffp_blocks", "tffp_dft", "tffp_gather", "gptq_update",
                 "gptq_update_lazy", "gptq_update_span", "gptq_block", "chol_syrk", "chol_potrf", "chol_trsm", "q_", "split_bf16",
                 "syrk_reduce", "dequant", "pack2"]


def make_inputs(wl, li):
    import torch
    from fq_inputs import gen
    L = wl.layers[li]
    t0 = time.time()
    Xs = gen.make_x(wl, L.d_in)
    Ws = gen.make_weight(wl, li)
    tf = time.time()
    Po64, Pi64 = gen.make_frames(wl, li)
    frames_host_s = time.time() - tf
    Po, Pi = gen.frame_f32(Po64), gen.frame_f32(Pi64)
    del Po64, Pi64

    def up(a, dt):
        t = torch.from_numpy(a)
        if dt == "bf16":
            t = t.view(torch.bfloat16)
        return t.cuda()

    dev = dict(X=up(Xs, wl.x_dtype), W=up(Ws, wl.w_dtype), P_out=up(Po, "f32"),
               P_in=up(Pi, "f32"))
    host = dict(X=Xs, W=Ws, P_out=Po, P_in=Pi, frames_host_s=frames_host_s)
    print(f"[bench] inputs generated and uploaded in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    return dev, host


def cpu_baseline(wl, li, host, budget_rows=1024, sample_tokens=8192):
    """Time the oracle on a bounded sample of the same layer and extrapolate per stage:
    H over one 8,192-token chunk (x n / 8192); D, OPTQ and W^ on `budget_rows` sampled
    rows (x rows / budget_rows); H~ and the factor U in full."""
    import oracle as O
    from fq_inputs import gen
    try:
        from threadpoolctl import threadpool_info
        cores = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:
        cores = len(os.sched_getaffinity(0))
    L = wl.layers[li]
    n = wl.n_tokens
    X = host["X"]
    W64 = gen.storage_to_f32(host["W"], wl.w_dtype).astype(np.float64)
    Po = host["P_out"].astype(np.float64)
    Pi = host["P_in"].astype(np.float64)
    K_out, K_in = Po.shape[1], Pi.shape[1]
    rng = np.random.default_rng(0)
    t = {}
    s0 = time.perf_counter()
    Xc = gen.storage_to_f32(X[:sample_tokens], wl.x_dtype).astype(np.float64)
    H = O.hessian(Xc) * (n / sample_tokens)
    t["hessian"] = (time.perf_counter() - s0) * (n / sample_tokens)
    rows = np.sort(rng.choice(K_out, size=min(budget_rows, K_out), replace=False))
    s0 = time.perf_counter()
    D_rows = (Po[:, rows].T @ W64) @ Pi
    t["analysis_D"] = (time.perf_counter() - s0) * (K_out / len(rows))
    s0 = time.perf_counter()
    _, Ht = O.frame_analysis(np.zeros((1, L.d_in)), np.zeros((1, 1)), Pi, H)
    t["analysis_Ht"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    U, dead, _ = O.gptq_prepare(Ht, wl.damp)
    t["factor"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    mu, sigma, lo, hi = O.clip_bounds(D_rows, wl.clip_sigmas)
    Dc = O.apply_clip(D_rows, lo, hi)
    sc, z = O.row_grid(Dc)
    r = O.gptq(Dc, U, sc, z, wl.bits, wl.block, dead)
    O.pack2(r["codes"])
    t["gptq"] = (time.perf_counter() - s0) * (K_out / len(rows))
    orow = np.sort(rng.choice(L.d_out, size=min(budget_rows, L.d_out), replace=False))
    Dh = O.dequant(r["codes"], sc, z)
    # rows of W^ = (P_l[rows, :] D^) P_prev^T; the sampled rows of D^ stand in for all of it
    s0 = time.perf_counter()
    Mr = Po[orow][:, rows] @ Dh
    t["synthesis_1"] = (time.perf_counter() - s0) * (L.d_out / len(orow)) * (K_out / len(rows))
    s0 = time.perf_counter()
    _ = Mr @ Pi.T
    t["synthesis_2"] = (time.perf_counter() - s0) * (L.d_out / len(orow))
    total = sum(t.values())
    return {"value": L.d_out * L.d_in / total, "unit": "weights/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"float64 numpy oracle: H on {sample_tokens} of {n} tokens (x{n // sample_tokens}); "
                       f"D, OPTQ and synthesis on {len(rows)} of {K_out} FF rows (scaled to all rows); "
                       f"H~ and its Cholesky factor in full; extrapolated total {total:.1f} s"),
            "stage_seconds": {k: round(v, 3) for k, v in t.items()}}


def apply_bytes(nt, d_out, d_in, K_out, K_in, x_bytes):
    """Algorithmic HBM bytes of one fq_frame_apply call per kernel group: every operand
    read once per block of up to 8 tokens (P_in, codes + scale + zero, P_out), X read
    and Y written once."""
    blocks = -(-nt // 8)
    nwords = -(-K_in // 16)
    return {"apply_in": blocks * d_in * K_in * 4 + nt * d_in * x_bytes,
            "apply_codes": blocks * (K_out * nwords * 4 + 2 * K_out * 4),
            "apply_out": blocks * d_out * K_out * 4 + nt * d_out * 4}


def apply_tff_bytes(nt, d_out, d_in, K_out, K_in, x_bytes, rot_floats):
    """Algorithmic HBM bytes of one fq_frame_apply_tff call: the codes + scale + zero once
    per block of up to 8 tokens, the rotation factors, X read and Y written once (the frames
    themselves are never read)."""
    blocks = -(-nt // 8)
    nwords = -(-K_in // 16)
    return (blocks * (K_out * nwords * 4 + 2 * K_out * 4) + rot_floats * 4 + nt * d_in * x_bytes
            + nt * d_out * 4)


def _time_calls(torch, call, stream, iters):
    for _ in range(10):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(iters):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / iters


def _kernel_us(fq, torch, call, names, iters):
    fq.fq_profile_reset()
    fq.fq_profile_enable(True)
    for _ in range(iters):
        call()
    torch.cuda.synchronize()
    fq.fq_profile_enable(False)
    out = {}
    for name in names:
        cnt, tot = fq.fq_profile_query(name)
        out[name] = {"launches_per_call": cnt / iters, "us_per_call": round(tot * 1e3 / iters, 2)}
    fq.fq_profile_reset()
    return out


def structured_bench(fq, torch, dev, bufs, wl, li, K_out, K_in, tokens=(1, 8), iters=200):
    """fq_frame_apply_tff: the same layer outputs with both frames applied from their
    construction (rotation factors + DFT blocks), for 1 and 8 tokens."""
    from fq_inputs import gen
    L = wl.layers[li]
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, li)
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    Fo = fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o))
    Fi = fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i))
    assert (Fo.K, Fi.K) == (K_out, K_in)
    rot_floats = sum(r.size for r in (R1o, R2o, R1i, R2i))
    stream = torch.cuda.current_stream()
    ws = torch.empty(fq.fq_frame_apply_tff_workspace_bytes(Fo, Fi), dtype=torch.uint8, device="cuda")
    rows = []
    for nt in tokens:
        X = dev["X"][:nt]
        Y = torch.empty((nt, L.d_out), dtype=torch.float32, device="cuda")

        def call():
            fq.fq_frame_apply_tff(X, bufs.codes, bufs.scale, bufs.zero, Fo, Fi, Y=Y, ws=ws,
                                  stream=stream)

        us = _time_calls(torch, call, stream, iters)
        # the same call captured once into a HIP graph and replayed (no host launch work
        # per kernel); the replay's output must equal the eager call's
        call()
        torch.cuda.synchronize()
        Y_eager = Y.clone()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fq.fq_frame_apply_tff(X, bufs.codes, bufs.scale, bufs.zero, Fo, Fi, Y=Y, ws=ws,
                                  stream=torch.cuda.current_stream())
        Y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        graph_equal = bool(torch.equal(Y, Y_eager))
        us_graph = _time_calls(torch, graph.replay, stream, iters)
        del graph
        kern = _kernel_us(fq, torch, call, ("tff_rotate", "tff_dft", "apply_codes"), iters)
        b = apply_tff_bytes(nt, L.d_out, L.d_in, K_out, K_in, dev["X"].element_size(), rot_floats)
        kc = kern["apply_codes"]
        kc["algorithmic_bytes"] = -(-nt // 8) * (K_out * (-(-K_in // 16)) * 4 + 2 * K_out * 4)
        kc["GB/s"] = round(kc["algorithmic_bytes"] / kc["us_per_call"] / 1e3, 1)
        rows.append({"tokens": nt, "us_per_call": round(us, 2),
                     "tokens_per_s": round(nt / (us / 1e6), 1), "algorithmic_bytes": b,
                     "GB/s": round(b / us / 1e3, 1), "kernels": kern,
                     "hip_graph": {"us_per_call": round(us_graph, 2),
                                   "tokens_per_s": round(nt / (us_graph / 1e6), 1),
                                   "output_equals_eager": graph_equal}})
        print(f"[bench] frame_apply_tff {nt} token(s): {us:.1f} us/call, {us_graph:.1f} us "
              f"replayed from a HIP graph", file=sys.stderr, flush=True)
    # the same with the frame representation of the inputs rounded to 8-bit integers
    wsq = torch.empty(fq.fq_frame_apply_tff_actq_workspace_bytes(Fo, Fi), dtype=torch.uint8,
                      device="cuda")
    qrows = []
    for nt in tokens:
        X = dev["X"][:nt]
        Y = torch.empty((nt, L.d_out), dtype=torch.float32, device="cuda")

        def callq():
            fq.fq_frame_apply_tff_actq(X, bufs.codes, bufs.scale, bufs.zero, Fo, Fi, 8, Y=Y, ws=wsq,
                                       stream=stream)

        us = _time_calls(torch, callq, stream, iters)
        kern = _kernel_us(fq, torch, callq, ("tff_rotate", "tff_dft", "act_quantize", "apply_codes"),
                          iters)
        qrows.append({"tokens": nt, "us_per_call": round(us, 2),
                      "tokens_per_s": round(nt / (us / 1e6), 1), "kernels": kern})
        print(f"[bench] frame_apply_tff_actq (8-bit activations) {nt} token(s): {us:.1f} us/call",
              file=sys.stderr, flush=True)
    return {"op": "fq_frame_apply_tff: the same outputs with P_in and P_l applied from their "
                  "construction (Kronecker rotation factors + length-k DFT blocks); no frame "
                  "matrix is read",
            "frames": {"out": {"d": L.d_out, "k": ko, "rho": ro, "d1": R1o.shape[0], "d2": R2o.shape[0]},
                       "in": {"d": L.d_in, "k": ki, "rho": ri, "d1": R1i.shape[0], "d2": R2i.shape[0]}},
            "per_tokens": rows,
            "int8_activations": {"op": "fq_frame_apply_tff_actq, act_bits 8: the analysis output "
                                       "rounded per token to int8, code products exact in int32 "
                                       "(v_dot4)", "per_tokens": qrows},
            "note": "about 7.6e7 FMAs per token (5.5e7 in the code GEMV) and 13.8 MB of codes "
                    "per block of 8 tokens: bound by launch and memory latency at 1 token, by "
                    "the code kernel's VALU work at 8"}


def grid_variants_bench(torch, dev, wl, li, L, K_out, K_in, n, steps, iters=200, frames=None):
    """The same pass with 3- and 4-bit grids (one warmup, then `steps` timed passes each;
    one stream), as quantized weights per second; then the 4-bit codes of that pass run
    through the integer inference path at 4-bit activations (W4/A4), 1 and 8 tokens."""
    import paper_2403_06082_amd as fq
    from fq_inputs import gen
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    out = {}
    for bits in (3, 4):
        b = LayerBuffers(L.d_out, L.d_in, K_out, K_in, dev["W"].dtype, dev["X"].dtype, n, wl.block,
                         bits=bits, frames=frames)

        def run():
            quantize_layer(dev["W"], dev["X"], dev["P_out"], dev["P_in"], b, bits=bits,
                           block=wl.block, damp=wl.damp, clip_sigmas=wl.clip_sigmas)

        run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            run()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        out[f"bits{bits}"] = {"ms_per_step": round(ms, 3),
                              "weights_per_s": round(L.d_out * L.d_in / (ms / 1e3), 1)}
        print(f"[bench] {bits}-bit pass: {ms:.2f} ms/step", file=sys.stderr, flush=True)
        if bits == 4:
            (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, li)
            up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
            Fo = fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o))
            Fi = fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i))
            stream = torch.cuda.current_stream()
            ws = torch.empty(fq.fq_frame_apply_tff_actq_workspace_bytes(Fo, Fi), dtype=torch.uint8,
                             device="cuda")
            rows = []
            for nt in (1, 8):
                X = dev["X"][:nt]
                Y = torch.empty((nt, L.d_out), dtype=torch.float32, device="cuda")

                def call():
                    fq.fq_frame_apply_tff_actq(X, b.codes, b.scale, b.zero, Fo, Fi, 4, Y=Y, ws=ws,
                                               stream=stream, bits=4)

                us = _time_calls(torch, call, stream, iters)
                rows.append({"tokens": nt, "us_per_call": round(us, 2),
                             "tokens_per_s": round(nt / (us / 1e6), 1)})
                print(f"[bench] W4/A4 structured inference {nt} token(s): {us:.1f} us/call",
                      file=sys.stderr, flush=True)
            out["w4a4_inference"] = {"op": "fq_frame_apply_tff_actq, bits 4, act_bits 4, on the "
                                           "4-bit pass's codes", "per_tokens": rows}
            wsf = torch.empty(fq.fq_frame_apply_tff_workspace_bytes(Fo, Fi), dtype=torch.uint8,
                              device="cuda")
            frows = []
            for nt in (1, 8):
                X = dev["X"][:nt]
                Y = torch.empty((nt, L.d_out), dtype=torch.float32, device="cuda")

                def callf():
                    fq.fq_frame_apply_tff(X, b.codes, b.scale, b.zero, Fo, Fi, Y=Y, ws=wsf,
                                          stream=stream, bits=4)

                us = _time_calls(torch, callf, stream, iters)
                frows.append({"tokens": nt, "us_per_call": round(us, 2),
                              "tokens_per_s": round(nt / (us / 1e6), 1)})
                print(f"[bench] W4 structured inference (float activations) {nt} token(s): "
                      f"{us:.1f} us/call", file=sys.stderr, flush=True)
            out["w4_inference"] = {"op": "fq_frame_apply_tff, bits 4, on the 4-bit pass's codes",
                                   "per_tokens": frows}
        del b
    return out


def frame_generation_bench(fq, torch, dev, wl, li, host, iters=5):
    """Both dense frames of the layer generated on the device from (k, rho, d) and their
    rotation factors (fq_tff_materialize), timed with HIP events, checked against the
    frames the pass used (generated on the host in float64 and rounded to float32)."""
    from fq_inputs import gen
    L = wl.layers[li]
    out = {}
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    stream = torch.cuda.current_stream()
    for name, d, (k, rho, R1, R2) in zip(("P_out", "P_in"), (L.d_out, L.d_in),
                                         gen.layer_frame_factors(wl, li)):
        F = fq.Frame(d, k, rho, up(R1), up(R2))
        P = torch.empty((d, F.K), dtype=torch.float32, device="cuda")
        ws = torch.empty(fq.fq_tff_materialize_workspace_bytes(F), dtype=torch.uint8, device="cuda")
        fq.fq_tff_materialize(F, P=P, ws=ws, stream=stream)
        torch.cuda.synchronize()
        err = float((P - dev[name]).abs().max())
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            fq.fq_tff_materialize(F, P=P, ws=ws, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        out[name] = {"shape": [d, F.K], "ms": round(e0.elapsed_time(e1) / iters, 3),
                     "max_abs_diff_vs_host_frame": err}
        # the same layer's rotation factors drawn on the device from a seed
        d1, d2 = R1.shape[0], R2.shape[0]
        wsr = torch.empty(fq.fq_tff_rotation_factors_workspace_bytes(d1, d2), dtype=torch.uint8,
                          device="cuda")
        S1 = torch.empty((d1, d1), dtype=torch.float32, device="cuda")
        S2 = torch.empty((d2, d2), dtype=torch.float32, device="cuda")
        fq.fq_tff_rotation_factors(wl.seed, d1, d2, R1=S1, R2=S2, ws=wsr, stream=stream)
        e0.record(stream)
        for _ in range(iters):
            fq.fq_tff_rotation_factors(wl.seed, d1, d2, R1=S1, R2=S2, ws=wsr, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        out[name]["seeded_factors"] = {"d1": d1, "d2": d2,
                                       "ms": round(e0.elapsed_time(e1) / iters, 3)}
        del P, ws, wsr
    out["host_float64_seconds_both"] = round(host["frames_host_s"], 2)
    return out


def inference_bench(fq, torch, dev, bufs, L, K_out, K_in, tokens=(1, 8), iters=200):
    """Layer outputs Y = X Theta^T from the pass's own codes and the frames (fq_frame_apply),
    for 1 and 8 tokens (rows of the calibration activations), timed with HIP events on the
    launch stream; per-kernel times from the library's kernel timers in a second run."""
    stream = torch.cuda.current_stream()
    ws = torch.empty(fq.fq_frame_apply_workspace_bytes(L.d_in, K_out, K_in), dtype=torch.uint8,
                     device="cuda")
    x_bytes = dev["X"].element_size()
    rows = []
    for nt in tokens:
        X = dev["X"][:nt]
        Y = torch.empty((nt, L.d_out), dtype=torch.float32, device="cuda")

        def call():
            fq.fq_frame_apply(X, bufs.codes, bufs.scale, bufs.zero, dev["P_out"], dev["P_in"],
                              Y=Y, ws=ws, stream=stream)

        for _ in range(10):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / iters
        fq.fq_profile_reset()
        fq.fq_profile_enable(True)
        for _ in range(iters):
            call()
        torch.cuda.synchronize()
        fq.fq_profile_enable(False)
        nbytes = apply_bytes(nt, L.d_out, L.d_in, K_out, K_in, x_bytes)
        kern = {}
        for name, b in nbytes.items():
            cnt, tot = fq.fq_profile_query(name)
            k_us = tot * 1e3 / iters
            kern[name] = {"launches_per_call": cnt / iters, "us_per_call": round(k_us, 2),
                          "algorithmic_bytes": b, "GB/s": round(b / k_us / 1e3, 1)}
        fq.fq_profile_reset()
        total = sum(nbytes.values())
        rows.append({"tokens": nt, "us_per_call": round(us, 2),
                     "tokens_per_s": round(nt / (us / 1e6), 1),
                     "algorithmic_bytes": total, "GB/s": round(total / us / 1e3, 1),
                     "frac_of_hbm_peak": round(total / us / 1e3 / PEAK["hbm"], 4),
                     "kernels": kern})
        print(f"[bench] frame_apply {nt} token(s): {us:.1f} us/call", file=sys.stderr, flush=True)
    k1 = rows[0]["kernels"]["apply_out"]
    roof = {"bound": "hbm", "kernel": "apply_out", "tokens": rows[0]["tokens"],
            "achieved": k1["GB/s"], "peak": PEAK["hbm"], "unit": "GB/s",
            "frac": round(k1["GB/s"] / PEAK["hbm"], 4), "traffic": measured_traffic("apply_out", "traffic_apply_out.json"),
            "avg_launch_us": k1["us_per_call"], "algorithmic_per_launch": k1["algorithmic_bytes"]}
    return {"op": "fq_frame_apply: Y = X Theta^T straight from the 2-bit codes and the two "
                  "fp32 frames (Theta^ never formed): U = X P_in, V = U (q - zero)^T diag(scale), "
                  "Y = V P_out^T",
            "workload": f"the benchmark layer ({L.d_out}x{L.d_in}, K {K_out}x{K_in}), codes of "
                        f"the pass just timed, X = first rows of its bf16 activations",
            "dtype": "fp32 (fp32 accumulation; split-K partials summed in fp64)",
            "per_tokens": rows, "roofline": roof}


def cpu_inference_baseline(host, codes, scale, zero, wl, li, sample_rows=512):
    """The oracle's layer output for one token on `sample_rows` sampled output channels;
    its row-proportional part is scaled to all channels, the dequantization counted once."""
    import oracle as O
    from fq_inputs import gen
    try:
        from threadpoolctl import threadpool_info
        cores = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:
        cores = len(os.sched_getaffinity(0))
    L = wl.layers[li]
    K_in = host["P_in"].shape[1]
    q = O.unpack2(codes.view(np.uint32), K_in)
    sc, z = scale.astype(np.float64), zero.astype(np.float64)
    X1 = gen.storage_to_f32(host["X"][:1], wl.x_dtype).astype(np.float64)
    rows = np.sort(np.random.default_rng(1).choice(L.d_out, size=min(sample_rows, L.d_out),
                                                    replace=False))
    s0 = time.perf_counter()
    O.dequant(q, sc, z)
    t_dq = time.perf_counter() - s0
    s0 = time.perf_counter()
    O.frame_apply(X1, q, sc, z, host["P_out"][rows], host["P_in"])
    t_rows = time.perf_counter() - s0
    total = t_dq + (t_rows - t_dq) * (L.d_out / len(rows))
    return {"value": round(1.0 / total, 4), "unit": "tokens/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"float64 numpy oracle frame_apply for 1 token on {len(rows)} of {L.d_out} "
                       f"output channels ({t_rows:.2f} s), the part beyond the dequantization "
                       f"({t_dq:.2f} s, counted once) scaled to all channels: {total:.1f} s")}


def measured_traffic(kernel, fname="traffic.json"):
    """HBM bytes per launch of `kernel` from a committed byte-counter profile, or None when
    there is none or the kernel source changed since it was taken."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    try:
        with open(os.path.join(here, "profiles", fname)) as f:
            t = json.load(f)
        if t.get("kernel") != kernel:
            return None
        with open(os.path.join(here, t["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != t["source_sha256"]:
                return None
        return t["hbm_bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llama7b")
    ap.add_argument("--layer", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=2, choices=(1, 2),
                    help="2 (default): D is formed on a second stream while the main stream "
                         "factors H~ (the factorization is a chain of small kernels that leaves "
                         "most CUs idle); 1: one stream.  The kernel-timer region always uses one")
    ap.add_argument("--frames", default="structured", choices=("structured", "dense"),
                    help="how the pass applies the frames in the analysis and the synthesis: "
                         "from their construction (default) or as the dense d x K matrices; "
                         "the other way is timed beside it")
    ap.add_argument("--pass-only", action="store_true",
                    help="time the pass only (no pass with the other frames, no inference, frame "
                         "generation or grid variants): the kernel trace then covers exactly "
                         "the warmup, timed and kernel-timer passes")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="device-to-device copy of this many MiB before the warmup, as the "
                         "known-size reference for hardware byte counters")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the per-layer pass runs on a single device in this "
              "build (no multi-GPU path); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2403_06082_amd as fq
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    from fq_inputs import WORKLOADS, gen

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    fq.lib()
    wl = WORKLOADS[args.workload]
    li = args.layer
    L = wl.layers[li]
    dev, host = make_inputs(wl, li)
    K_out, K_in = dev["P_out"].shape[1], dev["P_in"].shape[1]
    n = dev["X"].shape[0]
    (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, li)
    upf = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    tff_frames = (fq.Frame(L.d_out, ko, ro, upf(R1o), upf(R2o)),
                  fq.Frame(L.d_in, ki, ri, upf(R1i), upf(R2i)))
    frames = tff_frames if args.frames == "structured" else None
    bufs = LayerBuffers(L.d_out, L.d_in, K_out, K_in, dev["W"].dtype, dev["X"].dtype, n, wl.block,
                        frames=frames)
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream() if args.streams == 2 else None

    def step(two=args.streams == 2):
        quantize_layer(dev["W"], dev["X"], dev["P_out"], dev["P_in"], bufs, block=wl.block,
                       damp=wl.damp, clip_sigmas=wl.clip_sigmas, stream=stream,
                       side_stream=side if two else None)

    if args.copy_probe_mib > 0:
        nb = args.copy_probe_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        step()
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    # timed region: the pass alone
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1000.0 / args.steps
    print(f"[bench] {args.steps} timed steps: {ms:.2f} ms/step", file=sys.stderr, flush=True)
    # second timed region with the per-launch kernel timers (HIP events on the launch
    # stream around every kernel): the per-kernel breakdown and the roofline come from it.
    # One stream here, so that no two timed kernels overlap.
    fq.fq_profile_reset()
    fq.fq_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(two=False)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    fq.fq_profile_enable(False)
    ms_timed = (t1 - t0) * 1000.0 / args.steps
    print(f"[bench] {args.steps} steps with kernel timers: {ms_timed:.2f} ms/step", file=sys.stderr,
          flush=True)

    rot = (R1o.shape[0] + R2o.shape[0], R1i.shape[0] + R2i.shape[0])
    work = algorithmic_work(n, L.d_out, L.d_in, K_out, K_in, wl.block,
                            rho=wl.rho if frames is not None else None, rot=rot)
    passes = mfma_passes(wl.w_dtype)
    kernels = {}
    for name in KERNEL_GROUPS:
        cnt, tot = fq.fq_profile_query(name)
        if cnt == 0:
            continue
        e = {"launches_per_step": cnt / args.steps, "ms_per_step": round(tot / args.steps, 4)}
        if name in work:
            kind, amount = work[name]
            per_step_s = tot / args.steps / 1000.0
            if kind == "hbm":
                e["GB/s"] = round(amount / per_step_s / 1e9, 1)
                e["frac_of_peak"] = round(amount / per_step_s / 1e9 / PEAK["hbm"], 4)
            else:
                e["TFLOP/s"] = round(amount / per_step_s / 1e12, 2)
                e["frac_of_peak"] = round(amount / per_step_s / 1e12 / PEAK[kind], 4)
                e["peak"] = kind
                if name in passes:
                    # MFMA work actually executed: every bf16 pass of the split product
                    e["passes"] = passes[name]
                    e["executed_TFLOP/s"] = round(amount * passes[name] / per_step_s / 1e12, 2)
                    e["executed_frac_of_peak"] = round(amount * passes[name] / per_step_s / 1e12 / PEAK[kind], 4)
        kernels[name] = e
    cnt_all, tot_all = fq.fq_profile_query("")
    fq.fq_profile_reset()

    # dominant kernel with a defined algorithmic count ("gptq_update" is the sum of its
    # _lazy and _span launches, which run on two different kernels)
    dom = max((k for k in kernels if k in work and k != "gptq_update"),
              key=lambda k: kernels[k]["ms_per_step"])
    kind, amount = work[dom]
    launches = kernels[dom]["launches_per_step"]
    avg_ms = kernels[dom]["ms_per_step"] / launches
    per_launch = amount / launches
    if kind == "hbm":
        roof = {"bound": "hbm", "achieved": round(per_launch / (avg_ms / 1e3) / 1e9, 1),
                "peak": PEAK["hbm"], "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": round(per_launch / (avg_ms / 1e3) / 1e12, 2),
                "peak": PEAK[kind], "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom)
    roof["kernel"] = dom
    roof["avg_launch_ms"] = round(avg_ms, 4)
    roof["algorithmic_per_launch"] = per_launch

    # contraction fraction of S1 + S2 (the Hessian and, with dense frames, the analysis
    # contractions) at bf16 peak
    contr = [k for k in kernels if k.startswith("gemm_hessian") or k.startswith("gemm_analysis")]
    c_flops = sum(work[k][1] for k in contr)
    c_ms = sum(kernels[k]["ms_per_step"] for k in contr)
    contraction_frac = c_flops / (c_ms / 1e3) / 1e12 / PEAK["bf16"] if c_ms > 0 else None
    c_exec = sum(work[k][1] * passes[k] for k in contr)
    contraction_exec = c_exec / (c_ms / 1e3) / 1e12 / PEAK["bf16"] if c_ms > 0 else None

    out = {
        "metric": METRIC,
        "value": round(L.d_out * L.d_in / (ms / 1e3), 1),
        "unit": "weights/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "ms_per_step_with_kernel_timers": round(ms_timed, 3),
        "kernel_timer_streams": 1,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 MFMA (fp32 acc) + fp64",
        "data": "synthetic (seeded; Gaussian weights with 1% x10 outliers, Gaussian "
                "activations with 8 channels x100)",
        "config": {"workload": f"{wl.key} {L.name}_proj: W {L.d_out}x{L.d_in} {wl.w_dtype}, "
                               f"X {n}x{L.d_in} {wl.x_dtype}, frames K {K_out}x{K_in} "
                               f"(r={wl.r}, rho={wl.rho}), {wl.bits}-bit, block {wl.block}, "
                               f"damp {wl.damp}, clip {wl.clip_sigmas} sigma",
                   "d_out": L.d_out, "d_in": L.d_in, "n_tokens": n, "K_out": K_out,
                   "K_in": K_in, "streams": args.streams, "frames": args.frames},
        "roofline": roof,
        "contraction_mfma_frac": None if contraction_frac is None else round(contraction_frac, 4),
        "contraction_mfma_executed_frac": None if contraction_exec is None else round(contraction_exec, 4),
        "kernels": kernels,
        "kernel_ms_total_per_step": round(tot_all / args.steps, 3),
    }
    if args.pass_only:
        print(json.dumps(out), flush=True)
        return
    # the pass without S1: H given (it is shared by layers that read the same input, such
    # as q/k/v or gate/up), same frames and streams
    def gstep():
        quantize_layer(dev["W"], dev["X"], dev["P_out"], dev["P_in"], bufs, H=bufs.H,
                       block=wl.block, damp=wl.damp, clip_sigmas=wl.clip_sigmas, stream=stream,
                       side_stream=side)

    gstep()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        gstep()
    torch.cuda.synchronize()
    gms = (time.perf_counter() - t0) * 1000.0 / args.steps
    out["pass_given_H"] = {"ms_per_step": round(gms, 3),
                           "weights_per_s": round(L.d_out * L.d_in / (gms / 1e3), 1),
                           "note": "S2 -> S4 with H from the headline pass"}
    print(f"[bench] pass with H given: {gms:.2f} ms/step", file=sys.stderr, flush=True)
    # the pass with the frames applied the other way, same inputs (one warmup, `steps` timed)
    other = "dense" if args.frames == "structured" else "structured"
    ob = LayerBuffers(L.d_out, L.d_in, K_out, K_in, dev["W"].dtype, dev["X"].dtype, n, wl.block,
                      frames=tff_frames if other == "structured" else None)

    def ostep():
        quantize_layer(dev["W"], dev["X"], dev["P_out"], dev["P_in"], ob, block=wl.block,
                       damp=wl.damp, clip_sigmas=wl.clip_sigmas, stream=stream)

    ostep()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ostep()
    torch.cuda.synchronize()
    oms = (time.perf_counter() - t0) * 1000.0 / args.steps
    out["other_frames"] = {"frames": other, "ms_per_step": round(oms, 3),
                           "weights_per_s": round(L.d_out * L.d_in / (oms / 1e3), 1),
                           "codes_differing_frac_vs_headline_pass": float(sum(
                               (((ob.codes >> (2 * j)) & 3) != ((bufs.codes >> (2 * j)) & 3))
                               .sum().item() for j in range(16)) / (K_out * K_in))}
    print(f"[bench] pass with {other} frames: {oms:.2f} ms/step", file=sys.stderr, flush=True)
    del ob
    inf = inference_bench(fq, torch, dev, bufs, L, K_out, K_in)
    inf["structured"] = structured_bench(fq, torch, dev, bufs, wl, li, K_out, K_in)
    out["inference"] = inf
    out["frame_generation"] = frame_generation_bench(fq, torch, dev, wl, li, host)
    out["grid_variants"] = grid_variants_bench(torch, dev, wl, li, L, K_out, K_in, n, args.steps,
                                               frames=frames)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, li, host)
        inf["cpu_baseline"] = cpu_inference_baseline(host, bufs.codes.cpu().numpy(),
                                                     bufs.scale.cpu().numpy(),
                                                     bufs.zero.cpu().numpy(), wl, li)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
