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


def _tff_geom(d, K, rho):
    """Block geometry of a frame as the structured pass lays it out: nb = rho/2 blocks of
    2m real coordinates padded to pm and 2k frame coordinates padded to pk (multiples of
    32); the rotation factors d1 x d2 (d1 <= d2, d1 as close to sqrt(d) as possible)."""
    k, m = K // rho, d // rho
    d1 = max(a for a in range(1, int(d ** 0.5) + 1) if d % a == 0)
    return dict(k=k, m=m, nb=rho // 2, pm=-(-2 * m // 32) * 32, pk=-(-2 * k // 32) * 32,
                d1=d1, d2=d // d1)


def _rot_exec(g):
    """fp32 MFMA flops issued per vector by the rotation.  Fused kernel (d1 <= 128,
    d2 % 4 == 0, the operands within LDS): rows padded to 16 (5 and 7 tiles of 16 to 6 and
    8), k of the first factor padded to 16, output columns in blocks of 64 (128 when
    d2 >= 128); both factors on those padded shapes.  Otherwise the two-step kernels: 64 x 64
    output tiles, k steps of 16."""
    p16 = lambda x: -(-x // 16) * 16
    d1, d2 = g["d1"], g["d2"]
    mt = p16(d1) // 16
    mt = {5: 6, 7: 8}.get(mt, mt)
    m, k2 = 16 * mt, p16(d2)
    bj = 128 if k2 >= 128 else 64
    lds = (m * (max(k2, bj) + 4) + bj * (k2 + 4) + m * (m + 4)) * 4
    maxq = 16 if bj == 64 else 8
    if d1 <= 128 and d2 % 4 == 0 and d1 * (d2 // 4) <= (bj * 4) * maxq and lds <= 160 * 1024:
        cols = -(-d2 // bj) * bj
        return 2 * m * cols * (k2 + m)
    p64 = lambda x: -(-x // 64) * 64
    return 2 * p64(d1) * p64(d2) * (p16(d2) + p16(d1))


def algorithmic_work(n, d_out, d_in, K_out, K_in, block, rho=None, w_dtype="bf16"):
    """Work per kernel group and step: (peak kind, algorithmic amount, executed amount).
    Contractions count flops (one pass of the useful product for 'algorithmic'; every
    bf16 pass of a split product for 'executed'), streaming kernels bytes.
    With structured frames (rho given) the per-block DFT products cost 4 d k flops per
    transformed row (executed: 2 nb pm pk per row and pass, the padded block layout) and
    the rotations 2 d (d1 + d2) flops per row (executed: the padded 64 x 64 tiles).  The
    analysis (_an) transforms d_out rows of W, d_in rows of H and K_in rows of H P_in by
    the input frame, then K_in rows of W P_in by the output frame; the synthesis (_syn)
    transforms K_out code rows by the input frame (2 passes: exact codes), then d_in rows
    by the output frame."""
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
    chol = K_in ** 3 // 3                   # the factorization: n^3 / 3 flops
    work = {}
    if rho is not None:
        gi, go = _tff_geom(d_in, K_in, rho), _tff_geom(d_out, K_out, rho)
        dft_i = lambda rows, passes: (4 * d_in * gi["k"] * rows,
                                      passes * 2 * gi["nb"] * gi["pm"] * gi["pk"] * rows)
        dft_o = lambda rows, passes: (4 * d_out * go["k"] * rows,
                                      passes * 2 * go["nb"] * go["pm"] * go["pk"] * rows)
        rot_i = lambda rows: (2 * d_in * (gi["d1"] + gi["d2"]) * rows, _rot_exec(gi) * rows)
        rot_o = lambda rows: (2 * d_out * (go["d1"] + go["d2"]) * rows, _rot_exec(go) * rows)
        add = lambda a, b: (a[0] + b[0], a[1] + b[1])
        a1, a2 = dft_i(d_out + d_in + K_in, 3), dft_o(K_in, 3)
        work["tffp_dft_an"] = ("bf16",) + add(a1, a2)
        # the synthesis from the left: the code matrix's K_in columns through P_out (exact
        # integer operand: 2 passes), then the d_out rows through P_in
        work["tffp_dft_syn"] = ("bf16",) + add(dft_o(K_in, 2), dft_i(d_out, 3))
        work["tffp_rotate_an"] = ("f32",) + add(rot_i(d_out + d_in + K_in), rot_o(K_in))
        work["tffp_rotate_syn"] = ("f32",) + add(rot_o(K_in), rot_i(d_out))
    hess_tiles = (-(-d_in // 256)) * (-(-d_in // 256) + 1) // 2
    passes = {"gemm_hessian": 1, "gemm_analysis_w1": 2 if w_dtype == "bf16" else 3,
              "gemm_analysis_w2": 3, "gemm_analysis_h1": 3, "gemm_analysis_h2": 3,
              "gemm_synthesis_1": 2, "gemm_synthesis_2": 3}
    dense = {"gemm_hessian": n * d_in * (d_in + 1),
             "gemm_analysis_w1": 2 * K_out * d_out * d_in,
             "gemm_analysis_w2": 2 * K_out * d_in * K_in,
             "gemm_analysis_h1": 2 * d_in * d_in * K_in,
             "gemm_analysis_h2": K_in * (K_in + 1) * d_in,
             "gemm_synthesis_1": 2 * d_out * K_out * K_in,
             "gemm_synthesis_2": 2 * d_out * K_in * d_in}
    for k, v in dense.items():
        ex = passes[k] * v
        if k == "gemm_hessian":        # upper 256 x 256 tiles of the symmetric product
            ex = hess_tiles * 256 * 256 * 2 * n
        work[k] = ("bf16", v, ex)
    work.update({
        "gptq_update": ("f64", gptq_lazy, gptq_lazy),
        "gptq_update_lazy": ("f64", gptq_lazy, gptq_lazy),
        "chol": ("f64", chol, None),
        # the rounding kernel: the in-span products (the span's earlier chunks into each
        # chunk, fp64 MFMA) plus the in-block FMAs (upper bound)
        "gptq_block": ("f64", gptq_upd - gptq_lazy + K_out * K_in * 128, None),
        "pack2": ("hbm", K_out * K_in + K_out * ((K_in + 15) // 16) * 4, None),
    })
    return work


# contraction groups of the spec MFMA target: S1 and the frame transforms of S2
# (analysis) and S4 (synthesis)
CONTRACTIONS_S2 = ["gemm_analysis_w1", "gemm_analysis_w2", "gemm_analysis_h1",
                   "gemm_analysis_h2", "tffp_dft_an", "tffp_rotate_an"]
CONTRACTIONS_S4 = ["gemm_synthesis_1", "gemm_synthesis_2", "tffp_dft_syn", "tffp_rotate_syn"]

KERNEL_GROUPS = ["gemm_hessian", "gemm_analysis_w1", "gemm_analysis_w2", "gemm_analysis_h1",
                 "gemm_analysis_h2", "gemm_synthesis_1", "gemm_synthesis_2", "tffp_rotate_an",
                 "tffp_rotate_syn", "tffp_blocks", "tffp_dft_an", "tffp_dft_syn", "tffp_gather",
                 "gptq_update", "gptq_update_lazy", "gptq_block", "chol",
                 "chol_syrk", "chol_potrf", "chol_trsm", "q_", "split_bf16", "syrk_reduce",
                 "dequant", "pack2"]


def kernel_table(fq, work, steps):
    """Per kernel group: launches, ms per step and, where the work is defined, the rate
    against its own peak (algorithmic and executed), from the library's kernel timers."""
    kernels = {}
    for name in KERNEL_GROUPS:
        cnt, tot = fq.fq_profile_query(name)
        if cnt == 0:
            continue
        e = {"launches_per_step": cnt / steps, "ms_per_step": round(tot / steps, 4)}
        if name in work:
            kind, amount, executed = work[name]
            sec = tot / steps / 1000.0
            if kind == "hbm":
                e["GB/s"] = round(amount / sec / 1e9, 1)
                e["frac_of_peak"] = round(amount / sec / 1e9 / PEAK["hbm"], 4)
            else:
                e["peak"] = kind
                e["TFLOP/s"] = round(amount / sec / 1e12, 2)
                e["frac_of_peak"] = round(amount / sec / 1e12 / PEAK[kind], 4)
                if executed is not None and executed != amount:
                    e["executed_TFLOP/s"] = round(executed / sec / 1e12, 2)
                    e["executed_frac_of_peak"] = round(executed / sec / 1e12 / PEAK[kind], 4)
        kernels[name] = e
    return kernels


def contraction_summary(kernels, work, groups):
    """Combined MFMA fraction of several contraction groups, each against its own dtype's
    peak: (sum of work / peak) / (sum of time), i.e. the time the work takes at peak rate
    over the time it took.  Algorithmic and executed (every bf16 pass) separately."""
    used = [g for g in groups if g in kernels and g in work]
    t = sum(kernels[g]["ms_per_step"] for g in used) / 1e3
    if t <= 0:
        return None
    alg = sum(work[g][1] / (PEAK[work[g][0]] * 1e12) for g in used)
    exe = sum((work[g][2] if work[g][2] is not None else work[g][1]) / (PEAK[work[g][0]] * 1e12)
              for g in used)
    return {"groups": used, "ms_per_step": round(t * 1e3, 4), "algorithmic_frac": round(alg / t, 4),
            "executed_frac": round(exe / t, 4)}


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


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:
        return len(os.sched_getaffinity(0))


def cpu_baseline(wl, li, host, chunk=8192):
    """The float64 oracle's whole pass on the same layer and inputs, nothing sampled or
    extrapolated: H over every calibration token (chunks of `chunk` tokens upcast to
    float64), D and H~ with the dense float64-exact frames, OPTQ's preparation (literal
    U = chol(H~^-1)), clip, grid and rounding of every row, packing, and W^."""
    import oracle as O
    from fq_inputs import gen
    L = wl.layers[li]
    X = host["X"]
    n = X.shape[0]
    t = {}
    s0 = time.perf_counter()
    H = O.hessian(gen.storage_to_f32(X[c:c + chunk], wl.x_dtype) for c in range(0, n, chunk))
    t["hessian"] = time.perf_counter() - s0
    W64 = gen.storage_to_f32(host["W"], wl.w_dtype).astype(np.float64)
    Po = host["P_out"].astype(np.float64)
    Pi = host["P_in"].astype(np.float64)
    s0 = time.perf_counter()
    D, _ = O.frame_analysis(W64, Po, Pi, None)
    t["analysis_D"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    _, Ht = O.frame_analysis(W64[:0], Po[:0, :0], Pi, H)
    t["analysis_Ht"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    U, dead, _ = O.gptq_prepare(Ht, wl.damp)
    t["factor"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    mu, sigma, lo, hi = O.clip_bounds(D, wl.clip_sigmas)
    Dc = O.apply_clip(D, lo, hi)
    sc, z = O.row_grid(Dc, wl.bits)
    r = O.gptq(Dc, U, sc, z, wl.bits, wl.block, dead)
    t["clip_grid_optq"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    O.pack2(r["codes"])
    t["pack"] = time.perf_counter() - s0
    s0 = time.perf_counter()
    O.synthesis(r["codes"], sc, z, Po, Pi)
    t["synthesis"] = time.perf_counter() - s0
    total = sum(t.values())
    return {"value": L.d_out * L.d_in / total, "unit": "weights/s", "cores": int(_blas_threads()),
            "kind": "oracle", "cpu_model": _cpu_model(),
            "sample": (f"the whole pass on the benchmark layer, nothing sampled: H over all {n} "
                       f"tokens, D and H~, OPTQ on all {D.shape[0]} x {D.shape[1]} frame "
                       f"coefficients, pack, W^ ({total:.1f} s in float64 numpy/LAPACK)"),
            "seconds": round(total, 2),
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


def wiener_bench(fq, torch, bufs, K_out, K_in, steps):
    """The diagonal Wiener gains of the headline layer (fq_wiener_gains on the pass's own
    D, H~ and codes), timed with HIP events on the launch stream; the product (q - zero) H~
    runs as 2 bf16 passes of 2 K_out K_in^2 flops each."""
    stream = torch.cuda.current_stream()
    ws = torch.empty(fq.lib().fq_wiener_gains_workspace_bytes(K_out, K_in), dtype=torch.uint8,
                     device="cuda")
    g = torch.empty((K_out,), dtype=torch.float32, device="cuda")
    so = torch.empty_like(g)

    def call():
        fq.fq_wiener_gains(bufs.D, bufs.Ht, bufs.codes, bufs.scale, bufs.zero, gain=g,
                           scale_out=so, ws=ws, stream=stream)

    us = _time_calls(torch, call, stream, max(steps, 5))
    kern = _kernel_us(fq, torch, call, ("gemm_wiener", "wiener_rows", "dequant", "split_bf16"),
                      max(steps, 5))
    flops = 2.0 * K_out * K_in * K_in
    gu = kern["gemm_wiener"]["us_per_call"]
    kern["gemm_wiener"]["TFLOP/s"] = round(flops / (gu * 1e-6) / 1e12, 1)
    kern["gemm_wiener"]["frac_of_bf16_peak"] = round(flops / (gu * 1e-6) / 1e12 / PEAK["bf16"], 4)
    kern["gemm_wiener"]["executed_frac_of_bf16_peak"] = round(2 * flops / (gu * 1e-6) / 1e12 / PEAK["bf16"], 4)
    gh = g.cpu()
    print(f"[bench] Wiener gains: {us / 1e3:.2f} ms/call", file=sys.stderr, flush=True)
    return {"op": "fq_wiener_gains: per-row gains of the diagonal Wiener filter from D, H~ and "
                  "the codes, folded into the scale", "ms_per_call": round(us / 1e3, 3),
            "gain_range": [round(float(gh.min()), 4), round(float(gh.max()), 4)],
            "kernels": kern}


def prepare_bench(fq, torch, bufs, wl, K_out, K_in, steps):
    """fq_quantize_prepare on the headline pass's H~ (damping, Cholesky factor, R and its
    diagonal), timed with HIP events on the launch stream with nothing beside it: the
    factorization's trailing updates then run on the library's auxiliary stream beside the
    panel chain, so this is the critical path that the kernel timers (which serialize every
    launch on one stream) overstate."""
    stream = torch.cuda.current_stream()

    def call():
        fq.fq_quantize_prepare(bufs.Ht, K_out, bufs.ws_q, block=wl.block, damp=wl.damp,
                               stream=stream)

    us = _time_calls(torch, call, stream, max(steps, 5))
    kern = _kernel_us(fq, torch, call, ("chol_block", "chol_syrk", "q_"), max(steps, 5))
    flops = K_in ** 3 / 3.0
    print(f"[bench] prepare (factorization): {us / 1e3:.2f} ms/call", file=sys.stderr,
          flush=True)
    return {"op": "fq_quantize_prepare: damped H~, its Cholesky factor and R (H~ = R R^T), "
                  "trailing updates on the auxiliary stream", "K_in": K_in,
            "ms_per_call": round(us / 1e3, 3),
            "chol_TFLOP/s_wall": round(flops / (us * 1e-6) / 1e12, 2),
            "kernels_serialized": kern}


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


def roofline_of(kernels, work):
    """The dominant kernel group with a defined algorithmic count ("gptq_update" sums its
    _lazy and _span launches, which run on two different kernels; "chol" has no single
    kernel), against its own peak."""
    cands = [k for k in kernels if k in work and k not in ("gptq_update", "chol")]
    dom = max(cands, key=lambda k: kernels[k]["ms_per_step"])
    kind, amount, _ = work[dom]
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
    roof["kernel"] = dom
    roof["avg_launch_ms"] = round(avg_ms, 4)
    roof["algorithmic_per_launch"] = per_launch
    return roof


def timed_steps(torch, step, steps):
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1000.0 / steps


def profiled_steps(torch, fq, step, steps, work):
    """`steps` more passes under the kernel timers (one stream): (ms per step, kernel
    table, total kernel ms per step)."""
    fq.fq_profile_reset()
    fq.fq_profile_enable(True)
    ms = timed_steps(torch, step, steps)
    fq.fq_profile_enable(False)
    kernels = kernel_table(fq, work, steps)
    _, tot = fq.fq_profile_query("")
    fq.fq_profile_reset()
    return ms, kernels, tot / steps


def contraction_block(kernels, work):
    return {"S1_S2": contraction_summary(kernels, work, ["gemm_hessian"] + CONTRACTIONS_S2),
            "S1_S2_S4": contraction_summary(kernels, work,
                                            ["gemm_hessian"] + CONTRACTIONS_S2 + CONTRACTIONS_S4),
            "S2_S4": contraction_summary(kernels, work, CONTRACTIONS_S2 + CONTRACTIONS_S4)}


CONFIG_LAYERS = [("tiny256", 0), ("vitb", 0), ("vitb", 1), ("opt1b3", 0), ("llama7b", 0),
                 ("llama7b", 1), ("llama70b_r1.0", 0), ("llama70b_r1.1", 0)]


def configs_bench(torch, fq, headline, side, steps_small=5, steps_big=3):
    """Every workload layer through the same pass (structured frames, two streams): ms per
    step and weights per second from HIP-synchronized wall time around `steps` passes
    (more for small layers, about 30 ms in all) after one warmup, then one pass under the
    kernel timers for the dominant kernel's
    roofline and the contraction fractions.  The headline layer's entry repeats the
    headline figures.  GPU only (the oracle is timed on the headline layer alone)."""
    from paper_2403_06082_amd.pipeline import LayerBuffers, quantize_layer
    from fq_inputs import WORKLOADS, gen
    out = {}
    for key, li in CONFIG_LAYERS:
        wl = WORKLOADS[key]
        L = wl.layers[li]
        name = f"{key}:{L.name}"
        if (key, li) == headline[0]:
            out[name] = headline[1]
            continue
        t0 = time.time()
        Xs = gen.make_x(wl, L.d_in)
        X = torch.from_numpy(Xs)
        X = (X.view(torch.bfloat16) if wl.x_dtype == "bf16" else X).cuda()
        del Xs
        Ws = gen.make_weight(wl, li)
        W = torch.from_numpy(Ws)
        W = (W.view(torch.bfloat16) if wl.w_dtype == "bf16" else W).cuda()
        (ko, ro, R1o, R2o), (ki, ri, R1i, R2i) = gen.layer_frame_factors(wl, li)
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
        F = (fq.Frame(L.d_out, ko, ro, up(R1o), up(R2o)), fq.Frame(L.d_in, ki, ri, up(R1i), up(R2i)))
        K_out, K_in = F[0].K, F[1].K
        n = X.shape[0]
        bufs = LayerBuffers(L.d_out, L.d_in, K_out, K_in, W.dtype, X.dtype, n, wl.block, frames=F)
        stream = torch.cuda.current_stream()

        def step(two=True):
            quantize_layer(W, X, None, None, bufs, block=wl.block, damp=wl.damp,
                           clip_sigmas=wl.clip_sigmas, stream=stream,
                           side_stream=side if two else None)

        steps = steps_big if K_in > 10000 else steps_small
        step()
        # small layers run long enough (about 30 ms) that host-side noise averages out
        est = timed_steps(torch, step, 1)
        if est > 0:
            steps = max(steps, min(200, int(30.0 / est) + 1))
        ms = timed_steps(torch, step, steps)
        work = algorithmic_work(n, L.d_out, L.d_in, K_out, K_in, wl.block, rho=wl.rho,
                                w_dtype=wl.w_dtype)
        ms_t, kernels, _ = profiled_steps(torch, fq, lambda: step(False), 1, work)
        roof = roofline_of(kernels, work)
        e = {"workload": f"{key} {L.name}: W {L.d_out}x{L.d_in} {wl.w_dtype}, X {n}x{L.d_in} "
                         f"{wl.x_dtype}, K {K_out}x{K_in} (r={wl.r}, rho={wl.rho}), {wl.bits}-bit, "
                         f"block {wl.block}",
             "ms_per_step": round(ms, 3), "steps": steps,
             "weights_per_s": round(L.d_out * L.d_in / (ms / 1e3), 1),
             "roofline": roof, "contractions": contraction_block(kernels, work),
             "kernel_ms": {k: v["ms_per_step"] for k, v in kernels.items()}}
        out[name] = e
        print(f"[bench] config {name}: {ms:.2f} ms/step ({e['weights_per_s']:.3g} weights/s), "
              f"dominant {roof['kernel']} at {roof['frac']:.3f} of peak "
              f"({time.time() - t0:.1f}s with input generation)", file=sys.stderr, flush=True)
        del bufs, X, W, F
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama7b")
    ap.add_argument("--layer", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload section (every other layer shape)")
    ap.add_argument("--streams", type=int, default=2, choices=(1, 2),
                    help="2 (default): D is formed on a second stream while the main stream "
                         "factors H~ (the factorization is a chain of small kernels that leaves "
                         "most CUs idle); 1: one stream.  The kernel-timer region always uses one")
    ap.add_argument("--reserve-cus", type=int, default=144,
                    help="with two streams, the second is made by fq_side_stream_create and its "
                         "kernels stay off this many compute units, which the factorization's "
                         "chain keeps for itself (0: an ordinary second stream)")
    ap.add_argument("--frames", default="structured", choices=("structured", "dense"),
                    help="how the pass applies the frames in the analysis and the synthesis: "
                         "from their construction (default) or as the dense d x K matrices; "
                         "the other way is timed beside it")
    ap.add_argument("--pass-only", action="store_true",
                    help="time the pass only (no pass with the other frames, no inference, frame "
                         "generation, grid variants or other workloads): the kernel trace then "
                         "covers exactly the warmup, timed and kernel-timer passes")
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
    # everything runs on a non-blocking stream of its own: the side stream that
    # fq_side_stream_create makes synchronizes with the legacy default stream, so work on
    # the default stream would not overlap it
    torch.cuda.set_stream(torch.cuda.Stream())
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
    side_handle = fq.SideStream(args.reserve_cus) if args.streams == 2 else None
    side = side_handle.stream if side_handle is not None else None

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
    # timed region: the pass alone
    ms = timed_steps(torch, step, args.steps)
    print(f"[bench] {args.steps} timed steps: {ms:.2f} ms/step", file=sys.stderr, flush=True)
    # second timed region with the per-launch kernel timers (HIP events on the launch
    # stream around every kernel): the per-kernel breakdown and the roofline come from it.
    # One stream here (the library keeps its own look-ahead on the caller's stream while
    # the timers are on), so that no two timed kernels overlap.
    work = algorithmic_work(n, L.d_out, L.d_in, K_out, K_in, wl.block,
                            rho=wl.rho if frames is not None else None, w_dtype=wl.w_dtype)
    ms_timed, kernels, k_total = profiled_steps(torch, fq, lambda: step(False), args.steps, work)
    print(f"[bench] {args.steps} steps with kernel timers: {ms_timed:.2f} ms/step", file=sys.stderr,
          flush=True)
    roof = roofline_of(kernels, work)
    roof["traffic"] = measured_traffic(roof["kernel"])
    contr = contraction_block(kernels, work)

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
        "dtype": "bf16 MFMA (fp32 acc) + fp32 MFMA (rotations) + fp64",
        "data": "synthetic (seeded; Gaussian weights with 1% x10 outliers, Gaussian "
                "activations with 8 channels x100)",
        "config": {"workload": f"{wl.key} {L.name}_proj: W {L.d_out}x{L.d_in} {wl.w_dtype}, "
                               f"X {n}x{L.d_in} {wl.x_dtype}, frames K {K_out}x{K_in} "
                               f"(r={wl.r}, rho={wl.rho}), {wl.bits}-bit, block {wl.block}, "
                               f"damp {wl.damp}, clip {wl.clip_sigmas} sigma",
                   "d_out": L.d_out, "d_in": L.d_in, "n_tokens": n, "K_out": K_out,
                   "K_in": K_in, "streams": args.streams,
                   "side_stream_reserved_cus": args.reserve_cus if args.streams == 2 else None,
                   "frames": args.frames},
        "roofline": roof,
        # combined MFMA fraction of the Hessian and the frame-transform contractions of
        # the analysis (S1 + S2), each group against its own dtype's peak
        "contraction_mfma_frac": contr["S1_S2"]["algorithmic_frac"] if contr["S1_S2"] else None,
        "contraction_mfma_executed_frac": contr["S1_S2"]["executed_frac"] if contr["S1_S2"] else None,
        "contractions": contr,
        "kernels": kernels,
        "kernel_ms_total_per_step": round(k_total, 3),
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
    gms = timed_steps(torch, gstep, args.steps)
    out["pass_given_H"] = {"ms_per_step": round(gms, 3),
                           "weights_per_s": round(L.d_out * L.d_in / (gms / 1e3), 1),
                           "note": "S2 -> S4 with H from the headline pass"}
    print(f"[bench] pass with H given: {gms:.2f} ms/step", file=sys.stderr, flush=True)
    # the pass with the frames applied the other way, same inputs (one warmup, `steps`
    # timed, then `steps` under the kernel timers)
    other = "dense" if args.frames == "structured" else "structured"
    ob = LayerBuffers(L.d_out, L.d_in, K_out, K_in, dev["W"].dtype, dev["X"].dtype, n, wl.block,
                      frames=tff_frames if other == "structured" else None)

    def ostep():
        quantize_layer(dev["W"], dev["X"], dev["P_out"], dev["P_in"], ob, block=wl.block,
                       damp=wl.damp, clip_sigmas=wl.clip_sigmas, stream=stream)

    ostep()
    oms = timed_steps(torch, ostep, args.steps)
    owork = algorithmic_work(n, L.d_out, L.d_in, K_out, K_in, wl.block,
                             rho=wl.rho if other == "structured" else None, w_dtype=wl.w_dtype)
    _, okern, _ = profiled_steps(torch, fq, ostep, args.steps, owork)
    out["other_frames"] = {"frames": other, "ms_per_step": round(oms, 3),
                           "weights_per_s": round(L.d_out * L.d_in / (oms / 1e3), 1),
                           "codes_differing_frac_vs_headline_pass": float(sum(
                               (((ob.codes >> (2 * j)) & 3) != ((bufs.codes >> (2 * j)) & 3))
                               .sum().item() for j in range(16)) / (K_out * K_in)),
                           "contractions": contraction_block(okern, owork),
                           "kernels": okern}
    print(f"[bench] pass with {other} frames: {oms:.2f} ms/step", file=sys.stderr, flush=True)
    del ob
    inf = inference_bench(fq, torch, dev, bufs, L, K_out, K_in)
    inf["structured"] = structured_bench(fq, torch, dev, bufs, wl, li, K_out, K_in)
    out["inference"] = inf
    out["frame_generation"] = frame_generation_bench(fq, torch, dev, wl, li, host)
    out["grid_variants"] = grid_variants_bench(torch, dev, wl, li, L, K_out, K_in, n, args.steps,
                                               frames=frames)
    out["wiener_filter"] = wiener_bench(fq, torch, bufs, K_out, K_in, args.steps)
    out["quantize_prepare"] = prepare_bench(fq, torch, bufs, wl, K_out, K_in, args.steps)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on the whole pass", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, li, host)
        print(f"[bench] CPU oracle: {out['cpu_baseline']['seconds']} s", file=sys.stderr,
              flush=True)
        inf["cpu_baseline"] = cpu_inference_baseline(host, bufs.codes.cpu().numpy(),
                                                     bufs.scale.cpu().numpy(),
                                                     bufs.zero.cpu().numpy(), wl, li)
    if not args.no_configs:
        headline = ((args.workload, li),
                    {"workload": out["config"]["workload"], "ms_per_step": out["ms_per_step"],
                     "steps": args.steps, "weights_per_s": out["value"], "roofline": roof,
                     "contractions": contr, "note": "the headline pass above"})
        del bufs, dev, host
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        out["configs"] = configs_bench(torch, fq, headline, side if side is not None else torch.cuda.Stream())
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
