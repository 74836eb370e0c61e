"""The whole per-layer pass (Alg. 1) as the four ABI calls in order, on device tensors.

    H      = fq_hessian_accumulate(X)              (skipped when H is given)
    D, Ht  = fq_frame_analysis(W, P_out, P_in, H)  (Ht skipped when given)
    codes  = fq_quantize_frames(D, Ht)
    W_hat  = fq_frame_synthesis(codes, ...)

Workspaces are allocated once per call site with torch and reused.

With frames given by their construction (LayerBuffers(..., frames=(F_out, F_in)), fq.Frame
objects), the analysis and the synthesis are fq_frame_analysis_tff / fq_frame_synthesis_tff
and the dense P_out, P_in are not read (pass None).

With a second stream (side_stream), D = P_out^T W P_in is formed there, followed by the
part of the rounding that reads D only (fq_quantize_grid: clip bounds, per-row grid),
while the main stream factors the damped H~ (fq_quantize_prepare): the Cholesky
factorization, a chain of small dependent kernels, then overlaps the D contractions.  The
main stream then rounds (fq_quantize_round_async) and synthesizes, and reads the checks
at the end (fq_quantize_status), so that no synchronization sits between the rounding and
the synthesis.  Outputs are identical.
A side stream from fq.SideStream keeps the D kernels off part of the device, so that the
chain always finds free compute units; it synchronizes with the legacy default stream, so
the main stream must then be another stream (torch.cuda.Stream()).
"""
from __future__ import annotations

from . import fq as _fq


class LayerBuffers:
    """Device outputs and workspaces for one layer shape (reused across calls)."""

    def __init__(self, d_out, d_in, K_out, K_in, w_dtype, x_dtype, n_tokens, block=128,
                 device="cuda", bits=2, frames=None):
        import torch
        f32 = torch.float32
        self.H = torch.empty((d_in, d_in), dtype=f32, device=device)
        self.D = torch.empty((K_out, K_in), dtype=f32, device=device)
        self.Ht = torch.empty((K_in, K_in), dtype=f32, device=device)
        self.bits = bits
        self.codes = torch.empty((K_out, _fq.words_per_row(K_in, bits)), dtype=torch.int32,
                                 device=device)
        self.scale = torch.empty((K_out,), dtype=f32, device=device)
        self.zero = torch.empty((K_out,), dtype=f32, device=device)
        self.W_hat = torch.empty((d_out, d_in), dtype=f32, device=device)
        dt = {torch.float32: _fq.FQ_F32, torch.float16: _fq.FQ_F16,
              torch.bfloat16: _fq.FQ_BF16}
        u8 = torch.uint8
        self.ws_h = torch.empty(_fq.fq_hessian_workspace_bytes(dt[x_dtype], n_tokens, d_in),
                                dtype=u8, device=device)
        self.frames = frames
        if frames is None:
            na = _fq.fq_frame_analysis_workspace_bytes(dt[w_dtype], d_out, d_in, K_out, K_in)
            ns = _fq.fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in)
        else:
            fo, fi = frames
            if (fo.d, fi.d, fo.K, fi.K) != (d_out, d_in, K_out, K_in):
                raise ValueError("frames do not match the layer shape")
            na = _fq.fq_frame_analysis_tff_workspace_bytes(dt[w_dtype], fo, fi)
            ns = _fq.fq_frame_synthesis_tff_workspace_bytes(fo, fi)
        self.ws_a = torch.empty(na, dtype=u8, device=device)
        self.ws_a2 = None      # second analysis workspace, for the two-stream order
        self.ws_q = torch.empty(_fq.fq_quantize_frames_workspace_bytes(K_out, K_in, block),
                                dtype=u8, device=device)
        self.ws_s = torch.empty(ns, dtype=u8, device=device)


def _analysis(W, P_out, P_in, bufs, H, D, Ht, ws, stream):
    if bufs.frames is None:
        _fq.fq_frame_analysis(W, P_out, P_in, H, D, Ht, ws=ws, stream=stream)
    else:
        _fq.fq_frame_analysis_tff(W if D is not None else None, bufs.frames[0], bufs.frames[1],
                                  H, D, Ht, ws=ws, stream=stream)


def _synthesis(P_out, P_in, bufs, bits, stream):
    if bufs.frames is None:
        _fq.fq_frame_synthesis(bufs.codes, bufs.scale, bufs.zero, P_out, P_in, bufs.W_hat,
                               ws=bufs.ws_s, stream=stream, bits=bits)
    else:
        _fq.fq_frame_synthesis_tff(bufs.codes, bufs.scale, bufs.zero, bufs.frames[0],
                                   bufs.frames[1], bufs.W_hat, ws=bufs.ws_s, stream=stream,
                                   bits=bits)


def quantize_layer(W, X, P_out, P_in, bufs: LayerBuffers, H=None, Ht=None, bits=2, block=128,
                   damp=0.01, clip_sigmas=2.0, stream=None, side_stream=None):
    """Run the pass; returns bufs (H, D, Ht, codes, scale, zero, W_hat filled in)."""
    if side_stream is not None:
        return _quantize_layer_two_streams(W, X, P_out, P_in, bufs, H, Ht, bits, block, damp,
                                           clip_sigmas, stream, side_stream)
    if H is None:
        _fq.fq_hessian_accumulate(X, bufs.H, ws=bufs.ws_h, stream=stream)
        H = bufs.H
    if Ht is None:
        _analysis(W, P_out, P_in, bufs, H, bufs.D, bufs.Ht, bufs.ws_a, stream)
        Ht = bufs.Ht
    else:
        _analysis(W, P_out, P_in, bufs, None, bufs.D, None, bufs.ws_a, stream)
    # fq_quantize_frames in its parts, the checks read after the synthesis
    _fq.fq_quantize_prepare(Ht, bufs.D.shape[0], bufs.ws_q, block=block, damp=damp, stream=stream)
    _fq.fq_quantize_grid(bufs.D, bufs.scale, bufs.zero, bufs.ws_q, bits=bits, block=block,
                         clip_sigmas=clip_sigmas, stream=stream)
    _fq.fq_quantize_round_async(bufs.D, bufs.codes, bufs.ws_q, bits=bits, block=block,
                                stream=stream)
    _synthesis(P_out, P_in, bufs, bits, stream)
    _fq.fq_quantize_status(bufs.D.shape[0], bufs.D.shape[1], bufs.ws_q, block=block, stream=stream)
    return bufs


def _quantize_layer_two_streams(W, X, P_out, P_in, bufs, H, Ht, bits, block, damp,
                                clip_sigmas, stream, side):
    import torch
    main = torch.cuda.current_stream() if stream is None else stream
    if bufs.ws_a2 is None:
        bufs.ws_a2 = torch.empty_like(bufs.ws_a)
    if H is None and Ht is None:
        _fq.fq_hessian_accumulate(X, bufs.H, ws=bufs.ws_h, stream=main)
        H = bufs.H
    if Ht is None:
        _analysis(W, P_out, P_in, bufs, H, None, bufs.Ht, bufs.ws_a, main)
        Ht = bufs.Ht
    # D on the side stream, started once H~ is done (so that it does not delay H~)
    ready = torch.cuda.Event()
    ready.record(main)
    side.wait_event(ready)
    _analysis(W, P_out, P_in, bufs, None, bufs.D, None, bufs.ws_a2, side)
    _fq.fq_quantize_grid(bufs.D, bufs.scale, bufs.zero, bufs.ws_q, bits=bits, block=block,
                         clip_sigmas=clip_sigmas, stream=side)
    d_done = torch.cuda.Event()
    d_done.record(side)
    _fq.fq_quantize_prepare(Ht, bufs.D.shape[0], bufs.ws_q, block=block, damp=damp, stream=main)
    main.wait_event(d_done)
    # the synthesis follows the rounding on the stream; the checks come after both
    _fq.fq_quantize_round_async(bufs.D, bufs.codes, bufs.ws_q, bits=bits, block=block,
                                stream=main)
    _synthesis(P_out, P_in, bufs, bits, main)
    _fq.fq_quantize_status(bufs.D.shape[0], bufs.D.shape[1], bufs.ws_q, block=block, stream=main)
    return bufs
