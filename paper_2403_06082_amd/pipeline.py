"""The whole per-layer pass (Alg. 1) as the four ABI calls in order, on device tensors.

    H      = fq_hessian_accumulate(X)              (skipped when H is given)
    D, Ht  = fq_frame_analysis(W, P_out, P_in, H)  (Ht skipped when given)
    codes  = fq_quantize_frames(D, Ht)
    W_hat  = fq_frame_synthesis(codes, ...)

Workspaces are allocated once per call site with torch and reused.
"""
from __future__ import annotations

from . import fq as _fq


class LayerBuffers:
    """Device outputs and workspaces for one layer shape (reused across calls)."""

    def __init__(self, d_out, d_in, K_out, K_in, w_dtype, x_dtype, n_tokens, block=128,
                 device="cuda"):
        import torch
        f32 = torch.float32
        self.H = torch.empty((d_in, d_in), dtype=f32, device=device)
        self.D = torch.empty((K_out, K_in), dtype=f32, device=device)
        self.Ht = torch.empty((K_in, K_in), dtype=f32, device=device)
        self.codes = torch.empty((K_out, (K_in + 15) // 16), dtype=torch.int32, device=device)
        self.scale = torch.empty((K_out,), dtype=f32, device=device)
        self.zero = torch.empty((K_out,), dtype=f32, device=device)
        self.W_hat = torch.empty((d_out, d_in), dtype=f32, device=device)
        dt = {torch.float32: _fq.FQ_F32, torch.float16: _fq.FQ_F16,
              torch.bfloat16: _fq.FQ_BF16}
        u8 = torch.uint8
        self.ws_h = torch.empty(_fq.fq_hessian_workspace_bytes(dt[x_dtype], n_tokens, d_in),
                                dtype=u8, device=device)
        self.ws_a = torch.empty(_fq.fq_frame_analysis_workspace_bytes(dt[w_dtype], d_out, d_in,
                                                                      K_out, K_in),
                                dtype=u8, device=device)
        self.ws_q = torch.empty(_fq.fq_quantize_frames_workspace_bytes(K_out, K_in, block),
                                dtype=u8, device=device)
        self.ws_s = torch.empty(_fq.fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in),
                                dtype=u8, device=device)


def quantize_layer(W, X, P_out, P_in, bufs: LayerBuffers, H=None, Ht=None, bits=2, block=128,
                   damp=0.01, clip_sigmas=2.0, stream=None):
    """Run the pass; returns bufs (H, D, Ht, codes, scale, zero, W_hat filled in)."""
    if H is None:
        _fq.fq_hessian_accumulate(X, bufs.H, ws=bufs.ws_h, stream=stream)
        H = bufs.H
    if Ht is None:
        _fq.fq_frame_analysis(W, P_out, P_in, H, bufs.D, bufs.Ht, ws=bufs.ws_a, stream=stream)
        Ht = bufs.Ht
    else:
        _fq.fq_frame_analysis(W, P_out, P_in, None, bufs.D, None, ws=bufs.ws_a, stream=stream)
    _fq.fq_quantize_frames(bufs.D, Ht, bufs.codes, bufs.scale, bufs.zero, bits=bits, block=block,
                           damp=damp, clip_sigmas=clip_sigmas, ws=bufs.ws_q, stream=stream)
    _fq.fq_frame_synthesis(bufs.codes, bufs.scale, bufs.zero, P_out, P_in, bufs.W_hat,
                           ws=bufs.ws_s, stream=stream)
    return bufs
