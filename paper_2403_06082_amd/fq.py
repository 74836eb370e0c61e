"""Thin Python binding of libfq (the C ABI in include/fq.h).

Argument marshalling only: every function here checks tensor placement, shape and dtype,
turns tensors into device pointers, allocates the caller-side workspace with torch when
none is given, and calls the library.  All arithmetic of the pass runs in libfq's HIP
kernels; nothing here falls back to another implementation.  Loading fails loudly when
libfq.so has not been built.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfq.so")

FQ_F32, FQ_F16, FQ_BF16 = 0, 1, 2
STATUS = {0: "FQ_OK", 1: "FQ_ERR_INVALID_ARG", 2: "FQ_ERR_UNSUPPORTED",
          3: "FQ_ERR_NOT_POSITIVE_DEFINITE", 4: "FQ_ERR_NONFINITE",
          5: "FQ_ERR_WORKSPACE_TOO_SMALL", 6: "FQ_ERR_HIP"}



def words_per_row(K_in: int, bits: int = 2) -> int:
    """uint32 words of one row of packed codes: floor(32 / bits) codes per word."""
    cpw = 32 // bits
    return (K_in + cpw - 1) // cpw


class TFF(ctypes.Structure):
    """struct fq_tff: a tight fusion frame given by (d, k, rho) and its rotation factors."""
    _fields_ = [("d", ctypes.c_int64), ("k", ctypes.c_int64), ("rho", ctypes.c_int64),
                ("R1", ctypes.c_void_p), ("d1", ctypes.c_int64),
                ("R2", ctypes.c_void_p), ("d2", ctypes.c_int64)]


_tp = ctypes.POINTER(TFF)

# exported symbols of include/fq.h: name -> (restype, argtypes)
_vp, _i64, _i, _sz, _d = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t, ctypes.c_double
SIGNATURES = {
    "fq_hessian_accumulate": (_i, [_vp, _vp, _i, _i64, _i64, _i64, _vp, _i, _vp, _sz]),
    "fq_hessian_workspace_bytes": (_sz, [_i, _i64, _i64]),
    "fq_frame_analysis": (_i, [_vp, _vp, _i, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp,
                               _vp, _sz]),
    "fq_frame_analysis_workspace_bytes": (_sz, [_i, _i64, _i64, _i64, _i64]),
    "fq_quantize_frames": (_i, [_vp, _vp, _vp, _i64, _i64, _i, _i, _d, _d, _vp, _vp, _vp, _vp,
                                _sz]),
    "fq_quantize_frames_workspace_bytes": (_sz, [_i64, _i64, _i]),
    "fq_quantize_prepare": (_i, [_vp, _vp, _i64, _i64, _i, _d, _vp, _sz]),
    "fq_quantize_apply": (_i, [_vp, _vp, _i64, _i64, _i, _i, _d, _vp, _vp, _vp, _vp, _sz]),
    "fq_quantize_grid": (_i, [_vp, _vp, _i64, _i64, _i, _i, _d, _vp, _vp, _vp, _sz]),
    "fq_quantize_round": (_i, [_vp, _vp, _i64, _i64, _i, _i, _vp, _vp, _sz]),
    "fq_quantize_round_async": (_i, [_vp, _vp, _i64, _i64, _i, _i, _vp, _vp, _sz]),
    "fq_quantize_status": (_i, [_vp, _i64, _i64, _i, _vp, _sz]),
    "fq_frame_synthesis": (_i, [_vp, _vp, _vp, _vp, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _vp,
                                _sz]),
    "fq_frame_synthesis_workspace_bytes": (_sz, [_i64, _i64, _i64, _i64]),
    "fq_frame_synthesis_nbit": (_i, [_vp, _vp, _i, _vp, _vp, _i64, _i64, _vp, _i64, _vp, _i64,
                                     _vp, _vp, _sz]),
    "fq_frame_apply": (_i, [_vp, _vp, _i, _i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _vp, _i64,
                            _vp, _vp, _vp, _sz]),
    "fq_frame_apply_workspace_bytes": (_sz, [_i64, _i64, _i64]),
    "fq_tff_analysis": (_i, [_vp, _vp, _i, _i64, _i64, _tp, _vp, _vp, _sz]),
    "fq_tff_analysis_workspace_bytes": (_sz, [_i64, _tp]),
    "fq_tff_synthesis": (_i, [_vp, _vp, _i64, _tp, _vp, _vp, _sz]),
    "fq_tff_synthesis_workspace_bytes": (_sz, [_i64, _tp]),
    "fq_frame_apply_tff": (_i, [_vp, _vp, _i, _i64, _i64, _vp, _vp, _vp, _tp, _tp, _vp, _vp,
                                _sz]),
    "fq_frame_apply_tff_workspace_bytes": (_sz, [_tp, _tp]),
    "fq_tff_materialize": (_i, [_vp, _tp, _vp, _i64, _vp, _sz]),
    "fq_tff_materialize_workspace_bytes": (_sz, [_tp]),
    "fq_frame_analysis_tff": (_i, [_vp, _vp, _i, _tp, _tp, _vp, _vp, _vp, _vp, _sz]),
    "fq_frame_analysis_tff_workspace_bytes": (_sz, [_i, _tp, _tp]),
    "fq_frame_synthesis_tff": (_i, [_vp, _vp, _i, _vp, _vp, _tp, _tp, _vp, _vp, _sz]),
    "fq_frame_synthesis_tff_workspace_bytes": (_sz, [_tp, _tp]),
    "fq_tff_rotation_factors": (_i, [_vp, ctypes.c_uint64, _i64, _i64, _vp, _vp, _vp, _sz]),
    "fq_frame_apply_nbit": (_i, [_vp, _vp, _i, _i64, _i64, _i64, _vp, _i, _vp, _vp, _i64, _i64,
                                 _vp, _i64, _vp, _vp, _vp, _sz]),
    "fq_frame_apply_tff_nbit": (_i, [_vp, _vp, _i, _i64, _i64, _vp, _i, _vp, _vp, _tp, _tp, _vp,
                                     _vp, _sz]),
    "fq_frame_apply_tff_noalloc": (_i, [_vp, _vp, _i, _i64, _i64, _vp, _i, _vp, _vp, _tp, _tp,
                                        _vp]),
    "fq_tff_rotation_factors_workspace_bytes": (_sz, [_i64, _i64]),
    "fq_act_quantize": (_i, [_vp, _vp, _i64, _i64, _i, _vp, _vp]),
    "fq_wiener_gains": (_i, [_vp, _vp, _vp, _vp, _i, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _sz]),
    "fq_wiener_gains_workspace_bytes": (_sz, [_i64, _i64]),
    "fq_tff_frame_valid": (_i, [_i64, _i64, _i64]),
    "fq_tff_choose": (_i, [_i64, _d, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                           ctypes.POINTER(_i64)]),
    "fq_frame_apply_tff_actq": (_i, [_vp, _vp, _i, _i64, _i64, _vp, _i, _vp, _vp, _tp, _tp, _i,
                                     _vp, _vp, _sz]),
    "fq_frame_apply_tff_actq_workspace_bytes": (_sz, [_tp, _tp]),
    "fq_side_stream_create": (_i, [_i, ctypes.POINTER(_vp)]),
    "fq_side_stream_destroy": (_i, [_vp]),
    "fq_status_string": (ctypes.c_char_p, [_i]),
    "fq_last_error": (ctypes.c_char_p, []),
    "fq_profile_enable": (None, [_i]),
    "fq_profile_reset": (None, []),
    "fq_profile_query": (_i, [ctypes.c_char_p, ctypes.POINTER(_i), ctypes.POINTER(_d)]),
}

_lib = None


class FQError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded libfq.so (raises ImportError when it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it first "
                              "(python -m paper_2403_06082_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise FQError(status, lib().fq_last_error().decode())


def _torch():
    import torch
    return torch


def _dt(t) -> int:
    torch = _torch()
    return {torch.float32: FQ_F32, torch.float16: FQ_F16, torch.bfloat16: FQ_BF16}[t.dtype]


def _dev(t, name, dtype=None, shape=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ws(nbytes, ws, device):
    torch = _torch()
    if ws is None:
        ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    return ws, ctypes.c_void_p(ws.data_ptr()), ws.numel() * ws.element_size()


# ------------------------------------------------------------------ workspace queries
def fq_hessian_workspace_bytes(xt: int, n_tokens: int, d_in: int) -> int:
    return lib().fq_hessian_workspace_bytes(xt, n_tokens, d_in)


def fq_frame_analysis_workspace_bytes(wt, d_out, d_in, K_out, K_in) -> int:
    return lib().fq_frame_analysis_workspace_bytes(wt, d_out, d_in, K_out, K_in)


def fq_quantize_frames_workspace_bytes(K_out, K_in, block) -> int:
    return lib().fq_quantize_frames_workspace_bytes(K_out, K_in, block)


def fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in) -> int:
    return lib().fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in)


# ------------------------------------------------------------------ the four calls
def fq_hessian_accumulate(X, H, accumulate: bool = False, ws=None, stream=None):
    """H (+)= X^T X.  X: (n, d_in) f32/f16/bf16 device tensor, H: (d_in, d_in) f32."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    n, d = X.shape
    _dev(H, "H", torch.float32, (d, d))
    ws, wp, wb = _ws(fq_hessian_workspace_bytes(_dt(X), n, d), ws, X.device)
    _check(lib().fq_hessian_accumulate(_stream(stream), _ptr(X), _dt(X), n, d, X.stride(0),
                                       _ptr(H), int(bool(accumulate)), wp, wb))
    return H


def fq_frame_analysis(W, P_out, P_in, H=None, D=None, Ht=None, ws=None, stream=None):
    """D = P_out^T W P_in and Ht = P_in^T H P_in (each optional)."""
    torch = _torch()
    d_out, d_in = W.shape
    _dev(W, "W")
    _dev(P_out, "P_out", torch.float32)
    _dev(P_in, "P_in", torch.float32)
    K_out, K_in = P_out.shape[1], P_in.shape[1]
    if P_out.shape[0] != d_out or P_in.shape[0] != d_in:
        raise ValueError("frame shapes do not match W")
    _dev(H, "H", torch.float32, (d_in, d_in))
    _dev(D, "D", torch.float32, (K_out, K_in))
    _dev(Ht, "Ht", torch.float32, (K_in, K_in))
    ws, wp, wb = _ws(fq_frame_analysis_workspace_bytes(_dt(W), d_out, d_in, K_out, K_in), ws,
                     W.device)
    _check(lib().fq_frame_analysis(_stream(stream), _ptr(W), _dt(W), d_out, d_in, _ptr(P_out),
                                   K_out, _ptr(P_in), K_in, _ptr(H), _ptr(D), _ptr(Ht), wp, wb))
    return D, Ht


def fq_quantize_frames(D, Ht, codes, scale, zero, bits: int = 2, block: int = 128,
                       damp: float = 0.01, clip_sigmas: float = 2.0, ws=None, stream=None):
    """codes (K_out, words_per_row(K_in, bits)) int32 view of uint32 words, scale/zero (K_out,)."""
    torch = _torch()
    K_out, K_in = D.shape
    _dev(D, "D", torch.float32)
    _dev(Ht, "Ht", torch.float32, (K_in, K_in))
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    ws, wp, wb = _ws(fq_quantize_frames_workspace_bytes(K_out, K_in, block), ws, D.device)
    _check(lib().fq_quantize_frames(_stream(stream), _ptr(D), _ptr(Ht), K_out, K_in, bits, block,
                                    float(damp), float(clip_sigmas), _ptr(codes), _ptr(scale),
                                    _ptr(zero), wp, wb))
    return codes, scale, zero


def fq_quantize_prepare(Ht, K_out: int, ws, block: int = 128, damp: float = 0.01,
                        stream=None):
    """H~ phase of fq_quantize_frames (damping, Cholesky factor) into the workspace ws."""
    torch = _torch()
    K_in = Ht.shape[0]
    _dev(Ht, "Ht", torch.float32, (K_in, K_in))
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_prepare(_stream(stream), _ptr(Ht), int(K_out), K_in, block,
                                     float(damp), _ptr(ws), ws.numel()))
    return ws


def fq_quantize_apply(D, codes, scale, zero, ws, bits: int = 2, block: int = 128,
                      clip_sigmas: float = 2.0, stream=None):
    """D phase of fq_quantize_frames, after fq_quantize_prepare on the same workspace."""
    torch = _torch()
    K_out, K_in = D.shape
    _dev(D, "D", torch.float32)
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_apply(_stream(stream), _ptr(D), K_out, K_in, bits, block,
                                   float(clip_sigmas), _ptr(codes), _ptr(scale), _ptr(zero),
                                   _ptr(ws), ws.numel()))
    return codes, scale, zero


def fq_quantize_grid(D, scale, zero, ws, bits: int = 2, block: int = 128,
                     clip_sigmas: float = 2.0, stream=None):
    """First part of fq_quantize_apply (D only: clip bounds, per-row grid, working copy of
    the clipped D); may run beside fq_quantize_prepare on another stream."""
    torch = _torch()
    K_out, K_in = D.shape
    _dev(D, "D", torch.float32)
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_grid(_stream(stream), _ptr(D), K_out, K_in, bits, block,
                                  float(clip_sigmas), _ptr(scale), _ptr(zero), _ptr(ws),
                                  ws.numel()))
    return scale, zero


def fq_quantize_round(D, codes, ws, bits: int = 2, block: int = 128, stream=None):
    """Second part of fq_quantize_apply (rounding with error feedback, packing, checks),
    after fq_quantize_prepare and fq_quantize_grid on the same workspace."""
    torch = _torch()
    K_out, K_in = D.shape
    _dev(D, "D", torch.float32)
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_round(_stream(stream), _ptr(D), K_out, K_in, bits, block,
                                   _ptr(codes), _ptr(ws), ws.numel()))
    return codes


def fq_quantize_round_async(D, codes, ws, bits: int = 2, block: int = 128, stream=None):
    """fq_quantize_round without the synchronization: launches the rounding and packing;
    the checks are reported by a later fq_quantize_status on the same stream."""
    torch = _torch()
    K_out, K_in = D.shape
    _dev(D, "D", torch.float32)
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_round_async(_stream(stream), _ptr(D), K_out, K_in, bits, block,
                                         _ptr(codes), _ptr(ws), ws.numel()))
    return codes


def fq_quantize_status(K_out: int, K_in: int, ws, block: int = 128, stream=None):
    """Synchronize the stream and raise FQError for the checks recorded in the workspace by
    fq_quantize_prepare, fq_quantize_grid and fq_quantize_round_async."""
    torch = _torch()
    _dev(ws, "ws", torch.uint8)
    _check(lib().fq_quantize_status(_stream(stream), int(K_out), int(K_in), block, _ptr(ws),
                                    ws.numel()))


class SideStream:
    """A stream from fq_side_stream_create (kernels kept off `reserve_cus` compute units),
    usable wherever a torch stream is (`.stream` is a torch.cuda.ExternalStream).  Released
    with the object."""

    def __init__(self, reserve_cus: int = 144, device=None):
        torch = _torch()
        dev = torch.device("cuda", torch.cuda.current_device() if device is None else device)
        self._h = None
        with torch.cuda.device(dev):
            h = ctypes.c_void_p()
            _check(lib().fq_side_stream_create(int(reserve_cus), ctypes.byref(h)))
        self._h = h.value
        self.reserve_cus = int(reserve_cus)
        self.stream = torch.cuda.ExternalStream(self._h, device=dev)

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.fq_side_stream_destroy(ctypes.c_void_p(self._h))
            self._h = None


def fq_frame_synthesis(codes, scale, zero, P_out, P_in, W_hat, ws=None, stream=None, bits=2):
    """W_hat = P_out diag(scale) (codes - zero) P_in^T (codes of 2, 3 or 4 bits)."""
    torch = _torch()
    K_out, K_in = P_out.shape[1], P_in.shape[1]
    d_out, d_in = P_out.shape[0], P_in.shape[0]
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    _dev(P_out, "P_out", torch.float32)
    _dev(P_in, "P_in", torch.float32)
    _dev(W_hat, "W_hat", torch.float32, (d_out, d_in))
    ws, wp, wb = _ws(fq_frame_synthesis_workspace_bytes(K_out, K_in, d_out, d_in), ws,
                     W_hat.device)
    _check(lib().fq_frame_synthesis_nbit(_stream(stream), _ptr(codes), bits, _ptr(scale),
                                         _ptr(zero), K_out, K_in, _ptr(P_out), d_out, _ptr(P_in),
                                         d_in, _ptr(W_hat), wp, wb))
    return W_hat


def fq_wiener_gains(D, Ht, codes, scale, zero, gain=None, scale_out=None, ws=None, stream=None,
                    bits=2):
    """Per-row gains of the diagonal Wiener filter, g_i = (D H~ D^^T)_ii / (D^ H~ D^^T)_ii
    (D the unclipped analysis output, H~ undamped); scale_out (optional, may be scale)
    receives scale * g.  Returns gain."""
    torch = _torch()
    _dev(D, "D", torch.float32)
    if D.dim() != 2:
        raise ValueError("D must be 2-D")
    K_out, K_in = D.shape
    _dev(Ht, "Ht", torch.float32, (K_in, K_in))
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    if gain is None:
        gain = torch.empty((K_out,), dtype=torch.float32, device=D.device)
    _dev(gain, "gain", torch.float32, (K_out,))
    _dev(scale_out, "scale_out", torch.float32, (K_out,))
    ws, wp, wb = _ws(lib().fq_wiener_gains_workspace_bytes(K_out, K_in), ws, D.device)
    _check(lib().fq_wiener_gains(_stream(stream), _ptr(D), _ptr(Ht), _ptr(codes), bits, _ptr(scale),
                                 _ptr(zero), K_out, K_in, _ptr(gain), _ptr(scale_out), wp, wb))
    return gain


# ------------------------------------------------------------------ kernel timer
def fq_profile_enable(on: bool = True):
    lib().fq_profile_enable(int(bool(on)))


def fq_profile_reset():
    lib().fq_profile_reset()


def fq_profile_query(prefix: str = ""):
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    if lib().fq_profile_query(prefix.encode(), ctypes.byref(n), ctypes.byref(ms)) != 0:
        raise FQError(6, "event query failed")
    return n.value, ms.value


def fq_frame_apply_workspace_bytes(d_in, K_out, K_in) -> int:
    return lib().fq_frame_apply_workspace_bytes(d_in, K_out, K_in)


def fq_frame_apply(X, codes, scale, zero, P_out, P_in, Y=None, ws=None, stream=None, bits=2):
    """Y = X Theta^T from the codes (2 or 4 bits) and the frames (small token counts)."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D with unit column stride")
    n, d_in = X.shape
    if not X.is_cuda:
        raise ValueError("X must be a device tensor")
    K_out, K_in = P_out.shape[1], P_in.shape[1]
    d_out = P_out.shape[0]
    if P_in.shape[0] != d_in:
        raise ValueError("P_in must have d_in rows")
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    _dev(P_out, "P_out", torch.float32)
    _dev(P_in, "P_in", torch.float32)
    if Y is None:
        Y = torch.empty((n, d_out), dtype=torch.float32, device=X.device)
    _dev(Y, "Y", torch.float32, (n, d_out))
    ws, wp, wb = _ws(fq_frame_apply_workspace_bytes(d_in, K_out, K_in), ws, X.device)
    _check(lib().fq_frame_apply_nbit(_stream(stream), _ptr(X), _dt(X), n, X.stride(0), d_in,
                                     _ptr(codes), bits, _ptr(scale), _ptr(zero), K_out, K_in,
                                     _ptr(P_out), d_out, _ptr(P_in), _ptr(Y), wp, wb))
    return Y


class Frame:
    """A tight fusion frame by its construction: dimension d, k subspaces of dimension rho,
    rotation factors R1 (d1 x d1) and R2 (d2 x d2) as fp32 device tensors, d1 * d2 = d.
    Keeps the factor tensors alive while the descriptor is in use."""

    def __init__(self, d, k, rho, R1, R2):
        torch = _torch()
        _dev(R1, "R1", torch.float32)
        _dev(R2, "R2", torch.float32)
        if R1.dim() != 2 or R1.shape[0] != R1.shape[1] or R2.dim() != 2 or R2.shape[0] != R2.shape[1]:
            raise ValueError("R1 and R2 must be square")
        self.d, self.k, self.rho = int(d), int(k), int(rho)
        self.R1, self.R2 = R1, R2
        self.c = TFF(self.d, self.k, self.rho, R1.data_ptr(), R1.shape[0], R2.data_ptr(),
                     R2.shape[0])

    @property
    def K(self):
        return self.k * self.rho

    @classmethod
    def from_seed(cls, d, r, rho, seed, stream=None, device="cuda"):
        """The constructible frame nearest redundancy r (fq_tff_choose: k lowered until the
        modulation is tight) with its rotation factors drawn on the device from a 64-bit
        seed (fq_tff_rotation_factors): (d, r, rho, seed) regenerate the whole frame."""
        k, d1, d2 = fq_tff_choose(d, r, rho)
        R1, R2 = fq_tff_rotation_factors(seed, d1, d2, stream=stream, device=device)
        return cls(d, k, rho, R1, R2)


def fq_tff_analysis_workspace_bytes(n, frame: Frame) -> int:
    return lib().fq_tff_analysis_workspace_bytes(n, ctypes.byref(frame.c))


def fq_tff_synthesis_workspace_bytes(n, frame: Frame) -> int:
    return lib().fq_tff_synthesis_workspace_bytes(n, ctypes.byref(frame.c))


def fq_frame_apply_tff_workspace_bytes(frame_out: Frame, frame_in: Frame) -> int:
    return lib().fq_frame_apply_tff_workspace_bytes(ctypes.byref(frame_out.c),
                                                    ctypes.byref(frame_in.c))


def fq_tff_analysis(X, frame: Frame, U=None, ws=None, stream=None):
    """U = X P (rows P^T x) with P given by its construction."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1 or not X.is_cuda:
        raise ValueError("X must be a 2-D device tensor with unit column stride")
    n = X.shape[0]
    if X.shape[1] != frame.d:
        raise ValueError("X must have d columns")
    if U is None:
        U = torch.empty((n, frame.K), dtype=torch.float32, device=X.device)
    _dev(U, "U", torch.float32, (n, frame.K))
    ws, wp, wb = _ws(fq_tff_analysis_workspace_bytes(n, frame), ws, X.device)
    _check(lib().fq_tff_analysis(_stream(stream), _ptr(X), _dt(X), n, X.stride(0),
                                 ctypes.byref(frame.c), _ptr(U), wp, wb))
    return U


def fq_tff_synthesis(V, frame: Frame, Y=None, ws=None, stream=None):
    """Y = V P^T (rows P v) with P given by its construction."""
    torch = _torch()
    _dev(V, "V", torch.float32)
    if V.dim() != 2 or V.shape[1] != frame.K:
        raise ValueError("V must be n x (k rho)")
    n = V.shape[0]
    if Y is None:
        Y = torch.empty((n, frame.d), dtype=torch.float32, device=V.device)
    _dev(Y, "Y", torch.float32, (n, frame.d))
    ws, wp, wb = _ws(fq_tff_synthesis_workspace_bytes(n, frame), ws, V.device)
    _check(lib().fq_tff_synthesis(_stream(stream), _ptr(V), n, ctypes.byref(frame.c), _ptr(Y),
                                  wp, wb))
    return Y


def fq_frame_apply_tff(X, codes, scale, zero, frame_out: Frame, frame_in: Frame, Y=None, ws=None,
                       stream=None, bits=2):
    """Y = X Theta^T from the codes (2 or 4 bits), both frames given by their construction."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1 or not X.is_cuda:
        raise ValueError("X must be a 2-D device tensor with unit column stride")
    n, d_in = X.shape
    if d_in != frame_in.d:
        raise ValueError("X must have frame_in.d columns")
    K_out, K_in = frame_out.K, frame_in.K
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    if Y is None:
        Y = torch.empty((n, frame_out.d), dtype=torch.float32, device=X.device)
    _dev(Y, "Y", torch.float32, (n, frame_out.d))
    ws, wp, wb = _ws(fq_frame_apply_tff_workspace_bytes(frame_out, frame_in), ws, X.device)
    _check(lib().fq_frame_apply_tff_nbit(_stream(stream), _ptr(X), _dt(X), n, X.stride(0),
                                         _ptr(codes), bits, _ptr(scale), _ptr(zero),
                                         ctypes.byref(frame_out.c), ctypes.byref(frame_in.c),
                                         _ptr(Y), wp, wb))
    return Y


def fq_frame_apply_tff_noalloc(X, codes, scale, zero, frame_out: Frame, frame_in: Frame, Y,
                               stream=None, bits=2):
    """fq_frame_apply_tff without a workspace: the library's own per-device scratch array
    (FQ_NOALLOC_SCRATCH_BYTES) is used and nothing is allocated; Y (n x d_out fp32) is the
    caller's.  Calls that overlap on one GPU race on that array."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1 or not X.is_cuda:
        raise ValueError("X must be a 2-D device tensor with unit column stride")
    n, d_in = X.shape
    if d_in != frame_in.d:
        raise ValueError("X must have frame_in.d columns")
    K_out, K_in = frame_out.K, frame_in.K
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    _dev(Y, "Y", torch.float32, (n, frame_out.d))
    _check(lib().fq_frame_apply_tff_noalloc(_stream(stream), _ptr(X), _dt(X), n, X.stride(0),
                                            _ptr(codes), bits, _ptr(scale), _ptr(zero),
                                            ctypes.byref(frame_out.c), ctypes.byref(frame_in.c),
                                            _ptr(Y)))
    return Y


def fq_act_quantize(U, act_bits=8, Cq=None, delta=None, stream=None):
    """Per-token rounding of U (n x K fp32) to act_bits-bit integers: (Cq int8, delta)."""
    torch = _torch()
    _dev(U, "U", torch.float32)
    if U.dim() != 2:
        raise ValueError("U must be 2-D")
    n, K = U.shape
    if Cq is None:
        Cq = torch.empty((n, K), dtype=torch.int8, device=U.device)
    if delta is None:
        delta = torch.empty((n,), dtype=torch.float32, device=U.device)
    _dev(Cq, "Cq", torch.int8, (n, K))
    _dev(delta, "delta", torch.float32, (n,))
    _check(lib().fq_act_quantize(_stream(stream), _ptr(U), n, K, act_bits, _ptr(Cq), _ptr(delta)))
    return Cq, delta


def fq_frame_apply_tff_actq_workspace_bytes(frame_out: Frame, frame_in: Frame) -> int:
    return lib().fq_frame_apply_tff_actq_workspace_bytes(ctypes.byref(frame_out.c),
                                                         ctypes.byref(frame_in.c))


def fq_frame_apply_tff_actq(X, codes, scale, zero, frame_out: Frame, frame_in: Frame, act_bits=8,
                            Y=None, ws=None, stream=None, bits=2):
    """fq_frame_apply_tff with the inputs' frame representation rounded per token to
    act_bits-bit integers and the code products in integer arithmetic."""
    torch = _torch()
    if X.dim() != 2 or X.stride(1) != 1 or not X.is_cuda:
        raise ValueError("X must be a 2-D device tensor with unit column stride")
    n, d_in = X.shape
    if d_in != frame_in.d:
        raise ValueError("X must have frame_in.d columns")
    K_out, K_in = frame_out.K, frame_in.K
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    if Y is None:
        Y = torch.empty((n, frame_out.d), dtype=torch.float32, device=X.device)
    _dev(Y, "Y", torch.float32, (n, frame_out.d))
    ws, wp, wb = _ws(fq_frame_apply_tff_actq_workspace_bytes(frame_out, frame_in), ws, X.device)
    _check(lib().fq_frame_apply_tff_actq(_stream(stream), _ptr(X), _dt(X), n, X.stride(0),
                                         _ptr(codes), bits, _ptr(scale), _ptr(zero),
                                         ctypes.byref(frame_out.c), ctypes.byref(frame_in.c),
                                         act_bits, _ptr(Y), wp, wb))
    return Y


def fq_tff_materialize_workspace_bytes(frame: Frame) -> int:
    return lib().fq_tff_materialize_workspace_bytes(ctypes.byref(frame.c))


def fq_tff_materialize(frame: Frame, P=None, ws=None, stream=None):
    """The dense frame P (d x k rho fp32) generated on the device from its construction."""
    torch = _torch()
    dev = frame.R1.device
    if P is None:
        P = torch.empty((frame.d, frame.K), dtype=torch.float32, device=dev)
    _dev(P, "P", torch.float32, (frame.d, frame.K))
    ws, wp, wb = _ws(fq_tff_materialize_workspace_bytes(frame), ws, dev)
    _check(lib().fq_tff_materialize(_stream(stream), ctypes.byref(frame.c), _ptr(P), P.stride(0),
                                    wp, wb))
    return P


def fq_frame_analysis_tff_workspace_bytes(wt: int, frame_out: Frame, frame_in: Frame) -> int:
    return lib().fq_frame_analysis_tff_workspace_bytes(wt, ctypes.byref(frame_out.c),
                                                       ctypes.byref(frame_in.c))


def fq_frame_analysis_tff(W, frame_out: Frame, frame_in: Frame, H=None, D=None, Ht=None, ws=None,
                          stream=None):
    """D = P_out^T W P_in and Ht = P_in^T H P_in (each optional), both frames given by their
    construction.  W: (frame_out.d, frame_in.d) f32/f16/bf16 or None when D is None."""
    torch = _torch()
    d_out, d_in = frame_out.d, frame_in.d
    if W is not None:
        _dev(W, "W", None, (d_out, d_in))
    _dev(H, "H", torch.float32, (d_in, d_in))
    _dev(D, "D", torch.float32, (frame_out.K, frame_in.K))
    _dev(Ht, "Ht", torch.float32, (frame_in.K, frame_in.K))
    dev = next(t.device for t in (W, H, D, Ht) if t is not None)
    wt = _dt(W) if W is not None else 0
    ws, wp, wb = _ws(fq_frame_analysis_tff_workspace_bytes(wt, frame_out, frame_in), ws, dev)
    _check(lib().fq_frame_analysis_tff(_stream(stream), _ptr(W), wt, ctypes.byref(frame_out.c),
                                       ctypes.byref(frame_in.c), _ptr(H), _ptr(D), _ptr(Ht), wp,
                                       wb))
    return D, Ht


def fq_frame_synthesis_tff_workspace_bytes(frame_out: Frame, frame_in: Frame) -> int:
    return lib().fq_frame_synthesis_tff_workspace_bytes(ctypes.byref(frame_out.c),
                                                        ctypes.byref(frame_in.c))


def fq_frame_synthesis_tff(codes, scale, zero, frame_out: Frame, frame_in: Frame, W_hat=None,
                           ws=None, stream=None, bits=2):
    """W_hat = P_out diag(scale) (codes - zero) P_in^T, both frames given by their
    construction (codes of 2, 3 or 4 bits)."""
    torch = _torch()
    K_out, K_in = frame_out.K, frame_in.K
    _dev(codes, "codes", torch.int32, (K_out, words_per_row(K_in, bits)))
    _dev(scale, "scale", torch.float32, (K_out,))
    _dev(zero, "zero", torch.float32, (K_out,))
    if W_hat is None:
        W_hat = torch.empty((frame_out.d, frame_in.d), dtype=torch.float32, device=codes.device)
    _dev(W_hat, "W_hat", torch.float32, (frame_out.d, frame_in.d))
    ws, wp, wb = _ws(fq_frame_synthesis_tff_workspace_bytes(frame_out, frame_in), ws, codes.device)
    _check(lib().fq_frame_synthesis_tff(_stream(stream), _ptr(codes), bits, _ptr(scale),
                                        _ptr(zero), ctypes.byref(frame_out.c),
                                        ctypes.byref(frame_in.c), _ptr(W_hat), wp, wb))
    return W_hat


def fq_tff_frame_valid(d: int, k: int, rho: int) -> bool:
    """Whether the modulated spectral-tetris frame (k, rho, d) is tight (host check)."""
    return bool(lib().fq_tff_frame_valid(d, k, rho))


def fq_tff_choose(d: int, r: float, rho: int):
    """(k, d1, d2): the constructible frame nearest redundancy r = k rho / d (k lowered until
    valid) and the split d = d1 d2 of its Kronecker rotation (host computation)."""
    k, d1, d2 = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().fq_tff_choose(d, float(r), rho, ctypes.byref(k), ctypes.byref(d1),
                               ctypes.byref(d2)))
    return k.value, d1.value, d2.value


def fq_tff_rotation_factors_workspace_bytes(d1: int, d2: int) -> int:
    return lib().fq_tff_rotation_factors_workspace_bytes(d1, d2)


def fq_tff_rotation_factors(seed: int, d1: int, d2: int, R1=None, R2=None, ws=None, stream=None,
                            device="cuda"):
    """(R1, R2): the rotation factors (d1 x d1, d2 x d2 fp32) drawn on the device from a
    64-bit seed."""
    torch = _torch()
    if R1 is None:
        R1 = torch.empty((d1, d1), dtype=torch.float32, device=device)
    if R2 is None:
        R2 = torch.empty((d2, d2), dtype=torch.float32, device=device)
    _dev(R1, "R1", torch.float32, (d1, d1))
    _dev(R2, "R2", torch.float32, (d2, d2))
    ws, wp, wb = _ws(fq_tff_rotation_factors_workspace_bytes(d1, d2), ws, R1.device)
    _check(lib().fq_tff_rotation_factors(_stream(stream), ctypes.c_uint64(seed & (2 ** 64 - 1)),
                                         d1, d2, _ptr(R1), _ptr(R2), wp, wb))
    return R1, R2
