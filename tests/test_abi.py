"""Host-side checks of the C ABI: the library loads, exports every declared entry point,
answers workspace queries, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fq.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fq_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    from paper_2403_06082_amd import fq
    return fq.lib()


def test_header_and_binding_agree():
    from paper_2403_06082_amd import fq
    assert _declared() == sorted(fq.SIGNATURES)


def test_exports_every_symbol(L):
    for name in _declared():
        assert hasattr(L, name), name


def test_status_strings(L):
    assert L.fq_status_string(0) == b"FQ_OK"
    assert L.fq_status_string(3) == b"FQ_ERR_NOT_POSITIVE_DEFINITE"
    assert L.fq_status_string(99) == b"FQ_UNKNOWN_STATUS"


def test_workspace_queries(L):
    # llama-7B up_proj shapes
    wq = L.fq_quantize_frames_workspace_bytes(12112, 4512, 128)
    assert wq >= 12112 * 4512 * 8 + 2 * 4512 * 4512 * 8
    wa = L.fq_frame_analysis_workspace_bytes(2, 11008, 4096, 12112, 4512)
    assert wa >= 2 * 11008 * 12112 * 2
    wh = L.fq_hessian_workspace_bytes(2, 262144, 4096)
    assert wh > 0
    ws = L.fq_frame_synthesis_workspace_bytes(12112, 4512, 11008, 4096)
    assert ws >= 12112 * 4512 * 2
    assert L.fq_quantize_frames_workspace_bytes(-1, 5, 128) == 0
    assert L.fq_quantize_frames_workspace_bytes(5, 5, 0) == 0


def test_invalid_arguments_rejected_before_launch(L):
    n = None
    # bad dtype / negative size / ldx < d_in
    assert L.fq_hessian_accumulate(n, n, 7, 10, 10, 10, n, 0, n, 0) == 1
    assert L.fq_hessian_accumulate(n, n, 2, -1, 10, 10, n, 0, n, 0) == 1
    assert L.fq_hessian_accumulate(n, n, 2, 10, 10, 5, n, 0, n, 0) == 1
    assert b"ldx" in L.fq_last_error()
    # NULL H
    assert L.fq_hessian_accumulate(n, n, 2, 10, 10, 10, n, 0, n, 0) == 1
    # workspace too small
    assert L.fq_hessian_accumulate(n, ctypes.c_void_p(64), 2, 10, 10, 10, ctypes.c_void_p(64), 0,
                                   ctypes.c_void_p(64), 0) == 5
    # frames narrower than the space
    assert L.fq_frame_analysis(n, n, 2, 10, 10, n, 9, n, 10, n, n, n, n, 0) == 1
    # unsupported bit width, bad block, bad damp / clip
    args = (n, ctypes.c_void_p(64), ctypes.c_void_p(64), 4, 4)
    outs = (ctypes.c_void_p(64), ctypes.c_void_p(64), ctypes.c_void_p(64), n, 0)
    assert L.fq_quantize_frames(*args, 5, 128, 0.01, 2.0, *outs) == 2
    assert L.fq_quantize_frames(*args, 1, 128, 0.01, 2.0, *outs) == 2
    assert L.fq_quantize_frames(*args, 2, 0, 0.01, 2.0, *outs) == 1
    assert L.fq_quantize_frames(*args, 2, 128, -1.0, 2.0, *outs) == 1
    assert L.fq_quantize_frames(*args, 2, 128, 0.01, 0.0, *outs) == 1
    assert L.fq_quantize_frames(*args, 2, 128, 0.01, float("nan"), *outs) == 1
    assert L.fq_quantize_frames(*args, 2, 128, 0.01, 2.0, *outs) == 5
    # the two phases check the same arguments in the same order
    assert L.fq_quantize_prepare(n, ctypes.c_void_p(64), 4, 4, 0, 0.01, n, 0) == 1
    assert L.fq_quantize_prepare(n, ctypes.c_void_p(64), 4, 4, 128, float("inf"), n, 0) == 1
    assert L.fq_quantize_prepare(n, n, 4, 4, 128, 0.01, n, 0) == 1
    assert L.fq_quantize_prepare(n, ctypes.c_void_p(64), 4, 4, 128, 0.01, n, 0) == 5
    aouts = (ctypes.c_void_p(64), ctypes.c_void_p(64), ctypes.c_void_p(64), n, 0)
    assert L.fq_quantize_apply(n, ctypes.c_void_p(64), 4, 4, 5, 128, 2.0, *aouts) == 2
    assert L.fq_quantize_apply(n, ctypes.c_void_p(64), 4, 4, 2, 128, -2.0, *aouts) == 1
    assert L.fq_quantize_apply(n, ctypes.c_void_p(64), -4, 4, 2, 128, 2.0, *aouts) == 1
    assert L.fq_quantize_apply(n, ctypes.c_void_p(64), 4, 4, 2, 128, 2.0, *aouts) == 5
    # apply's two parts check their own arguments the same way
    gouts = (ctypes.c_void_p(64), ctypes.c_void_p(64), n, 0)
    assert L.fq_quantize_grid(n, ctypes.c_void_p(64), 4, 4, 5, 128, 2.0, *gouts) == 2
    assert L.fq_quantize_grid(n, ctypes.c_void_p(64), 4, 4, 2, 0, 2.0, *gouts) == 1
    assert L.fq_quantize_grid(n, ctypes.c_void_p(64), 4, 4, 2, 128, 0.0, *gouts) == 1
    assert L.fq_quantize_grid(n, n, 4, 4, 2, 128, 2.0, *gouts) == 1
    assert L.fq_quantize_grid(n, ctypes.c_void_p(64), 4, 4, 2, 128, 2.0, *gouts) == 5
    routs = (ctypes.c_void_p(64), n, 0)
    assert L.fq_quantize_round(n, ctypes.c_void_p(64), 4, 4, 1, 128, *routs) == 2
    assert L.fq_quantize_round(n, ctypes.c_void_p(64), -4, 4, 2, 128, *routs) == 1
    assert L.fq_quantize_round(n, ctypes.c_void_p(64), 4, 4, 2, 128, n, n, 0) == 1
    assert L.fq_quantize_round(n, ctypes.c_void_p(64), 4, 4, 2, 128, *routs) == 5
    assert L.fq_quantize_round_async(n, ctypes.c_void_p(64), 4, 4, 1, 128, *routs) == 2
    assert L.fq_quantize_round_async(n, ctypes.c_void_p(64), 4, 4, 2, 128, n, n, 0) == 1
    assert L.fq_quantize_round_async(n, ctypes.c_void_p(64), 4, 4, 2, 128, *routs) == 5
    assert L.fq_quantize_status(n, -1, 4, 128, n, 0) == 1
    assert L.fq_quantize_status(n, 4, 4, 0, n, 0) == 1
    assert L.fq_quantize_status(n, 4, 4, 128, n, 0) == 5
    # empty problems are no-ops
    assert L.fq_quantize_frames(n, n, n, 0, 5, 2, 128, 0.01, 2.0, n, n, n, n, 0) == 0
    assert L.fq_quantize_prepare(n, n, 0, 5, 128, 0.01, n, 0) == 0
    assert L.fq_quantize_apply(n, n, 5, 0, 2, 128, 2.0, n, n, n, n, 0) == 0
    assert L.fq_quantize_grid(n, n, 5, 0, 2, 128, 2.0, n, n, n, 0) == 0
    assert L.fq_quantize_round(n, n, 0, 5, 2, 128, n, n, 0) == 0
    assert L.fq_quantize_round_async(n, n, 0, 5, 2, 128, n, n, 0) == 0
    assert L.fq_quantize_status(n, 0, 5, 128, n, 0) == 0
    assert L.fq_frame_synthesis(n, n, n, n, 5, 5, n, 0, n, 5, n, n, 0) == 0


def test_tff_frames_validated_before_launch(L):
    """Structured frames: the workspace query answers 0 and every entry point returns its
    status before any launch for frames outside the supported set."""
    from paper_2403_06082_amd.fq import TFF
    p, n = ctypes.c_void_p(64), None
    good = TFF(4096, 282, 16, 64, 64, 64, 64)
    assert L.fq_tff_analysis_workspace_bytes(1, ctypes.byref(good)) >= 4096 * 4
    assert L.fq_frame_apply_tff_workspace_bytes(ctypes.byref(good), ctypes.byref(good)) > 0
    cases = [
        (TFF(4096, 282, 15, 64, 64, 64, 64), 1),     # odd rho
        (TFF(4096, 282, 24, 64, 64, 64, 64), 2),     # d not divisible by rho
        (TFF(4096, 200, 16, 64, 64, 64, 64), 1),     # d / rho > k: modulation not tight
        (TFF(4096, 282, 16, 64, 64, 64, 32), 1),     # d1 d2 != d
        (TFF(4096, 282, 16, None, 64, 64, 64), 1),   # NULL rotation factor
        (TFF(4096, 4000, 2, 64, 64, 64, 64), 2),     # k above the LDS limit
        (TFF(8192, 600, 16, 64, 1, 64, 8192), 2),    # d2 above the LDS limit
    ]
    for f, st in cases:
        fp = ctypes.byref(f)
        if f.R1 is not None:
            assert L.fq_tff_analysis_workspace_bytes(1, fp) == 0
        assert L.fq_tff_analysis(n, p, 0, 1, 4096, fp, p, p, 1 << 30) == st
        assert L.fq_tff_synthesis(n, p, 1, fp, p, p, 1 << 30) == st
        assert L.fq_frame_apply_tff(n, p, 0, 1, 4096, p, p, p, fp, ctypes.byref(good), p, p,
                                    1 << 30) == st
        assert b"frame" in L.fq_last_error()
    # ldx < d, bad dtype, empty input, too small a workspace
    gp = ctypes.byref(good)
    assert L.fq_tff_analysis(n, p, 0, 1, 4095, gp, p, p, 1 << 30) == 1
    assert L.fq_tff_analysis(n, p, 5, 1, 4096, gp, p, p, 1 << 30) == 1
    assert L.fq_tff_analysis(n, n, 0, 0, 4096, gp, n, n, 0) == 0
    assert L.fq_tff_analysis(n, p, 0, 1, 4096, gp, p, p, 64) == 5
    assert L.fq_frame_apply_tff(n, p, 0, 1, 4096, p, p, p, gp, gp, p, p, 64) == 5


def test_structured_pass_arguments(L):
    """fq_frame_analysis_tff / fq_frame_synthesis_tff: frames, sizes, bits, NULL arrays and
    the workspace are checked before any launch."""
    from paper_2403_06082_amd.fq import TFF
    p, n = ctypes.c_void_p(64), None
    good = TFF(4096, 282, 16, 64, 64, 64, 64)
    gp = ctypes.byref(good)
    need_a = L.fq_frame_analysis_tff_workspace_bytes(2, gp, gp)
    need_s = L.fq_frame_synthesis_tff_workspace_bytes(gp, gp)
    assert need_a >= 4512 * 4512 * 4 and need_s >= 4096 * 4512 * 4
    assert L.fq_frame_analysis_tff_workspace_bytes(3, gp, gp) == 0
    big = TFF(1 << 22, 3968, 2048, 64, 1 << 11, 64, 1 << 11)     # d above 2^21, else valid
    bp = ctypes.byref(big)
    assert L.fq_frame_analysis_tff_workspace_bytes(2, bp, gp) == 0
    assert L.fq_frame_analysis_tff(n, p, 2, bp, gp, p, p, p, p, 1 << 40) == 2
    assert L.fq_frame_synthesis_tff(n, p, 2, p, p, gp, bp, p, p, 1 << 40) == 2
    wide = ctypes.byref(TFF(1 << 20, 3968, 1024, 64, 256, 64, 4096))   # K = 3968 * 1024 > 65535 * 32
    assert L.fq_frame_analysis_tff_workspace_bytes(2, wide, gp) == 0
    assert L.fq_frame_analysis_tff(n, p, 2, wide, gp, p, p, p, p, 1 << 40) == 2
    bad = ctypes.byref(TFF(4096, 282, 15, 64, 64, 64, 64))
    assert L.fq_frame_analysis_tff(n, p, 2, bad, gp, p, p, p, p, 1 << 40) == 1
    assert b"frame_out" in L.fq_last_error()
    assert L.fq_frame_analysis_tff(n, p, 5, gp, gp, p, p, p, p, 1 << 40) == 1    # bad dtype
    assert L.fq_frame_analysis_tff(n, n, 2, gp, gp, p, p, p, p, need_a) == 1     # W NULL with D
    assert L.fq_frame_analysis_tff(n, p, 2, gp, gp, n, p, p, p, need_a) == 1     # H NULL with Ht
    assert L.fq_frame_analysis_tff(n, p, 2, gp, gp, p, p, p, p, need_a - 1) == 5
    assert L.fq_frame_analysis_tff(n, n, 2, gp, gp, n, n, n, p, need_a) == 0     # nothing asked
    assert L.fq_frame_synthesis_tff(n, p, 5, p, p, gp, gp, p, p, need_s) == 2    # bits
    assert L.fq_frame_synthesis_tff(n, p, 2, p, p, gp, bad, p, p, need_s) == 1
    assert b"frame_in" in L.fq_last_error()
    assert L.fq_frame_synthesis_tff(n, n, 2, p, p, gp, gp, p, p, need_s) == 1    # codes NULL
    assert L.fq_frame_synthesis_tff(n, p, 2, p, p, gp, gp, p, p, need_s - 1) == 5


def test_rotation_factor_arguments(L):
    p, n = ctypes.c_void_p(64), None
    need = L.fq_tff_rotation_factors_workspace_bytes(86, 128)
    assert need >= 2 * 128 * 128 * 8
    assert L.fq_tff_rotation_factors_workspace_bytes(0, 4) == 0
    assert L.fq_tff_rotation_factors_workspace_bytes(4, 1025) == 0
    assert L.fq_tff_rotation_factors(n, 7, 0, 4, p, p, p, need) == 1
    assert L.fq_tff_rotation_factors(n, 7, 4, 1025, p, p, p, 1 << 40) == 2
    assert L.fq_tff_rotation_factors(n, 7, 86, 128, n, p, p, need) == 1
    assert L.fq_tff_rotation_factors(n, 7, 86, 128, p, p, p, need - 1) == 5
    assert L.fq_tff_rotation_factors(n, 7, 86, 128, p, p, n, need) == 1


def test_act_quantize_arguments(L):
    p, n = ctypes.c_void_p(64), None
    assert L.fq_act_quantize(n, p, 4, 8, 1, p, p) == 1
    assert L.fq_act_quantize(n, p, 4, 8, 9, p, p) == 1
    assert L.fq_act_quantize(n, n, 0, 8, 8, n, n) == 0
    assert L.fq_act_quantize(n, n, 4, 8, 8, p, p) == 1
    from paper_2403_06082_amd.fq import TFF
    good = ctypes.byref(TFF(4096, 282, 16, 64, 64, 64, 64))
    assert L.fq_frame_apply_tff_actq_workspace_bytes(good, good) > \
        L.fq_frame_apply_tff_workspace_bytes(good, good)
    assert L.fq_frame_apply_tff_actq(n, p, 0, 1, 4096, p, 2, p, p, good, good, 9, p, p, 1 << 30) == 1
    assert L.fq_frame_apply_tff_actq(n, p, 0, 1, 4096, p, 3, p, p, good, good, 8, p, p, 1 << 30) == 2
    assert L.fq_frame_apply_tff_actq(n, p, 0, 1, 4096, p, 2, p, p, good, good, 8, p, p, 64) == 5


def test_frame_choice_matches_the_oracle(L):
    """fq_tff_frame_valid against the oracle's definition of tightness on every small real
    triple, and fq_tff_choose against the oracle's choice (support rule at the workloads'
    sizes) and against the frames the workloads use."""
    import numpy as np
    import oracle as O
    from fq_inputs import WORKLOADS, configs
    for rho in range(2, 13, 2):
        for d in range(rho, 3 * rho + 6, 2):
            for k in range(1, d // 2 + 3):
                assert L.fq_tff_frame_valid(d, k, rho) == int(O.tff_frame_valid(d, k, rho)), (d, k, rho)
    assert L.fq_tff_frame_valid(256, 16, 18) == 0 and L.fq_tff_frame_valid(256, 18, 16) == 1
    assert L.fq_tff_frame_valid(21, 5, 8) == 0 and L.fq_tff_frame_valid(22, 5, 7) == 0

    def support_valid(d, k, rho):
        F = O.spectral_tetris_untf(rho // 2, d // 2)
        return F is not None and O.untf_max_row_support(F) <= k

    k, d1, d2 = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    for wl in WORKLOADS.values():
        for lay in wl.layers:
            for d in (lay.d_out, lay.d_in):
                if d in wl.k_override:
                    continue
                assert L.fq_tff_choose(d, wl.r, wl.rho, ctypes.byref(k), ctypes.byref(d1),
                                       ctypes.byref(d2)) == 0
                assert k.value == O.tff_choose_k(d, wl.r, wl.rho, support_valid)
                assert k.value == configs.frame_k(wl, d)
                assert d1.value * d2.value == d and d1.value <= d2.value
    # the 256 x 256 layer's stated (k, rho) = (16, 18): no k <= 16 is valid with rho = 18
    assert L.fq_tff_choose(256, 1.125, 18, ctypes.byref(k), None, None) == 2
    assert L.fq_tff_choose(256, 1.125, 16, ctypes.byref(k), None, None) == 0 and k.value == 18
    assert L.fq_tff_choose(22, 1.9, 8, ctypes.byref(k), None, None) == 0 and k.value == 5
    assert L.fq_tff_choose(22, 1.1, 8, ctypes.byref(k), None, None) == 2
    assert L.fq_tff_choose(255, 1.1, 16, ctypes.byref(k), None, None) == 1
    assert L.fq_tff_choose(256, -1.0, 16, ctypes.byref(k), None, None) == 1
