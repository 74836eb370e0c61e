"""FrameQuant's per-layer quantization pass on AMD Instinct MI355X (gfx950).

The computation lives in libfq.so (HIP kernels behind the C ABI of include/fq.h); this
package holds the sources, the build script and a thin ctypes binding.
"""
from .fq import (  # noqa: F401
    FQ_F32, FQ_F16, FQ_BF16, FQError, lib,
    fq_hessian_accumulate, fq_frame_analysis, fq_quantize_frames, fq_frame_synthesis,
    fq_quantize_prepare, fq_quantize_apply, fq_quantize_grid, fq_quantize_round,
    fq_quantize_round_async, fq_quantize_status, fq_frame_apply,
    fq_frame_apply_workspace_bytes,
    Frame, fq_tff_analysis, fq_tff_synthesis, fq_frame_apply_tff, fq_frame_apply_tff_noalloc,
    fq_tff_analysis_workspace_bytes,
    fq_tff_synthesis_workspace_bytes, fq_frame_apply_tff_workspace_bytes,
    fq_act_quantize, fq_frame_apply_tff_actq, fq_frame_apply_tff_actq_workspace_bytes,
    fq_tff_materialize, fq_tff_materialize_workspace_bytes,
    fq_frame_analysis_tff, fq_frame_analysis_tff_workspace_bytes,
    fq_frame_synthesis_tff, fq_frame_synthesis_tff_workspace_bytes,
    fq_tff_rotation_factors, fq_tff_rotation_factors_workspace_bytes, fq_tff_choose,
    fq_tff_frame_valid,
    fq_hessian_workspace_bytes, fq_frame_analysis_workspace_bytes,
    fq_quantize_frames_workspace_bytes, fq_frame_synthesis_workspace_bytes,
    fq_profile_enable, fq_profile_reset, fq_profile_query, fq_wiener_gains, SideStream,
)
