"""Workload table: synthetic layers shaped like the paper's ViT / OPT / Llama workloads.

The paper quantizes real pretrained layers with real calibration sets (ImageNet images,
LLM text); neither is available, so seeded synthetic layers with the same shapes and the
same qualitative structure (Gaussian weights with a sparse set of large outliers,
Gaussian activations with a few outlier channels) stand in for them.

Frame convention: rho = 16 real dimensions per subspace and k = round(r * d / rho)
subspaces, so every d used here has d / rho integral and the modulated spectral-tetris
frame is tight (k >= d / rho).  The 256 x 256 layer is given k = 18, rho = 16
(r = 1.125): the triple k = 16, rho = 18 has a spectral-tetris row whose support
is 17 columns long, wider than k = 16, so its modulation is not tight.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Layer:
    name: str
    d_out: int
    d_in: int
    w_sigma: float
    outlier_frac: float = 0.01      # fraction of weights scaled by outlier_scale
    outlier_scale: float = 10.0
    t4_frac: float = 0.0            # fraction of weights drawn from sigma * Student-t(4)


@dataclass(frozen=True)
class Workload:
    key: str
    description: str
    layers: tuple
    n_tokens: int
    x_outlier_channels: int
    x_outlier_scale: float
    w_dtype: str                    # "f32" | "f16" | "bf16"
    x_dtype: str
    r: float = 1.1
    rho: int = 16
    k_override: dict = field(default_factory=dict)   # d -> k
    bits: int = 2
    block: int = 128
    damp: float = 0.01
    clip_sigmas: float = 2.0
    seed: int = 0


TINY = Workload(
    key="tiny256",
    description="single 256x256 linear layer, fp32; X 512x256 fp32 with 4 outlier "
                "channels x20; frames k=18, rho=16 (r=1.125)",
    layers=(Layer("w", 256, 256, 0.02),),
    n_tokens=512, x_outlier_channels=4, x_outlier_scale=20.0,
    w_dtype="f32", x_dtype="f32", r=1.125, k_override={256: 18},
)

VIT_B = Workload(
    key="vitb",
    description="ViT-B-shaped qkv 2304x768 and fc1 3072x768 fp32 sharing one input; "
                "X = 128 x 197 tokens x 768 fp32 with 6 outlier channels x20; r = 1.1",
    layers=(Layer("qkv", 2304, 768, 0.02), Layer("fc1", 3072, 768, 0.02)),
    n_tokens=128 * 197, x_outlier_channels=6, x_outlier_scale=20.0,
    w_dtype="f32", x_dtype="f32",
)

OPT_1B3 = Workload(
    key="opt1b3",
    description="OPT-1.3B-shaped fc1 8192x2048 fp16 (Gaussian sigma 0.02 with a 5% "
                "Student-t(4) mixture); X = 128 x 2048 tokens x 2048 fp16 with 2 outlier "
                "channels x50; r = 1.1",
    layers=(Layer("fc1", 8192, 2048, 0.02, outlier_frac=0.0, t4_frac=0.05),),
    n_tokens=128 * 2048, x_outlier_channels=2, x_outlier_scale=50.0,
    w_dtype="f16", x_dtype="f16",
)

LLAMA_7B = Workload(
    key="llama7b",
    description="Llama-2-7B-shaped q_proj 4096x4096 and up_proj 11008x4096 bf16 sharing "
                "one input; X = 128 x 2048 tokens x 4096 bf16 with 8 massive-activation "
                "channels x100; r = 1.1",
    layers=(Layer("q", 4096, 4096, 0.02), Layer("up", 11008, 4096, 0.02)),
    n_tokens=128 * 2048, x_outlier_channels=8, x_outlier_scale=100.0,
    w_dtype="bf16", x_dtype="bf16",
)

LLAMA_70B_R10 = Workload(
    key="llama70b_r1.0",
    description="Llama-2-70B-shaped down_proj 8192x28672 bf16 (sigma 0.015); X = 128 x "
                "2048 tokens x 28672 bf16 with 16 outlier channels x50; r = 1.0",
    layers=(Layer("down", 8192, 28672, 0.015),),
    n_tokens=128 * 2048, x_outlier_channels=16, x_outlier_scale=50.0,
    w_dtype="bf16", x_dtype="bf16", r=1.0,
)

LLAMA_70B_R11 = Workload(
    key="llama70b_r1.1",
    description=LLAMA_70B_R10.description.replace("r = 1.0", "r = 1.1"),
    layers=LLAMA_70B_R10.layers,
    n_tokens=LLAMA_70B_R10.n_tokens, x_outlier_channels=16, x_outlier_scale=50.0,
    w_dtype="bf16", x_dtype="bf16", r=1.1,
)

WORKLOADS = {w.key: w for w in (TINY, VIT_B, OPT_1B3, LLAMA_7B, LLAMA_70B_R10, LLAMA_70B_R11)}


def frame_k(wl: Workload, d: int) -> int:
    from .tff import choose_k
    if d in wl.k_override:
        return wl.k_override[d]
    return choose_k(d, wl.r, wl.rho)
