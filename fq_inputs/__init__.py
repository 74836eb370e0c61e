"""Seeded synthetic inputs for the FrameQuant per-layer quantization pass.

Shared by the oracle tests, the device tests and the benchmark.  Holds random draws,
rounding to device dtypes and the tight-fusion-frame construction that defines the frame
inputs; none of the quantization method's arithmetic lives here.
"""
from .configs import WORKLOADS, Workload, Layer, frame_k  # noqa: F401
from . import tff, gen  # noqa: F401
