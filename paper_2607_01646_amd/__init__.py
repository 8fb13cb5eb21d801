"""MI355X-native in-memory checkpoint hot path (PHOENIX, D2H phase).

libckpt (C ABI in include/ckpt.h, HIP kernels for gfx950) packs one rank's
training state with per-chunk word-sums into device staging, streams it to
ping-pong pinned host images off the critical path, gates the optimizer step
at chunk granularity, and restores / verifies on the GPU.  This package is
the thin Python binding over that library.
"""
from .ckpt import *  # noqa: F401,F403
from .ckpt import Checkpointer, CkptError, lib  # noqa: F401
