"""MI355X-native in-memory checkpoint hot path (PHOENIX, D2H and H2H phases).

libckpt (C ABI in include/ckpt.h, HIP kernels for gfx950) packs one rank's
training state with per-chunk word-sums into device staging, streams it to
ping-pong host images off the critical path, gates the optimizer step at
chunk granularity, and restores / verifies on the GPU.  It also replicates
the optimizer chunks to k ring peers (Peer), lets a replacement rank restore
from a peer's replica, and keeps crash-surviving image files.  This package
is the thin Python binding over that library (Checkpointer, Peer); the
analytic models and replica placement are in `disruption` and `placement`.
"""
from .ckpt import *  # noqa: F401,F403
from .ckpt import Checkpointer, CkptError, Peer, PeerError, lib  # noqa: F401
