"""Seeded synthetic training-state shards.

This package only generates inputs: model shapes, fragment lists, value
distributions and fault-injection positions.  It holds none of the snapshot
arithmetic (layout, pack, checksum, restore), so both the GPU library's tests
and the CPU oracle can take their inputs from it.
"""
from .shards import *  # noqa: F401,F403
