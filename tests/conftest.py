import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# One hardware queue per stream for the test process.  HIP gives a process 4
# queues by default; streams beyond that share a queue and run in submission
# order, which hides a missing wait instead of exposing it.  The race tests
# (an update on another stream with and without the gate) need streams that
# really run side by side.  Read by the HIP runtime when it first starts,
# which is after this file is loaded.
os.environ["GPU_MAX_HW_QUEUES"] = "16"
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; runs through the C-ABI library")
    config.addinivalue_line("markers", "slow: full-size shard; minutes of GPU time")
