"""CPU checks of the benchmark's bookkeeping: the minimal-byte formulas reproduce the
per-op figures worked out for the Mamba-1.4B workload (8 x 4096 tokens, d_inner 4096,
d_state 16, width 4, bf16), the sequence listing reads starts from the position
indices, and more than one GPU is refused before anything touches a device."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_minimal_bytes_at_the_headline_shape():
    import bench
    mb = bench.minimal_bytes(8, 4096, 4096, 16, 4, 2)
    want = {"conv_fwd": 0.5371e9, "scan_fwd": 1.0763e9, "scan_bwd": 1.8861e9, "conv_bwd": 0.8056e9}
    for k, v in want.items():
        assert abs(mb[k] - v) <= 5e4, (k, mb[k], v)
    assert abs(sum(mb.values()) - 4.3050e9) <= 1e6
    # scan forward: u, delta, z in and y out per element; B, C and the index per token; A, D, bias
    E, T = 8 * 4096 * 4096, 8 * 4096
    assert mb["scan_fwd"] == E * 8 + T * (2 * 16 * 2 + 4) + 4 * (4096 * 16 + 2 * 4096)


def test_sequences_from_positions():
    import bench
    pos = np.array([[0, 1, 2, 0, 0, 1], [0, 1, 2, 3, 4, 5]], dtype=np.int32)
    assert bench.sequences(pos) == [(0, 0, 3), (0, 3, 1), (0, 4, 2), (1, 0, 6)]


def test_more_than_one_gpu_is_refused():
    env = dict(os.environ, WORLD_SIZE="1")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, env=env, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_stored_traffic_only_for_the_measured_shape():
    """The counter-based traffic is reported only for the shape the counters were taken on
    (and only while the kernel source is unchanged)."""
    import bench
    shape = {"batch": 8, "seqlen": 4096, "dim": 4096, "dstate": 16, "storage": "bf16"}
    t = bench.stored_traffic(shape)
    assert t is None or (t["shape"] == shape and t["kernel_hash"] == bench.kernel_hash())
    for other in ({**shape, "dim": 5120}, {**shape, "storage": "f32"}, {**shape, "batch": 4, "seqlen": 2048}):
        assert bench.stored_traffic(other) is None
